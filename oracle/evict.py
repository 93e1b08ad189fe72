"""The Random Attention eviction rule, written out plainly (oracle side).

TEST INFRASTRUCTURE ONLY (see the package header).

What the paper fixes
--------------------
* Periodic eviction (Section 2, "Periodic eviction with budget K and buffer
  r", Eq. 1): each decode step appends one pair; the candidate set holds every
  cached position outside the buffer of the r most recent pairs; the K
  highest-scoring candidates are kept and the rest are discarded for good.
* Random Attention's score (Section 3): +infinity for prompt positions,
  i.i.d. Uniform(0,1) for every other candidate, drawn independently per KV
  head at every eviction.  Eq. 1 then keeps the prompt and a uniformly random
  subset of the rest.
* Engine details (Appendix F): the trigger fires every r=64 decode steps
  once the cache exceeds K+r; keep-sets are sorted chronologically; grouped
  query heads share their KV head's keep-set; eviction is monotonic.

Readings where the paper is silent (each is also listed in the design notes)
--------------------------------------------------------------------------
* Budget convention.  In Eq. 1 the prompt competes with score +infinity, so
  K counts the prompt (``TOTAL``: k_keep = K - lp, defined only when the
  prompt fits, Appendix H "Budgets and long prompts").  The workloads measured
  here instead fix K as the number of kept non-prompt, non-buffer entries
  (``EVICTABLE``: k_keep = K).  Both are supported; they keep identical sets
  for the same k_keep.
* Trigger.  Evict at the end of decode step t iff t mod R == 0 and the
  evictable entries (cached - prompt - r) exceed k_keep, with R = r = 64 as
  in Appendix F; R = 1 gives the "whenever they exceed" reading.
* Uniform score.  A uniform draw is represented by a 64-bit unsigned integer
  (a uniform on a 2^-64 grid); keeping the k_keep largest is the same as
  keeping the k_keep largest Uniform(0,1) scores.  The key of position p at
  event e of layer l, KV head g, for request (seed, request_id) is word
  (p mod 4) of Philox4x64-10 at counter (floor(p/4), e, l, g) and key
  (seed, request_id).  The key is tied to the position, not the memory slot.
* Ties.  Candidates are ordered by (key, position); the m = |C| - k_keep
  smallest are dropped, so among equal keys the earlier position goes first.
* Event index e counts the evictions performed on the sequence so far
  (0-based), shared by all its layers and KV heads.

Diagnostic policies (the paper's controls, on the same trigger and select)
--------------------------------------------------------------------------
Only the key of a candidate changes; the m smallest (key, position) pairs
are still the ones dropped.
* Shared draw (Section 5, Appendix D): the same random positions in every
  head.  Reading: the key of p is the Random Attention key with the layer and
  KV head fixed at 0, so every (layer, head) keeps the set that (0, 0) keeps.
* Block-wise (Section 5): history kept in contiguous blocks of B tokens.
  Reading: blocks are aligned at the end of the prompt, block b covering
  positions lp + bB .. lp + bB + B - 1, and every position takes the key of
  its block's first position, so whole blocks go together (the one block that
  straddles the cut loses its earliest positions first) and B = 1 is Random
  Attention.
* Recency + prompt (Section 4.1): the prompt plus the contiguous recent
  window.  The key is the position itself, so the oldest candidates go and
  the cache is always the prompt plus the last k_keep + r positions.

Parity: pinned by the tests against brute-force subset enumeration, the
exact subset law and marginal inclusion (chi-square), cross-head and
cross-event independence, the survival law of Appendix D, the structural
invariants, and the TOTAL/EVICTABLE equivalence.  The particular subset a
given seed yields has no paper value to pin it (any uniform K-subset is
correct); that choice is this generator's, reproduced bit-exactly by the GPU.
"""

import numpy as np

from .philox import philox4x64_10_np

BUDGET_EVICTABLE = 0
BUDGET_TOTAL = 1

POLICY_RANDOM = 0
POLICY_SHARED = 1
POLICY_BLOCK = 2
POLICY_RECENCY = 3


def keep_count(budget_k, prompt_len, mode):
    """Number of evictable (non-prompt, non-buffer) entries a head keeps."""
    if mode == BUDGET_EVICTABLE:
        return int(budget_k)
    if mode == BUDGET_TOTAL:
        k = int(budget_k) - int(prompt_len)
        if k < 0:
            raise ValueError("prompt does not fit in the budget")
        return k
    raise ValueError("unknown budget mode")


def position_keys(positions, seed, request_id, event, layer, kv_head):
    """Uniform 64-bit scores of the given positions for one eviction event."""
    p = np.asarray(positions, dtype=np.uint64)
    words = philox4x64_10_np(p >> np.uint64(2), event, layer, kv_head,
                             seed, request_id)
    lane = (p & np.uint64(3)).astype(np.int64)
    return np.choose(lane, words)


def policy_keys(policy, candidates, prompt_len, seed, request_id, event,
                layer, kv_head, block=1):
    """Keys of the candidates under one of the policies above."""
    cand = np.asarray(candidates, dtype=np.int64)
    if policy == POLICY_RANDOM:
        return position_keys(cand, seed, request_id, event, layer, kv_head)
    if policy == POLICY_SHARED:
        return position_keys(cand, seed, request_id, event, 0, 0)
    if policy == POLICY_BLOCK:
        if block < 1:
            raise ValueError("block size must be >= 1")
        first = prompt_len + (cand - prompt_len) // block * block
        return position_keys(first, seed, request_id, event, layer, kv_head)
    if policy == POLICY_RECENCY:
        return cand.astype(np.uint64)
    raise ValueError("unknown policy")


def drop_set(candidates, keys, m):
    """Indices (into candidates) of the m smallest (key, position) pairs."""
    candidates = np.asarray(candidates)
    order = np.lexsort((candidates, keys))     # by key, then position
    return np.sort(order[:m])


def eviction_due(step, n_cached, prompt_len, recent_r, k_keep, every):
    """Trigger at the end of decode step ``step`` (1-based count)."""
    return step % every == 0 and n_cached - prompt_len - recent_r > k_keep


def evict_head(P, prompt_len, recent_r, k_keep, seed, request_id, event,
               layer, kv_head, policy=POLICY_RANDOM, block=1):
    """One eviction of one (layer, KV head) cache.

    P: ascending positions currently cached.  Returns the new ascending
    list: prompt, then the kept candidates in chronological order, then the
    r most recent positions.  If the candidates do not exceed k_keep the
    list is returned unchanged.
    """
    P = np.asarray(P, dtype=np.int64)
    n = P.shape[0]
    cand = P[prompt_len:n - recent_r]
    m = cand.shape[0] - k_keep
    if m <= 0:
        return P.copy()
    keys = policy_keys(policy, cand, prompt_len, seed, request_id, event,
                       layer, kv_head, block)
    keep = np.ones(cand.shape[0], dtype=bool)
    keep[drop_set(cand, keys, m)] = False
    return np.concatenate([P[:prompt_len], cand[keep], P[n - recent_r:]])


class SequenceReplay:
    """Index-only replay of one sequence: positions of every (layer, head).

    Appends one position per decode step to every head and applies the
    periodic eviction; no key or value rows are involved.
    """

    def __init__(self, prompt_len, k_keep, recent_r, every, seed, request_id,
                 heads, policy=POLICY_RANDOM, block=1):
        self.policy = int(policy)
        self.block = int(block)
        self.lp = int(prompt_len)
        self.k_keep = int(k_keep)
        self.r = int(recent_r)
        self.every = int(every)
        self.seed = int(seed)
        self.rid = int(request_id)
        self.heads = list(heads)                  # [(layer, kv_head), ...]
        self.step = 0
        self.event = 0
        self.P = {h: np.arange(self.lp, dtype=np.int64) for h in self.heads}
        self.log = []                             # (step, event) per eviction

    def append(self):
        """Decode step: every head caches the new position lp + step."""
        p = self.lp + self.step
        for h in self.heads:
            self.P[h] = np.append(self.P[h], p)
        self.step += 1

    def end_step(self):
        """End-of-step trigger; returns True when an eviction happened."""
        n = self.P[self.heads[0]].shape[0]
        if not eviction_due(self.step, n, self.lp, self.r, self.k_keep,
                            self.every):
            return False
        self.evict_now()
        return True

    def evict_now(self):
        """Apply one eviction event to every head (if anything is evictable)."""
        n = self.P[self.heads[0]].shape[0]
        if n - self.lp - self.r <= self.k_keep:
            return False
        for (layer, g) in self.heads:
            self.P[(layer, g)] = evict_head(self.P[(layer, g)], self.lp,
                                            self.r, self.k_keep, self.seed,
                                            self.rid, self.event, layer, g,
                                            self.policy, self.block)
        self.log.append((self.step, self.event))
        self.event += 1
        return True

    def advance(self, n_steps):
        """Run n_steps decode steps (append then trigger), positions only.

        The trigger can only fire on multiples of ``every``, so the steps in
        between are appended as one run; the result is identical to calling
        ``append`` and ``end_step`` once per step.
        """
        target = self.step + int(n_steps)
        while self.step < target:
            nxt = min(target, (self.step // self.every + 1) * self.every)
            run = np.arange(self.lp + self.step, self.lp + nxt, dtype=np.int64)
            for h in self.heads:
                self.P[h] = np.concatenate([self.P[h], run])
            self.step = nxt
            self.end_step()
