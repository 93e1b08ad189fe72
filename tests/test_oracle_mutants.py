"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of an oracle function -- a wrong
selection direction or tie order, a dropped term, a wrong index or counter
field, a transposed axis -- on the CPU, and runs the pins that should see it:
at least one of them must fail.  The oracle itself is untouched (pytest's
monkeypatch restores every name after the case).
"""

import sys

import numpy as np
import pytest

import oracle.attention as att
import oracle.evict as ev
import oracle.scored as sc
import oracle.window_score as ws
from oracle.philox import philox4x64_10_np

import test_oracle_attention as pin_att
import test_oracle_evict as pin_ev
import test_oracle_philox as pin_philox
import test_oracle_policies as pin_pol
import test_oracle_scored as pin_sc
import test_oracle_window as pin_ws


def plant(monkeypatch, module, name, fn):
    """Replace module.name, and every pin module's imported copy of it."""
    orig = getattr(module, name)
    monkeypatch.setattr(module, name, fn)
    for m in list(sys.modules.values()):
        if getattr(m, "__name__", "").startswith("test_oracle") and getattr(m, name, None) is orig:
            monkeypatch.setattr(m, name, fn)


def failing(pins):
    """Names of the pins (callables) that fail (any exception: a pin that
    cannot even complete has not passed)."""
    out = []
    for pin in pins:
        try:
            pin()
        except Exception:            # noqa: BLE001 -- every failure counts
            out.append(getattr(pin, "__name__", repr(pin)))
    return out


def _brute_force_pins():
    return [lambda t=t: pin_ev.test_drop_set_matches_brute_force(t) for t in range(12)]


def _invariant_pins():
    return [lambda a=a: pin_ev.test_invariants_every_event(*a)
            for a in [(0, 8, 4, 4), (5, 20, 8, 8), (12, 64, 16, 16)]]


def _evict_head_variant(cand_of):
    """evict_head with the candidate slice [lo, hi) = cand_of(n, lp, r)."""
    def evict_head(P, prompt_len, recent_r, k_keep, seed, request_id, event,
                   layer, kv_head, policy=ev.POLICY_RANDOM, block=1):
        P = np.asarray(P, dtype=np.int64)
        lo, hi = cand_of(P.shape[0], prompt_len, recent_r)
        cand = P[lo:hi]
        m = cand.shape[0] - k_keep
        if m <= 0:
            return P.copy()
        keys = ev.policy_keys(policy, cand, prompt_len, seed, request_id, event,
                              layer, kv_head, block)
        keep = np.ones(cand.shape[0], dtype=bool)
        keep[ev.drop_set(cand, keys, m)] = False
        return np.concatenate([P[:lo], cand[keep], P[hi:]])
    return evict_head


MUTANTS = {
    # selection
    "drop the largest keys": (ev, "drop_set",
        lambda c, k, m: np.sort(np.lexsort((np.asarray(c), k))[::-1][:m]), _brute_force_pins),
    "ties drop the later position": (ev, "drop_set",
        lambda c, k, m: np.sort(np.lexsort((-np.asarray(c), k))[:m]), _brute_force_pins),
    # the key of a position
    "layer and KV head swapped in the counter": (ev, "position_keys",
        lambda p, s, rid, e, l, g: pin_philox_free_keys(p, s, rid, e, g, l),
        lambda: [lambda t=t: pin_philox.test_position_keys_follow_the_counter_layout(t)
                 for t in range(3)]),
    "counter p / 2 instead of p / 4": (ev, "position_keys",
        lambda p, s, rid, e, l, g: pin_philox_free_keys(p, s, rid, e, l, g, shift=1),
        lambda: [lambda t=t: pin_philox.test_position_keys_follow_the_counter_layout(t)
                 for t in range(3)]),
    "seed and request id swapped in the key": (ev, "position_keys",
        lambda p, s, rid, e, l, g: pin_philox_free_keys(p, rid, s, e, l, g),
        lambda: [lambda t=t: pin_philox.test_position_keys_follow_the_counter_layout(t)
                 for t in range(3)]),
    # the candidate set
    "recent buffer among the candidates": (ev, "evict_head",
        _evict_head_variant(lambda n, lp, r: (lp, n)), _invariant_pins),
    "prompt among the candidates": (ev, "evict_head",
        _evict_head_variant(lambda n, lp, r: (0, n - r)), _invariant_pins),
    "candidates one short of the buffer": (ev, "evict_head",
        _evict_head_variant(lambda n, lp, r: (lp, n - r - 1)), _invariant_pins),
    # trigger and budget
    "trigger one step early": (ev, "eviction_due",
        lambda step, n, lp, r, k, every: (step + 1) % every == 0 and n - lp - r > k,
        lambda: [pin_ev.test_trigger_schedule_tiny_case]),
    "TOTAL budget off by one": (ev, "keep_count",
        lambda K, lp, mode: int(K) if mode == ev.BUDGET_EVICTABLE else int(K) - int(lp) + 1,
        lambda: [pin_ev.test_budget_modes]),
    # attention
    "no 1/sqrt(d) scale": (att, "softmax_attention",
        lambda q, K, V: _softmax_attention(q, K, V, scale=False),
        lambda: [lambda n=n: pin_att.test_matches_torch_sdpa_float64(n) for n in (2, 31)]),
    "weights not normalised": (att, "softmax_attention",
        lambda q, K, V: _softmax_attention(q, K, V, normalise=False),
        lambda: [pin_att.test_equal_keys_give_mean_value, pin_att.test_zero_query_gives_mean_value]),
    "GQA map h mod Hkv": (att, "gqa_decode",
        lambda q, Ks, Vs: np.stack([att.softmax_attention(q[h], Ks[h % len(Ks)], Vs[h % len(Ks)])
                                    for h in range(np.asarray(q).shape[0])]),
        lambda: [pin_att.test_gqa_map_contiguous_groups]),
    # policies
    "shared draw keeps the layer": (ev, "policy_keys",
        lambda policy, cand, lp, s, rid, e, l, g, block=1: (
            ev.position_keys(np.asarray(cand, dtype=np.int64), s, rid, e, l, 0)
            if policy == ev.POLICY_SHARED else
            _policy_keys_orig(policy, cand, lp, s, rid, e, l, g, block)),
        lambda: [pin_pol.test_shared_draw_same_set_in_every_head]),
    "blocks aligned at position 0": (ev, "policy_keys",
        lambda policy, cand, lp, s, rid, e, l, g, block=1: (
            ev.position_keys(np.asarray(cand, dtype=np.int64) // block * block, s, rid, e, l, g)
            if policy == ev.POLICY_BLOCK else
            _policy_keys_orig(policy, cand, lp, s, rid, e, l, g, block)),
        lambda: [lambda a=a: pin_pol.test_block_drops_whole_aligned_blocks(*a)
                 for a in [(5, 4, 40, 8, 8), (3, 8, 64, 16, 16)]]),
    # observation-window scorer
    "no causal mask": (ws, "window_scores",
        lambda Qw, qpos, K, kpos: _window_scores_unmasked(Qw, K),
        lambda: [pin_ws.test_scores_sum_to_query_count_and_respect_the_mask]),
    "max-pool over 5 rows": (ws, "max_pool",
        lambda s, kernel=7: _max_pool_orig(s, max(1, kernel - 2)),
        lambda: [pin_ws.test_max_pool_against_direct_windows]),
    # scored evictors
    "fill keys log(u) * w": (sc, "es_keys",
        lambda u, w: np.where(np.asarray(w) > 0, np.log(np.asarray(u, dtype=np.float64))
                              * np.asarray(w, dtype=np.float64), -np.inf),
        lambda: [pin_sc.test_es_single_draw_is_proportional]),
    "redundancy divided by n": (sc, "rkv_redundancy",
        lambda K, pos, threshold=0.9, recent_dups=1: _rkv_orig(K, pos, threshold, recent_dups)
        * (np.asarray(K).shape[0] - 1) / np.asarray(K).shape[0],
        lambda: [pin_sc.test_redundancy_closed_form_three_copies]),
    "value range over the rows": (sc, "value_range",
        lambda V: np.asarray(V, dtype=np.float64).max(axis=0)[:np.asarray(V).shape[0]]
        - np.asarray(V, dtype=np.float64).min(axis=0)[:np.asarray(V).shape[0]],
        lambda: [pin_sc.test_value_range_hand_rows]),
}

_policy_keys_orig = ev.policy_keys
_max_pool_orig = ws.max_pool
_rkv_orig = sc.rkv_redundancy


def pin_philox_free_keys(positions, seed, rid, event, layer, head, shift=2):
    """position_keys written out again with its arguments as given."""
    p = np.asarray(positions, dtype=np.uint64)
    words = philox4x64_10_np(p >> np.uint64(shift), event, layer, head, seed, rid)
    return np.choose((p & np.uint64(3)).astype(np.int64), words)


def _softmax_attention(q, K, V, scale=True, normalise=True):
    q, K, V = (np.asarray(x, dtype=np.float64) for x in (q, K, V))
    logits = K @ q
    if scale:
        logits = logits / np.sqrt(q.shape[-1])
    w = np.exp(logits - logits.max())
    if normalise:
        w = w / w.sum()
    return w @ V


def _window_scores_unmasked(Qw, K):
    Qw, K = np.asarray(Qw, dtype=np.float64), np.asarray(K, dtype=np.float64)
    logits = (Qw @ K.T) / np.sqrt(Qw.shape[1])
    w = np.exp(logits - logits.max(axis=1, keepdims=True))
    return (w / w.sum(axis=1, keepdims=True)).sum(axis=0)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(name, monkeypatch):
    module, attr, fn, pins = MUTANTS[name]
    plant(monkeypatch, module, attr, fn)
    failed = failing(pins())
    assert failed, "no pin caught the planted mistake: %s" % name


def test_unplanted_oracle_passes_the_same_pins():
    """The pins used above pass on the oracle as written."""
    for name in sorted(MUTANTS):
        assert failing(MUTANTS[name][3]()) == [], name
