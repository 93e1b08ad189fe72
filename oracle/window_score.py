"""Observation-window attention score of a score-based evictor (oracle side).

TEST INFRASTRUCTURE ONLY (see the package header).  This is not part of
Random Attention: it is the scoring pass that Random Attention removes, timed
for comparison on the ragged Phi-4-shaped workload.

Section 2 ("Baselines as choices of s") gives SnapKV's score of a cached
position as the sum of the attention weights that the last w queries give
it, max-pooled over neighbouring positions; Eq. 1 then keeps the top-scoring
candidates, the candidates being every cached position outside the buffer of
the r most recent.

Readings (the paper gives no more detail):
* w = 64, the window of the measured workload; the queries are those of the
  last 64 decode steps of every query head of the KV head's group, so a KV
  head's score sums over G * 64 queries;
* the weights are recomputed at eviction time against the current cache,
  each window query seeing only the cached positions at or before its own
  (causal mask by position), softmax over q.k / sqrt(d);
* max-pooling over a window of 7 neighbouring cached rows, clipped at the
  ends of the cache;
* candidates are cached rows 0 .. len - r - 1 (the prompt competes, as in
  Eq. 1 for a scored policy); the number dropped is the same m as Random
  Attention drops at the same event; ties are broken by slot, lower first.

Parity: pinned by the tests (a single query reproduces plain softmax
attention weights; every query's weights sum to one, so the scores sum to the
number of queries; the mask; pooling against a direct loop).
"""

import numpy as np


def window_scores(Qw, qpos, K, kpos):
    """Sum over window queries of their attention weights on each cached row.

    Qw: [nq, d] queries; qpos: [nq] their positions; K: [N, d] cached keys;
    kpos: [N] their positions.  Returns [N] float64.
    """
    Qw = np.asarray(Qw, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    d = Qw.shape[1]
    logits = (Qw @ K.T) / np.sqrt(d)
    visible = np.asarray(kpos)[None, :] <= np.asarray(qpos)[:, None]
    logits = np.where(visible, logits, -np.inf)
    logits = logits - logits.max(axis=1, keepdims=True)
    w = np.where(visible, np.exp(logits), 0.0)
    w = w / w.sum(axis=1, keepdims=True)
    return w.sum(axis=0)


def max_pool(s, kernel=7):
    """out[j] = max(s[j - kernel//2 .. j + kernel//2]), clipped at the ends."""
    s = np.asarray(s, dtype=np.float64)
    half = kernel // 2
    n = s.shape[0]
    return np.array([s[max(0, j - half):min(n, j + half + 1)].max() for j in range(n)])


def window_drop_set(pooled, n_candidates, m):
    """Slots of the m lowest (pooled score, slot) among slots 0..n_candidates-1."""
    pooled = np.asarray(pooled[:n_candidates])
    order = np.lexsort((np.arange(n_candidates), pooled))
    return np.sort(order[:m])
