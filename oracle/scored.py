"""Score-based evictors of the paper's comparison (oracle side).

TEST INFRASTRUCTURE ONLY (see the package header).  These are not Random
Attention: they are the scored rounds whose cost Random Attention avoids,
built to price the selection signal (the eviction-cost comparison).

Section 2 ("Baselines as choices of s") defines the scores; Eq. 1 keeps the
top-scoring candidates.  In these methods the prompt competes with the
generated trace (Figure 1a), so the candidates of a round are every cached
row outside the r most recent, and a round keeps `budget` of them (lp + k_keep
rows, the same count Random Attention keeps).

* SnapKV: the pooled observation-window score (oracle/window_score.py).
* R-KV: s_i = lam * snap_i - (1 - lam) * softmax_i(cbar), cbar_i the mean
  cosine similarity of key i to the other cached keys, its most recent
  near-duplicates not counted.
* VaSE: keep the n_large candidates of largest value range
  (max_j v_ij - min_j v_ij over channels j), then fill the rest of the
  budget by sampling the other candidates without replacement with
  probability proportional to their SnapKV score.

Readings (the paper gives no more detail; each is listed in the design notes):
* R-KV: the cached keys compared with key i are all cached rows (the buffer
  included) other than i; the near-duplicates of i are the rows j with
  cos(k_i, k_j) > threshold; the `recent_dups` of them with the largest
  positions are not counted (their similarity counts as 0); cbar_i is the sum
  over the rest divided by n - 1; the softmax runs over the candidates;
  lam = 0.1, threshold 0.9, recent_dups = 1 by default.
* VaSE: n_large = half the budget by default; the large set is the n_large
  largest (range, position); the proportional fill uses the
  Efraimidis-Spirakis keys log(u_i) / w_i (the largest are kept), u_i in
  (0, 1] taken as ((x >> 11) + 1) * 2^-53 from word (p mod 4) of Philox4x64-10
  at counter (p / 4, e, l, g) with key (seed, request id), w_i the pooled
  SnapKV score; a zero score gives -inf (dropped first).
* Ties everywhere by position: among equal keys the earlier position is
  dropped first.

Parity: pinned by the tests (brute force on tiny inputs; the definition of
the value range on hand-made rows; the Efraimidis-Spirakis inclusion law
against the successive-sampling closed form by chi-square; cosine
properties of duplicated keys).
"""

import numpy as np

from .evict import position_keys


def lowest(keys, positions, m):
    """Indices of the m smallest (key, position) pairs, ascending."""
    order = np.lexsort((np.asarray(positions), np.asarray(keys)))
    return np.sort(order[:m])


def cosine_matrix(K):
    """cos(k_i, k_j) for all pairs, float64."""
    K = np.asarray(K, dtype=np.float64)
    nrm = np.linalg.norm(K, axis=1)
    return (K @ K.T) / np.outer(nrm, nrm)


def rkv_redundancy(K, positions, threshold=0.9, recent_dups=1):
    """cbar_i for every cached row i (see the module readings)."""
    C = cosine_matrix(K)
    n = C.shape[0]
    pos = np.asarray(positions)
    cbar = np.empty(n)
    for i in range(n):
        row = C[i].copy()
        row[i] = 0.0
        dups = [j for j in range(n) if j != i and C[i, j] > threshold]
        dups.sort(key=lambda j: pos[j], reverse=True)
        for j in dups[:recent_dups]:
            row[j] = 0.0
        cbar[i] = row.sum() / (n - 1)
    return cbar


def softmax(x):
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(x - x.max())
    return e / e.sum()


def rkv_scores(snap_pooled, cbar, n_candidates, lam=0.1):
    """R-KV's score of the candidates (rows 0 .. n_candidates - 1)."""
    s = np.asarray(snap_pooled[:n_candidates], dtype=np.float64)
    return lam * s - (1.0 - lam) * softmax(cbar[:n_candidates])


def value_range(V):
    """max_j v_ij - min_j v_ij over the channels of every row, float64."""
    V = np.asarray(V, dtype=np.float64)
    return V.max(axis=1) - V.min(axis=1)


def es_uniform(positions, seed, request_id, event, layer, kv_head):
    """u in (0, 1] from the 64-bit Philox word of each position."""
    x = position_keys(positions, seed, request_id, event, layer, kv_head)
    return ((x >> np.uint64(11)).astype(np.float64) + 1.0) * 2.0 ** -53


def es_keys(u, w):
    """Efraimidis-Spirakis keys log(u) / w (largest kept); w = 0 gives -inf."""
    u = np.asarray(u, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    with np.errstate(divide="ignore"):
        return np.where(w > 0, np.log(u) / np.where(w > 0, w, 1.0), -np.inf)


def vase_drops(vrange, snap_pooled, positions, n_candidates, budget, n_large, u):
    """Rows dropped by one VaSE round (indices into the candidates).

    The n_large largest (range, position) candidates are kept; the other
    candidates compete for budget - n_large places by the keys log(u)/w.
    """
    pos = np.asarray(positions[:n_candidates])
    rng_ = np.asarray(vrange[:n_candidates], dtype=np.float64)
    m = n_candidates - budget
    if m <= 0:
        return np.zeros(0, dtype=np.int64)
    small = lowest(rng_, pos, n_candidates - n_large)     # not in the large set
    keys = es_keys(np.asarray(u)[small], np.asarray(snap_pooled)[small])
    # -inf keys rank below every finite key; map them to a key below the min
    finite = np.isfinite(keys)
    floor = (keys[finite].min() - 1.0) if finite.any() else -1.0
    keys = np.where(finite, keys, floor)
    return np.sort(small[lowest(keys, pos[small], m)])
