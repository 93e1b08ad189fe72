"""Pins of the oracle's score-based evictors (R-KV, VaSE; measurement only).

Section 2 gives the scores; what they fix is pinned here: brute-force
selection with ties, closed forms of the redundancy term on duplicated keys,
the limits of the R-KV mix, the value range on hand-made rows, and the
Efraimidis-Spirakis proportional fill against the successive-sampling law
(chi-square).
"""

import itertools

import numpy as np
import pytest
from scipy import stats

from oracle.scored import (cosine_matrix, es_keys, es_uniform, lowest, rkv_redundancy,
                           rkv_scores, softmax, value_range, vase_drops)


@pytest.mark.parametrize("trial", range(30))
def test_lowest_matches_brute_force(trial):
    rng = np.random.default_rng(trial)
    n = int(rng.integers(1, 8))
    m = int(rng.integers(0, n + 1))
    keys = rng.integers(0, 3, n).astype(float)
    pos = np.sort(rng.choice(100, n, replace=False))
    got = set(lowest(keys, pos, m).tolist())
    rank = lambda i: (keys[i], pos[i])
    found = [set(s) for s in itertools.combinations(range(n), m)
             if all(rank(a) < rank(b) for a in s for b in range(n) if b not in s)]
    assert found == [got]


def test_cosine_of_duplicates_and_orthogonal_rows():
    K = np.array([[1.0, 2, 0, 0], [2.0, 4, 0, 0], [0, 0, 3.0, 0], [-1.0, -2, 0, 0]])
    C = cosine_matrix(K)
    assert np.allclose(np.diag(C), 1)
    assert abs(C[0, 1] - 1) < 1e-15 and abs(C[0, 2]) < 1e-15 and abs(C[0, 3] + 1) < 1e-15


def _three_copies(n_other=5):
    """Rows 0, 2, 5 hold the same key (positions 10, 12, 15); the others are
    mutually orthogonal to it and to each other."""
    n = 3 + n_other
    K = np.zeros((n, n + 1))
    copies = [0, 2, 5]
    for i in copies:
        K[i, 0] = 1.0
    others = [i for i in range(n) if i not in copies]
    for c, i in enumerate(others):
        K[i, c + 1] = 1.0
    pos = 10 + np.arange(n)
    return K, pos, copies, others


def test_redundancy_closed_form_three_copies():
    K, pos, copies, others = _three_copies()
    n = K.shape[0]
    # no exclusion: each copy sees the other two copies
    c0 = rkv_redundancy(K, pos, threshold=0.9, recent_dups=0)
    assert np.allclose(c0[copies], 2 / (n - 1)) and np.allclose(c0[others], 0)
    # the most recent near-duplicate is not counted: each copy sees one
    c1 = rkv_redundancy(K, pos, threshold=0.9, recent_dups=1)
    assert np.allclose(c1[copies], 1 / (n - 1)) and np.allclose(c1[others], 0)
    # which one is skipped: for the oldest copy it is the newest one, so
    # moving the newest copy's key elsewhere changes nothing for it
    K2 = K.copy()
    K2[5] = 0
    K2[5, -1] = 1.0
    c2 = rkv_redundancy(K2, pos, threshold=0.9, recent_dups=1)
    assert np.isclose(c2[0], 0) and np.isclose(c2[2], 0)     # one duplicate left, skipped
    c3 = rkv_redundancy(K2, pos, threshold=0.9, recent_dups=0)
    assert np.isclose(c3[0], 1 / (n - 1)) and np.isclose(c3[2], 1 / (n - 1))


def test_redundancy_counts_dissimilar_keys_fully():
    rng = np.random.default_rng(3)
    K = rng.standard_normal((9, 16))
    C = cosine_matrix(K)
    want = (C.sum(axis=1) - 1.0) / 8                   # nothing above 0.99
    assert np.all(np.abs(C - np.eye(9)) < 0.99)
    assert np.allclose(rkv_redundancy(K, np.arange(9), threshold=0.99, recent_dups=2), want)


def test_rkv_mix_limits():
    rng = np.random.default_rng(4)
    snap = rng.random(12)
    cbar = rng.standard_normal(12)
    assert np.allclose(rkv_scores(snap, cbar, 10, lam=1.0), snap[:10])
    assert np.allclose(rkv_scores(snap, cbar, 10, lam=0.0), -softmax(cbar[:10]))
    assert abs(softmax(cbar[:10]).sum() - 1) < 1e-15


def test_value_range_hand_rows():
    V = np.array([[0.5, -1.0, 2.0, 0.0], [3.0, 3.0, 3.0, 3.0], [-4.0, -2.0, -8.0, -1.0]])
    assert np.array_equal(value_range(V), [3.0, 0.0, 7.0])


def test_es_uniform_range_and_resolution():
    u = es_uniform(np.arange(4000), 5, 6, 0, 1, 2)
    assert np.all(u > 0) and np.all(u <= 1)
    assert abs(u.mean() - 0.5) < 0.02
    assert len(np.unique(u)) == 4000


def test_es_single_draw_is_proportional():
    """Keep 1 of 4 with weights 1:2:3:4: P(i) = w_i / 10 (chi-square)."""
    w = np.array([1.0, 2.0, 3.0, 4.0])
    S = 20000
    counts = np.zeros(4)
    for s in range(S):
        u = es_uniform(np.arange(4), s, 1, 0, 0, 0)
        counts[np.argmax(es_keys(u, w))] += 1
    assert stats.chisquare(counts, S * w / w.sum()).pvalue > 1e-3


def test_es_two_draws_follow_successive_sampling():
    """Keep 2 of 4: P({i, j}) = w_i/W w_j/(W-w_i) + w_j/W w_i/(W-w_j)."""
    w = np.array([1.0, 2.0, 3.0, 4.0])
    W = w.sum()
    S = 20000
    pairs = list(itertools.combinations(range(4), 2))
    law = np.array([w[i] / W * w[j] / (W - w[i]) + w[j] / W * w[i] / (W - w[j])
                    for i, j in pairs])
    assert abs(law.sum() - 1) < 1e-12
    counts = dict.fromkeys(pairs, 0)
    for s in range(S):
        u = es_uniform(np.arange(4), s, 2, 0, 0, 0)
        kept = tuple(sorted(np.argsort(es_keys(u, w))[-2:].tolist()))
        counts[kept] += 1
    obs = np.array([counts[p] for p in pairs])
    assert stats.chisquare(obs, S * law).pvalue > 1e-3


def test_vase_keeps_the_large_set_and_fills_by_score():
    rng = np.random.default_rng(7)
    n, budget, n_large = 20, 12, 5
    vr = rng.permutation(n).astype(float)           # distinct ranges
    snap = rng.random(n) + 0.1
    snap[3] = 0.0                                    # never sampled
    pos = 100 + np.arange(n)
    u = es_uniform(pos, 11, 0, 0, 0, 0)
    d = vase_drops(vr, snap, pos, n, budget, n_large, u)
    assert d.shape[0] == n - budget
    large = np.argsort(vr)[-n_large:]
    assert not set(d.tolist()) & set(large.tolist())
    rest = np.setdiff1d(np.arange(n), large)
    keys = es_keys(u[rest], snap[rest])
    assert 3 in d                                     # zero score goes first
    thr = np.sort(keys)[n - budget - 1]
    kept_rest = np.setdiff1d(rest, d)
    assert np.all(es_keys(u[d], snap[d]) <= thr)
    assert np.all(es_keys(u[kept_rest], snap[kept_rest]) >= thr)


def test_vase_fill_is_proportional_over_seeds():
    """No large set, keep 1 of 3 with scores 1:1:2 -> kept 1/4, 1/4, 1/2."""
    snap = np.array([1.0, 1.0, 2.0])
    pos = np.arange(3)
    S = 12000
    counts = np.zeros(3)
    for s in range(S):
        u = es_uniform(pos, s, 3, 0, 0, 0)
        d = vase_drops(np.zeros(3), snap, pos, 3, 1, 0, u)
        counts[np.setdiff1d(pos, d)] += 1
    assert stats.chisquare(counts, S * snap / snap.sum()).pvalue > 1e-3
