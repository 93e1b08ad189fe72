"""Pins of the observation-window scorer's oracle (measurement only)."""

import numpy as np
import torch

from oracle.window_score import max_pool, window_drop_set, window_scores


def test_single_query_is_softmax_weights():
    rng = np.random.default_rng(0)
    q = rng.standard_normal((1, 64))
    k = rng.standard_normal((30, 64))
    s = window_scores(q, [100], k, np.arange(30))
    logits = torch.from_numpy(k @ q[0] / 8.0)
    assert np.allclose(s, torch.softmax(logits, 0).numpy(), atol=1e-14)


def test_scores_sum_to_query_count_and_respect_the_mask():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((12, 32))
    k = rng.standard_normal((40, 32))
    kpos = np.arange(40) * 2
    qpos = np.arange(12) * 3 + 40
    s = window_scores(q, qpos, k, kpos)
    assert abs(s.sum() - 12) < 1e-12
    # rows after every query's position receive nothing
    assert np.all(s[kpos > qpos.max()] == 0)
    # a row visible to exactly one query gets that query's weight only
    j = np.where(kpos > qpos[-2])[0]
    j = j[kpos[j] <= qpos[-1]]
    sole = window_scores(q[-1:], qpos[-1:], k, kpos)
    assert np.allclose(s[j], sole[j])


def test_max_pool_against_direct_windows():
    rng = np.random.default_rng(2)
    s = rng.random(23)
    p = max_pool(s, 7)
    for j in range(23):
        assert p[j] == max(s[max(0, j - 3):j + 4])
    assert np.array_equal(max_pool(s, 1), s)


def test_drop_set_lowest_with_slot_ties():
    pooled = np.array([0.5, 0.1, 0.1, 0.9, 0.1, 0.3, 7.0])
    assert window_drop_set(pooled, 6, 2).tolist() == [1, 2]
    assert window_drop_set(pooled, 6, 4).tolist() == [1, 2, 4, 5]
