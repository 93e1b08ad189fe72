"""Pins of the oracle's softmax attention (Section 2, "Notation").

Special cases with closed forms, permutation invariance, the GQA map, and a
cross-check against an independent library routine
(torch.nn.functional.scaled_dot_product_attention in float64 on the CPU).
"""

import numpy as np
import pytest
import torch

from oracle.attention import gqa_decode, softmax_attention
from oracle.decode import run_decode
from oracle.evict import SequenceReplay


def test_single_row_returns_its_value():
    rng = np.random.default_rng(0)
    v = rng.standard_normal((1, 128))
    o = softmax_attention(rng.standard_normal(128), rng.standard_normal((1, 128)), v)
    assert np.allclose(o, v[0], rtol=0, atol=1e-15)


def test_equal_keys_give_mean_value():
    rng = np.random.default_rng(1)
    k = np.tile(rng.standard_normal(128), (37, 1))
    v = rng.standard_normal((37, 128))
    o = softmax_attention(rng.standard_normal(128), k, v)
    assert np.allclose(o, v.mean(0), atol=1e-13)


def test_zero_query_gives_mean_value():
    rng = np.random.default_rng(2)
    v = rng.standard_normal((50, 64))
    o = softmax_attention(np.zeros(64), rng.standard_normal((50, 64)), v)
    assert np.allclose(o, v.mean(0), atol=1e-13)


def test_dominant_logit_selects_its_value():
    rng = np.random.default_rng(3)
    k = rng.standard_normal((20, 128)) * 0.01
    q = np.zeros(128)
    q[0] = 1.0
    k[7, 0] = 2000.0                      # logit 2000/sqrt(128) ~ 177
    v = rng.standard_normal((20, 128))
    assert np.allclose(softmax_attention(q, k, v), v[7], atol=1e-12)


def test_permutation_invariance():
    rng = np.random.default_rng(4)
    q, k, v = rng.standard_normal(128), rng.standard_normal((90, 128)), rng.standard_normal((90, 128))
    perm = rng.permutation(90)
    assert np.allclose(softmax_attention(q, k, v), softmax_attention(q, k[perm], v[perm]), atol=1e-13)


@pytest.mark.parametrize("n", [1, 2, 31, 300, 2049])
def test_matches_torch_sdpa_float64(n):
    rng = np.random.default_rng(n)
    q = rng.standard_normal(128)
    k = rng.standard_normal((n, 128)) * rng.uniform(0.5, 2, 128)
    v = rng.standard_normal((n, 128)) * rng.uniform(0.5, 2, 128)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).view(1, 1, 1, 128), torch.from_numpy(k).view(1, 1, n, 128),
        torch.from_numpy(v).view(1, 1, n, 128)).view(128).numpy()
    assert np.allclose(softmax_attention(q, k, v), ref, rtol=0, atol=1e-12)


def test_gqa_map_contiguous_groups():
    rng = np.random.default_rng(5)
    Ks = [rng.standard_normal((10 + g, 16)) for g in range(3)]
    Vs = [rng.standard_normal((10 + g, 16)) for g in range(3)]
    q = rng.standard_normal((12, 16))
    out = gqa_decode(q, Ks, Vs)
    for h in range(12):
        g = h // 4
        assert np.allclose(out[h], softmax_attention(q[h], Ks[g], Vs[g]))


def test_decode_loop_composes_parts():
    """The decode loop equals an explicit replay plus per-step attention:
    before the first event every position is attended; after it, exactly
    the replayed kept set plus the new position."""
    rng = np.random.default_rng(6)
    L, Hq, Hkv, d, lp = 2, 4, 2, 16, 5
    table_k = rng.standard_normal((L, Hkv, 400, d))
    table_v = rng.standard_normal((L, Hkv, 400, d))
    table_q = rng.standard_normal((L, 400, Hq, d))
    qf = lambda l, s: table_q[l, s]
    kf = lambda l, g, P: table_k[l, g, P]
    vf = lambda l, g, P: table_v[l, g, P]
    outs, rep = run_decode(L, Hq, Hkv, lp, 60, 12, 4, 8, 9, 2, qf, kf, vf)
    # step index 0: cache = prompt + position lp
    P0 = np.arange(lp + 1)
    ref0 = gqa_decode(table_q[1, 0], [table_k[1, g, P0] for g in range(Hkv)],
                      [table_v[1, g, P0] for g in range(Hkv)])
    assert np.allclose(outs[0][1], ref0)
    # replay separately and check the last step's attended set
    rep2 = SequenceReplay(lp, 12, 4, 8, 9, 2, [(l, g) for l in range(L) for g in range(Hkv)])
    rep2.advance(59)
    rep2.append()
    ref = gqa_decode(table_q[0, 59], [table_k[0, g, rep2.P[(0, g)]] for g in range(Hkv)],
                     [table_v[0, g, rep2.P[(0, g)]] for g in range(Hkv)])
    assert np.allclose(outs[59][0], ref)
    rep2.end_step()
    for h in rep.P:
        assert np.array_equal(rep.P[h], rep2.P[h])
