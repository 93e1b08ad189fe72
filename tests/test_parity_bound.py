"""The bf16 attention bound of the GPU parity tests can tell a wrong kernel
from a right one at the full sizes (CPU only; mistakes are planted in the
oracle's output, never on the GPU).

The GPU tests accept a bf16 output element when |got - want| <= 2^-8 |want|
+ floor (one half-ulp of bf16 rounding plus a small floor) besides the
workloads' absolute 2e-2.  On a Qwen3-14B-shaped head at the end of a 32k
generation (9,313 cached rows, scaled keys and values, five query heads of
one group, every row distinct) the correctly rounded exact output passes,
while an output that skips one 32-key block or reads one 32-row block from
the wrong rows fails it for every block tried.  The absolute 2e-2 alone
accepts all of them.
"""

import numpy as np
import pytest
import torch

from gpu_harness import BF16_FLOOR, BF16_HALF_ULP, TOL
from oracle.attention import softmax_attention
from paper_2609_03430_amd import binding as B
from paper_2609_03430_amd.synth import Workload

N, LP, G = 9313, 1024, 5


def _bf16(x):
    return torch.from_numpy(x).float().bfloat16().double().numpy()


def _ratio(got, want):
    return float(np.max(np.abs(got - want) / (BF16_HALF_ULP * np.abs(want) + BF16_FLOOR)))


def _attend(Q, K, V):
    return np.stack([softmax_attention(q, K, V) for q in Q])


@pytest.fixture(scope="module")
def head():
    wl = Workload(1002, 40, 40, 8, 128, torch.bfloat16, True)
    pos = torch.arange(N)
    K = wl.k_rows(3, 17, 5, pos, LP).double().numpy()
    V = wl.v_rows(3, 17, 5, pos, LP).double().numpy()
    Q = wl.q_rows(3, 17, torch.arange(5 * G, 6 * G), 32000).double().numpy()
    return Q, K, V, _attend(Q, K, V)


def test_correct_output_passes(head):
    Q, K, V, want = head
    assert _ratio(_bf16(want), want) <= 1.0
    # one bf16 half-ulp is the most that rounding moves an element
    assert np.all(np.abs(_bf16(want) - want) <= BF16_HALF_ULP * np.abs(want))


@pytest.mark.parametrize("block", [0, 32 * 40, 32 * 150, 32 * 290 - 64])
def test_skipped_key_block_fails(head, block):
    Q, K, V, want = head
    keep = np.r_[0:block, block + 32:N]
    got = _bf16(_attend(Q, K[keep], V[keep]))
    assert np.max(np.abs(got - want)) <= TOL[B.RA_BF16]   # the absolute bound alone passes it
    assert _ratio(got, want) > 1.0


@pytest.mark.parametrize("block", [0, 32 * 77, 32 * 200, 32 * 290 - 64])
def test_wrong_row_gather_fails(head, block):
    Q, K, V, want = head
    K2, V2 = K.copy(), V.copy()
    K2[block:block + 32] = K[block + 32:block + 64]
    V2[block:block + 32] = V[block + 32:block + 64]
    got = _bf16(_attend(Q, K2, V2))
    assert np.max(np.abs(got - want)) <= TOL[B.RA_BF16]
    assert _ratio(got, want) > 1.0
