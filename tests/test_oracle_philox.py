"""Pins of the oracle's Philox4x64-10 against an independent implementation.

numpy ships Philox4x64-10 (``numpy.random.Philox``), written from the same
published definition (Salmon et al., SC'11).  numpy increments its 256-bit
counter before producing a block, so its first four raw outputs from counter
c are the block at c + 1 (established empirically, checked here).
"""

import numpy as np
import pytest

from oracle.philox import philox4x64_10, philox4x64_10_np

_MASK = (1 << 64) - 1


def _numpy_block(counter, key):
    """Block at ``counter`` from numpy's generator (undo its pre-increment)."""
    c = sum(int(w) << (64 * i) for i, w in enumerate(counter))
    c = (c - 1) % (1 << 256)
    words = [(c >> (64 * i)) & _MASK for i in range(4)]
    # uint64 arrays: numpy would round Python ints above 2^53 through float
    gen = np.random.Philox(counter=np.array(words, dtype=np.uint64),
                           key=np.array([int(k) for k in key], dtype=np.uint64))
    return tuple(int(x) for x in gen.random_raw(4))


def test_zero_block_matches_numpy():
    assert philox4x64_10((0, 0, 0, 0), (0, 0)) == _numpy_block((0, 0, 0, 0), (0, 0))


@pytest.mark.parametrize("trial", range(40))
def test_scalar_matches_numpy(trial):
    rng = np.random.default_rng(1234 + trial)
    ctr = [int(x) for x in rng.integers(0, 2**63, 4, dtype=np.uint64) * 2
           + rng.integers(0, 2, 4, dtype=np.uint64)]
    key = [int(x) for x in rng.integers(0, 2**63, 2, dtype=np.uint64) * 2 + 1]
    if trial % 4 == 0:                     # small counters like the sampler's
        ctr = [trial * 97, trial % 5, trial % 3, trial % 7]
    assert philox4x64_10(ctr, key) == _numpy_block(ctr, key)


def test_vectorised_matches_scalar():
    rng = np.random.default_rng(7)
    n = 257
    c = rng.integers(0, 2**63, (4, n), dtype=np.uint64) * np.uint64(2)
    k0 = rng.integers(0, 2**63, n, dtype=np.uint64)
    k1 = rng.integers(0, 2**63, n, dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    out = philox4x64_10_np(c[0], c[1], c[2], c[3], k0, k1)
    for i in range(n):
        ref = philox4x64_10([c[j, i] for j in range(4)], [k0[i], k1[i]])
        assert tuple(int(o[i]) for o in out) == ref


def test_vectorised_broadcasts_scalars():
    out = philox4x64_10_np(np.arange(5, dtype=np.uint64), 3, 2, 1, 99, 2**63 + 5)
    for i in range(5):
        assert tuple(int(o[i]) for o in out) == philox4x64_10((i, 3, 2, 1), (99, 2**63 + 5))


@pytest.mark.parametrize("trial", range(6))
def test_position_keys_follow_the_counter_layout(trial):
    """The key of position p at event e, layer l, KV head g of request
    (seed, request id) is word p mod 4 of the Philox4x64-10 block at counter
    (p / 4, e, l, g) under key (seed, request id): checked word by word
    against numpy's generator, so a wrong counter field, key order or word
    choice fails here (the uniformity pins cannot see such a mistake)."""
    from oracle.evict import position_keys
    rng = np.random.default_rng(99 + trial)
    seed = int(rng.integers(0, 2**63)) * 2 + trial % 2
    rid = int(rng.integers(0, 2**40))
    event, layer, head = int(rng.integers(0, 500)), int(rng.integers(0, 64)), int(rng.integers(0, 16))
    p = np.sort(rng.choice(40000, 24, replace=False))
    got = position_keys(p, seed, rid, event, layer, head)
    for pi, key in zip(p.tolist(), got.tolist()):
        block = _numpy_block((pi // 4, event, layer, head), (seed, rid))
        assert key == block[pi % 4], (pi, event, layer, head)
