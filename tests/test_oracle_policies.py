"""Pins of the oracle's diagnostic eviction policies (Sections 4.1 and 5,
Appendix D): shared draw, block-wise and recency + prompt.

Each policy changes only the key that Eq. 1 ranks; the pins check what the
paper's description fixes: recency keeps exactly the prompt and a contiguous
recent window (closed form); the shared draw keeps one set for every head and
that set is still a uniform subset; block-wise eviction drops whole blocks
(aligned at the end of the prompt) chosen uniformly, and with blocks of one
token it is Random Attention itself.
"""

import itertools

import numpy as np
import pytest
from scipy import stats

from oracle.evict import (POLICY_BLOCK, POLICY_RANDOM, POLICY_RECENCY,
                          POLICY_SHARED, SequenceReplay, evict_head)

HEADS = [(0, 0), (0, 1), (1, 0), (3, 2)]


def _replay(policy, lp, k, r, every, steps, seed=21, block=1, heads=HEADS):
    rep = SequenceReplay(lp, k, r, every, seed, 4, heads, policy=policy,
                         block=block)
    snaps = []
    for _ in range(steps):
        rep.append()
        if rep.end_step():
            snaps.append({h: rep.P[h].copy() for h in heads})
    return rep, snaps


@pytest.mark.parametrize("policy,block", [(POLICY_SHARED, 1), (POLICY_BLOCK, 4),
                                          (POLICY_BLOCK, 64), (POLICY_RECENCY, 1)])
@pytest.mark.parametrize("lp,k,r,every", [(0, 16, 8, 8), (5, 40, 4, 4),
                                           (13, 64, 16, 16), (7, 9, 3, 1)])
def test_policy_invariants(policy, block, lp, k, r, every):
    """Prompt pinned, buffer kept, monotone, back to budget -- as for Random
    Attention (Appendix F), since only the key differs."""
    rep = SequenceReplay(lp, k, r, every, 3, 1, HEADS, policy=policy, block=block)
    prev = {h: set(range(lp)) for h in HEADS}
    for _ in range(300):
        rep.append()
        newest = lp + rep.step - 1
        fired = rep.end_step()
        for h in HEADS:
            P = rep.P[h]
            assert np.all(np.diff(P) > 0)
            assert set(range(lp)) <= set(P.tolist())
            assert set(range(max(lp, newest - r + 1), newest + 1)) <= set(P.tolist())
            assert set(P.tolist()) <= prev[h] | {newest}
            prev[h] = set(P.tolist())
            if fired:
                assert P.shape[0] == lp + k + r


# --- recency + prompt -------------------------------------------------------

@pytest.mark.parametrize("lp,k,r,every", [(0, 32, 8, 8), (9, 50, 16, 16),
                                           (4, 7, 2, 1), (30, 0, 4, 4)])
def test_recency_is_prompt_plus_recent_window(lp, k, r, every):
    """Section 4.1: the cache is the prompt plus a contiguous recent window;
    after an event that window is exactly the last k + r positions."""
    _, snaps = _replay(POLICY_RECENCY, lp, k, r, every, 400)
    assert snaps
    rep, _ = _replay(POLICY_RECENCY, lp, k, r, every, 400, seed=999)
    for h in HEADS:
        P = rep.P[h]
        tail = P[lp:]
        assert np.array_equal(P[:lp], np.arange(lp))
        assert np.all(np.diff(tail) == 1)               # contiguous window
        assert tail[-1] == lp + rep.step - 1
    rep2, snaps2 = _replay(POLICY_RECENCY, lp, k, r, every, 400)
    for snap in snaps2:
        for h in HEADS:
            P = snap[h]
            assert P.shape[0] == lp + k + r
            assert np.array_equal(P[lp:], np.arange(P[-1] - k - r + 1, P[-1] + 1))


def test_recency_ignores_seed_and_head():
    a, _ = _replay(POLICY_RECENCY, 6, 20, 8, 8, 200, seed=1)
    b, _ = _replay(POLICY_RECENCY, 6, 20, 8, 8, 200, seed=2)
    for h in HEADS:
        assert np.array_equal(a.P[h], b.P[h])
        assert np.array_equal(a.P[h], a.P[HEADS[0]])


# --- shared draw -------------------------------------------------------------

def test_shared_draw_same_set_in_every_head():
    """Section 5 / Appendix D control: the same random positions in every
    head -- and that set is the one Random Attention draws for (0, 0)."""
    rep, snaps = _replay(POLICY_SHARED, 11, 48, 16, 16, 500)
    rnd, _ = _replay(POLICY_RANDOM, 11, 48, 16, 16, 500)
    assert len(snaps) >= 5
    for snap in snaps:
        for h in HEADS:
            assert np.array_equal(snap[h], snap[HEADS[0]])
    assert np.array_equal(rep.P[(0, 0)], rnd.P[(0, 0)])
    # Random Attention's heads differ from each other (independent draws)
    assert not np.array_equal(rnd.P[(0, 1)], rnd.P[(0, 0)])


def _one_event_sets(policy, C, k, seeds, layer, head, block=1, lp=0):
    P = np.arange(lp + C + 1)
    return [tuple(evict_head(P, lp, 1, k, int(s), 11, 0, layer, head, policy,
                             block)[lp:lp + k].tolist()) for s in seeds]


def test_shared_draw_subset_law_and_full_dependence():
    """C=6, keep 3: every 3-subset equally likely (the draw is still
    uniform), and two heads always agree (no cross-head independence)."""
    S = 20000
    a = _one_event_sets(POLICY_SHARED, 6, 3, range(S), 0, 0)
    b = _one_event_sets(POLICY_SHARED, 6, 3, range(S), 2, 5)
    assert a == b
    cells = {s: 0 for s in itertools.combinations(range(6), 3)}
    for s in a:
        cells[s] += 1
    assert stats.chisquare(np.array(list(cells.values()))).pvalue > 1e-3


# --- block-wise --------------------------------------------------------------

def test_block_size_one_is_random_attention():
    for lp in (0, 7):
        a, _ = _replay(POLICY_BLOCK, lp, 40, 8, 8, 300, block=1)
        b, _ = _replay(POLICY_RANDOM, lp, 40, 8, 8, 300)
        for h in HEADS:
            assert np.array_equal(a.P[h], b.P[h])


@pytest.mark.parametrize("lp,B,k,r,every", [(5, 4, 40, 8, 8), (0, 16, 64, 16, 16),
                                             (13, 64, 128, 64, 64), (3, 3, 10, 5, 1)])
def test_block_drops_whole_aligned_blocks(lp, B, k, r, every):
    """At every event the dropped positions are whole blocks (aligned at the
    end of the prompt), except at most one block that loses only its
    earliest candidates."""
    rep = SequenceReplay(lp, k, r, every, 8, 2, HEADS, policy=POLICY_BLOCK, block=B)
    checked = 0
    for _ in range(600):
        rep.append()
        before = {h: rep.P[h].copy() for h in HEADS}
        if not rep.end_step():
            continue
        n = before[HEADS[0]].shape[0]
        for h in HEADS:
            cand = before[h][lp:n - r]
            dropped = np.setdiff1d(cand, rep.P[h])
            blocks = (cand - lp) // B
            partial = 0
            for b in np.unique((dropped - lp) // B):
                in_block = cand[blocks == b]
                gone = np.intersect1d(in_block, dropped)
                if gone.shape[0] < in_block.shape[0]:
                    partial += 1
                    assert np.array_equal(gone, in_block[:gone.shape[0]])
            assert partial <= 1
            checked += 1
    assert checked > 10


def test_block_choice_is_uniform_over_blocks():
    """Candidates = 5 whole blocks of 4, keep 8 (2 blocks): each of the 10
    pairs of blocks is kept equally often (chi-square, 9 dof)."""
    lp, B = 3, 4
    sets = _one_event_sets(POLICY_BLOCK, 20, 8, range(12000), 1, 1, block=B, lp=lp)
    cells = {s: 0 for s in itertools.combinations(range(5), 2)}
    for s in sets:
        kept = np.asarray(s)
        blocks = tuple(sorted(set(((kept - lp) // B).tolist())))
        assert len(blocks) == 2
        cells[blocks] += 1
    assert stats.chisquare(np.array(list(cells.values()))).pvalue > 1e-3
