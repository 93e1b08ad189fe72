"""Pins of the oracle's eviction rule (Eq. 1, Section 3, Appendices B, D, F).

No paper table prints a kept set, so the rule is pinned by what the paper
and the mathematics fix: brute-force selection on tiny inputs, the
structural invariants, uniformity (chi-square on the exact subset law, on
marginal inclusion and on cross-head independence), the survival law of
Appendix D and the printed constants in tests/golden/paper_constants.json.
"""

import itertools
import json
import os

import numpy as np
import pytest
from scipy import stats

from oracle import evict
from oracle.evict import (BUDGET_EVICTABLE, BUDGET_TOTAL, SequenceReplay,
                          drop_set, evict_head, eviction_due, keep_count,
                          position_keys)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


# --- selection given the keys -------------------------------------------

@pytest.mark.parametrize("trial", range(60))
def test_drop_set_matches_brute_force(trial):
    """The m dropped candidates are exactly the subset whose every member
    ranks below every kept one in (key, position) order."""
    rng = np.random.default_rng(trial)
    c = int(rng.integers(1, 9))
    m = int(rng.integers(0, c + 1))
    cand = np.sort(rng.choice(1000, c, replace=False))
    keys = rng.integers(0, 4, c).astype(np.uint64)     # many ties on purpose
    got = set(drop_set(cand, keys, m).tolist())
    rank = lambda i: (int(keys[i]), int(cand[i]))
    found = []
    for sub in itertools.combinations(range(c), m):
        kept = [i for i in range(c) if i not in sub]
        if all(rank(a) < rank(b) for a in sub for b in kept):
            found.append(set(sub))
    assert found == [got]


def test_keys_depend_on_every_counter_field():
    p = np.arange(40)
    base = position_keys(p, 5, 9, 0, 0, 0)
    for args in ((6, 9, 0, 0, 0), (5, 10, 0, 0, 0), (5, 9, 1, 0, 0),
                 (5, 9, 0, 1, 0), (5, 9, 0, 0, 1)):
        other = position_keys(p, *args)
        assert np.count_nonzero(other == base) == 0
    assert len(set(base.tolist())) == 40


# --- trigger and budget readings ------------------------------------------

def test_trigger_schedule_tiny_case():
    """Prompt 128, K=256, r=64, every 64: first event at step 384, then one
    event every 64 steps (11 events in 1024 steps)."""
    rep = SequenceReplay(128, 256, 64, 64, 1000, 0, [(0, 0), (0, 1)])
    rep.advance(1024)
    steps = [s for s, _ in rep.log]
    assert steps[0] == 384 and steps == list(range(384, 1025, 64))
    assert [e for _, e in rep.log] == list(range(11))


def test_trigger_matches_golden_period():
    g = _golden()["trigger"]
    assert eviction_due(g["every"], 10**6, 0, g["recent_r"], 0, g["every"])
    assert not eviction_due(g["every"] + 1, 10**6, 0, g["recent_r"], 0, g["every"])


def test_budget_modes():
    assert keep_count(4096, 100, BUDGET_EVICTABLE) == 4096
    assert keep_count(4096, 100, BUDGET_TOTAL) == 3996
    assert keep_count(4096, 4096, BUDGET_TOTAL) == 0
    with pytest.raises(ValueError):
        keep_count(1024, 2048, BUDGET_TOTAL)


def test_modes_keep_identical_sets():
    """TOTAL with K_total = K + lp keeps exactly EVICTABLE's sets with K."""
    lp, K, r = 37, 50, 16
    heads = [(0, 0), (1, 1)]
    a = SequenceReplay(lp, keep_count(K, lp, BUDGET_EVICTABLE), r, 16, 3, 4, heads)
    b = SequenceReplay(lp, keep_count(K + lp, lp, BUDGET_TOTAL), r, 16, 3, 4, heads)
    a.advance(500)
    b.advance(500)
    for h in heads:
        assert np.array_equal(a.P[h], b.P[h])


# --- structural invariants --------------------------------------------------

@pytest.mark.parametrize("lp,k,r,every", [(0, 8, 4, 4), (5, 20, 8, 8),
                                           (30, 0, 4, 1), (12, 64, 16, 16),
                                           (3, 7, 1, 3)])
def test_invariants_every_event(lp, k, r, every):
    heads = [(0, 0), (0, 1), (2, 0)]
    rep = SequenceReplay(lp, k, r, every, 77, 5, heads)
    seen = {h: set(range(lp)) for h in heads}
    for _ in range(400):
        rep.append()
        for h in heads:
            seen[h].add(rep.lp + rep.step - 1)
        fired = rep.end_step()
        for h in heads:
            P = rep.P[h]
            assert np.all(np.diff(P) > 0)                        # distinct, in order
            assert set(range(lp)) <= set(P.tolist())             # prompt pinned
            newest = rep.lp + rep.step - 1
            recent = range(max(lp, newest - r + 1), newest + 1)
            assert set(recent) <= set(P.tolist())                # buffer kept
            assert set(P.tolist()) <= seen[h]                    # monotonic
            seen[h] = set(P.tolist())
            if fired:
                assert P.shape[0] == lp + k + r                  # back to budget
                assert P.shape[0] - lp - r == k                  # exactly k evictable


def test_no_eviction_when_not_over_budget():
    P = np.arange(30)
    assert np.array_equal(evict_head(P, 10, 4, 16, 1, 1, 0, 0, 0), P)


# --- uniformity -------------------------------------------------------------

def _keep_sets(C, k, seeds, event=0, layer=0, head=0, lp=0):
    cand = np.arange(lp, lp + C)
    P = np.arange(lp + C + 1)              # one recent entry after the candidates
    out = []
    for s in seeds:
        newP = evict_head(P, lp, 1, k, int(s), 11, event, layer, head)
        out.append(tuple(newP[lp:lp + k].tolist()))
    return out


def test_exact_subset_law():
    """C=6, keep 3: all 20 subsets equally likely (chi-square, 19 dof)."""
    sets = _keep_sets(6, 3, range(20000))
    cells = {s: 0 for s in itertools.combinations(range(6), 3)}
    for s in sets:
        cells[s] += 1
    obs = np.array(list(cells.values()))
    assert obs.sum() == 20000 and len(cells) == 20
    p = stats.chisquare(obs).pvalue
    assert p > 1e-3, p


def test_marginal_inclusion():
    """C=320, keep 256 (the tiny case's first event): each candidate is kept
    with probability 256/320.  The statistic ((C-1)/C) * sum (n_p - S pi)^2 /
    (S pi (1-pi)) is chi-square with C-1 dof under sampling without
    replacement."""
    C, k, S = 320, 256, 8000
    lp = 128
    counts = np.zeros(C)
    P = np.arange(lp + C + 64)
    for s in range(S):
        newP = evict_head(P, lp, 64, k, 1000 + s, 0, 0, 0, 0)
        counts[newP[lp:lp + k] - lp] += 1
    pi = k / C
    X = (C - 1) / C * np.sum((counts - S * pi) ** 2) / (S * pi * (1 - pi))
    p = stats.chi2.sf(X, C - 1)
    assert 1e-3 < p < 1 - 1e-3, p


def test_cross_head_independence():
    """Two KV heads, C=4, keep 2: the 36 joint outcomes are equally likely."""
    S = 18000
    a = _keep_sets(4, 2, range(S), head=0)
    b = _keep_sets(4, 2, range(S), head=1)
    subs = list(itertools.combinations(range(4), 2))
    idx = {s: i for i, s in enumerate(subs)}
    tab = np.zeros((6, 6))
    for x, y in zip(a, b):
        tab[idx[x], idx[y]] += 1
    p = stats.chisquare(tab.ravel()).pvalue
    assert p > 1e-3, p


def _survival(lp, k_keep, r, every, n_events, seeds, mode_total_k=None):
    first = None
    fracs = np.zeros((len(seeds), n_events))
    for si, s in enumerate(seeds):
        rep = SequenceReplay(lp, k_keep, r, every, s, 3, [(0, 0)])
        while not rep.log:
            rep.advance(every)
        first = rep.log[0][0]
        # candidates of event 0 that survived it
        tracked = set(rep.P[(0, 0)][lp:lp + k_keep].tolist())
        base = len(tracked)
        for n in range(n_events):
            rep.advance(every)
            alive = tracked & set(rep.P[(0, 0)].tolist())
            fracs[si, n] = len(alive) / base
    return first, fracs


def test_survival_law_matches_appendix_d():
    """Appendix D: after n further evictions a trace position survives with
    ((K - lp) / (K + r - lp))^n; about 0.94 per event at K=1024, r=64."""
    g = _golden()["age_bias"]
    K, r = g["budget_k"], g["recent_r"]
    ratio = K / (K + r)                            # lp = 0 here
    assert round(ratio, g["printed_digits"]) == g["printed_per_event_survival"]
    first, fr = _survival(0, K, r, r, 4, range(120))
    assert first == K + 2 * r                      # first event at step 1152
    mean = fr.mean(axis=0)
    se = fr.std(axis=0, ddof=1) / np.sqrt(fr.shape[0])
    for n in range(4):
        expect = ratio ** (n + 1)
        assert abs(mean[n] - expect) < 5 * se[n] + 1e-4, (n, mean[n], expect)


def test_survival_law_total_mode_with_prompt():
    """Same law with the prompt counted in K (Eq. 1 convention)."""
    lp, K_total, r = 40, 136, 16
    k_keep = keep_count(K_total, lp, BUDGET_TOTAL)
    ratio = (K_total - lp) / (K_total + r - lp)
    _, fr = _survival(lp, k_keep, r, r, 6, range(300))
    mean = fr.mean(axis=0)
    se = fr.std(axis=0, ddof=1) / np.sqrt(fr.shape[0])
    for n in range(6):
        assert abs(mean[n] - ratio ** (n + 1)) < 5 * se[n] + 1e-4


def test_planted_fact_survival_closed_form():
    """Appendix B: with no protection rule a planted copy survives E eviction
    events with probability (1024/1088)^E.  In steady state (K = 1024 kept,
    64 new candidates per event, so 1088 candidates) the fraction of the
    positions kept by one event that are still cached E events later matches
    the closed form at the printed E, within a binomial interval over the
    tracked positions; fresh draws make events independent (the overlap of
    two events' drop sets is hypergeometric)."""
    g = _golden()["planted_fact_survival"]
    C, k = g["candidates"], g["kept"]
    P = np.arange(C + 1)
    newP = evict_head(P, 0, 1, k, 5, 5, 0, 0, 0)
    assert newP.shape[0] - 1 == k
    seeds = range(24)
    _, fr = _survival(0, k, C - k, C - k, max(g["events"]), seeds)
    tracked = len(seeds) * k
    for E in g["events"]:
        p = (k / C) ** E
        half = 4.5 * np.sqrt(p * (1 - p) / tracked)
        assert abs(fr[:, E - 1].mean() - p) < half, (E, fr[:, E - 1].mean(), p)
    # independence across events: the overlap of two events' drop sets over
    # the same candidates matches the hypergeometric mean m^2 / C
    m = C - k
    overl = []
    for s in range(200):
        a = set(np.setdiff1d(P[:C], evict_head(P, 0, 1, k, s, 1, 0, 0, 0)).tolist())
        b = set(np.setdiff1d(P[:C], evict_head(P, 0, 1, k, s, 1, 1, 0, 0)).tolist())
        overl.append(len(a & b))
    assert abs(np.mean(overl) - m * m / C) < 0.6
