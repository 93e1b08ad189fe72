"""Score-based eviction rounds (measurement only) against the oracle.

A cache with the external policy decodes without end-of-step eviction; at
every 64th step a scored round (Section 2: SnapKV, R-KV or VaSE; the prompt
competes) drops the rows over budget.  The GPU's drop set must be a valid
selection under the oracle's fp64 scores: lowest-m of the SnapKV or R-KV
score up to near-ties within the bf16 / fp32 tolerance; for VaSE the large
set (value ranges are exact) bit-exact and the proportional fill consistent
with the oracle's keys log(u)/w for every w within the score tolerance.  The
surviving rows must be exactly the rows of the kept positions in
chronological order, sequences under budget must be left as they are, and
attention after the round must match the oracle on the kept rows.
"""

import numpy as np
import pytest
import torch

from gpu_harness import Run, log, max_abs
from oracle.attention import gqa_decode
from oracle.scored import es_uniform, lowest, rkv_redundancy, rkv_scores, value_range
from oracle.window_score import max_pool, window_scores
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu


def _qwin(run, steps_done):
    qw = torch.zeros(run.max_seqs, run.L, run.Hq, 64, 128, dtype=torch.bfloat16, device="cuda")
    heads = torch.arange(run.Hq, device="cuda").view(-1, 1)
    for b in range(run.n):
        st = torch.arange(steps_done[b] - 64, steps_done[b], device="cuda").view(1, -1)
        for l in range(run.L):
            qw[b, l] = run.wl.q_rows(run.rids[b], l, heads, st)
    return qw


def _valid_lowest(pooled, drops, n_cand, m, where, tol=None):
    d = np.asarray(drops)
    assert d.shape[0] == m and np.all(np.diff(d) > 0) and d.min() >= 0 and d.max() < n_cand, where
    thr = np.sort(pooled[:n_cand])[m - 1]
    if tol is None:
        tol = 4e-3 + 2e-3 * thr
    kept = np.setdiff1d(np.arange(n_cand), d)
    assert np.all(pooled[d] <= thr + tol), where
    assert np.all(pooled[kept] >= thr - tol), where


def _valid_vase(pooled, vr, u, P, drops, n_cand, budget, n_large, m, where):
    d = np.asarray(drops)
    assert d.shape[0] == m and np.all(np.diff(d) > 0), where
    small = lowest(vr[:n_cand], P[:n_cand], n_cand - n_large)
    large = np.setdiff1d(np.arange(n_cand), small)
    assert not set(d.tolist()) & set(large.tolist()), where     # large set kept exactly
    assert set(d.tolist()) <= set(small.tolist()), where
    w = pooled[:n_cand]
    delta = 4e-3 + 2e-3 * w
    lo = np.log(u[:n_cand]) / np.maximum(w - delta, 1e-12)      # keys log(u)/w over the
    hi = np.log(u[:n_cand]) / (w + delta)                       # tolerance interval of w
    kept_small = np.setdiff1d(small, d)
    assert lo[d].max() <= hi[kept_small].min(), where


SCORERS = [(B.RA_SCORER_SNAPKV, "snapkv"), (B.RA_SCORER_RKV, "rkv"), (B.RA_SCORER_VASE, "vase")]


@pytest.mark.parametrize("scorer,name", SCORERS)
@pytest.mark.parametrize("Hq,Hkv,lps,K", [(8, 2, [40, 7, 0], 100), (10, 2, [150, 3], 60)])
def test_scored_rounds(Hq, Hkv, lps, K, scorer, name):
    log("%s rounds Hq=%d Hkv=%d lps=%s K=%d" % (name, Hq, Hkv, lps, K))
    L, r, every = 2, 64, 64
    run = Run(L=L, Hq=Hq, Hkv=Hkv, K=K, lps=lps, r=r, every=every,
              policy=B.RA_POLICY_EXTERNAL)
    G = run.G
    wl = run.wl.to("cpu")
    scratch = torch.empty(B.ra_scored_scratch_bytes(run.cfg, max(lps)) // 4 + 1,
                          dtype=torch.int32, device="cuda")
    lam, thr_dup, n_dups, vseed = 0.1, 0.9, 1, 4242
    prm = B.make_scorer(scorer, rkv_lambda=lam, rkv_threshold=thr_dup,
                        rkv_recent_dups=n_dups, vase_n_large=-1, vase_seed=vseed)
    # the oracle's view: positions per (slot, layer, head)
    P = {(b, l, g): np.arange(lps[b]) for b in range(run.n) for l in range(L) for g in range(Hkv)}
    rounds = 0
    for t in range(1, 5 * 64 + 1):
        outs, ev = run.step()
        assert ev == 0                              # no end-of-step eviction
        for key in P:
            P[key] = np.append(P[key], lps[key[0]] + t - 1)
        if t % 64 == 0:
            due = [b for b in range(run.n)
                   if P[(b, 0, 0)].shape[0] - r > lps[b] + K]
            qw = _qwin(run, [t] * run.n)
            before = {b: B.ra_get_seq_info(run.h, b) for b in range(run.n)}
            B.ra_scored_evict(run.h, 0, run.n, prm, qw, scratch)
            torch.cuda.synchronize()
            for b in range(run.n):
                info = B.ra_get_seq_info(run.h, b)
                if b not in due:
                    assert info.len == before[b].len
                    continue
                n = P[(b, 0, 0)].shape[0]
                m = n - r - lps[b] - K
                assert info.len == n - m and info.event == before[b].event + 1
                for l in range(L):
                    for g in range(Hkv):
                        Pold = P[(b, l, g)]
                        k = wl.k_rows(run.rids[b], l, g, torch.as_tensor(Pold), lps[b])
                        q = wl.q_rows(run.rids[b], l, torch.arange(g * G, (g + 1) * G).view(-1, 1),
                                      torch.arange(t - 64, t).view(1, -1))
                        qpos = np.repeat((lps[b] + np.arange(t - 64, t))[None, :], G, 0)
                        sc = window_scores(q.reshape(-1, 128).double().numpy(), qpos.reshape(-1),
                                           k.double().numpy(), Pold)
                        pooled = max_pool(sc, 7)
                        got = run.positions(b, l, g)
                        drops = np.setdiff1d(np.arange(n), np.searchsorted(Pold, got))
                        assert np.all(np.diff(got) > 0), (b, l, g)
                        where = (name, t, b, l, g)
                        budget = lps[b] + K
                        if scorer == B.RA_SCORER_SNAPKV:
                            _valid_lowest(pooled, drops, n - r, m, where)
                        elif scorer == B.RA_SCORER_RKV:
                            cbar = rkv_redundancy(k.double().numpy(), Pold, thr_dup, n_dups)
                            s = rkv_scores(pooled, cbar, n - r, lam)
                            # the SnapKV term carries the scorer's tolerance, scaled by lambda
                            tol = lam * (4e-3 + 2e-3 * pooled.max()) + 1e-5
                            _valid_lowest(s, drops, n - r, m, where, tol)
                        else:
                            v = wl.v_rows(run.rids[b], l, g, torch.as_tensor(Pold), lps[b])
                            u = es_uniform(Pold, vseed, run.rids[b], before[b].event, l, g)
                            _valid_vase(pooled, value_range(v.double().numpy()), u, Pold,
                                        drops, n - r, budget, budget // 2, m, where)
                        P[(b, l, g)] = got.astype(np.int64)
                        kg, vg = run.rows(b, l, g)
                        kw = wl.k_rows(run.rids[b], l, g, torch.as_tensor(got), lps[b])
                        vw = wl.v_rows(run.rids[b], l, g, torch.as_tensor(got), lps[b])
                        assert torch.equal(kg, kw) and torch.equal(vg, vw), (t, b, l, g)
                rounds += 1
        elif t % 64 == 1 and t > 64:
            # the step after a round attends over the kept rows
            outs = outs.float().cpu()
            for b in range(run.n):
                for l in range(L):
                    q = wl.q_rows(run.rids[b], l, torch.arange(Hq), t - 1).double().numpy()
                    Ks, Vs = [], []
                    for g in range(Hkv):
                        pp = torch.as_tensor(P[(b, l, g)])
                        Ks.append(wl.k_rows(run.rids[b], l, g, pp, lps[b]).double().numpy())
                        Vs.append(wl.v_rows(run.rids[b], l, g, pp, lps[b]).double().numpy())
                    err = max_abs(outs[l, b], gqa_decode(q, Ks, Vs))
                    assert err <= 2e-2, (t, b, l, err)
    log("  %d sequence rounds" % rounds)
    assert rounds >= 6
    run.close()
