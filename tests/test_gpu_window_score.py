"""The observation-window scorer (measurement only) against its oracle.

Scores must agree with the fp64 oracle within 2e-3 absolute plus 1e-3
relative (bf16 inputs, fp32 accumulation); the drop set must be a valid
lowest-m selection of the oracle's pooled scores, i.e. unique up to
near-ties within that tolerance.
"""

import numpy as np
import pytest
import torch

from gpu_harness import OracleSeq, Run, log
from oracle.window_score import max_pool, window_scores
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu


def _qwin(run, steps_done):
    L, Hq = run.L, run.Hq
    qw = torch.empty(run.max_seqs, L, Hq, 64, 128, dtype=torch.bfloat16, device="cuda")
    heads = torch.arange(Hq, device="cuda").view(-1, 1)
    steps = torch.arange(steps_done - 64, steps_done, device="cuda").view(1, -1)
    for b in range(run.n):
        for l in range(L):
            qw[b, l] = run.wl.q_rows(run.rids[b], l, heads, steps)
    return qw


@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (10, 2), (4, 4), (16, 2), (32, 2)])
def test_window_scores_and_selection(Hq, Hkv):
    log("window scorer Hq=%d Hkv=%d" % (Hq, Hkv))
    L, K, r, every = 2, 200, 64, 64
    lps = [40, 7, 150]
    run = Run(L=L, Hq=Hq, Hkv=Hkv, K=K, lps=lps, r=r, every=every)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    n_steps = 300
    for _ in range(n_steps):
        run.step()
        for o in oracles:
            o.rep.append()
            o.rep.end_step()
    qw = _qwin(run, n_steps)
    stride = 1024
    scores = torch.zeros(run.n, L, Hkv, stride, dtype=torch.float32, device="cuda")
    drops = torch.full((run.n, L, Hkv, every), -1, dtype=torch.int32, device="cuda")
    B.ra_window_select(run.h, 0, run.n, qw, scores, stride, drops)
    torch.cuda.synchronize()
    scores, drops = scores.cpu().numpy(), drops.cpu().numpy()
    G = run.G
    for o in oracles:
        b = o.slot
        info = B.ra_get_seq_info(run.h, b)
        n = info.len
        m = n - o.lp - r - run.k_keep(b)
        assert m > 0
        for l in range(L):
            for g in range(Hkv):
                P = o.rep.P[(l, g)]
                k, _ = o.rows(l, g, P)
                q = o.wl.q_rows(o.rid, l, torch.arange(g * G, (g + 1) * G).view(-1, 1),
                                torch.arange(n_steps - 64, n_steps).view(1, -1))
                qpos = (o.lp + np.arange(n_steps - 64, n_steps))[None, :].repeat(G, 0)
                want = window_scores(q.reshape(-1, 128).double().numpy(), qpos.reshape(-1),
                                     k.double().numpy(), P)
                got = scores[b, l, g, :n]
                assert np.all(np.abs(got - want) <= 2e-3 + 1e-3 * np.abs(want)), (b, l, g)
                pooled = max_pool(want, 7)[: n - r]
                d = drops[b, l, g, :m]
                assert np.all(np.diff(d) > 0) and d.min() >= 0 and d.max() < n - r
                thr = np.sort(pooled)[m - 1]
                tol = 4e-3 + 2e-3 * thr
                kept = np.setdiff1d(np.arange(n - r), d)
                assert np.all(pooled[d] <= thr + tol), (b, l, g)
                assert np.all(pooled[kept] >= thr - tol), (b, l, g)
    run.close()
