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
    _select_and_check(run, oracles, n_steps, stride=1024)
    run.close()


def _select_and_check(run, oracles, n_steps, stride):
    """Run the scorer on every slot of `run` after `n_steps` decode steps and
    check its raw scores against the fp64 oracle and its drops as a valid
    lowest-m selection of the oracle's pooled scores."""
    L, Hkv, r, every = run.L, run.Hkv, run.r, run.every
    qw = _qwin(run, n_steps)
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


@pytest.mark.parametrize("K,lps,steps,Hq,Hkv", [
    (4096, [1024, 300], 4190, 8, 2),       # 5,214 rows: the 16-keys-per-thread build
    (8192, [2048, 100], 8300, 8, 2),       # 10,348 rows: the 32-keys-per-thread build
    (8192, [2048, 100], 8300, 10, 2),      #   the same with G = 5 (three tiles per wave)
])
def test_window_select_large_caches(K, lps, steps, Hq, Hkv):
    """Caches of the Phi-4-shaped batch's size (prompts up to 2,048, K = 8,192):
    the selection holds 16 or 32 keys per thread.  The state is reached by a
    positions-only fast forward to a step before the next trigger, so the
    rows over budget (steps - r - K) are fewer than evict_every, and the
    cached rows are materialised from the generator."""
    log("window scorer large caches K=%d lps=%s steps=%d Hq=%d" % (K, lps, steps, Hq))
    run = Run(L=2, Hq=Hq, Hkv=Hkv, K=K, lps=lps, r=64, every=64, write_prompt=False,
              wl_seed=1004)
    run.fast_forward(steps)
    for b in range(run.n):
        run.materialise(b)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    for o in oracles:
        o.advance(steps)
    _select_and_check(run, oracles, steps, stride=16384)
    run.close()
