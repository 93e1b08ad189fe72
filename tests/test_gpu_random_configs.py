"""GPU parity on seeded random small configurations.

Each case draws a configuration from its own seed: layers, KV heads and
group size (1..16), dtype, budget K (0 included) and budget mode, recent
buffer r (0 included), trigger period (every step included), row layout,
eviction policy, and ragged prompt lengths for 1-3 sequences.  The HIP path
then decodes long enough for several events; every step's attention output
of every query head is checked against the fp64 oracle (2e-2 bf16, 1e-5
fp32), the kept positions after every event, and the compacted rows at every
eighth event and at the end.  A last set of cases runs the drawn
configurations in bf16 and the chronological layout with one work item per
head, where events of every sequence at once leave their row moves to the
next step's attention; their rows are checked after the step that moved
them.
"""

import numpy as np
import pytest

from gpu_harness import OracleSeq, Run, attn_err, check_heads, log
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu

N_CASES = 12


def draw_config(case):
    rng = np.random.default_rng(9000 + case)
    c = {}
    c["dtype"] = [B.RA_BF16, B.RA_F32][int(rng.integers(0, 2))]
    c["L"] = int(rng.integers(1, 4))
    c["Hkv"] = int(rng.choice([1, 2, 3, 5]))
    c["G"] = int(rng.choice([1, 2, 3, 4, 7, 8, 16]))
    c["layout"] = int(rng.integers(0, 2))
    c["policy"] = int(rng.choice([B.RA_POLICY_RANDOM, B.RA_POLICY_RANDOM, B.RA_POLICY_SHARED,
                                  B.RA_POLICY_BLOCK, B.RA_POLICY_RECENCY]))
    c["block"] = int(rng.integers(1, 20)) if c["policy"] == B.RA_POLICY_BLOCK else 1
    c["mode"] = [B.RA_BUDGET_EVICTABLE, B.RA_BUDGET_TOTAL][int(rng.integers(0, 2))]
    c["r"] = int(rng.choice([0, 1, 7, 16, 64, 80]))
    c["every"] = int(rng.choice([1, 3, 16, 64]))
    c["K"] = int(rng.integers(0, 200))
    n = int(rng.integers(1, 4))
    lps = rng.integers(0, 150, n)
    if c["mode"] == B.RA_BUDGET_TOTAL:
        lps = np.minimum(lps, c["K"])
    c["lps"] = [int(x) for x in lps]
    budget = c["K"] if c["mode"] == B.RA_BUDGET_EVICTABLE else c["K"] - min(c["lps"])
    c["T"] = int(min(360, budget + c["r"] + 3 * c["every"] + rng.integers(5, 60)))
    return c


def _run_config(case, c, page_rows=32, attn_split=0):
    """Decode the drawn configuration, checking every output.  After an event
    the kept sets are checked at once; its rows too at every eighth event,
    or, when the event left its row moves to the next step's attention, once
    that step has moved them (reading rows would move them first)."""
    run = Run(L=c["L"], Hq=c["Hkv"] * c["G"], Hkv=c["Hkv"], K=c["K"], lps=c["lps"],
              r=c["r"], every=c["every"], dtype=c["dtype"], mode=c["mode"],
              layout=c["layout"], policy=c["policy"], block=c["block"],
              seeds=[case * 7919 + s for s in range(len(c["lps"]))],
              rids=[case * 31 + s for s in range(len(c["lps"]))], wl_seed=500 + case,
              page_rows=page_rows, attn_split=attn_split)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    worst, events, deferred, moved = 0.0, 0, 0, False
    for t in range(c["T"]):
        outs, ev = run.step()
        outs = outs.float().cpu()
        for o in oracles:
            o.rep.append()
            for layer in range(run.L):
                err = attn_err(outs[layer, o.slot], o.attend(layer, t), c["dtype"],
                               (case, t, o.slot, layer))
                worst = max(worst, err)
            o.rep.end_step()
        if moved and not ev:
            check_heads(run, oracles)          # rows moved by this step's attention
        moved = False
        if ev:
            events += 1
            pending = any(B.ra_get_seq_info(run.h, o.slot).move_pending for o in oracles)
            deferred += pending
            moved = pending and deferred % 4 == 1
            check_heads(run, oracles, rows=not pending and events % 8 == 1)
    check_heads(run, oracles, rows=True)
    log("  steps=%d events=%d deferred=%d worst=%.3g" % (c["T"], events, deferred, worst))
    assert events >= 1
    run.close()
    return deferred


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_config_parity(case):
    c = draw_config(case)
    log("random config %d: %s" % (case, c))
    _run_config(case, c)


@pytest.mark.parametrize("case", range(6))
def test_random_config_parity_paged(case):
    """The same drawn configurations in the paged layout, with pages of 32,
    64 or 128 rows."""
    c = draw_config(case)
    c["layout"] = B.RA_LAYOUT_PAGED
    page_rows = (32, 64, 128)[case % 3]
    log("random config %d paged (%d-row pages): %s" % (case, page_rows, c))
    _run_config(case, c, page_rows)


@pytest.mark.parametrize("case", range(100, 108))
def test_random_config_parity_deferred(case):
    """Drawn configurations in bf16 and the chronological layout with one
    attention work item per head, so that an event of every active sequence
    at once leaves its row moves to the next step's attention (the moving
    attention; whole blocks of dropped rows included, where budgets are small
    or there is no recent buffer)."""
    c = draw_config(case)
    c["dtype"], c["layout"] = B.RA_BF16, B.RA_LAYOUT_CHRONOLOGICAL
    log("random config %d deferred: %s" % (case, c))
    assert _run_config(case, c, attn_split=4096) >= 1
