"""GPU parity on seeded random small configurations.

Each case draws a configuration from its own seed: layers, KV heads and
group size (1..16), dtype, budget K (0 included) and budget mode, recent
buffer r (0 included), trigger period (every step included), row layout,
eviction policy, and ragged prompt lengths for 1-3 sequences.  The HIP path
then decodes long enough for several events; every step's attention output
of every query head is checked against the fp64 oracle (2e-2 bf16, 1e-5
fp32), the kept positions after every event, and the compacted rows at every
eighth event and at the end.
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


def _run_config(case, c, page_rows=32):
    run = Run(L=c["L"], Hq=c["Hkv"] * c["G"], Hkv=c["Hkv"], K=c["K"], lps=c["lps"],
              r=c["r"], every=c["every"], dtype=c["dtype"], mode=c["mode"],
              layout=c["layout"], policy=c["policy"], block=c["block"],
              seeds=[case * 7919 + s for s in range(len(c["lps"]))],
              rids=[case * 31 + s for s in range(len(c["lps"]))], wl_seed=500 + case,
              page_rows=page_rows)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    worst, events = 0.0, 0
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
        if ev:
            events += 1
            check_heads(run, oracles, rows=events % 8 == 1)
    check_heads(run, oracles, rows=True)
    log("  steps=%d events=%d worst=%.3g" % (c["T"], events, worst))
    assert events >= 1
    run.close()


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
