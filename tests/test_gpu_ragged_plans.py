"""Ragged batches at mid sizes, across the attention plan's branches.

Each case draws a batch (1-90 sequences, 1-8 KV heads, group 1-8, budgets of
200-9,500 rows, prompts of 0-1,000, r in {0, 16, 64}, a trigger every 16 or
64 steps, any layout, mostly bf16) and forwards every sequence on its own
(ra_seq_fast_forward) to its own step, a little before or after one of its
events, so the batch holds caches of many lengths.  The cases are chosen so
that together they run every branch of the launch plan -- 1, 4, 8 and 12
wavefronts per work item, one or several work items per head (merged by the
last split, or by the merge kernel for fp32), in each layout -- and each case
asserts the plan it was chosen for.  Then a trigger period of steps: sampled
outputs against the fp64 oracle at every fifth step and at every step with an
event, and the kept sets and rows of sampled sequences at the end.
"""

import numpy as np
import pytest

from gpu_harness import OracleSeq, Run, attn_err, check_heads, log
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu

# seed: (wavefronts per item, several items per head)
CASES = {102: (1, True), 41: (1, True), 119: (1, True), 64: (1, True), 93: (1, True),
         96: (4, False), 110: (4, False), 67: (4, False), 79: (4, True), 52: (4, True),
         53: (4, True), 115: (8, False), 103: (8, True), 83: (8, True), 97: (12, False),
         100: (12, False)}


def draw(seed):
    rng = np.random.default_rng(5000 + seed)
    c = dict(L=int(rng.integers(1, 3)), Hkv=int(rng.choice([1, 2, 4, 8])),
             G=int(rng.choice([1, 2, 4, 5, 8])))
    n = int(rng.choice([1, 2, 5, 12, 16, 32, 40, 90]))
    c["n"] = max(1, 400 // c["Hkv"]) if n * c["Hkv"] > 400 else n
    c["K"] = int(rng.integers(200, 9501))
    c["r"] = int(rng.choice([0, 16, 64]))
    c["every"] = int(rng.choice([16, 64]))
    c["layout"] = int(rng.integers(0, 3))
    c["dtype"] = B.RA_BF16 if rng.integers(0, 5) else B.RA_F32
    c["lps"] = [int(x) for x in rng.integers(0, 1001, c["n"])]
    c["page_rows"] = int(rng.choice([32, 64, 256]))
    return c, rng


@pytest.mark.parametrize("seed", sorted(CASES))
def test_ragged_batch_plan_branches(seed):
    c, rng = draw(seed)
    L, n, dtype = c["L"], c["n"], c["dtype"]
    run = Run(L=L, Hq=c["Hkv"] * c["G"], Hkv=c["Hkv"], K=c["K"], lps=c["lps"], r=c["r"],
              every=c["every"], dtype=dtype, layout=c["layout"], wl_seed=900 + seed,
              page_rows=c["page_rows"])
    oracles = [OracleSeq(run, s) for s in range(n)]
    for s in range(n):
        target = int(rng.integers(0, c["K"] + c["r"] + 3 * c["every"]))
        B.ra_seq_fast_forward(run.h, s, target)
        oracles[s].advance(target)
        run.steps[s] = target
        run.materialise(s)
    plan = B.ra_attention_plan(run.h)
    log("ragged batch %d: %s plan %s" % (seed, {k: v for k, v in c.items() if k != "lps"},
                                          plan))
    assert (plan[2], plan[1] > 1) == CASES[seed]
    worst, events = 0.0, 0
    for t in range(c["every"] + 4):
        outs, ev = run.step()
        check = t % 5 == 0 or ev
        pick = set(rng.choice(n, size=min(n, 4), replace=False).tolist()) if check else set()
        if check:
            outs = outs.float().cpu()
        for o in oracles:
            o.rep.append()
            if o.slot in pick:
                for layer in range(L):
                    worst = max(worst, attn_err(outs[layer, o.slot],
                                                o.attend(layer, o.rep.step - 1), dtype,
                                                (seed, t, o.slot, layer)))
            o.rep.end_step()
        events += bool(ev)
    check_heads(run, [oracles[i] for i in rng.choice(n, size=min(n, 3), replace=False)])
    log("  events %d worst %.3g" % (events, worst))
    run.close()
