"""Serving with requests that finish and are replaced (continuous batching).

Requests with their own prompt and generation lengths occupy a few slots; a
finished request releases its rows (the free list merges neighbours) and
the next request of the queue begins in that slot with its prompt written.
Every live request must keep decoding exactly as the oracle says (kept sets
bit-exact after its events, outputs within the bf16 tolerance) whatever the
other slots do, and the released rows must be reusable.
"""

import numpy as np
import pytest
import torch

from gpu_harness import OracleSeq, Run, attn_err, log
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu


def _check_sets(run, o):
    for (layer, g) in o.heads:
        got = run.positions(o.slot, layer, g)
        if run.layout == B.RA_LAYOUT_HOLE_FILL:
            got = np.sort(got)
        assert np.array_equal(got, o.rep.P[(layer, g)]), (o.slot, o.rid, layer, g, o.rep.step)


@pytest.mark.parametrize("layout", [B.RA_LAYOUT_CHRONOLOGICAL, B.RA_LAYOUT_HOLE_FILL, B.RA_LAYOUT_PAGED])
def test_requests_finish_and_are_replaced(layout):
    log("serving churn layout=%d" % layout)
    rng = np.random.default_rng(31)
    slots, K, r, every = 4, 40, 16, 16
    n_req = 12
    reqs = [dict(lp=int(rng.integers(0, 60)), gen=int(rng.integers(40, 220)),
                 seed=1000 + i, rid=500 + i) for i in range(n_req)]
    # room for every slot at the largest prompt, and no more
    probe = B.make_config(2, 4, 2, K, r, every, B.RA_BUDGET_EVICTABLE, B.RA_BF16, slots,
                          layout=layout, page_rows=32, max_prompt_len=60)
    pool = slots * B.ra_seq_rows(probe, 60)
    run = Run(L=2, Hq=4, Hkv=2, K=K, lps=[0] * slots, r=r, every=every, begin=False,
              max_seqs=slots, pool_rows=pool, layout=layout, page_rows=32,
              max_prompt_len=60)
    queue = list(range(n_req))
    live, oracles, done = {}, {}, []

    def admit(slot):
        i = queue.pop(0)
        q = reqs[i]
        run.lps[slot], run.seeds[slot], run.rids[slot] = q["lp"], q["seed"], q["rid"]
        run.begin(slot)
        live[slot] = i
        oracles[slot] = OracleSeq(run, slot)

    for s in range(slots):
        admit(s)
    steps = 0
    worst = 0.0
    while live:
        outs, _ = run.step()
        steps += 1
        check = steps % 7 == 0
        if check:
            outs = outs.float().cpu()
        for s, o in oracles.items():
            o.rep.append()
            if check:
                for layer in range(run.L):
                    err = attn_err(outs[layer, s], o.attend(layer, o.rep.step - 1),
                                   B.RA_BF16, (s, o.rid, layer))
                    worst = max(worst, err)
            if o.rep.end_step():
                _check_sets(run, o)
        for s in list(live):
            if run.steps[s] == reqs[live[s]]["gen"]:
                _check_sets(run, oracles[s])
                run.end(s)
                done.append(live.pop(s))
                del oracles[s]
                if queue:
                    admit(s)
    assert sorted(done) == list(range(n_req))
    assert B.ra_pool_info(run.h) == (0, pool)      # every row was returned
    if layout != B.RA_LAYOUT_PAGED:
        # and the free list merged it: one sequence of the whole pool fits
        big = pool // (run.L * run.Hkv) - (K + r + every)
        big = big - big % 32 - 32
        assert B.ra_seq_rows(run.cfg, big) <= pool
        run.lps[0] = big
        run.begin(0)
        assert B.ra_get_seq_info(run.h, 0).base == 0
    log("  %d requests over %d steps, worst %.3g" % (n_req, steps, worst))
    run.close()


def test_released_rows_merge_with_neighbours():
    """First fit over a fragmented pool: a request larger than any hole is
    refused until a neighbour finishes and the holes merge."""
    K, r, every = 64, 16, 16
    cfg = B.make_config(1, 2, 2, K, r, every, B.RA_BUDGET_EVICTABLE, B.RA_BF16, 4)
    small = B.ra_seq_rows(cfg, 0)
    run = Run(L=1, Hq=2, Hkv=2, K=K, lps=[0, 0, 0, 0], r=r, every=every, begin=False,
              max_seqs=4, pool_rows=4 * small)
    for s in range(4):
        run.begin(s)
    run.end(1)                                    # a hole of one small region
    run.lps[1] = 40                               # needs more than one region
    assert B.ra_seq_rows(cfg, 40) > small
    with pytest.raises(B.RandAttnError) as e:
        run.begin(1)
    assert e.value.status == B.RA_ERR_CAPACITY
    run.end(2)                                    # the neighbour: holes merge
    run.begin(1)
    assert B.ra_get_seq_info(run.h, 1).base == small      # in the merged hole
    run.close()
