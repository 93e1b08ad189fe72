"""A request preempted from a live batch and resumed later (Appendix G:
eviction under paging has to stay correct across preemption).

The request's rows are read head by head and its slot ended; the rest of the
batch keeps decoding; then the request begins again (in its old slot or
another free one) with the same prompt length, seed and request id, is
advanced positions-only by the steps it had decoded (ra_seq_fast_forward,
which leaves every other slot alone), and gets its saved rows back
(ra_write_rows).  Its kept positions depend only on its seed, request id and
step, so the resumed state must be the one it left: the same length, step,
event count and positions, the oracle's kept sets and rows; and every request
then decodes as the oracle says (outputs within tolerance, kept sets and rows
bit-exact at the end).
"""

import numpy as np
import pytest
import torch

from gpu_harness import OracleSeq, Run, attn_err, check_heads, log
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu


def _decode(run, oracles, n, dtype, check_every=5):
    worst = 0.0
    for t in range(n):
        outs, _ = run.step()
        check = t % check_every == check_every - 1 or t == n - 1
        if check:
            outs = outs.float().cpu()
        for o in oracles:
            o.rep.append()
            if check:
                for layer in range(run.L):
                    worst = max(worst, attn_err(outs[layer, o.slot],
                                                o.attend(layer, o.rep.step - 1), dtype,
                                                (o.slot, o.rep.step, layer)))
            o.rep.end_step()
    return worst


ONE_SPLIT = 4096          # keys per work item: every head is one item, so events defer moves


@pytest.mark.parametrize("layout,dtype,t1,target,split", [
    (B.RA_LAYOUT_CHRONOLOGICAL, B.RA_BF16, 64, 3, ONE_SPLIT),   # preempted, its moves deferred
    (B.RA_LAYOUT_CHRONOLOGICAL, B.RA_BF16, 61, 1, 0),           # resumed in its own slot
    (B.RA_LAYOUT_HOLE_FILL, B.RA_BF16, 61, 3, 0),
    (B.RA_LAYOUT_PAGED, B.RA_BF16, 64, 1, 0),
    (B.RA_LAYOUT_PAGED, B.RA_BF16, 61, 3, 0),
    (B.RA_LAYOUT_CHRONOLOGICAL, B.RA_F32, 61, 3, 0),
])
def test_preempted_request_resumes_where_it_left(layout, dtype, t1, target, split):
    log("preempt layout=%d dtype=%d t1=%d target=%d split=%d" % (layout, dtype, t1, target,
                                                                 split))
    lps = [5, 17, 9, 17]                # slot 3 starts free, sized for the request of slot 1
    run = Run(L=2, Hq=8, Hkv=2, K=40, lps=lps, r=8, every=8, dtype=dtype, layout=layout,
              begin=False, max_seqs=4, page_rows=32, attn_split=split)
    for s in range(3):
        run.begin(s)
    oracles = {s: OracleSeq(run, s) for s in range(3)}
    worst = _decode(run, oracles.values(), t1, dtype)   # events at steps 56 and 64
    assert B.ra_get_seq_info(run.h, 1).event >= 1
    if split == ONE_SPLIT and t1 % 8 == 0:
        assert B.ra_get_seq_info(run.h, 1).move_pending      # moves ride on the next step

    # preempt the request of slot 1: its positions and rows, then its slot
    info = B.ra_get_seq_info(run.h, 1)
    n = info.len
    pos = torch.empty(run.L * run.Hkv * n, dtype=torch.int32, device="cuda")
    B.ra_export_positions(run.h, 1, pos)
    ks = torch.empty(run.L, run.Hkv, n, 128, dtype=run.tdtype, device="cuda")
    vs = torch.empty_like(ks)
    for layer in range(run.L):
        for g in range(run.Hkv):
            B.ra_read_rows(run.h, 1, layer, g, ks[layer, g], vs[layer, g])
    torch.cuda.synchronize()
    saved = (info.len, info.step, info.event, info.k_keep)
    req = oracles.pop(1)
    run.end(1)

    # the others decode on without it (its phase falls behind theirs)
    worst = max(worst, _decode(run, oracles.values(), 13, dtype))

    # resume: same prompt length, seed and request id; positions forwarded,
    # rows written back
    run.lps[target], run.seeds[target], run.rids[target] = run.lps[1], run.seeds[1], run.rids[1]
    before = {s: (B.ra_get_seq_info(run.h, s).len, B.ra_get_seq_info(run.h, s).step)
              for s in oracles}
    B.ra_seq_begin(run.h, target, run.lps[target], run.seeds[target], run.rids[target],
                   None, None)
    B.ra_seq_fast_forward(run.h, target, saved[1])
    B.ra_write_rows(run.h, target, ks, vs)
    run.active.add(target)
    run.steps[target] = saved[1]
    now = B.ra_get_seq_info(run.h, target)
    assert (now.len, now.step, now.event, now.k_keep) == saved
    for s in oracles:                    # the other slots were not advanced
        i = B.ra_get_seq_info(run.h, s)
        assert (i.len, i.step) == before[s]
    pos2 = torch.empty_like(pos)
    B.ra_export_positions(run.h, target, pos2)
    assert torch.equal(pos.cpu(), pos2.cpu())
    req.slot = target
    oracles[target] = req
    check_heads(run, [req])

    # every request decodes on as the oracle says
    worst = max(worst, _decode(run, oracles.values(), 30, dtype))
    check_heads(run, oracles.values())
    log("  worst %.3g" % worst)
    run.close()


def test_seq_fast_forward_leaves_other_slots_alone():
    """Forwarding one slot advances only it (the other slots' records,
    positions and rows unchanged, their deferred moves still pending), and
    is refused for an inactive slot, inside a step and for a negative count."""
    run = Run(L=2, Hq=4, Hkv=2, K=40, lps=[5, 17, 11], r=8, every=8, begin=False, max_seqs=3,
              attn_split=ONE_SPLIT)
    run.begin(0)
    run.begin(1)
    oracles = [OracleSeq(run, s) for s in range(2)]
    _decode(run, oracles, 64, B.RA_BF16)           # ends on a deferred event
    assert all(B.ra_get_seq_info(run.h, s).move_pending for s in range(2))
    info0 = B.ra_get_seq_info(run.h, 0)
    for bad in ((2, 5), (1, -1), (3, 1)):
        with pytest.raises(B.RandAttnError) as e:
            B.ra_seq_fast_forward(run.h, *bad)
        assert e.value.status in (B.RA_ERR_STATE, B.RA_ERR_INVALID_ARG)
    run.seeds[2], run.rids[2] = 99, 77
    run.begin(2)
    late = OracleSeq(run, 2)
    B.ra_seq_fast_forward(run.h, 2, 61)            # through its own event at step 56
    late.advance(61)
    run.steps[2] = 61
    assert B.ra_get_seq_info(run.h, 2).event == 1
    assert all(B.ra_get_seq_info(run.h, s).move_pending for s in range(2))   # carried
    i0 = B.ra_get_seq_info(run.h, 0)
    assert (i0.len, i0.step, i0.event) == (info0.len, info0.step, info0.event)
    assert np.array_equal(run.positions(0, 1, 1), oracles[0].rep.P[(1, 1)])
    run.materialise(2)                   # writing rows moves the pending rows first
    oracles.append(late)
    _decode(run, oracles, 12, B.RA_BF16, check_every=1)
    check_heads(run, oracles)
    # inside a step
    q, k, v = run.step_inputs(0)
    out = torch.empty(run.max_seqs, run.Hq, 128, dtype=torch.bfloat16, device="cuda")
    run.cache.decode(0, q, k, v, out)
    with pytest.raises(B.RandAttnError) as e:
        B.ra_seq_fast_forward(run.h, 0, 1)
    assert e.value.status == B.RA_ERR_STATE
    q, k, v = run.step_inputs(1)
    run.cache.decode(1, q, k, v, out)
    B.ra_end_step(run.h)
    run.close()
