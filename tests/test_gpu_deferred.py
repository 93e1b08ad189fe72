"""Eviction events whose row moves ride on the next step's attention.

In the bf16 chronological layout, when every active sequence evicts at the
same step and every head is one attention work item, the end-of-step event
selects and compacts the positions only; the next
step's attention reads each head's rows in the order before the event,
masks the dropped ones, and moves every survivor down to its compacted slot
while it attends.  Kept sets are the oracle's right after the event; rows
must be the oracle's after that next step, and every output within the
tolerance, through every event.  An event in which some active sequence is
not due moves its rows at once.  Any call that reads or writes rows or plans
another event in between moves the rows first (the same end state), and so
does a step whose attention needs more than one work item per head.
"""

import numpy as np
import pytest
import torch

from gpu_harness import OracleSeq, Run, attn_err, check_heads, log
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu

ONE_SPLIT = 4096          # keys per work item: every head of these runs is one item


def _step(run, oracles, t):
    outs, ev = run.step()
    outs = outs.float().cpu()
    for o in oracles:
        o.rep.append()
        for layer in range(run.L):
            attn_err(outs[layer, o.slot], o.attend(layer, o.rep.step - 1), B.RA_BF16,
                     (t, o.slot, layer))
        o.rep.end_step()
    return ev


def _pending(run):
    return [B.ra_get_seq_info(run.h, s).move_pending for s in range(run.n)]


@pytest.mark.parametrize("policy,block", [(B.RA_POLICY_RANDOM, 1), (B.RA_POLICY_SHARED, 1),
                                          (B.RA_POLICY_BLOCK, 4), (B.RA_POLICY_RECENCY, 1)])
@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (10, 2), (16, 1)])
def test_moves_ride_on_the_next_attention(policy, block, Hq, Hkv):
    """Events every 8 steps on ragged prompts; after each event the sets are
    the oracle's while the moves are pending, and after the next step (whose
    attention moved the rows) every row is the oracle's."""
    log("deferred moves policy=%d block=%d Hq=%d Hkv=%d" % (policy, block, Hq, Hkv))
    run = Run(L=2, Hq=Hq, Hkv=Hkv, K=40, lps=[5, 0, 17], r=8, every=8, attn_split=ONE_SPLIT,
              policy=policy, block=block)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    events = 0
    after_event = False
    for t in range(150):
        ev = _step(run, oracles, t)
        if after_event and not ev:
            assert not any(_pending(run))
            check_heads(run, oracles)                 # moved by the attention
        if ev:
            events += 1
            pend = _pending(run)
            assert any(pend)
            for o in oracles:                         # sets final at once
                for (layer, g) in o.heads:
                    assert np.array_equal(run.positions(o.slot, layer, g), o.rep.P[(layer, g)])
        after_event = bool(ev)
    assert events >= 10
    run.close()


def test_calls_between_event_and_next_step_move_rows_first():
    """Between an event and the next step: reading rows, writing rows, an
    explicit event, a fast forward, ending the pending sequence and beginning
    another, and the window scorer each leave the same state as a full event
    (rows as the oracle's), and decoding goes on as the oracle says."""
    log("deferred moves: calls in between")
    cfg = B.make_config(2, 8, 2, 60, 16, 16, B.RA_BUDGET_EVICTABLE, B.RA_BF16, 4,
                        attn_split=ONE_SPLIT)
    pool = sum(B.ra_seq_rows(cfg, lp) for lp in (5, 30, 12, ONE_SPLIT + 100))
    run = Run(L=2, Hq=8, Hkv=2, K=60, lps=[5, 30, 12], r=16, every=16,
              attn_split=ONE_SPLIT, max_seqs=4, pool_rows=pool)
    oracles = {s: OracleSeq(run, s) for s in range(run.n)}

    staggered = []

    def until_event():
        """Step to the next event whose moves are deferred.  An event in which
        some active sequence is not due moves its rows at once."""
        for t in range(200):
            if _step(run, list(oracles.values()), t):
                if any(_pending(run)):
                    return
                staggered.append(t)
                check_heads(run, list(oracles.values()))
        raise AssertionError("no deferred event")

    until_event()
    check_heads(run, list(oracles.values()))          # read_rows moves them
    assert not any(_pending(run))
    until_event()
    for s in range(run.n):                            # write_rows: same rows back
        info = B.ra_get_seq_info(run.h, s)
        if not info.move_pending:
            continue
        k = torch.empty(run.L, run.Hkv, info.len, 128, dtype=torch.bfloat16, device="cuda")
        v = torch.empty_like(k)
        o = oracles[s]
        for l in range(run.L):
            for g in range(run.Hkv):
                kk, vv = o.rows(l, g, o.rep.P[(l, g)])
                k[l, g], v[l, g] = kk.to("cuda"), vv.to("cuda")
        B.ra_write_rows(run.h, s, k, v)
        break
    for t in range(20):
        _step(run, list(oracles.values()), t)
    check_heads(run, list(oracles.values()))
    until_event()
    B.ra_evict_now(run.h, 1)                          # an explicit event first moves rows
    oracles[1].rep.evict_now()
    check_heads(run, list(oracles.values()))
    until_event()
    run.fast_forward(5)                               # moves rows first, then positions only
    for o in oracles.values():
        o.advance(5)
    for s in range(run.n):
        run.materialise(s)                             # positions-only steps: rows rewritten
    check_heads(run, list(oracles.values()))
    until_event()
    pend = _pending(run)
    s_end = int(np.argmax(pend))
    run.end(s_end)                                    # a pending sequence ends
    run.lps[s_end], run.seeds[s_end], run.rids[s_end] = 9, 4242, 77
    run.begin(s_end)
    oracles[s_end] = OracleSeq(run, s_end)
    for t in range(40):
        _step(run, list(oracles.values()), t)
    check_heads(run, list(oracles.values()))
    # a new sequence long enough to need two work items per head: the
    # pending moves run on their own before the step's attention
    until_event()
    assert staggered          # the restarted sequence not yet due: moved at once
    run.lps.append(ONE_SPLIT + 100)
    run.seeds.append(99)
    run.rids.append(99)
    run.n += 1
    run.slots.append(3)
    run.steps.append(0)
    run.begin(3)
    assert B.ra_attention_plan(run.h)[1] == 2
    oracles[3] = OracleSeq(run, 3)
    for t in range(20):
        _step(run, list(oracles.values()), t)
    check_heads(run, list(oracles.values()))
    run.close()


@pytest.mark.parametrize("K,lps", [(1500, [3, 50, 211]), (3000, [0, 1, 33])])
def test_moves_across_many_rounds(K, lps):
    """Caches of 1.6k-3.2k rows, so the moving attention works through 7-13
    rounds of 256 rows and destination value tiles shared by neighbouring
    rounds: after each of two events the rows are the oracle's once the next
    step has run, and every output is within tolerance."""
    log("deferred moves over many rounds K=%d" % K)
    run = Run(L=2, Hq=8, Hkv=2, K=K, lps=lps, r=64, every=64, attn_split=ONE_SPLIT)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    t0 = 64 * ((K + 128) // 64 + 1) - 3          # three steps before an event
    run.fast_forward(t0)
    for o in oracles:
        o.advance(t0)
    for s in range(run.n):
        run.materialise(s)
    assert B.ra_attention_plan(run.h)[1] == 1
    events = 0
    for t in range(3 + 64 + 2):
        ev = _step(run, oracles, t)
        if ev:
            events += 1
            assert all(_pending(run))
        elif t > 0 and t in (3, 3 + 64):
            assert not any(_pending(run))
            check_heads(run, oracles)                 # moved by the attention
    assert events == 2
    check_heads(run, oracles)
    run.close()


@pytest.mark.parametrize("r,every", [(0, 8), (0, 1), (8, 1)])
def test_moves_with_no_buffer_or_every_step(r, every):
    """No buffer of recent pairs (the newest rows are candidates too), and an
    event at every step (each step's attention moves the previous event's
    rows while the step's own event defers the next moves): rows and sets
    the oracle's, outputs within tolerance, throughout."""
    log("deferred moves r=%d every=%d" % (r, every))
    run = Run(L=2, Hq=8, Hkv=2, K=30, lps=[4, 0, 13], r=r, every=every, attn_split=ONE_SPLIT)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    events = 0
    for t in range(90):
        ev = _step(run, oracles, t)
        events += bool(ev)
        if ev:
            assert all(_pending(run))
        if t % 17 == 16:
            check_heads(run, oracles)                 # reading rows moves them first
    assert events >= (6 if every > 1 else 50)     # from step ~31 on
    check_heads(run, oracles)
    run.close()


@pytest.mark.parametrize("K,lps,mode,every", [
    (35, [35, 7, 35], B.RA_BUDGET_TOTAL, 64),      # two of the heads keep no generated row
    (0, [0, 5, 32], B.RA_BUDGET_EVICTABLE, 64),    # nothing kept; the first has no prompt
    (2, [0, 33, 64], B.RA_BUDGET_EVICTABLE, 32),
])
def test_moves_when_whole_blocks_are_dropped(K, lps, mode, every):
    """Events that drop whole 32-row blocks, so that a wavefront of the
    moving attention sees only dropped rows in its first block (or in all of
    its blocks): its softmax state must stay empty rather than turn NaN, and
    the outputs, sets and rows stay the oracle's through every event."""
    log("deferred moves, whole blocks dropped: K=%d lps=%s mode=%d every=%d" % (K, lps, mode,
                                                                             every))
    run = Run(L=2, Hq=8, Hkv=2, K=K, lps=lps, r=0, every=every, mode=mode,
              attn_split=ONE_SPLIT)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    events = 0
    after_event = False
    for t in range(3 * every + 8):
        ev = _step(run, oracles, t)               # every output within tolerance
        if after_event:
            check_heads(run, oracles)
        if ev:
            events += 1
            assert all(_pending(run))
        after_event = bool(ev)
    assert events >= 3
    run.close()


@pytest.mark.parametrize("layout,every,r,split", [
    (B.RA_LAYOUT_CHRONOLOGICAL, 1024, 0, ONE_SPLIT),   # up to 1,024 drops per head, deferred
    (B.RA_LAYOUT_CHRONOLOGICAL, 256, 64, 0),           # split heads: moved on their own first
    (B.RA_LAYOUT_HOLE_FILL, 1024, 16, 0),
    (B.RA_LAYOUT_PAGED, 512, 64, 0),
])
def test_large_trigger_periods(layout, every, r, split):
    """Trigger periods up to the largest allowed (1,024 steps), so that an
    event drops up to ~1,000 rows per head: the drop lists, the moving
    attention's scan of them across many blocks, the hole-fill moves and the
    paged rewrite at that size.  Outputs checked every eighth step and at
    the step after each event, sets and rows after each event."""
    log("large trigger period layout=%d every=%d r=%d split=%d" % (layout, every, r, split))
    run = Run(L=1, Hq=8, Hkv=2, K=100, lps=[5, 40], r=r, every=every, layout=layout,
              attn_split=split, page_rows=64)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    events, after = 0, False
    for t in range(2 * every + 3):
        outs, ev = run.step()
        check = after or t % 8 == 0
        if check:
            outs = outs.float().cpu()
        for o in oracles:
            o.rep.append()
            if check:
                attn_err(outs[0, o.slot], o.attend(0, o.rep.step - 1), B.RA_BF16, (t, o.slot))
            o.rep.end_step()
        if after:
            check_heads(run, oracles)
        if ev:
            events += 1
            if split == ONE_SPLIT:
                assert all(_pending(run))
        after = bool(ev)
    assert events == 2
    check_heads(run, oracles)
    run.close()
