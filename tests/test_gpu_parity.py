"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Kept-position sets and the compacted key/value rows must match bit-exactly;
attention outputs within max abs error 1e-5 (fp32) / 2e-2 (bf16) of the
fp64 oracle, the tolerances the workloads fix.  Inputs come from the seeded
workload generator; the oracle computes its own kept sets from the seeds.
"""

import numpy as np
import pytest
import torch

from gpu_harness import TOL, attn_err, OracleSeq, Run, log, max_abs
from gpu_harness import check_heads as _check_heads
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu

@pytest.mark.parametrize("layout", [B.RA_LAYOUT_CHRONOLOGICAL, B.RA_LAYOUT_HOLE_FILL, B.RA_LAYOUT_PAGED])
@pytest.mark.parametrize("dtype", [B.RA_BF16, B.RA_F32])
def test_small_decode_parity(dtype, layout):
    """Three sequences (prompts 5, 0, 17), r=8, every=8, K=40, 150 steps:
    every output, and every head's positions and rows after every event."""
    log("small decode parity dtype=%d layout=%d" % (dtype, layout))
    run = Run(L=2, Hq=4, Hkv=2, K=40, lps=[5, 0, 17], r=8, every=8, dtype=dtype,
              layout=layout)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    worst = 0.0
    events = 0
    for t in range(150):
        outs, ev = run.step()
        outs = outs.float().cpu()
        for o in oracles:
            o.rep.append()
            for layer in range(run.L):
                want = o.attend(layer, t)
                err = attn_err(outs[layer, o.slot], want, dtype, (t, o.slot, layer,))
                worst = max(worst, err)
            o.rep.end_step()
        if ev:
            events += 1
            _check_heads(run, oracles)
    log("  events=%d worst=%.3g" % (events, worst))
    assert events >= 10
    run.close()


@pytest.mark.parametrize("lp,K,r,every,mode,layout", [
    (37, 100, 16, 16, B.RA_BUDGET_EVICTABLE, 0),
    (0, 64, 0, 1, B.RA_BUDGET_EVICTABLE, 0),
    (300, 300, 64, 64, B.RA_BUDGET_TOTAL, 0),        # k_keep = 0
    (5, 1000, 64, 64, B.RA_BUDGET_EVICTABLE, 0),
    (129, 8192, 64, 64, B.RA_BUDGET_EVICTABLE, 0),   # 8256 candidates
    (37, 100, 16, 16, B.RA_BUDGET_EVICTABLE, 1),
    (3, 50, 40, 8, B.RA_BUDGET_EVICTABLE, 1),        # r > every: recent rows move
    (0, 64, 0, 1, B.RA_BUDGET_EVICTABLE, 1),
    (129, 8192, 64, 64, B.RA_BUDGET_EVICTABLE, 1),
    (37, 100, 16, 16, B.RA_BUDGET_EVICTABLE, 2),
    (0, 64, 0, 1, B.RA_BUDGET_EVICTABLE, 2),
    (300, 300, 64, 64, B.RA_BUDGET_TOTAL, 2),
    (129, 8192, 64, 64, B.RA_BUDGET_EVICTABLE, 2),
])
def test_fast_forward_and_evict_now(lp, K, r, every, mode, layout):
    """Positions-only fast forward and explicit events at arbitrary steps
    keep the same sets as the oracle; rows written afterwards are compacted
    exactly by a full event."""
    log("fast forward lp=%d K=%d r=%d every=%d mode=%d layout=%d" % (lp, K, r, every, mode, layout))
    run = Run(L=2, Hq=2, Hkv=2, K=K, lps=[lp, max(0, lp - 3)], r=r, every=every, mode=mode,
              seeds=[2**63 + 11, 5], rids=[2**40 + 1, 9], layout=layout)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    rng = np.random.default_rng(lp + K)
    for rep in range(3 if K <= 1000 else 1):
        n = int(rng.integers(1, 2 * (K + r + every)))
        run.fast_forward(n)
        for o in oracles:
            o.advance(n)
        _check_heads(run, oracles, rows=False)
        for s in range(run.n):
            run.materialise(s)
        # append a few rows so the event has candidates, then evict now
        for _ in range(int(rng.integers(1, max(2, every)))):
            run.step()
            for o in oracles:
                o.rep.append()
                o.rep.end_step()
        for s in range(run.n):
            B.ra_evict_now(run.h, s)
            oracles[s].rep.evict_now()
        _check_heads(run, oracles, rows=True)
    run.close()


POLICIES = [(B.RA_POLICY_SHARED, 1), (B.RA_POLICY_BLOCK, 4), (B.RA_POLICY_BLOCK, 64),
            (B.RA_POLICY_RECENCY, 1)]


@pytest.mark.parametrize("layout", [B.RA_LAYOUT_CHRONOLOGICAL, B.RA_LAYOUT_HOLE_FILL, B.RA_LAYOUT_PAGED])
@pytest.mark.parametrize("policy,block", POLICIES)
def test_policy_decode_parity(policy, block, layout):
    """The diagnostic policies (shared draw, block-wise, recency + prompt):
    same kept sets, rows and attention outputs as the oracle."""
    log("policy decode parity policy=%d block=%d layout=%d" % (policy, block, layout))
    run = Run(L=2, Hq=4, Hkv=2, K=40, lps=[5, 0, 17], r=8, every=8, layout=layout,
              policy=policy, block=block)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    worst, events = 0.0, 0
    for t in range(120):
        outs, ev = run.step()
        outs = outs.float().cpu()
        for o in oracles:
            o.rep.append()
            for layer in range(run.L):
                err = attn_err(outs[layer, o.slot], o.attend(layer, t), B.RA_BF16, (t, o.slot, layer,))
                worst = max(worst, err)
            o.rep.end_step()
        if ev:
            events += 1
            _check_heads(run, oracles)
    log("  events=%d worst=%.3g" % (events, worst))
    assert events >= 8
    run.close()


@pytest.mark.parametrize("layout", [B.RA_LAYOUT_CHRONOLOGICAL, B.RA_LAYOUT_HOLE_FILL, B.RA_LAYOUT_PAGED])
@pytest.mark.parametrize("policy,block", POLICIES + [(B.RA_POLICY_BLOCK, 16)])
def test_policy_large_select(policy, block, layout):
    """8256 candidates per head (the 1024-thread select): kept sets after a
    fast forward and an explicit event, with rows compacted exactly."""
    log("policy large select policy=%d block=%d layout=%d" % (policy, block, layout))
    run = Run(L=2, Hq=2, Hkv=2, K=8192, lps=[129, 40], r=64, every=64, layout=layout,
              policy=policy, block=block, seeds=[2**63 + 11, 5], rids=[2**40 + 1, 9])
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    n = 8192 + 3 * 64 + 17
    run.fast_forward(n)
    for o in oracles:
        o.advance(n)
    _check_heads(run, oracles, rows=False)
    for s in range(run.n):
        run.materialise(s)
    for _ in range(5):
        run.step()
        for o in oracles:
            o.rep.append()
            o.rep.end_step()
    for s in range(run.n):
        B.ra_evict_now(run.h, s)
        oracles[s].rep.evict_now()
    _check_heads(run, oracles, rows=True)
    run.close()


@pytest.mark.parametrize("K,layout", [
    (20000, B.RA_LAYOUT_CHRONOLOGICAL),
    (20000, B.RA_LAYOUT_HOLE_FILL),
    (32704, B.RA_LAYOUT_CHRONOLOGICAL),   # K + every = 32768 candidates, the largest
    (32640, B.RA_LAYOUT_HOLE_FILL),       # K + every + r = 32768
    (32704, B.RA_LAYOUT_PAGED),
])
def test_largest_select(K, layout):
    """More than 16,384 candidates per head (the 1024-thread select with 32
    keys per thread, up to the largest candidate count the library accepts):
    kept sets after a positions-only fast forward through several events and
    after an explicit event, with the rows compacted exactly."""
    log("largest select K=%d layout=%d" % (K, layout))
    run = Run(L=1, Hq=2, Hkv=2, K=K, lps=[129, 3], r=64, every=64, layout=layout,
              seeds=[2**63 + 11, 5], rids=[2**40 + 1, 9])
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    n = K + 5 * 64 + 17
    run.fast_forward(n)
    for o in oracles:
        o.advance(n)
    assert oracles[0].rep.event >= 3
    _check_heads(run, oracles, rows=False)
    for s in range(run.n):
        run.materialise(s)
    for _ in range(5):
        run.step()
        for o in oracles:
            o.rep.append()
            o.rep.end_step()
    for s in range(run.n):
        B.ra_evict_now(run.h, s)
        oracles[s].rep.evict_now()
    _check_heads(run, oracles, rows=True)
    run.close()


@pytest.mark.parametrize("C,layout", [
    (c, B.RA_LAYOUT_CHRONOLOGICAL) for c in
    (1024, 1025, 2048, 2049, 3072, 3073, 5120, 5121, 9216, 9217, 16384, 16385)
] + [(3073, B.RA_LAYOUT_HOLE_FILL), (16385, B.RA_LAYOUT_HOLE_FILL),
      (5121, B.RA_LAYOUT_PAGED), (16385, B.RA_LAYOUT_PAGED)])
def test_select_size_boundaries(C, layout):
    """An explicit event with exactly C candidates per head, on and just past
    each boundary of the selection's scores-per-thread builds (1,024 threads
    x 1, 2, 3, 5, 9, 16): kept sets and compacted rows as the oracle's.  With
    a trigger period of 1,024 steps nothing is evicted during the positions-
    only fast forward of C + r steps, so the event sees all C positions."""
    log("select size boundary C=%d layout=%d" % (C, layout))
    r = 64
    run = Run(L=1, Hq=2, Hkv=2, K=C - 64, lps=[129, 3], r=r, every=1024, layout=layout,
              seeds=[2**63 + 11, 5], rids=[2**40 + 1, 9])
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    run.fast_forward(C + r)
    for o in oracles:
        o.advance(C + r)
        assert o.rep.event == 0
    for s in range(run.n):
        run.materialise(s)
        info = B.ra_get_seq_info(run.h, s)
        assert info.len - info.prompt_len - r == C
    for s in range(run.n):
        B.ra_evict_now(run.h, s)
        oracles[s].rep.evict_now()
    _check_heads(run, oracles, rows=True)
    run.close()


def test_evict_now_rejects_oversize_selection():
    """Under the external policy rows pile up past the budget; an explicit
    event that would examine more than 32,768 slots is refused on the host
    (nothing is launched) and leaves the state as it was."""
    cfg = B.make_config(1, 2, 1, 32704, 64, 64, B.RA_BUDGET_EVICTABLE, B.RA_BF16, 1,
                        policy=B.RA_POLICY_EXTERNAL)
    cache = B.Cache(cfg, B.ra_seq_rows(cfg, 1))
    h = cache.handle
    B.ra_seq_begin(h, 0, 1, 3, 0, None, None)
    info = B.ra_get_seq_info(h, 0)
    B.ra_fast_forward(h, info.cap - info.len)
    before = B.ra_get_seq_info(h, 0)
    assert before.len == before.cap
    with pytest.raises(B.RandAttnError) as err:
        B.ra_evict_now(h, 0)
    assert err.value.status == B.RA_ERR_UNSUPPORTED
    after = B.ra_get_seq_info(h, 0)
    assert (after.len, after.event) == (before.len, before.event)
    cache.close()


# (tag, KV heads, group, batch, K, wavefronts per item the plan must pick,
#  layout)
PLAN_CASES = [
    ("12 wavefronts, 1 split", 8, 2, 25, 7600, 12, B.RA_LAYOUT_CHRONOLOGICAL),
    ("12 wavefronts, 2 splits", 8, 2, 16, 15400, 12, B.RA_LAYOUT_CHRONOLOGICAL),
    ("12 wavefronts, 2 splits, paged", 8, 2, 16, 15400, 12, B.RA_LAYOUT_PAGED),
    ("8 wavefronts, 2 splits", 8, 2, 16, 4000, 8, B.RA_LAYOUT_CHRONOLOGICAL),
    ("8 wavefronts, 2 splits, paged", 8, 2, 16, 4000, 8, B.RA_LAYOUT_PAGED),
    ("4 wavefronts, 4 splits", 4, 2, 16, 2000, 4, B.RA_LAYOUT_CHRONOLOGICAL),
    ("320 heads", 8, 2, 40, 600, 4, B.RA_LAYOUT_CHRONOLOGICAL),
    ("800 heads", 8, 1, 100, 300, 4, B.RA_LAYOUT_CHRONOLOGICAL),
]


def _arrivals_zero(run):
    """The split arrival counters (the tail of the metadata buffer, one int32
    per slot and KV head, rounded up to 256 bytes) are zero between launches:
    the last split of every head reset its counter."""
    torch.cuda.synchronize()
    n = -(-4 * run.max_seqs * run.Hkv // 256) * 256
    return int(run.cache.meta[-n:].count_nonzero()) == 0


@pytest.mark.parametrize("tag,Hkv,G,Bsz,K,waves,layout", PLAN_CASES)
def test_attention_plans(tag, Hkv, G, Bsz, K, waves, layout):
    """Each branch of the attention launch plan, on a ragged batch (prompts
    and generated lengths differ per sequence): every query head of every
    sequence against the oracle for two steps, the second after the
    sequences that were due have evicted.  Heads of several splits are merged
    by their last split (or, in the contiguous 12-wavefront build, by the
    merge kernel); the split counters are zero afterwards."""
    log("attention plan: %s" % tag)
    rng = np.random.default_rng(Bsz * 31 + K)
    lps = rng.integers(0, 300, Bsz).tolist()
    gens = sorted(rng.integers(K + 70, K + 700, Bsz).tolist(), reverse=True)
    run = Run(L=1, Hq=Hkv * G, Hkv=Hkv, K=K, lps=lps, r=64, every=64, begin=False,
              write_prompt=False, wl_seed=77, layout=layout, page_rows=64)
    for b in range(Bsz):
        run.begin(b)
        nxt = gens[b + 1] if b + 1 < Bsz else 0
        if gens[b] > nxt:
            run.fast_forward(gens[b] - nxt)
    for b in range(Bsz):
        run.materialise(b)
    _, _, w = B.ra_attention_plan(run.h)
    assert w == waves, (tag, w)
    oracles = [OracleSeq(run, b, heads=[(0, g) for g in range(Hkv)]) for b in range(Bsz)]
    for b, o in enumerate(oracles):
        o.advance(gens[b])
    worst = 0.0
    for i in range(66):
        outs, _ = run.step()
        check = i in (0, 65)
        if check:
            outs = outs.float().cpu()
        for b, o in enumerate(oracles):
            o.rep.append()
            if check:
                err = attn_err(outs[0, b], o.attend(0, gens[b] + i), B.RA_BF16, (tag, i, b,))
                worst = max(worst, err)
            o.rep.end_step()
    assert _arrivals_zero(run)
    log("  worst %.3g" % worst)
    run.close()


def test_batching_invariance():
    """A request keeps the same sets alone in slot 0 and inside a batch in
    slot 3 (the scores depend on the request, not on the memory slot)."""
    log("batching invariance")
    alone = Run(L=1, Hq=4, Hkv=4, K=50, lps=[20], r=8, every=8, seeds=[99], rids=[4242])
    batch = Run(L=1, Hq=4, Hkv=4, K=50, lps=[3, 40, 7, 20], r=8, every=8,
                seeds=[1, 2, 3, 99], rids=[1, 2, 3, 4242])
    for _ in range(200):
        alone.step()
        batch.step()
    for g in range(4):
        assert np.array_equal(alone.positions(0, 0, g), batch.positions(3, 0, g))
        ka, va = alone.rows(0, 0, g)
        kb, vb = batch.rows(3, 0, g)
        assert torch.equal(ka, kb) and torch.equal(va, vb)
    alone.close()
    batch.close()


@pytest.mark.parametrize("dtype", [B.RA_BF16, B.RA_F32])
@pytest.mark.parametrize("Hq,Hkv,split", [(1, 1, 32), (4, 2, 64), (10, 2, 0),
                                          (8, 1, 32), (16, 1, 96), (40, 8, 0)])
def test_attention_shapes(dtype, Hq, Hkv, split):
    """Group sizes 1..16, forced small splits (many partials merged), ragged
    lengths within a batch, and a first step with a single cached row."""
    log("attention shapes dtype=%d Hq=%d Hkv=%d split=%d" % (dtype, Hq, Hkv, split))
    lps = [0, 1, 31, 32, 33, 250]
    run = Run(L=1, Hq=Hq, Hkv=Hkv, K=200, lps=lps, r=16, every=16, dtype=dtype,
              attn_split=split)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    checked = 0
    for t in range(70):
        outs, _ = run.step()
        outs = outs.float().cpu()
        for o in oracles:
            o.rep.append()
            if t in (0, 1, 2, 31, 32, 47, 69):
                err = attn_err(outs[0, o.slot], o.attend(0, t), dtype, (t, o.slot,))
                checked += 1
            o.rep.end_step()
    assert checked == 7 * len(lps)
    assert _arrivals_zero(run)
    run.close()


@pytest.mark.parametrize("every,n_events", [(64, 11), (1, 704)])
def test_tiny_config_full_run(every, n_events):
    """The tiny single-layer case in full: 1 sequence, 4 query / 2 KV heads,
    fp32, prompt 128, r=64, K=256, 1024 decode steps, evicting once over
    budget -- at every 64th step (the paper's periodic trigger, the headline
    reading: 11 events) or at every step (the case's own "whenever the
    evictable entries exceed K": 704 events, from step 321 on).  Every output
    of every step within 1e-5 of the fp64 oracle; kept sets and rows
    bit-exact after every event."""
    log("tiny config full run, trigger every %d" % every)
    run = Run(L=1, Hq=4, Hkv=2, K=256, lps=[128], r=64, every=every, dtype=B.RA_F32,
              scaled=False, seeds=[1000], rids=[0])
    o = OracleSeq(run, 0)
    worst = 0.0
    events = 0
    for t in range(1024):
        outs, ev = run.step()
        o.rep.append()
        err = attn_err(outs[0, 0].cpu(), o.attend(0, t), B.RA_F32, (t,))
        worst = max(worst, err)
        o.rep.end_step()
        if ev:
            events += 1
            _check_heads(run, [o])
    log("  events=%d worst=%.3g" % (events, worst))
    assert events == n_events
    run.close()


def test_external_policy_evict_now_bounds():
    """Under the external policy nothing evicts at the end of a step; an
    explicit event with up to 1024 rows over budget uses Random Attention's
    keys (same set as the oracle), and more than that is refused before any
    launch."""
    log("external policy: evict-now bounds")
    from oracle.evict import SequenceReplay
    run = Run(L=1, Hq=2, Hkv=1, K=8, lps=[3], r=4, every=1024,
              policy=B.RA_POLICY_EXTERNAL, seeds=[17], rids=[5])
    for _ in range(1030):
        _, ev = run.step()
        assert ev == 0
    B.ra_evict_now(run.h, 0)                        # 1033 rows: 1018 over budget
    rep = SequenceReplay(3, 8, 4, 10 ** 9, 17, 5, [(0, 0)])   # no end-of-step trigger
    rep.advance(1030)
    rep.evict_now()
    assert np.array_equal(run.positions(0, 0, 0), rep.P[(0, 0)])
    for _ in range(1030):                           # 1030 more rows: 1042 over budget
        run.step()
    with pytest.raises(B.RandAttnError) as e:
        B.ra_evict_now(run.h, 0)
    assert e.value.status == B.RA_ERR_STATE
    run.close()
