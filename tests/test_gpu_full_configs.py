"""Parity at the full sizes of the measured workloads, in the launch
configuration bench.py times (all sequences, all layers, the library's own
split choice).

Each case fast-forwards every sequence (positions only) to shortly before
step 32768 of a 32k-token generation, materialises the kept rows from the
seeded generator, then decodes the last steps, which include an eviction
event.  Sampled (sequence, layer, KV head) sites are replayed by the oracle
from the seeds alone: their kept positions must match bit-exactly after the
event, and every query head of the sampled sites must be within 2e-2 of the
fp64 oracle and within one bf16 half-ulp of it plus a small floor, element by
element.  Every cached position has its own key and value row (no input
ring), and queries come from their own pool, so no query meets a copy of
itself among the keys.
"""

import numpy as np
import pytest
import torch

from gpu_harness import OracleSeq, Run, attn_err, log, note
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu

# (layers, q heads, kv heads, batch, prompt, K, seed)
SHAPES = {
    "qwen3-4b": (36, 32, 8, 16, 512, 8192, 1001),
    "qwen3-14b": (40, 40, 8, 32, 1024, 8192, 1002),
    "qwen3-32b": (64, 64, 8, 16, 4096, 4096, 1003),
}
T = 32768
WINDOW = 72          # steps decoded on the GPU (events at 32704 and 32768)


@pytest.mark.parametrize("name,layout,graph", [(n, 0, False) for n in sorted(SHAPES)] +
                         [("qwen3-14b", 1, False), ("qwen3-14b", 2, False),
                          ("qwen3-14b", 0, True)])
def test_full_size(name, layout, graph):
    """`graph`: the window decoded in graph mode (the plan fixed from the
    regions' capacity, every head's eviction launched at the end of every
    step and decided on the device), as the per-step HIP graphs of bench.py
    --graph run it."""
    L, Hq, Hkv, Bsz, lp, K, seed = SHAPES[name]
    log("full size %s layout %d graph %d: L=%d Hq=%d Hkv=%d B=%d lp=%d K=%d"
        % (name, layout, graph, L, Hq, Hkv, Bsz, lp, K))
    run = Run(L=L, Hq=Hq, Hkv=Hkv, K=K, lps=[lp] * Bsz, r=64, every=64,
              seeds=[seed * 1000003 + b for b in range(Bsz)], rids=list(range(Bsz)),
              wl_seed=seed, write_prompt=False, layout=layout, page_rows=64)
    t0 = T - WINDOW
    run.fast_forward(t0)
    for b in range(Bsz):
        run.materialise(b)
    log("  state at step %d materialised" % t0)
    sites = [(0, 0, 0), (Bsz - 1, L - 1, Hkv - 1), (Bsz // 2, L // 2, 1),
             (1, L - 2, Hkv // 2), (Bsz - 2, 3, Hkv - 2), (Bsz // 3, L // 3, 3)]
    heads = {}
    for b, l, g in sites:
        heads.setdefault(b, []).append((l, g))
    oracles = {b: OracleSeq(run, b, heads=h) for b, h in heads.items()}
    for o in oracles.values():
        o.advance(t0)
    log("  oracle replay done")
    check_steps = {0, 8, 31, 32, 33, WINDOW - 1}   # 8: right after the event at step 32704
    worst = 0.0
    if graph:
        B.ra_graph_mode(run.h, 1)
    for i in range(WINDOW):
        outs, ev = run.step()
        for o in oracles.values():
            o.rep.append()
        if i in check_steps:
            for b, l, g in sites:
                o = oracles[b]
                want = o.attend_group(l, g, t0 + i)
                got = outs[l, b, g * run.G:(g + 1) * run.G].float().cpu()
                err = attn_err(got, want, B.RA_BF16, (name, i, b, l, g))
                worst = max(worst, err)
        for o in oracles.values():
            o.rep.end_step()
    if graph:
        B.ra_graph_mode(run.h, 0)          # the device's records back into the mirror
        info = B.ra_get_seq_info(run.h, 0)
        assert (info.step, info.event) == (oracles[0].rep.step, oracles[0].rep.event)
    for b, l, g in sites:
        got = (run.sorted_positions(b, l, g) if layout == B.RA_LAYOUT_HOLE_FILL
               else run.positions(b, l, g))
        want = oracles[b].rep.P[(l, g)]
        assert np.array_equal(got, want), (name, b, l, g)
    assert oracles[0].rep.event >= 2
    note("events", oracles[0].rep.event)
    log("  %s ok: worst %.3g, events %d" % (name, worst, oracles[0].rep.event))
    run.close()
    torch.cuda.empty_cache()


def test_full_size_phi4_ragged():
    """Phi-4-reasoning-shaped ragged batch: 40 layers, 40 Q / 10 KV heads,
    128 sequences with prompts ~U[64, 2048] and generated lengths
    ~U[4096, 32768] (seeded), K=8192, r=64.  Sequences are begun longest
    first and fast-forwarded between begins, so each reaches its own step
    count through the real sampler; the decoded window then evicts every
    sequence on its own phase."""
    L, Hq, Hkv, Bsz, K, seed = 40, 40, 10, 128, 8192, 1004
    rng = np.random.default_rng(seed)
    lps = rng.integers(64, 2049, Bsz).tolist()
    gens = sorted(rng.integers(4096, 32769, Bsz).tolist(), reverse=True)
    log("phi4 ragged: prompts %d..%d, generated %d..%d" % (min(lps), max(lps), gens[-1], gens[0]))
    run = Run(L=L, Hq=Hq, Hkv=Hkv, K=K, lps=lps, r=64, every=64,
              seeds=[seed * 1000003 + b for b in range(Bsz)], rids=list(range(Bsz)),
              wl_seed=seed, write_prompt=False, begin=False)
    for b in range(Bsz):
        run.begin(b)
        nxt = gens[b + 1] if b + 1 < Bsz else 0
        if gens[b] - nxt > 0:
            run.fast_forward(gens[b] - nxt)
    assert run.steps == gens
    for b in range(Bsz):
        run.materialise(b)
    log("  snapshot materialised")
    sites = [(0, 0, 0), (Bsz - 1, L - 1, Hkv - 1), (Bsz // 2, 7, 5), (31, L - 1, 0),
             (100, 20, 9), (77, 1, 3)]
    heads = {}
    for b, l, g in sites:
        heads.setdefault(b, []).append((l, g))
    oracles = {b: OracleSeq(run, b, heads=h) for b, h in heads.items()}
    for b, o in oracles.items():
        o.advance(gens[b])
    log("  oracle replay done")
    window = 72
    check_steps = {0, 40, window - 1}
    events = 0
    for i in range(window):
        outs, ev = run.step()
        events += ev
        for o in oracles.values():
            o.rep.append()
        if i in check_steps:
            for b, l, g in sites:
                want = oracles[b].attend_group(l, g, gens[b] + i)
                got = outs[l, b, g * run.G:(g + 1) * run.G].float().cpu()
                attn_err(got, want, B.RA_BF16, ("phi4", i, b, l, g))
        for o in oracles.values():
            o.rep.end_step()
    for b, l, g in sites:
        assert np.array_equal(run.positions(b, l, g), oracles[b].rep.P[(l, g)]), (b, l, g)
    # a sequence is evicted at step t iff t is a multiple of 64 and its
    # evictable rows (t - r during growth, k_keep + 64 in steady state)
    # exceed k_keep, i.e. t > k_keep + r
    expected = sum(1 for g0 in gens for t in range(g0 + 1, g0 + window + 1)
                   if t % 64 == 0 and t > K + 64)
    assert events == expected, (events, expected)
    log("  phi4 ok: %d sequence-events in the window" % events)
    run.close()
    torch.cuda.empty_cache()
