"""Decode steps captured into a HIP graph and replayed (ra_graph_mode).

In graph mode the launches of a step depend on no host state: the attention
plan is fixed for every state the caches can reach, and the end of the step
launches the advance and every head's eviction, each eviction workgroup
reading on the device whether its sequence is due.  One captured step (every
layer's attention and the end of the step) therefore replays correctly at
every later step.  Each replay is checked against the same step issued
directly, in graph mode, on a twin cache (outputs bit-exact: the same kernels
and plan on the same data), with the program's own input copies and a
synchronisation between replays, and against the oracle; leaving graph mode
reads the device's records back into the host mirror, after which the kept
sets and rows are the oracle's and eager decoding goes on.
"""

import numpy as np
import pytest
import torch

from gpu_harness import OracleSeq, Run, attn_err, check_heads, log
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu


def _buffers(run):
    q = torch.zeros(run.L, run.max_seqs, run.Hq, 128, dtype=run.tdtype, device="cuda")
    k = torch.zeros(run.L, run.max_seqs, run.Hkv, 128, dtype=run.tdtype, device="cuda")
    return q, k, torch.zeros_like(k), torch.zeros_like(q)


def _load(run, q, k, v):
    for layer in range(run.L):
        ql, kl, vl = run.step_inputs(layer)
        q[layer].copy_(ql)
        k[layer].copy_(kl)
        v[layer].copy_(vl)


def _issue(run, q, k, v, out, noalloc=False):
    for layer in range(run.L):
        if noalloc:
            run.cache.decode_noalloc(layer, q[layer], k[layer], v[layer], out[layer])
        else:
            run.cache.decode(layer, q[layer], k[layer], v[layer], out[layer])
    return B.ra_end_step(run.h)


def _status(fn, *args):
    try:
        fn(*args)
    except B.RandAttnError as e:
        return e.status
    return B.RA_OK


@pytest.mark.parametrize("layout", [B.RA_LAYOUT_CHRONOLOGICAL, B.RA_LAYOUT_HOLE_FILL])
@pytest.mark.parametrize("dtype,Hq,Hkv,noalloc", [(B.RA_BF16, 8, 2, False),
                                                  (B.RA_BF16, 10, 2, True),
                                                  (B.RA_F32, 4, 2, False)])
def test_graph_replays_match_direct_steps_and_oracle(layout, dtype, Hq, Hkv, noalloc):
    log("graph replays layout=%d dtype=%d Hq=%d noalloc=%d" % (layout, dtype, Hq, noalloc))
    kw = dict(L=2, Hq=Hq, Hkv=Hkv, K=40, lps=[5, 0, 17], r=8, every=8, dtype=dtype,
              layout=layout)
    direct, graph = Run(**kw), Run(**kw)
    oracles = [OracleSeq(graph, s) for s in range(graph.n)]
    for _ in range(64):           # ends on an event step: a deferred move is pending
        direct.step()
        graph.step()
        for o in oracles:
            o.rep.append()
            o.rep.end_step()
    entry = [B.ra_get_seq_info(graph.h, s) for s in range(graph.n)]
    B.ra_graph_mode(direct.h, 1)
    B.ra_graph_mode(graph.h, 1)
    B.ra_graph_mode(graph.h, 1)   # a second entry is a no-op
    assert B.ra_attention_plan(direct.h) == B.ra_attention_plan(graph.h)
    qd, kd, vd, od = _buffers(direct)
    qg, kg, vg, og = _buffers(graph)
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        _issue(graph, qg, kg, vg, og, noalloc)
    worst = 0.0
    for t in range(100):
        _load(direct, qd, kd, vd)
        _load(graph, qg, kg, vg)
        _issue(direct, qd, kd, vd, od, noalloc)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(od, og), t
        outs = og.float().cpu()
        for o in oracles:
            o.rep.append()
            if t % 9 == 0 or t > 95:
                for layer in range(graph.L):
                    worst = max(worst, attn_err(outs[layer, o.slot], o.attend(layer, o.rep.step - 1),
                                                dtype, (t, o.slot, layer)))
            o.rep.end_step()
        direct.steps = [x + 1 for x in direct.steps]
        graph.steps = [x + 1 for x in graph.steps]
    # the mirror is that of the entry until graph mode ends
    for s in range(graph.n):
        info = B.ra_get_seq_info(graph.h, s)
        assert (info.len, info.step, info.event) == (entry[s].len, entry[s].step, entry[s].event)
    B.ra_graph_mode(graph.h, 0)
    B.ra_graph_mode(direct.h, 0)
    B.ra_graph_mode(graph.h, 0)   # a second exit is a no-op
    for o in oracles:
        info = B.ra_get_seq_info(graph.h, o.slot)
        assert info.step == o.rep.step and info.event == o.rep.event
        assert info.len == len(o.rep.P[(0, 0)])
    check_heads(graph, oracles)
    for s in range(graph.n):
        for layer in range(graph.L):
            for h in range(graph.Hkv):
                assert np.array_equal(direct.positions(s, layer, h), graph.positions(s, layer, h))
    # eager decoding goes on from the read-back mirror
    for t in range(20):
        outs, _ = graph.step()
        outs = outs.float().cpu()
        for o in oracles:
            o.rep.append()
            for layer in range(graph.L):
                attn_err(outs[layer, o.slot], o.attend(layer, o.rep.step - 1), dtype, ("after", t))
            o.rep.end_step()
    check_heads(graph, oracles)
    log("  worst %.3g" % worst)
    direct.close()
    graph.close()


def test_graph_mode_refusals():
    """Calls that need the host mirror are refused in graph mode, graph mode
    cannot be entered or left inside a step, the paged layout and the
    external policy cannot enter it; after leaving it every call works and
    the sequences are still the oracle's."""
    log("graph mode refusals")
    run = Run(L=2, Hq=4, Hkv=2, K=40, lps=[5, 17], r=8, every=8)
    oracles = [OracleSeq(run, s) for s in range(run.n)]
    for _ in range(10):
        run.step()
        for o in oracles:
            o.rep.append()
            o.rep.end_step()
    B.ra_graph_mode(run.h, 1)
    st = B.RA_ERR_STATE
    k = torch.empty(run.L, run.Hkv, 40, 128, dtype=torch.bfloat16, device="cuda")
    assert _status(B.ra_seq_end, run.h, 0) == st
    assert _status(B.ra_evict_now, run.h, 0) == st
    assert _status(B.ra_fast_forward, run.h, 1) == st
    assert _status(B.ra_read_rows, run.h, 0, 0, 0, k[0, 0], None) == st
    assert _status(B.ra_read_positions, run.h, 0, 0, 0, 64) == st
    assert _status(B.ra_write_rows, run.h, 0, k, k) == st
    q, kk, v = run.step_inputs(0)
    out = torch.empty(run.max_seqs, run.Hq, 128, dtype=torch.bfloat16, device="cuda")
    run.cache.decode(0, q, kk, v, out)
    assert _status(B.ra_graph_mode, run.h, 0) == st             # inside a step
    q, kk, v = run.step_inputs(1)
    run.cache.decode(1, q, kk, v, out)
    B.ra_end_step(run.h)
    run.steps = [x + 1 for x in run.steps]
    for o in oracles:
        o.rep.append()
        o.rep.end_step()
    B.ra_graph_mode(run.h, 0)
    check_heads(run, oracles)
    run.end(1)
    run.close()
    for layout, policy in ((B.RA_LAYOUT_PAGED, B.RA_POLICY_RANDOM),
                           (B.RA_LAYOUT_CHRONOLOGICAL, B.RA_POLICY_EXTERNAL)):
        other = Run(L=1, Hq=4, Hkv=2, K=40, lps=[5], r=8, every=8, layout=layout,
                    policy=policy)
        assert _status(B.ra_graph_mode, other.h, 1) == B.RA_ERR_UNSUPPORTED
        other.close()
