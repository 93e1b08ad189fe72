#!/usr/bin/env python
"""Decode throughput of the Random Attention hot path on one MI355X.

A step is one decode step of the whole attention stack for every sequence
of the batch: for each layer, append the new key/value and run GQA decode
attention over the compressed cache; then the end-of-step eviction (every
64 steps, per KV head, uniform random, with compaction).  Model projections
and MLPs are not part of the path and are not run.

Default workload: the Qwen3-14B-shaped headline case (40 layers, 40 query /
8 KV heads, head_dim 128, bf16, batch 32, prompt 1024, K=8192, r=64,
eviction every 64 steps) in its steady state at the end of a 32k-token
generation: the state at step 32768 - warmup - steps is reached with the
positions-only fast forward (the same sampler and trigger), the kept rows
are materialised from the seeded generator, then `warmup` untimed and
`steps` timed decode steps run up to step 32768.  Inputs (a 64-step ring of
q, k_new, v_new for every layer) are resident in HBM before timing.
--workload selects the other shapes (Qwen3-4B, Qwen3-32B, and the ragged
Phi-4 batch whose sequences start from their own generated lengths).

Prints one JSON line.  `value` is tokens/s = batch * steps / wall time.
"""

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("decode tokens/s incl. eviction at 32k gen; attention+compaction "
          "HBM GB/s vs peak")
PEAK_HBM_GBS = 8000.0     # MI355X HBM3E, AMD published

WORKLOADS = {
    "qwen3-14b": dict(L=40, Hq=40, Hkv=8, B=32, lp=1024, T=32768, K=8192,
                      desc="Qwen3-14B-shaped attention stack: 40 layers, 40 Q / 8 KV "
                           "heads, head_dim 128, bf16, batch 32, prompt 1024, 32768 "
                           "generated tokens, K=8192, r=64, evict every 64 steps"),
    "qwen3-4b": dict(L=36, Hq=32, Hkv=8, B=16, lp=512, T=32768, K=8192,
                     desc="Qwen3-4B-shaped attention stack: 36 layers, 32 Q / 8 KV "
                          "heads, head_dim 128, bf16, batch 16, prompt 512, 32768 "
                          "generated tokens, K=8192, r=64, evict every 64 steps"),
    "qwen3-32b": dict(L=64, Hq=64, Hkv=8, B=16, lp=4096, T=32768, K=4096,
                      desc="Qwen3-32B-shaped attention stack: 64 layers, 64 Q / 8 KV "
                           "heads, head_dim 128, bf16, batch 16, prompt 4096, 32768 "
                           "generated tokens, K=4096, r=64, evict every 64 steps"),
    "phi4-ragged": dict(L=40, Hq=40, Hkv=10, B=128, lp=None, T=None, K=8192,
                        desc="Phi-4-reasoning-shaped ragged batch: 40 layers, 40 Q / 10 KV "
                             "heads, head_dim 128, bf16, 128 sequences, prompts ~U[64,2048], "
                             "generated lengths ~U[4096,32768] at the window start, K=8192, "
                             "r=64, evict every 64 steps (each sequence on its own phase)"),
}
SEEDS = {"qwen3-4b": 1001, "qwen3-14b": 1002, "qwen3-32b": 1003, "phi4-ragged": 1004}


def sequence_plan(name, w, total, steps=None):
    """Per-sequence (prompt length, step at the start of the warm-up).

    The timed steps of a uniform workload end at the last step of the
    generation; a window shorter than two trigger periods is instead centred
    on the event one period before the end, so that it holds the event and
    the step after it (whose attention moves a deferred event's rows)."""
    import numpy as np
    if name == "phi4-ragged":
        rng = np.random.default_rng(SEEDS[name])
        lps = rng.integers(64, 2049, w["B"]).tolist()
        gens = sorted(rng.integers(4096, 32769, w["B"]).tolist(), reverse=True)
        return lps, gens
    start = w["T"] - total
    if steps is not None and steps < 2 * EVERY:
        start = w["T"] - EVERY - (total - steps) - steps // 2
    return [w["lp"]] * w["B"], [start] * w["B"]
R = 64
EVERY = 64
RING = 64


def code_of(text):
    """Source text without comments and blank space: what the compiler sees
    of it, so that a comment edit does not count as a kernel change."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash(read=None):
    """Hash of the code of the attention and eviction kernels (the traffic
    measured by rocprofv3 counters is reported only while it matches)."""
    h = hashlib.sha256()
    for name in ("attention.hip", "evict.hip"):
        if read is None:
            with open(os.path.join(ROOT, "paper_2609_03430_amd", "csrc", name)) as f:
                text = f.read()
        else:
            text = read(name)
        h.update(code_of(text).encode())
    return h.hexdigest()[:16]


def run_signature(args):
    """The settings that decide which launches a run times."""
    return {"workload": args.workload, "steps": args.steps, "warmup": args.warmup,
            "layout": args.layout, "policy": args.policy,
            "block": args.block if args.policy == "block" else None,
            "attn_split": args.attn_split,
            "page_rows": args.page_rows if args.layout == "paged" else None}


def read_traffic(signature):
    """HBM traffic per attention launch measured with rocprofv3 counters (the
    mean over the timed launches of one run), if a summary for the current
    kernel sources and for a run with the same settings exists under
    profiles/."""
    path = os.path.join(ROOT, "profiles", "attention_traffic_%s.json" % signature["workload"])
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    if d.get("run") != signature:
        return None
    return d.get("hbm_bytes_per_launch")


def host_cpu():
    """The host the CPU baseline ran on: CPUs this process may use, CPUs of
    the machine, and the CPU model."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return {"cpus_usable": len(os.sched_getaffinity(0)), "nproc": os.cpu_count(),
            "cpu_model": model,
            "note": "cores = the BLAS threads the numpy oracle ran with"}


def cpu_baseline(w, seed, lp, t0, steps):
    """The CPU oracle, untuned, on one sequence x one layer x all KV heads for
    `steps` steady-state decode steps (one eviction event included)."""
    import numpy as np
    import torch
    from oracle.attention import gqa_decode
    from oracle.evict import SequenceReplay
    from paper_2609_03430_amd.synth import Workload

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    L, Hq, Hkv, K = w["L"], w["Hq"], w["Hkv"], w["K"]
    wl = Workload(seed, L, Hq, Hkv, 128, torch.bfloat16, True, ring=RING)
    layer, rid = 0, 0
    heads = [(layer, g) for g in range(Hkv)]
    rep = SequenceReplay(lp, K, R, EVERY, seed, rid, heads)
    rep.advance(t0)
    # rows resident in RAM before timing, as the GPU's are in HBM
    new = np.arange(lp + t0, lp + t0 + steps)
    tables = []
    for g in range(Hkv):
        P = np.union1d(rep.P[(layer, g)], new)
        k = wl.k_rows(rid, layer, g, torch.as_tensor(P), lp).double().numpy()
        v = wl.v_rows(rid, layer, g, torch.as_tensor(P), lp).double().numpy()
        tables.append((P, k, v))
    qs = [wl.q_rows(rid, layer, torch.arange(Hq), t0 + s).double().numpy()
          for s in range(steps)]
    t_start = time.perf_counter()
    for s in range(steps):
        rep.append()
        Ks, Vs = [], []
        for g in range(Hkv):
            P, k, v = tables[g]
            idx = np.searchsorted(P, rep.P[(layer, g)])
            Ks.append(k[idx])
            Vs.append(v[idx])
        gqa_decode(qs[s], Ks, Vs)
        rep.end_step()
    elapsed = time.perf_counter() - t_start
    return {
        "value": steps / (elapsed * L),
        "unit": "tokens/s",
        "cores": int(threads),
        "kind": "oracle",
        "host": host_cpu(),
        "sample": ("1 sequence x 1 layer x %d KV heads (%d query heads), %d decode "
                   "steps at steps %d..%d incl. %d eviction event(s), numpy fp64; "
                   "tokens/s = steps / (time x %d layers), i.e. the oracle's rate on "
                   "the whole job" % (Hkv, Hq, steps, t0 + 1, t0 + steps,
                                      len([1 for st, _ in rep.log if st > t0]), L)),
        "seconds": elapsed,
    }


def evict_cost(B, torch, Workload, methods=("random", "snapkv")):
    """Per-layer eviction-round time of a single decoding sequence.

    The paper times one eviction round (scoring + compaction) per layer with
    CUDA events on an idle H200, K=1024, 4096 decode steps (its eviction-cost
    table).  Here: the Qwen3-4B and Qwen3-14B attention shapes, one sequence,
    budget K=1024 counting the prompt (Eq. 1), prompt 300, r=64, every 64:
    52 events in 4096 steps, i.e. 1872 / 2080 per-layer rounds, the paper's
    call counts (after an untimed 1,024-step warm-up copy of the run).  One event covers every layer; per-layer time = event time /
    layers.  Decode time = all attention launches + end-of-step work.
    Random Attention evicts at the end of the step; the score-based rounds
    (external policy) run right after it on the same steps, scored on the
    queries of the last 64 steps, and their time includes that end of step.
    """
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    scorers = {"snapkv": B.RA_SCORER_SNAPKV, "rkv": B.RA_SCORER_RKV,
               "vase": B.RA_SCORER_VASE}
    # "random-holefill": Random Attention's round with the hole-fill layout
    # (the same kept sets; only the surviving rows of the last m slots move)
    layouts = {"random-holefill": B.RA_LAYOUT_HOLE_FILL}
    res = {"metric": "eviction round ms per layer (scoring + selection + compaction)",
           "protocol": "1 sequence, K=1024 incl. prompt 300, r=64, every 64, 4096 "
                       "decode steps from the prompt, distinct rows every step, HIP events, "
                       "after an untimed 1024-step warm-up run per method",
           "shapes": {}}
    for name, (L, Hq, Hkv) in (("qwen3-4b", (36, 32, 8)), ("qwen3-14b", (40, 40, 8))):
        lp, K, steps = 300, 1024, 4096
        # every step's rows are distinct (no input ring): the redundancy term
        # of R-KV sees the near-duplicates of the generator's row collisions,
        # not a 64-step period
        wl = Workload(2000, L, Hq, Hkv, 128, torch.bfloat16, True, ring=None, device=dev)
        ls = torch.arange(L, device=dev).view(-1, 1, 1)
        gs = torch.arange(Hkv, device=dev).view(1, -1, 1)
        ps = torch.arange(lp, device=dev).view(1, 1, -1)
        kp = wl.k_rows(0, ls, gs, ps, lp).contiguous()
        vp = wl.v_rows(0, ls, gs, ps, lp).contiguous()
        zero = torch.zeros(steps, dtype=torch.long, device=dev)
        st = torch.arange(steps, device=dev)
        qs = torch.stack([wl.q_step(zero, l, st) for l in range(L)], 1)   # [T][L][Hq][128]
        ks = torch.empty(steps, L, Hkv, 128, dtype=torch.bfloat16, device=dev)
        vs = torch.empty_like(ks)
        for l in range(L):
            ks[:, l], vs[:, l] = wl.kv_step(zero, l, lp + st, zero + lp)
        out = torch.empty(1, Hq, 128, dtype=torch.bfloat16, device=dev)
        res["shapes"][name] = {"layers": L, "kv_heads": Hkv}
        for method, run_steps in [(m, n) for m in methods for n in (1024, steps)]:
            # each method first runs an untimed 1,024-step copy of the protocol
            # (4 rounds), so that no round pays a kernel's first-launch cost
            timed = run_steps == steps
            scored = method in scorers
            policy = B.RA_POLICY_EXTERNAL if scored else B.RA_POLICY_RANDOM
            cfg = B.make_config(L, Hq, Hkv, K, R, EVERY, B.RA_BUDGET_TOTAL, B.RA_BF16, 1,
                                policy=policy,
                                layout=layouts.get(method, B.RA_LAYOUT_CHRONOLOGICAL))
            cache = B.Cache(cfg, B.ra_seq_rows(cfg, lp), device=dev)
            h = cache.handle
            B.ra_seq_begin(h, 0, lp, 77, 0, kp, vp)
            if scored:
                prm = B.make_scorer(scorers[method], vase_seed=99)
                scratch = torch.empty(B.ra_scored_scratch_bytes(cfg, lp) // 4 + 1,
                                      dtype=torch.int32, device=dev)
            torch.cuda.synchronize()
            ev, dec = [], []
            for t in range(run_steps):
                due = False
                if scored and (t + 1) % EVERY == 0:
                    due = B.ra_get_seq_info(h, 0).len + 1 - R > K
                    if due:   # the window: queries of steps t - 63 .. t, oldest first
                        qwin = qs[t - 63:t + 1].permute(1, 2, 0, 3).unsqueeze(0).contiguous()
                a0 = torch.cuda.Event(enable_timing=True)
                a1 = torch.cuda.Event(enable_timing=True)
                a0.record(stream)
                for l in range(L):
                    B.ra_decode_attention(h, l, qs[t, l].unsqueeze(0), ks[t, l].unsqueeze(0),
                                          vs[t, l].unsqueeze(0), out, cache.workspace, stream)
                a1.record(stream)
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                n = B.ra_end_step(h, stream)
                if due:
                    B.ra_scored_evict(h, 0, 1, prm, qwin, scratch, stream)
                    n = 1
                e1.record(stream)
                dec.append((a0, a1))
                (ev if n else dec).append((e0, e1))
            torch.cuda.synchronize()
            if not timed:
                cache.close()
                continue
            ev_ms = [a.elapsed_time(b) for a, b in ev]
            dec_ms = sum(a.elapsed_time(b) for a, b in dec) + sum(ev_ms)
            res["shapes"][name][method] = {
                "events": len(ev_ms),
                "per_layer_rounds": len(ev_ms) * L,
                "ms_per_event_all_layers": sum(ev_ms) / len(ev_ms),
                "ms_per_layer_round": sum(ev_ms) / len(ev_ms) / L,
                "percent_of_decode": 100.0 * sum(ev_ms) / dec_ms,
            }
            cache.close()
            torch.cuda.empty_cache()
    return res


def tiny_cpu_baseline(lp, K, T, Hq, Hkv, seed, rid):
    """The CPU oracle, untuned, on the whole tiny run: the same 1024 steps and
    eviction events, fp64 attention over the kept rows (rows resident in RAM
    before timing)."""
    import numpy as np
    import torch
    from oracle.attention import gqa_decode
    from oracle.evict import SequenceReplay
    from paper_2609_03430_amd.synth import Workload

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    wl = Workload(1000, 1, Hq, Hkv, 128, torch.float32, False)
    allp = torch.arange(lp + T)
    k = [wl.k_rows(rid, 0, g, allp, lp).double().numpy() for g in range(Hkv)]
    v = [wl.v_rows(rid, 0, g, allp, lp).double().numpy() for g in range(Hkv)]
    qs = [wl.q_rows(rid, 0, torch.arange(Hq), t).double().numpy() for t in range(T)]
    rep = SequenceReplay(lp, K, R, EVERY, seed, rid, [(0, g) for g in range(Hkv)])
    t_start = time.perf_counter()
    for t in range(T):
        rep.append()
        gqa_decode(qs[t], [k[g][rep.P[(0, g)]] for g in range(Hkv)],
                   [v[g][rep.P[(0, g)]] for g in range(Hkv)])
        rep.end_step()
    seconds = time.perf_counter() - t_start
    return {"value": seconds * 1e6 / T, "unit": "us/step", "cores": threads,
            "kind": "oracle", "events": rep.event,
            "sample": "the whole tiny run (%d steps from the prompt, every eviction event), "
                      "numpy fp64" % T, "seconds": seconds}


def tiny_latency(B, torch, Workload, with_cpu=True, graph=False):
    """Per-step latency of the tiny case: 1 layer, 4 query / 2 KV heads,
    head_dim 128, fp32 N(0,1) rows, prompt 128, r=64, K=256, eviction every
    64 steps, 1024 decode steps from the pinned prompt (11 events).  A
    latency case, not a roofline one: the cache is under 1 MB."""
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    L, Hq, Hkv, K, lp, T = 1, 4, 2, 256, 128, 1024
    cfg = B.make_config(L, Hq, Hkv, K, R, EVERY, B.RA_BUDGET_EVICTABLE, B.RA_F32, 1)
    wl = Workload(1000, L, Hq, Hkv, 128, torch.float32, False, device=dev)
    ls = torch.arange(L, device=dev).view(-1, 1, 1)
    gs = torch.arange(Hkv, device=dev).view(1, -1, 1)
    ps = torch.arange(lp, device=dev).view(1, 1, -1)
    kp = wl.k_rows(0, ls, gs, ps, lp).contiguous()
    vp = wl.v_rows(0, ls, gs, ps, lp).contiguous()
    zero = torch.zeros(T, dtype=torch.long, device=dev)
    st = torch.arange(T, device=dev)
    qs = wl.q_step(zero, 0, st)                                # [T][Hq][128]
    ks, vs = wl.kv_step(zero, 0, lp + st, zero + lp)           # [T][Hkv][128]
    out = torch.empty(1, Hq, 128, dtype=torch.float32, device=dev)
    result = {}
    for run in ("warm-up", "timed"):
        cache = B.Cache(cfg, B.ra_seq_rows(cfg, lp), device=dev)
        h = cache.handle
        B.ra_seq_begin(h, 0, lp, 1000 * 1000003, 0, kp, vp)
        torch.cuda.synchronize()

        def issue(s):
            n = 0
            for t in range(T):
                B.ra_decode_attention(h, 0, qs[t].unsqueeze(0), ks[t].unsqueeze(0),
                                      vs[t].unsqueeze(0), out, cache.workspace, s)
                n += B.ra_end_step(h, s)
            return n

        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        if graph:
            # the whole run as one graph: in graph mode every step's launches
            # are independent of the host's state, so they can be recorded
            # before any of them runs
            B.ra_graph_mode(h, 1, stream)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                issue(None)
            torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        if graph:
            g.replay()
        else:
            events = issue(stream)
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        if graph:
            B.ra_graph_mode(h, 0, stream)
            events = B.ra_get_seq_info(h, 0).event
            del g
        cache.close()
        result = {
            "metric": "tiny-case decode step latency (append + attention + end of step)",
            "config": {"workload": "1 layer, 4 Q / 2 KV heads, head_dim 128, fp32, prompt 128, "
                                   "K=256, r=64, evict every 64, 1024 steps from the prompt"},
            "steps": T,
            "events": events,
            "graph": graph,
            "us_per_step_gpu": e0.elapsed_time(e1) * 1e3 / T,
            "us_per_step_wall": wall * 1e6 / T,
            "higher_is_better": False,
        }
    if with_cpu:
        result["cpu_baseline"] = tiny_cpu_baseline(lp, K, T, Hq, Hkv, 1000 * 1000003, 0)
    return result


def serving(B, torch, Workload, steps, log):
    """Continuous batching of a request stream (the paper's serving regime:
    staggered compressions, requests finishing and being replaced).

    Phi-4-reasoning attention shape (40 layers, 40 Q / 10 KV heads), 128
    slots, budget K = 2048 evictable rows per head (the paper's budget for its
    32k benchmark traces), r = 64, every 64; requests with prompts ~U[64, 2048]
    and a fixed 8192-token generation (the paper's shortest serving length).
    At the window start every slot holds a request at a uniformly drawn age
    (reached through the real sampler by staggered begins and fast forward),
    so compressions happen on every sequence's own phase and a request
    completes every ~64 steps on average; a finished request ends, and the
    next request of the stream begins in its slot with its prompt rows
    written (first fit over the released rows).  Timed: every decode step's
    launches, end-of-step evictions and the admissions, wall clock; the rows
    of the requests to admit are generated before the window.
    """
    import numpy as np
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    L, Hq, Hkv, S, K, GEN = 40, 40, 10, 128, 2048, 8192
    rng = np.random.default_rng(1005)
    n_req = S + 64
    lps = rng.integers(64, 2049, n_req).tolist()
    ages = rng.integers(0, GEN, S).tolist()
    cfg = B.make_config(L, Hq, Hkv, K, R, EVERY, B.RA_BUDGET_EVICTABLE, B.RA_BF16, S)
    pool = S * B.ra_seq_rows(cfg, 2048)
    cache = B.Cache(cfg, pool, device=dev)
    h = cache.handle
    wl = Workload(1005, L, Hq, Hkv, 128, torch.bfloat16, True, ring=RING, device=dev)
    ls = torch.arange(L, device=dev).view(-1, 1, 1)
    gs = torch.arange(Hkv, device=dev).view(1, -1, 1)
    hq = torch.arange(Hq, device=dev)

    def prompt(rid, lp):
        ps = torch.arange(lp, device=dev).view(1, 1, -1)
        return wl.k_rows(rid, ls, gs, ps, lp).contiguous(), wl.v_rows(rid, ls, gs, ps, lp).contiguous()

    def ring_of(rid, lp, step0):
        """[64][L][Hq|Hkv][128] inputs of steps step0 .. step0 + 63."""
        st = torch.arange(step0, step0 + RING, device=dev)
        rr = torch.full((RING,), rid, device=dev)
        q = torch.stack([wl.q_step(rr, l, st) for l in range(L)], 1)
        kv = [wl.kv_step(rr, l, lp + st, torch.full_like(st, lp)) for l in range(L)]
        return q, torch.stack([k for k, _ in kv], 1), torch.stack([v for _, v in kv], 1)

    # the snapshot: request s in slot s at age ages[s] (oldest begun first)
    t0 = time.time()
    order = sorted(range(S), key=lambda s: -ages[s])
    for i, s in enumerate(order):
        B.ra_seq_begin(h, s, lps[s], 7 * s + 1, s)
        nxt = ages[order[i + 1]] if i + 1 < S else 0
        if ages[s] > nxt:
            B.ra_fast_forward(h, ages[s] - nxt)
    for s in range(S):
        n = B.ra_get_seq_info(h, s).len
        posb = torch.empty(L * Hkv * n, dtype=torch.int32, device=dev)
        B.ra_export_positions(h, s, posb)
        posb = posb.view(L, Hkv, n).long()
        kr = torch.empty(L, Hkv, n, 128, dtype=torch.bfloat16, device=dev)
        vr = torch.empty_like(kr)
        for l in range(L):
            kr[l] = wl.k_rows(s, l, gs.view(-1, 1), posb[l], lps[s])
            vr[l] = wl.v_rows(s, l, gs.view(-1, 1), posb[l], lps[s])
        B.ra_write_rows(h, s, kr, vr)
        del posb, kr, vr
    # ring slot j = (iteration mod 64) holds every slot's inputs of the step it
    # decodes at that iteration (the generator's inputs repeat every 64 steps)
    q_ring = torch.empty(RING, L, S, Hq, 128, dtype=torch.bfloat16, device=dev)
    k_ring = torch.empty(RING, L, S, Hkv, 128, dtype=torch.bfloat16, device=dev)
    v_ring = torch.empty_like(k_ring)
    for s in range(S):
        q, k, v = ring_of(s, lps[s], ages[s])
        q_ring[:, :, s], k_ring[:, :, s], v_ring[:, :, s] = q, k, v
    # requests admitted during the window (a slot finishes at iteration
    # GEN - age - 1 and its successor decodes step 0 at iteration GEN - age),
    # prepared in advance, their rings rotated to that iteration
    finishing = sorted((GEN - a, s) for s, a in enumerate(ages) if GEN - a < steps)
    queued = {}
    for i, (ia, s) in enumerate(finishing):
        rid = S + i
        q, k, v = ring_of(rid, lps[rid], 0)
        queued[(ia, s)] = (rid, prompt(rid, lps[rid]),
                           tuple(torch.roll(x, ia % RING, 0) for x in (q, k, v)))
    out = torch.empty(S, Hq, 128, dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    log("serving snapshot ready (%.1fs); %d admissions expected in %d steps"
        % (time.time() - t0, len(finishing), steps))

    slot_step = list(ages)
    slot_lp = lps[:S]
    slot_len = [B.ra_get_seq_info(h, s).len for s in range(S)]
    kv_bytes = 0                      # algorithmic K/V bytes read by attention
    tokens = events = admissions = 0
    adm_ms = 0.0
    wall0 = time.perf_counter()
    for it in range(steps):
        j = it % RING
        for l in range(L):
            B.ra_decode_attention(h, l, q_ring[j, l], k_ring[j, l], v_ring[j, l], out,
                                  cache.workspace, stream)
        events += B.ra_end_step(h, stream)
        tokens += S
        kv_bytes += L * Hkv * 2 * 128 * 2 * sum(n + 1 for n in slot_len)
        slot_step = [st + 1 for st in slot_step]
        for s in range(S):
            slot_len[s] += 1                  # the host rule of the trigger
            if slot_step[s] % EVERY == 0 and slot_len[s] - slot_lp[s] - R > K:
                slot_len[s] = slot_lp[s] + K + R
            if slot_step[s] == GEN:
                a0 = time.perf_counter()
                rid, (kp, vp), (q, k, v) = queued.pop((it + 1, s))
                B.ra_seq_end(h, s, stream)
                B.ra_seq_begin(h, s, lps[rid], 7 * rid + 1, rid, kp, vp, stream)
                q_ring[:, :, s], k_ring[:, :, s], v_ring[:, :, s] = q, k, v
                slot_step[s] = 0
                slot_lp[s] = lps[rid]
                slot_len[s] = lps[rid]
                admissions += 1
                adm_ms += 1e3 * (time.perf_counter() - a0)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    res = {
        "metric": "serving decode tokens/s with staggered compressions and request churn",
        "value": tokens / wall, "unit": "tokens/s", "steps": steps,
        "ms_per_step": 1e3 * wall / steps,
        "config": {"workload": "Phi-4-reasoning-shaped attention stack, 128 slots, "
                               "prompts ~U[64,2048], 8192-token generations, K=2048, r=64, "
                               "evict every 64 steps, uniform request ages at the start"},
        "attention_kv_gbs": kv_bytes / wall / 1e9,
        "attention_kv_gbs_note": "every kept K and V row read once per step, over the "
                                 "whole wall time (evictions and admissions included)",
        "compressions_per_step": events / steps,
        "admissions": admissions,
        "admission_host_ms_avg": adm_ms / max(1, admissions),
    }
    cache.close()
    torch.cuda.empty_cache()
    return res


def serving_cap(B, torch, Workload, steps, log, layout_name, page_rows=64,
                watermark=0.02):
    """Serving at a fixed memory cap: contiguous regions against pages.

    Phi-4-reasoning attention shape (40 layers, 40 Q / 10 KV heads), K = 2048,
    r = 64, every 64, prompts ~U[64, 2048], 8192-token generations, up to 256
    slots, and one pool for both layouts: the rows 128 sequences with the
    longest prompt take in contiguous regions.  Requests come from a queue.
    Contiguous regions are sized by each request's own prompt and placed by
    first fit; a request is admitted while a region fits.  Pages are taken as
    rows are appended; a request is admitted while the free rows, less a
    watermark (2% of the pool), cover its prompt; a step whose new rows find
    no free page preempts the youngest request (its progress is lost and it
    returns to the head of the queue).  The pool starts filled by requests of
    staggered ages, reached through the real sampler.  Rows are not
    materialised and admitted prompts are positions only: the timing does not
    depend on the values, and the rows left in the pool are synthetic data
    either way.  Timed: every step's launches, end-of-step evictions,
    preemptions and admissions, wall clock.
    """
    import collections
    import numpy as np
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    L, Hq, Hkv, K, GEN, SLOTS = 40, 40, 10, 2048, 8192, 256
    layout = {"chronological": B.RA_LAYOUT_CHRONOLOGICAL, "paged": B.RA_LAYOUT_PAGED}[layout_name]
    ref = B.make_config(L, Hq, Hkv, K, R, EVERY, B.RA_BUDGET_EVICTABLE, B.RA_BF16, 128)
    pool = 128 * B.ra_seq_rows(ref, 2048)
    cfg = B.make_config(L, Hq, Hkv, K, R, EVERY, B.RA_BUDGET_EVICTABLE, B.RA_BF16, SLOTS,
                        layout=layout, page_rows=page_rows, max_prompt_len=2048)
    if layout == B.RA_LAYOUT_PAGED:
        pool -= pool % (L * Hkv * page_rows)
    cache = B.Cache(cfg, pool, device=dev)
    h = cache.handle
    rng = np.random.default_rng(1006)
    n_req = 1 << 14
    lps = rng.integers(64, 2049, n_req).tolist()
    queue = collections.deque(range(n_req))
    res = {}                           # slot -> [rid, step]
    group = L * Hkv * page_rows

    def rows_held(lp, age):
        # cached rows after `age` steps: growth until the first event (the
        # first multiple of 64 with more than K evictable rows), then K + r
        # plus the steps since the last event
        first = EVERY * ((K + R) // EVERY + 1)
        n = lp + age if age < first else lp + K + R + age % EVERY
        if layout == B.RA_LAYOUT_PAGED:
            return group * -(-n // page_rows)
        return B.ra_seq_rows(cfg, lp)

    def ages_for(n):
        return [int(GEN * (n - i - 0.5) / n) for i in range(n)]   # oldest first

    # the starting population: the most requests of uniformly spread ages
    # that fit the cap (less the watermark for pages)
    room = pool * (1 - watermark) if layout == B.RA_LAYOUT_PAGED else pool
    n_start = 1
    while n_start < SLOTS and sum(rows_held(lps[i], a) for i, a in
                                  enumerate(ages_for(n_start + 1))) <= room:
        n_start += 1
    ages = ages_for(n_start)

    def begin(slot, rid):
        try:
            B.ra_seq_begin(h, slot, lps[rid], 7 * rid + 1, rid, None, None, stream)
        except B.RandAttnError as e:
            if e.status != B.RA_ERR_CAPACITY:
                raise
            return False
        res[slot] = [rid, 0]
        return True

    # begun oldest first, with a fast forward between begins
    t0 = time.time()
    for i in range(n_start):
        if not begin(i, queue[0]):
            break
        queue.popleft()
        run = ages[i] - (ages[i + 1] if i + 1 < n_start else 0)
        try:
            B.ra_fast_forward(h, run, stream)
        except B.RandAttnError as e:
            if e.status != B.RA_ERR_CAPACITY:
                raise
            B.ra_seq_end(h, i, stream)
            queue.appendleft(res.pop(i)[0])
            break
        for s in res:
            res[s][1] += run
    start_resident = len(res)
    # per-slot input rings (inputs of a slot's request template; the values do
    # not change the timing)
    wl = Workload(1006, L, Hq, Hkv, 128, torch.bfloat16, True, ring=RING, device=dev)
    bidx = torch.arange(SLOTS, device=dev)
    lp_t = torch.tensor(lps[:SLOTS], device=dev)
    q_ring = torch.empty(RING, L, SLOTS, Hq, 128, dtype=torch.bfloat16, device=dev)
    k_ring = torch.empty(RING, L, SLOTS, Hkv, 128, dtype=torch.bfloat16, device=dev)
    v_ring = torch.empty_like(k_ring)
    for j in range(RING):
        st = torch.full((SLOTS,), j, device=dev)
        for l in range(L):
            q_ring[j, l] = wl.q_step(bidx, l, st)
            k, v = wl.kv_step(bidx, l, lp_t + st, lp_t)
            k_ring[j, l], v_ring[j, l] = k, v
    out = torch.empty(SLOTS, Hq, 128, dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    log("serving at a fixed cap (%s): %d requests resident at the start (%.1fs)"
        % (layout_name, start_resident, time.time() - t0))

    tokens = events = admissions = done = preempted = lost = 0
    resident_sum = 0
    kv_bytes = 0
    wall0 = time.perf_counter()
    for it in range(steps):
        j = it % RING
        while True:                   # the first layer takes the step's pages
            try:
                B.ra_decode_attention(h, 0, q_ring[j, 0], k_ring[j, 0], v_ring[j, 0], out,
                                      cache.workspace, stream)
                break
            except B.RandAttnError as e:
                if e.status != B.RA_ERR_CAPACITY or not res:
                    raise
                victim = min(res, key=lambda s: res[s][1])
                B.ra_seq_end(h, victim, stream)
                rid, step = res.pop(victim)
                queue.appendleft(rid)
                preempted += 1
                lost += step
        for l in range(1, L):
            B.ra_decode_attention(h, l, q_ring[j, l], k_ring[j, l], v_ring[j, l], out,
                                  cache.workspace, stream)
        events += B.ra_end_step(h, stream)
        tokens += len(res)
        resident_sum += len(res)
        for s in list(res):
            res[s][1] += 1
            kv_bytes += L * Hkv * 2 * 128 * 2 * B.ra_get_seq_info(h, s).len
            if res[s][1] == GEN:
                B.ra_seq_end(h, s, stream)
                del res[s]
                done += 1
        # admissions into free slots while the pool accepts them
        for slot in range(SLOTS):
            if slot in res or not queue:
                continue
            if layout == B.RA_LAYOUT_PAGED:
                _, free = B.ra_pool_info(h)
                if free - L * Hkv * (lps[queue[0]] + page_rows) < watermark * pool:
                    break
            if not begin(slot, queue[0]):
                break
            queue.popleft()
            admissions += 1
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    used, free = B.ra_pool_info(h)
    out_d = {
        "metric": "serving decode tokens/s at a fixed memory cap",
        "value": tokens / wall, "unit": "tokens/s", "steps": steps,
        "layout": layout_name + ("" if layout != B.RA_LAYOUT_PAGED else
                                 " (%d-row pages)" % page_rows),
        "pool_gb": pool * (2 * 128 * 2 + 4) / 1e9,
        "resident_start": start_resident,
        "resident_mean": resident_sum / steps,
        "preemptions": preempted, "steps_lost_to_preemption": lost,
        "admissions": admissions, "completions": done,
        "compressions_per_step": events / steps,
        "ms_per_step": 1e3 * wall / steps,
        "attention_kv_gbs": kv_bytes / wall / 1e9,
        "pool_used_at_end": used / (used + free),
        "config": {"workload": "Phi-4-reasoning-shaped attention stack, prompts ~U[64,2048], "
                               "8192-token generations, K=2048, r=64, evict every 64 steps, "
                               "up to 256 slots, pool = 128 contiguous regions at the "
                               "longest prompt"},
    }
    cache.close()
    torch.cuda.empty_cache()
    return out_d


def time_window_scorer(B, torch, h, wl, cfg, Bsz, L, Hq, Hkv, stream, comp, log):
    """One round of the observation-window scoring pass over every sequence
    (what a score-based evictor computes before it can evict, and Random
    Attention does not), timed with HIP events on the current state."""
    dev = torch.device("cuda:0")
    infos = [B.ra_get_seq_info(h, b) for b in range(Bsz)]
    qwin = torch.empty(Bsz, L, Hq, 64, 128, dtype=torch.bfloat16, device=dev)
    heads = torch.arange(Hq, device=dev).view(-1, 1)
    for b in range(Bsz):
        steps = torch.arange(infos[b].step - 64, infos[b].step, device=dev).view(1, -1)
        for l in range(L):
            qwin[b, l] = wl.q_rows(b, l, heads, steps)
    drops = torch.empty(Bsz, L, Hkv, cfg.evict_every, dtype=torch.int32, device=dev)
    B.ra_window_select(h, 0, Bsz, qwin, None, 0, drops, stream)     # warm-up
    times = []
    for _ in range(3):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        B.ra_window_select(h, 0, Bsz, qwin, None, 0, drops, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    ms = min(times)
    G = Hq // Hkv
    keys = sum(i.len for i in infos) * L * Hkv
    flops = 2 * 2 * keys * G * 64 * 128          # two logit passes, 2 flop per MAC
    kbytes = 2 * keys * 128 * 2                   # every cached key read in both passes
    rand_ms = None
    if comp and comp.get("sequence_events"):
        rand_ms = (comp["avg_ms_per_end_step_with_events"] * comp["end_steps_with_events"]
                   / comp["sequence_events"])
    log("window scorer: %.2f ms per round over %d sequences" % (ms, Bsz))
    out = {
        "what": "observation-window (last 64 queries x G heads) attention-score pass, "
                "max-pool 7 and lowest-m selection, every (sequence, layer, KV head)",
        "ms_per_round_all_sequences": ms,
        "ms_per_sequence": ms / Bsz,
        "tflops": flops / (ms * 1e-3) / 1e12,
        "key_read_gbs": kbytes / (ms * 1e-3) / 1e9,
        "random_eviction_ms_per_sequence_event": rand_ms,
    }
    if rand_ms:
        out["scorer_over_random_eviction"] = (ms / Bsz) / rand_ms
    del qwin, drops
    torch.cuda.empty_cache()
    return out


def build_parser():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=64)
    ap.add_argument("--workload", default="qwen3-14b", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-steps", type=int, default=384,
                    help="decode steps of the oracle's timed sample (about 10 s)")
    ap.add_argument("--attn-split", type=int, default=0)
    ap.add_argument("--layout", default="chronological",
                    choices=["chronological", "holefill", "paged"],
                    help="row order kept by eviction (chronological: the paper's)")
    ap.add_argument("--policy", default="random",
                    choices=["random", "shared", "block", "recency"],
                    help="eviction policy: Random Attention, or one of the paper's "
                         "controls (shared draw, block-wise, recency + prompt)")
    ap.add_argument("--block", type=int, default=64,
                    help="tokens per block for --policy block (a divisor of 64)")
    ap.add_argument("--evict-cost", action="store_true",
                    help="eviction-round cost of one sequence at K=1024 (budget counting "
                         "the prompt, prompt 300) over 4096 decode steps, as in the "
                         "paper's eviction-cost table; prints its own JSON line")
    ap.add_argument("--serving", action="store_true",
                    help="continuous batching of a request stream on the Phi-4 shape "
                         "(staggered compressions, requests finishing and replaced); "
                         "prints its own JSON line; --steps sets the window")
    ap.add_argument("--serving-cap", action="store_true",
                    help="serving at a fixed memory cap, the pool of 128 contiguous "
                         "regions, with --layout chronological or paged (--page-rows); "
                         "prints its own JSON line; --steps sets the window")
    ap.add_argument("--page-rows", type=int, default=64,
                    help="rows per page of --layout paged")
    ap.add_argument("--evict-cost-methods", default="random,snapkv",
                    help="comma-separated rounds timed by --evict-cost: random, "
                         "random-holefill (the hole-fill layout) and the score-based "
                         "snapkv, rkv, vase")
    ap.add_argument("--window-scorer", action="store_true",
                    help="also time the observation-window scoring pass (always on for "
                         "phi4-ragged)")
    ap.add_argument("--tiny", action="store_true",
                    help="per-step latency of the tiny fp32 case (1 layer, 4/2 heads, "
                         "prompt 128, K=256, 1024 steps); prints its own JSON line")
    ap.add_argument("--full-run", action="store_true",
                    help="time the whole generation from the prompt (steps 1..32768, no "
                         "warm-up) instead of the steady-state window at its end; about "
                         "four minutes on the Qwen3-14B shape")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device-to-device copy three times (the "
                         "known-size reference for the HBM byte counters)")
    ap.add_argument("--graph", action="store_true",
                    help="capture the decode steps into HIP graphs (ra_graph_mode) and "
                         "replay them: one graph of the layers' attention and one of the "
                         "end of the step per input-ring slot, or with --tiny the whole "
                         "run as one graph; events then move their rows themselves")
    ap.add_argument("--timeline-summary", metavar="TRACE_DIR",
                    help="read a rocprofv3 --kernel-trace CSV of a run with the same "
                         "--workload/--steps, and print per-layer attention, merge and "
                         "gap durations over the timed launches")
    ap.add_argument("--traffic-summary", nargs=4,
                    metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="CPU only: read the rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE "
                         "outputs of a bench run with the other arguments given here and "
                         "of --calibrate-copy, and write "
                         "profiles/attention_traffic_<workload>.json")
    return ap


def _counter_rows(d):
    """(dispatch id, kernel name, counter, value) rows of every rocprofv3
    counter-collection CSV under directory d; values summed per dispatch and
    counter."""
    import csv
    import glob
    acc = {}
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit("no counter_collection.csv under %s" % d)
    for path in files:
        with open(path, newline="") as f:
            for row in csv.DictReader(f):
                key = (int(row["Dispatch_Id"]), row["Kernel_Name"], row["Counter_Name"])
                acc[key] = acc.get(key, 0.0) + float(row["Counter_Value"])
    return sorted((k[0], k[1], k[2], v) for k, v in acc.items())


def _trace_rows(d):
    """(start ns, end ns, kernel name) of the library's dispatches in a
    rocprofv3 kernel-trace CSV under directory d, by start time."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    if not files:
        raise SystemExit("no kernel_trace.csv under %s" % d)
    rows = []
    for path in files:
        with open(path, newline="") as f:
            for r in csv.DictReader(f):
                if "ra::" in r["Kernel_Name"]:
                    rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]),
                                 r["Kernel_Name"]))
    return sorted(rows)


def timeline_summary(args):
    """Per-layer timeline of the timed launches of one bench run from its
    kernel trace: the attention kernel, the gap to the split merge kernel (if
    any), the merge, and the gap to the next layer's attention (launches
    within one step; the step's end-of-step kernels come after its last
    layer).  Steps whose attention moved a deferred event's rows
    (attn_bf16_move_kernel) are reported apart."""
    w = WORKLOADS[args.workload]
    L = w["L"]
    rows = _trace_rows(args.timeline_summary)
    attn = [i for i, r in enumerate(rows)
            if "attn_bf16_kernel" in r[2] or "attn_bf16_move_kernel" in r[2]]
    timed = attn[-args.steps * L:]
    acc = {"attention_us": [], "move_attention_us": [], "merge_us": [], "gap_to_merge_us": [],
           "gap_to_next_layer_us": [], "layer_span_us": []}
    for k, i in enumerate(timed):
        s0, e, name = rows[i]
        acc["move_attention_us" if "move" in name else "attention_us"].append((e - s0) / 1e3)
        j = i + 1
        if j < len(rows) and "combine" in rows[j][2]:
            acc["gap_to_merge_us"].append((rows[j][0] - e) / 1e3)
            acc["merge_us"].append((rows[j][1] - rows[j][0]) / 1e3)
            e = rows[j][1]
        if (k + 1) % L and k + 1 < len(timed):
            nxt = rows[timed[k + 1]][0]
            acc["gap_to_next_layer_us"].append((nxt - e) / 1e3)
            if "move" not in name:
                acc["layer_span_us"].append((nxt - s0) / 1e3)

    def stat(v):
        if not v:
            return None
        v = sorted(v)
        return {"n": len(v), "mean": sum(v) / len(v), "p10": v[len(v) // 10],
                "p50": v[len(v) // 2], "p90": v[(9 * len(v)) // 10]}

    out = {k: stat(v) for k, v in acc.items()}
    out["kernel"] = rows[timed[0]][2].replace("(anonymous namespace)::", "").split("(")[0]
    out["workload"] = args.workload
    out["launches"] = len(timed)
    print(json.dumps(out))


def traffic_summary(args):
    """Copy-calibrated HBM bytes per attention launch, and per eviction event,
    of the timed region of one bench run, from two counter runs.

    An event either moves its rows itself (a full evict_kernel dispatch) or
    selects only (the last positions-only evict_kernel dispatch: the fast
    forward's are earlier) and leaves the moves to the next step's attention
    (attn_bf16_move_kernel, one dispatch per layer); the latter's bytes above
    as many plain attention launches are the moves' share."""
    fetch_dir, write_dir, cfetch_dir, cwrite_dir = args.traffic_summary
    w = WORKLOADS[args.workload]

    def per_dispatch(d, counter, match):
        return [v for _, name, c, v in _counter_rows(d) if c == counter and match(name)]

    def copy_kib(d, counter):
        rows = [(v, name) for _, name, c, v in _counter_rows(d) if c == counter]
        top = max(v for v, _ in rows)
        big = [v for v, _ in rows if v > 0.5 * top]
        return sum(big) / len(big)

    copy_bytes = 1 << 30
    cf, cw = copy_kib(cfetch_dir, "FETCH_SIZE"), copy_kib(cwrite_dir, "WRITE_SIZE")
    fscale, wscale = copy_bytes / (cf * 1024), copy_bytes / (cw * 1024)
    attn = lambda n: "attn_bf16_kernel" in n
    move = lambda n: "attn_bf16_move_kernel" in n
    full_evict = lambda n: "evict_kernel" in n and "false" in n
    select_evict = lambda n: "evict_kernel" in n and "true" in n
    fm = per_dispatch(fetch_dir, "FETCH_SIZE", move)
    wm = per_dispatch(write_dir, "WRITE_SIZE", move)
    timed = args.steps * w["L"] - len(fm)
    fa = per_dispatch(fetch_dir, "FETCH_SIZE", attn)[-timed:]
    wa = per_dispatch(write_dir, "WRITE_SIZE", attn)[-timed:]
    fe = per_dispatch(fetch_dir, "FETCH_SIZE", full_evict)
    we = per_dispatch(write_dir, "WRITE_SIZE", full_evict)
    fb = sum(fa) / len(fa) * 1024 * fscale
    wb = sum(wa) / len(wa) * 1024 * wscale
    deferred = None
    if fm and wm:
        fs = per_dispatch(fetch_dir, "FETCH_SIZE", select_evict)[-1] * 1024 * fscale
        ws = per_dispatch(write_dir, "WRITE_SIZE", select_evict)[-1] * 1024 * wscale
        mf, mw = sum(fm) * 1024 * fscale, sum(wm) * 1024 * wscale
        deferred = {"select_fetch_bytes": fs, "select_write_bytes": ws,
                    "move_attention_launches": len(fm),
                    "move_attention_fetch_bytes": mf, "move_attention_write_bytes": mw,
                    "moves_fetch_bytes": mf - len(fm) * fb,
                    "moves_write_bytes": mw - len(wm) * wb}
    out = {
        "workload": args.workload,
        "kernel": "attn_bf16_kernel",
        "kernel_source_hash": kernel_source_hash(),
        "copy_calibration": {"bytes": copy_bytes, "fetch_kib_per_dispatch": cf,
                             "write_kib_per_dispatch": cw, "fetch_scale": fscale,
                             "write_scale": wscale},
        "fetch_bytes_per_launch": fb,
        "write_bytes_per_launch": wb,
        "hbm_bytes_per_launch": fb + wb,
        "launches_sampled": len(fa),
        "evict_full_events_sampled": len(fe),
        "evict_full_event": ({"fetch_bytes": sum(fe) / len(fe) * 1024 * fscale,
                              "write_bytes": sum(we) / len(we) * 1024 * wscale}
                             if fe and we else None),
        "evict_deferred_event": deferred,
        "run": run_signature(args),
    }
    path = os.path.join(ROOT, "profiles", "attention_traffic_%s.json" % args.workload)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def main():
    args = build_parser().parse_args()

    if args.gpus != 1:
        print("bench.py runs on one GPU only: the hot path has no cross-GPU step; "
              "--gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    if args.traffic_summary:
        traffic_summary(args)
        return
    if args.timeline_summary:
        timeline_summary(args)
        return

    import torch
    from paper_2609_03430_amd import binding as B
    from paper_2609_03430_amd.synth import Workload

    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": src.numel() * 4}))
        return

    if args.serving_cap:
        def clog(msg):
            print("[bench] " + msg, file=sys.stderr, flush=True)
        print(json.dumps(serving_cap(B, torch, Workload, args.steps, clog, args.layout,
                                     args.page_rows)), flush=True)
        return

    if args.serving:
        def slog(msg):
            print("[bench] " + msg, file=sys.stderr, flush=True)
        print(json.dumps(serving(B, torch, Workload, args.steps, slog)), flush=True)
        return

    if args.evict_cost:
        print(json.dumps(evict_cost(B, torch, Workload, tuple(args.evict_cost_methods.split(",")))),
              flush=True)
        return

    if args.tiny:
        print(json.dumps(tiny_latency(B, torch, Workload, not args.no_cpu_baseline, args.graph)),
              flush=True)
        return

    w = WORKLOADS[args.workload]
    L, Hq, Hkv, Bsz, K = (w[k] for k in ("L", "Hq", "Hkv", "B", "K"))
    if args.full_run:
        if w["T"] is None:
            print("--full-run needs a workload with one generation length", file=sys.stderr)
            sys.exit(2)
        args.warmup, args.steps = 0, w["T"]
    seed = SEEDS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    def log(msg):
        print("[bench] " + msg, file=sys.stderr, flush=True)

    total = args.warmup + args.steps
    lps, starts = sequence_plan(args.workload, w, total, None if args.full_run else args.steps)
    assert min(starts) >= 0
    layout = {"chronological": B.RA_LAYOUT_CHRONOLOGICAL, "holefill": B.RA_LAYOUT_HOLE_FILL,
              "paged": B.RA_LAYOUT_PAGED}[args.layout]
    policy = {"random": B.RA_POLICY_RANDOM, "shared": B.RA_POLICY_SHARED,
              "block": B.RA_POLICY_BLOCK, "recency": B.RA_POLICY_RECENCY}[args.policy]
    if policy == B.RA_POLICY_BLOCK and (args.block < 1 or EVERY % args.block):
        print("--block must divide %d" % EVERY, file=sys.stderr)
        sys.exit(2)
    cfg = B.make_config(L, Hq, Hkv, K, R, EVERY, B.RA_BUDGET_EVICTABLE, B.RA_BF16, Bsz,
                        attn_split=args.attn_split, layout=layout, policy=policy,
                        policy_block=args.block, page_rows=args.page_rows,
                        max_prompt_len=max(lps))
    rows = sum(B.ra_seq_rows(cfg, lp) for lp in lps)
    log("workload %s: pools %.1f GB" % (args.workload, rows * (128 * 2 * 2 + 4) / 1e9))
    cache = B.Cache(cfg, rows, device=dev)
    h = cache.handle
    wl = Workload(seed, L, Hq, Hkv, 128, torch.bfloat16, True, ring=RING, device=dev)
    t_ff = time.time()
    # begin the longest generations first and fast-forward between begins, so
    # that every sequence reaches its own step through the real sampler
    order = sorted(range(Bsz), key=lambda b: -starts[b])
    for i, b in enumerate(order):
        B.ra_seq_begin(h, b, lps[b], seed * 1000003 + b, b)
        nxt = starts[order[i + 1]] if i + 1 < Bsz else 0
        if starts[b] > nxt:
            B.ra_fast_forward(h, starts[b] - nxt)
    torch.cuda.synchronize()
    log("fast forward to steps %d..%d: %.2fs" % (min(starts), max(starts), time.time() - t_ff))
    gs = torch.arange(Hkv, device=dev).view(-1, 1)
    for b in range(Bsz):
        n = B.ra_get_seq_info(h, b).len
        pos = torch.empty(L * Hkv * n, dtype=torch.int32, device=dev)
        B.ra_export_positions(h, b, pos)
        pos = pos.view(L, Hkv, n).long()
        kr = torch.empty(L, Hkv, n, 128, dtype=torch.bfloat16, device=dev)
        vr = torch.empty_like(kr)
        for l in range(L):
            kr[l] = wl.k_rows(b, l, gs, pos[l], lps[b])
            vr[l] = wl.v_rows(b, l, gs, pos[l], lps[b])
        B.ra_write_rows(h, b, kr, vr)
        del pos, kr, vr
    torch.cuda.synchronize()
    log("rows materialised: %.2fs" % (time.time() - t_ff))

    # 64-step input ring for every layer, resident before timing: slot j holds
    # each sequence's inputs of its step starts[b] + j; iteration i of the
    # run uses slot i mod 64 (the generator's rows repeat with period 64)
    bidx = torch.arange(Bsz, device=dev)
    lp_t = torch.tensor(lps, device=dev)
    st_t = torch.tensor(starts, device=dev)
    q_ring = torch.empty(RING, L, Bsz, Hq, 128, dtype=torch.bfloat16, device=dev)
    k_ring = torch.empty(RING, L, Bsz, Hkv, 128, dtype=torch.bfloat16, device=dev)
    v_ring = torch.empty_like(k_ring)
    for j in range(RING):
        for l in range(L):
            q_ring[j, l] = wl.q_step(bidx, l, st_t + j)
            k, v = wl.kv_step(bidx, l, lp_t + st_t + j, lp_t)
            k_ring[j, l] = k
            v_ring[j, l] = v
    out = torch.empty(Bsz, Hq, 128, dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    split_keys, max_splits, waves = B.ra_attention_plan(h)
    log("inputs ready; attention split %d keys x %d, %d wavefronts per item"
        % (split_keys, max_splits, waves))

    def run_steps(first, n, timed, graphs=None, track=None):
        # HIP events bracket each step's L attention launches (one pair per
        # step: an event between every launch would add its own gap to the
        # timed region) and each end-of-step call.  With graphs, the step
        # replays the two graphs of its input-ring slot, and `track` follows
        # the lengths and events the device produces (the library's mirror
        # stays that of the entry into graph mode).
        rec = []
        for i in range(first, first + n):
            if timed and (i - first) % (2048 if n > 4096 else 64) == 0:
                log("step %d of %d enqueued" % (i - first, n))
            j = i % RING
            if not timed:
                lens = None
            elif track is not None:
                lens = [t["len"] for t in track]
            else:
                lens = [B.ra_get_seq_info(h, b).len for b in range(Bsz)]
            evs = []
            if timed:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
            if graphs is not None:
                graphs[j][0].replay()
            else:
                for l in range(L):
                    B.ra_decode_attention(h, l, q_ring[j, l], k_ring[j, l], v_ring[j, l], out,
                                          cache.workspace, stream)
            if timed:
                e1.record(stream)
                evs.append((e0, e1))
            if timed:
                x0 = torch.cuda.Event(enable_timing=True)
                x1 = torch.cuda.Event(enable_timing=True)
                x0.record(stream)
            if graphs is not None:
                graphs[j][1].replay()
                nev = 0
                for t in track:          # the end-of-step rule (trigger, then plan)
                    t["step"] += 1
                    t["len"] += 1
                    if t["step"] % EVERY == 0 and t["len"] - t["lp"] - R > t["k_keep"]:
                        t["len"] = t["lp"] + t["k_keep"] + R
                        t["event"] += 1
                        nev += 1
                deferred = False
            else:
                nev = B.ra_end_step(h, stream)
                deferred = nev > 0 and any(B.ra_get_seq_info(h, b).move_pending
                                           for b in range(Bsz))
            if timed:
                x1.record(stream)
                rec.append((lens, evs, (x0, x1), nev, deferred))
            last_event[0] = nev > 0
        return rec

    last_event = [False]     # whether the step before the next one ended in an event

    run_steps(0, args.warmup, False)
    post0 = last_event[0]    # the first timed step follows an event
    graphs = track = None
    if args.graph:
        B.ra_graph_mode(h, 1, stream)
        split_keys, max_splits, waves = B.ra_attention_plan(h)
        torch.cuda.synchronize()
        graphs = []
        for j in range(RING):
            ga, ge = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
            with torch.cuda.graph(ga):
                for l in range(L):
                    B.ra_decode_attention(h, l, q_ring[j, l], k_ring[j, l], v_ring[j, l], out,
                                          cache.workspace)
            with torch.cuda.graph(ge):
                B.ra_end_step(h)
            graphs.append((ga, ge))
        track = []
        for b in range(Bsz):
            info = B.ra_get_seq_info(h, b)
            track.append({"lp": lps[b], "k_keep": info.k_keep, "len": info.len,
                          "step": info.step, "event": info.event})
        torch.cuda.synchronize()
        log("captured %d + %d graphs; attention split %d keys x %d, %d wavefronts per item"
            % (RING, RING, split_keys, max_splits, waves))
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    rec = run_steps(args.warmup, args.steps, True, graphs, track)
    # an event at the last timed step left its row moves to the next step's
    # attention: they are part of the timed work, done here (a fast forward
    # of no steps moves them and does nothing else)
    pending = any(B.ra_get_seq_info(h, b).move_pending for b in range(Bsz))
    if pending:
        B.ra_fast_forward(h, 0, stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    tokens = Bsz * args.steps
    if args.graph:
        B.ra_graph_mode(h, 0, stream)
        for b in range(Bsz):
            info = B.ra_get_seq_info(h, b)
            assert (info.len, info.step, info.event) == (
                track[b]["len"], track[b]["step"], track[b]["event"]), (b, info.len, track[b])
        del graphs
    for b in range(Bsz):
        assert B.ra_get_seq_info(h, b).step == starts[b] + total

    # per-launch durations and algorithmic bytes
    s_el = 2
    attn_ms, attn_bytes = [], []
    ev_ms, ev_bytes = [], []
    ev_work = []             # per event: the bytes a separate compaction moves
    n_events = 0
    seq_events = 0
    C = K + EVERY                      # candidates at every event of these workloads
    m = EVERY
    # expected rows an event moves; drops fall on whole units of `unit` rows
    # (1 for the per-token draws, B for block-wise), m / unit of C / unit units
    unit = args.block if policy == B.RA_POLICY_BLOCK else 1
    if layout == B.RA_LAYOUT_HOLE_FILL:
        # the surviving rows among the last m slots fill the holes below the
        # new length (recency drops none of them), plus all slots' positions
        # read by the selection
        moved = m if policy == B.RA_POLICY_RECENCY else m * (1.0 - m / C)
        per_head = moved * (2 * 128 * s_el + 4) * 2 + (C + R) * 4
    else:
        # rows from the first drop to the end: recency drops the first
        # candidate; otherwise the first of j dropped units among n is
        # preceded by (n - j) / (j + 1) kept units on average
        n_u, j_u = C // unit, m // unit
        first = 0.0 if policy == B.RA_POLICY_RECENCY else unit * (n_u - j_u) / (j_u + 1)
        moved = K + R - first
        per_head = moved * (2 * 128 * s_el + 4) * 2 + C * 4
    # an event whose moves ride on the next attention: the candidates'
    # positions read and the moved rows written once (the attention's own
    # read of every row is counted with the attention)
    per_head_deferred = moved * (2 * 128 * s_el + 4) + C * 4
    post = []                # per timed step: it follows an event step
    prev = post0
    any_deferred = False
    for lens, evs, (x0, x1), nev, deferred in rec:
        post.append(prev)
        prev = nev > 0
        any_deferred = any_deferred or deferred
        per_launch = sum(Hkv * ((n + 1) * 2 * 128 * s_el + (2 * 128 * s_el + 4)) +
                         2 * Hq * 128 * s_el for n in lens)
        for e0, e1 in evs:            # one span = L launches
            attn_ms.append(e0.elapsed_time(e1))
            attn_bytes.append(per_launch * L)
        if nev:
            n_events += 1
            seq_events += nev
            ev_ms.append(x0.elapsed_time(x1))
            ev_bytes.append((per_head_deferred if deferred else per_head) * nev * L * Hkv)
            ev_work.append(per_head * nev * L * Hkv)
    # a deferred event's rows move in the next step's attention: its cost is
    # the end-of-step time plus that step's extra attention time
    plain = [ms for ms, p in zip(attn_ms, post) if not p]
    after = [ms for ms, p in zip(attn_ms, post) if p]
    post_extra = (sum(after) / len(after) - sum(plain) / len(plain)
                  if any_deferred and after and plain else 0.0)
    # the streaming kernel's figures: steps whose attention also moved the rows
    # of a deferred event ran the moving kernel (their time above the others'
    # is the event's, in event_ms)
    roof = [(ms, b) for ms, b, p in zip(attn_ms, attn_bytes, post) if not (any_deferred and p)]
    attn_avg_ms = sum(ms for ms, _ in roof) / (len(roof) * L)
    attn_gbs = sum(b for _, b in roof) / (sum(ms for ms, _ in roof) * 1e-3) / 1e9
    comp = None
    if ev_ms:
        end_ms = sum(ev_ms) / len(ev_ms)
        event_ms = end_ms + post_extra
        gbs = sum(ev_bytes) / len(ev_bytes) / (event_ms * 1e-3) / 1e9
        comp = {
            "end_steps_with_events": n_events,
            "sequence_events": seq_events,
            "avg_ms_per_end_step_with_events": end_ms,
            "rows_moved_by_next_attention": any_deferred,
            # the last timed step's event: its moves ran at the window's end
            # (counted in the wall time, not in event_ms)
            "last_event_moved_at_window_end": pending,
            "next_attention_extra_ms": post_extra if any_deferred else None,
            "event_ms": event_ms,
            "achieved_gbs": gbs,
            "peak_gbs": PEAK_HBM_GBS,
            "frac": gbs / PEAK_HBM_GBS,
            "bytes_per_event": sum(ev_bytes) / len(ev_bytes),
            # the event's work priced as a separate compaction (its rows read
            # and written): the rate at which that work completes, comparable
            # across events that move their rows themselves and events whose
            # moves ride on the next attention
            "separate_compaction_bytes_per_event": sum(ev_work) / len(ev_work),
            "separate_compaction_equivalent_gbs":
                sum(ev_work) / len(ev_work) / (event_ms * 1e-3) / 1e9,
            "bytes_note": "per (sequence, layer, KV head) event: expected rows moved by "
                          "the order-preserving shift (from the first drop to the end) x "
                          "(key + value + position), read and written (written only, when "
                          "the next step's attention moves the rows: it reads them "
                          "anyway), plus candidate positions read; over event_ms = the "
                          "end-of-step time plus, when the next step's attention moves the "
                          "rows, that step's attention time above the other steps' mean",
        }
    total_bytes = sum(attn_bytes) + sum(ev_bytes)
    # Steady-state rate: a window of `steps` steps holds round(steps / 64)
    # end-of-step events only on average, so the raw value over a short
    # window weighs the event by its position; the amortised figure charges
    # every step the mean attention span, the mean end-of-step time of steps
    # without events, and 1/64 of the mean event.
    amortised = None
    if ev_ms and len(set(starts)) == 1 and plain and (after or not any_deferred):
        quiet = [x0.elapsed_time(x1) for _, _, (x0, x1), nev, _ in rec if not nev]
        step_ms = (sum(plain) / len(plain) + (sum(quiet) / len(quiet) if quiet else 0.0) +
                   comp["event_ms"] / EVERY)
        amortised = {"value": Bsz / (step_ms * 1e-3), "unit": "tokens/s",
                     "ms_per_step": step_ms,
                     "note": "mean attention span of the steps that follow no event + "
                             "mean end-of-step time without an event + (the event's "
                             "end-of-step time + the next attention's extra time) / 64 "
                             "(GPU time from HIP events; the raw value is wall time over "
                             "the window)"}
    if len(set(starts)) == 1:
        window = ("decode steps %d..%d of %d (%d end-of-step eviction events)"
                  % (starts[0] + args.warmup + 1, starts[0] + total, w["T"], n_events))
    else:
        window = ("%d timed decode steps per sequence, sequence i from step "
                  "start_i + %d (start_i %d..%d), %d sequence eviction events"
                  % (args.steps, args.warmup + 1, min(starts), max(starts), seq_events))
    result = {
        "metric": METRIC,
        "value": tokens / wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w["desc"],
            "layout": args.layout + (" (%d-row pages)" % args.page_rows
                                     if layout == B.RA_LAYOUT_PAGED else ""),
            "policy": args.policy if policy != B.RA_POLICY_BLOCK
            else "block%d" % args.block,
            "timed_window": window,
            "global_batch": Bsz,
            "seq_len": max(lp + st + total for lp, st in zip(lps, starts)),
            "attn_split_keys": split_keys,
            "attn_splits": max_splits,
            "attn_waves_per_item": waves,
            "graph": bool(args.graph),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "attn_bf16_kernel",
            "achieved": attn_gbs,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": attn_gbs / PEAK_HBM_GBS,
            "traffic": read_traffic(run_signature(args)),
            "avg_launch_ms": attn_avg_ms,
            "avg_launch_note": "HIP events around each step's launches of all layers, "
                               "divided by the layer count (inter-kernel gaps included); "
                               "steps whose attention also moved a deferred event's rows "
                               "(attn_bf16_move_kernel) are left out",
            "bytes_per_launch": sum(b for _, b in roof) / (len(roof) * L),
        },
        "compaction": comp,
        "amortised": amortised,
        "end_to_end_gbs": total_bytes / wall / 1e9,
        "end_to_end_frac": total_bytes / wall / 1e9 / PEAK_HBM_GBS,
    }
    if layout != B.RA_LAYOUT_CHRONOLOGICAL and (args.workload == "phi4-ragged" or
                                               args.window_scorer):
        result["window_scorer"] = "not run: the scorer reads the contiguous chronological layout"
    elif args.workload == "phi4-ragged" or args.window_scorer:
        del q_ring, k_ring, v_ring
        torch.cuda.empty_cache()
        result["window_scorer"] = time_window_scorer(B, torch, h, wl, cfg, Bsz, L, Hq,
                                                     Hkv, stream, comp, log)
    cache.close()
    q_ring = k_ring = v_ring = None
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        # sequence 0, a sample of its last cpu_steps steps (> 64 steps, so
        # the sample contains eviction events)
        c0 = starts[0] + total - args.cpu_steps
        result["cpu_baseline"] = cpu_baseline(w, seed, lps[0], c0, args.cpu_steps)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
