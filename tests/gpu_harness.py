"""Helpers shared by the GPU parity tests (not collected by pytest).

A ``Run`` drives the HIP path through the C ABI (via the ctypes binding) on
seeded synthetic rows; ``OracleSeq`` replays the same sequence with the CPU
oracle on the same rows.  The two share only the workload generator.
"""

import json
import os
import time

import numpy as np
import torch

from oracle.attention import gqa_decode
from oracle.evict import SequenceReplay, keep_count
from paper_2609_03430_amd import binding as B
from paper_2609_03430_amd.synth import Workload

DEV = "cuda"


def log(msg):
    print(msg, flush=True)


class Run:
    """One cache with several sequences, stepped in lock-step."""

    def __init__(self, L, Hq, Hkv, K, lps, r=64, every=64, dtype=B.RA_BF16,
                 mode=B.RA_BUDGET_EVICTABLE, seeds=None, rids=None,
                 scaled=True, wl_seed=1000, ring=None, attn_split=0,
                 max_seqs=None, write_prompt=True, begin=True,
                 layout=B.RA_LAYOUT_CHRONOLOGICAL, policy=B.RA_POLICY_RANDOM,
                 block=1, pool_rows=None, page_rows=32, max_prompt_len=None):
        self.L, self.Hq, self.Hkv, self.K, self.r, self.every = L, Hq, Hkv, K, r, every
        self.G = Hq // Hkv
        self.lps = list(lps)
        n = len(self.lps)
        self.n = n
        self.max_seqs = max_seqs or n
        self.seeds = list(seeds) if seeds is not None else [7 + 13 * i for i in range(n)]
        self.rids = list(rids) if rids is not None else list(range(n))
        self.mode = mode
        self.tdtype = torch.bfloat16 if dtype == B.RA_BF16 else torch.float32
        self.layout = layout
        self.policy, self.block = policy, block
        self.cfg = B.make_config(L, Hq, Hkv, K, r, every, mode, dtype, self.max_seqs,
                                 attn_split=attn_split, layout=layout, policy=policy,
                                 policy_block=block, page_rows=page_rows,
                                 max_prompt_len=(max(self.lps, default=0)
                                                 if max_prompt_len is None else max_prompt_len))
        rows = pool_rows or sum(B.ra_seq_rows(self.cfg, lp) for lp in self.lps)
        self.cache = B.Cache(self.cfg, rows)
        self.h = self.cache.handle
        self.wl = Workload(wl_seed, L, Hq, Hkv, 128, self.tdtype, scaled, ring=ring,
                           device=DEV)
        self.slots = list(range(n))
        self.steps = [0] * n
        self.write_prompt = write_prompt
        if begin:
            for slot in range(n):
                self.begin(slot)

    def begin(self, slot):
        lp = self.lps[slot]
        kp = vp = None
        if self.write_prompt and lp > 0:
            kp, vp = self.prompt_rows(slot, lp)
        B.ra_seq_begin(self.h, slot, lp, self.seeds[slot], self.rids[slot], kp, vp)
        self.steps[slot] = 0
        self.active = getattr(self, "active", set()) | {slot}

    def end(self, slot):
        B.ra_seq_end(self.h, slot)
        self.active.discard(slot)

    def k_keep(self, slot):
        return keep_count(self.K, self.lps[slot], self.mode)

    def prompt_rows(self, slot, lp):
        l = torch.arange(self.L, device=DEV).view(-1, 1, 1)
        g = torch.arange(self.Hkv, device=DEV).view(1, -1, 1)
        p = torch.arange(lp, device=DEV).view(1, 1, -1)
        rid = self.rids[slot]
        return (self.wl.k_rows(rid, l, g, p, lp).contiguous(),
                self.wl.v_rows(rid, l, g, p, lp).contiguous())

    def step_inputs(self, layer):
        """q [max_seqs,Hq,d], k/v [max_seqs,Hkv,d] for the current step."""
        q = torch.zeros(self.max_seqs, self.Hq, 128, dtype=self.tdtype, device=DEV)
        k = torch.zeros(self.max_seqs, self.Hkv, 128, dtype=self.tdtype, device=DEV)
        v = torch.zeros_like(k)
        rids = torch.tensor([self.rids[s] for s in self.slots], device=DEV)
        steps = torch.tensor(self.steps, device=DEV)
        lps = torch.tensor(self.lps, device=DEV)
        q[: self.n] = self.wl.q_step(rids, layer, steps)
        kk, vv = self.wl.kv_step(rids, layer, lps + steps, lps)
        k[: self.n] = kk
        v[: self.n] = vv
        return q, k, v

    def step(self, noalloc=False):
        """One decode step of every sequence (through the allocation-free entry
        point if `noalloc`); returns out [L, max_seqs, Hq, d]."""
        outs = torch.empty(self.L, self.max_seqs, self.Hq, 128, dtype=self.tdtype,
                           device=DEV)
        for layer in range(self.L):
            q, k, v = self.step_inputs(layer)
            if noalloc:
                self.cache.decode_noalloc(layer, q, k, v, outs[layer])
            else:
                self.cache.decode(layer, q, k, v, outs[layer])
        evicted = B.ra_end_step(self.h)
        self.steps = [s + 1 for s in self.steps]
        return outs, evicted

    def fast_forward(self, n):
        """Positions-only advance of every begun sequence."""
        B.ra_fast_forward(self.h, n)
        self.steps = [s + n if slot in self.active else s
                      for slot, s in enumerate(self.steps)]

    def materialise(self, slot):
        """Write the rows of the currently cached positions (after a fast
        forward) from the workload generator, one layer at a time."""
        info = B.ra_get_seq_info(self.h, slot)
        n = info.len
        pos = torch.empty(self.L * self.Hkv * n, dtype=torch.int32, device=DEV)
        B.ra_export_positions(self.h, slot, pos)
        pos = pos.view(self.L, self.Hkv, n).long()
        g = torch.arange(self.Hkv, device=DEV).view(-1, 1)
        rid = self.rids[slot]
        lp = self.lps[slot]
        k = torch.empty(self.L, self.Hkv, n, 128, dtype=self.tdtype, device=DEV)
        v = torch.empty_like(k)
        for l in range(self.L):
            k[l] = self.wl.k_rows(rid, l, g, pos[l], lp)
            v[l] = self.wl.v_rows(rid, l, g, pos[l], lp)
        B.ra_write_rows(self.h, slot, k, v)
        torch.cuda.synchronize()
        del k, v, pos

    def positions(self, slot, layer, g):
        """Cached positions in row order (ascending only in the chronological
        layout)."""
        info = B.ra_get_seq_info(self.h, slot)
        return B.ra_read_positions(self.h, slot, layer, g, info.cap)

    def sorted_positions(self, slot, layer, g):
        return np.sort(self.positions(slot, layer, g))

    def rows(self, slot, layer, g, by_position=False):
        """Cached key and value rows in row order, or ordered by position."""
        info = B.ra_get_seq_info(self.h, slot)
        k = torch.empty(info.len, 128, dtype=self.tdtype, device=DEV)
        v = torch.empty_like(k)
        B.ra_read_rows(self.h, slot, layer, g, k, v)
        torch.cuda.synchronize()
        k, v = k.cpu(), v.cpu()
        if by_position:
            order = torch.from_numpy(np.argsort(self.positions(slot, layer, g), kind="stable"))
            k, v = k[order], v[order]
        return k, v

    def close(self):
        self.cache.close()


class OracleSeq:
    """The CPU oracle's view of one sequence of a Run (same rows)."""

    def __init__(self, run, slot, heads=None):
        self.run = run
        self.slot = slot
        self.lp = run.lps[slot]
        self.rid = run.rids[slot]
        self.heads = heads or [(l, g) for l in range(run.L) for g in range(run.Hkv)]
        self.rep = SequenceReplay(self.lp, run.k_keep(slot), run.r, run.every,
                                  run.seeds[slot], self.rid, self.heads,
                                  policy=run.policy, block=run.block)
        self.wl = run.wl.to("cpu")

    def advance(self, n):
        self.rep.advance(n)

    def rows(self, layer, g, P):
        k = self.wl.k_rows(self.rid, layer, g, torch.as_tensor(P), self.lp)
        v = self.wl.v_rows(self.rid, layer, g, torch.as_tensor(P), self.lp)
        return k, v

    def attend_group(self, layer, g, step0):
        """Outputs [G, d] float64 of the query heads of KV head g."""
        run = self.run
        G = run.G
        q = self.wl.q_rows(self.rid, layer, torch.arange(g * G, (g + 1) * G), step0)
        k, v = self.rows(layer, g, self.rep.P[(layer, g)])
        from oracle.attention import softmax_attention
        qd = q.double().numpy()
        kd, vd = k.double().numpy(), v.double().numpy()
        return np.stack([softmax_attention(qd[i], kd, vd) for i in range(G)])

    def attend(self, layer, step0):
        """Outputs [Hq, d] float64 of `layer` at 0-based step ``step0``; the
        replay must hold the cache after that step's append."""
        run = self.run
        q = self.wl.q_rows(self.rid, layer, torch.arange(run.Hq), step0)
        Ks, Vs = [], []
        for g in range(run.Hkv):
            k, v = self.rows(layer, g, self.rep.P[(layer, g)])
            Ks.append(k.double().numpy())
            Vs.append(v.double().numpy())
        return gqa_decode(q.double().numpy(), Ks, Vs)


def _f64(x):
    if isinstance(x, torch.Tensor):
        x = x.detach().to("cpu", torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


# Worst figures of the running test, appended to a JSON-lines record at its
# end (see conftest.py), in the repository's output folder for remote runs.
_WORST = {}
RECORD = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "gpurun_out", "parity_records.jsonl")


def note(name, value):
    """Keep the largest value of `name` seen in the running test."""
    value = float(value)
    if not (name in _WORST and _WORST[name] >= value):
        _WORST[name] = value


def reset_record():
    _WORST.clear()


def write_record(test, outcome):
    os.makedirs(os.path.dirname(RECORD), exist_ok=True)
    with open(RECORD, "a") as f:
        f.write(json.dumps({"test": test, "outcome": outcome, "time": time.time(),
                            "worst": dict(_WORST)}) + "\n")


def max_abs(a, b):
    err = float(np.max(np.abs(_f64(a) - _f64(b)))) if np.size(_f64(a)) else 0.0
    note("max_abs", err)
    return err


# Tolerances the workloads fix for attention against the fp64 oracle.
TOL = {B.RA_BF16: 2e-2, B.RA_F32: 1e-5}

# bf16 outputs, element by element: |got - want| <= HALF_ULP * |want| + FLOOR.
# Rounding to bf16 (8 significant bits, nearest even) moves a value by at most
# 2^-8 of its magnitude; FLOOR covers the fp32 accumulation and the two-part
# bf16 softmax weights before that rounding.
BF16_HALF_ULP = 2.0 ** -8
BF16_FLOOR = 1e-4


def attn_err(got, want, dtype, ctx=()):
    """Max abs error of attention outputs against the fp64 oracle, asserted
    within the workloads' absolute tolerance and, for bf16, within the
    output-scaled bound element by element; the worst figures are recorded
    (the scaled bound's ratio, and the error beyond one half-ulp of want)."""
    g, w = _f64(got), _f64(want)
    err = max_abs(g, w)
    assert err <= TOL[dtype], ("abs", err) + tuple(ctx)
    if dtype == B.RA_BF16 and g.size:
        d = np.abs(g - w)
        bound = BF16_HALF_ULP * np.abs(w) + BF16_FLOOR
        ratio = float(np.max(d / bound))
        note("scaled_ratio", ratio)
        note("excess_over_half_ulp", float(np.max(d - BF16_HALF_ULP * np.abs(w))))
        note("max_abs_want", float(np.max(np.abs(w))))
        assert ratio <= 1.0, ("scaled", ratio, err) + tuple(ctx)
    return err


def check_heads(run, oracles, rows=True):
    """Kept positions equal the oracle's (as a sorted list in the hole-fill
    layout, whose rows are unordered), and every row holds its position's
    key and value."""
    holefill = run.layout == B.RA_LAYOUT_HOLE_FILL
    for o in oracles:
        for (layer, g) in o.heads:
            got = run.positions(o.slot, layer, g)
            want = o.rep.P[(layer, g)]
            if holefill:
                assert len(set(got.tolist())) == len(got)
                got = np.sort(got)
            assert np.array_equal(got, want), (o.slot, layer, g, o.rep.step)
            if rows:
                k, v = run.rows(o.slot, layer, g, by_position=holefill)
                kw, vw = o.rows(layer, g, want)
                assert torch.equal(k, kw), (o.slot, layer, g)
                assert torch.equal(v, vw), (o.slot, layer, g)
