"""Seeded random call sequences on live caches, checked against the oracle.

Each case draws a small configuration (layers, heads, group size, budget and
budget mode, recent buffer, trigger period, dtype, all three layouts, the
four end-of-step policies, slots, one or several work items per head) and
then a random sequence of calls: decode steps (most of them; a quarter
through the allocation-free entry point), sequences
beginning and ending, explicit events, fast forwards of every sequence or
of one, a request preempted (rows read, slot ended; the others may decode
meanwhile) and resumed in a free slot, and graph mode entered (steps then run
in it) and left.  Every output of every step is checked against the fp64
oracle; the kept sets after every step with an event, and the rows after
explicit events, fast forwards, resumes, leaving graph mode, at a quarter of
the events and at the end.  Half of the paged cases get a pool of about 60%
of what their slots could hold; the refusals of steps for lack of pages are
met by ending a sequence, as a serving loop would.
"""

import numpy as np
import pytest
import torch

from gpu_harness import OracleSeq, Run, attn_err, check_heads, log
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu

N_CASES = 32
N_OPS = 80


class Fuzz:
    def __init__(self, seed):
        rng = self.rng = np.random.default_rng(7700 + seed)
        self.seed = seed
        self.L, self.Hkv = int(rng.integers(1, 3)), int(rng.integers(1, 3))
        G = int(rng.choice([1, 2, 4, 5]))
        K = int(rng.integers(0, 61))
        mode = int(rng.integers(0, 2))
        self.dtype = B.RA_BF16 if rng.integers(0, 4) else B.RA_F32
        self.layout = int(rng.integers(0, 3))
        policy = int(rng.integers(0, 4))
        self.max_seqs = int(rng.integers(2, 5))
        self.maxlp = 40 if mode == B.RA_BUDGET_EVICTABLE else min(40, K)
        self.cfg = dict(L=self.L, Hkv=self.Hkv, G=G, K=K, mode=mode, dtype=self.dtype,
                        layout=self.layout, policy=policy, max_seqs=self.max_seqs,
                        r=int(rng.choice([0, 4, 8])), every=int(rng.choice([1, 4, 8, 16])),
                        split=int(rng.choice([0, 4096])), page_rows=int(rng.choice([32, 64])))
        c = self.cfg
        pool = None
        if self.layout == B.RA_LAYOUT_PAGED and seed % 2:
            # the pool at ~60% of what every slot could hold: steps are refused
            # for lack of pages and a sequence is preempted, as a serving loop would
            probe = B.make_config(self.L, self.Hkv * G, self.Hkv, K, c["r"], c["every"], mode,
                                  self.dtype, self.max_seqs, layout=self.layout,
                                  page_rows=c["page_rows"], max_prompt_len=self.maxlp)
            group = self.L * self.Hkv * c["page_rows"]
            full = self.max_seqs * B.ra_seq_rows(probe, self.maxlp)
            pool = max(2 * group, int(full * 0.6) // group * group)
            c["pool"] = pool
        self.run = Run(L=self.L, Hq=self.Hkv * G, Hkv=self.Hkv, K=K, lps=[self.maxlp] * self.max_seqs,
                       r=c["r"], every=c["every"], dtype=self.dtype, mode=mode,
                       layout=self.layout, policy=policy,
                       block=int(rng.integers(1, 6)) if policy == B.RA_POLICY_BLOCK else 1,
                       begin=False, max_seqs=self.max_seqs, attn_split=c["split"],
                       page_rows=c["page_rows"], max_prompt_len=self.maxlp,
                       wl_seed=300 + seed, pool_rows=pool)
        self.run.active = set()
        self.oracles, self.explicit = {}, {}
        self.n_req = 0
        self.graph = False
        self.counts = {}
        self.worst = 0.0

    def count(self, what):
        self.counts[what] = self.counts.get(what, 0) + 1

    def free(self):
        return [s for s in range(self.max_seqs) if s not in self.oracles]

    def pick(self, xs):
        return xs[int(self.rng.integers(0, len(xs)))]

    def check(self, rows):
        check_heads(self.run, list(self.oracles.values()), rows=rows)

    def begin(self, slot):
        run = self.run
        run.lps[slot] = int(self.rng.integers(0, self.maxlp + 1))
        run.seeds[slot] = int(self.rng.integers(1, 1 << 40))
        run.rids[slot] = 1000 + self.n_req
        self.n_req += 1
        try:
            run.begin(slot)
        except B.RandAttnError as e:
            assert e.status == B.RA_ERR_CAPACITY, e           # no hole large enough
            return
        self.oracles[slot] = OracleSeq(run, slot)
        self.explicit[slot] = False
        self.count("begin")

    def end(self, slot):
        self.run.end(slot)
        del self.oracles[slot]

    def step(self, oracles, ctx):
        """One decode step; False if the paged pool refused it (nothing done)."""
        try:
            outs, ev = self.run.step(noalloc=self.rng.integers(0, 4) == 0)
        except B.RandAttnError as e:
            assert e.status == B.RA_ERR_CAPACITY and self.layout == B.RA_LAYOUT_PAGED, e
            return False, 0
        outs = outs.float().cpu()
        evs = 0
        for o in oracles:
            o.rep.append()
            for layer in range(self.L):
                self.worst = max(self.worst, attn_err(
                    outs[layer, o.slot], o.attend(layer, o.rep.step - 1), self.dtype,
                    (self.seed, ctx, o.slot, layer)))
            evs += bool(o.rep.end_step())
        if not self.graph:
            assert ev == evs, (ev, evs)
        return True, evs

    def op_step(self, op):
        if not self.oracles:
            if self.graph:
                B.ra_graph_mode(self.run.h, 0)
                self.graph = False
            if self.free():
                self.begin(self.free()[0])
            return
        done, evs = self.step(list(self.oracles.values()), op)
        if not done:                    # out of pages: preempt one for good
            self.end(self.pick(sorted(self.oracles)))
            self.count("refused")
            return
        self.count("step")
        if evs and not self.graph:
            self.check(rows=self.rng.integers(0, 4) == 0)

    def op_forward(self):
        act = sorted(self.oracles)
        n = int(self.rng.integers(0, 2 * self.cfg["every"] + 3))
        slots = act if self.rng.integers(0, 2) else [self.pick(act)]
        try:
            if len(slots) > 1 or len(act) == 1 and self.rng.integers(0, 2):
                B.ra_fast_forward(self.run.h, n)
                slots = act
            else:
                B.ra_seq_fast_forward(self.run.h, slots[0], n)
        except B.RandAttnError as e:
            assert e.status == B.RA_ERR_CAPACITY and self.layout == B.RA_LAYOUT_PAGED, e
            return
        for s in slots:
            self.oracles[s].advance(n)
            self.run.steps[s] += n
            self.run.materialise(s)      # positions-only steps: rows from the generator
        self.check(rows=True)
        self.count("forward")

    def op_resume(self, op):
        run = self.run
        s = self.pick(sorted(self.oracles))
        if self.explicit[s]:            # explicit events are not replayed by a forward
            return
        info = B.ra_get_seq_info(run.h, s)
        ks = torch.empty(self.L, self.Hkv, info.len, 128, dtype=run.tdtype, device="cuda")
        vs = torch.empty_like(ks)
        for layer in range(self.L):
            for g in range(self.Hkv):
                B.ra_read_rows(run.h, s, layer, g, ks[layer, g], vs[layer, g])
        req = self.oracles.pop(s)
        run.end(s)
        for _ in range(int(self.rng.integers(0, 4))):      # the others decode meanwhile
            if not self.oracles or not self.step(list(self.oracles.values()), (op, "p"))[0]:
                break
        t = self.pick(self.free())
        run.lps[t], run.seeds[t], run.rids[t] = req.lp, req.rep.seed, req.rid
        try:
            B.ra_seq_begin(run.h, t, req.lp, req.rep.seed, req.rid, None, None)
        except B.RandAttnError as e:
            assert e.status == B.RA_ERR_CAPACITY, e
            return
        run.active.add(t)
        try:
            B.ra_seq_fast_forward(run.h, t, info.step)
        except B.RandAttnError as e:
            assert e.status == B.RA_ERR_CAPACITY and self.layout == B.RA_LAYOUT_PAGED, e
            run.end(t)
            return
        B.ra_write_rows(run.h, t, ks, vs)
        now = B.ra_get_seq_info(run.h, t)
        assert (now.len, now.step, now.event) == (info.len, info.step, info.event)
        run.steps[t] = info.step
        req.slot = t
        self.oracles[t] = req
        self.explicit[t] = False
        self.check(rows=True)
        self.count("resume")

    def go(self, n_ops):
        rng = self.rng
        for s in range(self.max_seqs):
            if rng.integers(0, 3):
                self.begin(s)
        for op in range(n_ops):
            k = int(rng.integers(0, 100))
            if self.graph and k < 95:
                k = 0                    # in graph mode: steps, or leave it
            if k < 60 or not self.oracles and k < 95:
                self.op_step(op)
            elif k < 66:
                if self.free() and rng.integers(0, 2):
                    self.begin(self.pick(self.free()))
                else:
                    self.end(self.pick(sorted(self.oracles)))
                    self.count("end")
            elif k < 70:
                s = self.pick(sorted(self.oracles))
                B.ra_evict_now(self.run.h, s)
                self.oracles[s].rep.evict_now()
                self.explicit[s] = True
                self.check(rows=True)
                self.count("evict_now")
            elif k < 75:
                self.op_forward()
            elif k < 85:
                self.op_resume(op)
            elif k < 95:
                if self.layout != B.RA_LAYOUT_PAGED:
                    B.ra_graph_mode(self.run.h, 1)
                    self.graph = True
                    self.count("graph")
            elif self.graph:
                B.ra_graph_mode(self.run.h, 0)
                self.graph = False
                self.check(rows=True)
        if self.graph:
            B.ra_graph_mode(self.run.h, 0)
        self.check(rows=True)
        self.run.close()


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_protocol_matches_oracle(case):
    f = Fuzz(case)
    log("protocol fuzz %d: %s" % (case, f.cfg))
    f.go(N_OPS)
    log("  %s worst %.3g" % (f.counts, f.worst))
    assert f.counts.get("step", 0) > 0
