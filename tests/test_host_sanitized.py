"""The host library under AddressSanitizer and UndefinedBehaviorSanitizer,
driven by a seeded protocol fuzzer and checked against the oracle (CPU only).

api.cpp (the C ABI, the host mirror of every slot, the first-fit and paged
allocators, the deferred-move bookkeeping) is built for the host alone with
both sanitizers and linked with stand-ins for the device launches
(tests/host_fuzz/stub_launchers.cpp: they keep the slot records and block
tables in the caller's metadata buffer, check that every row a launch would
touch lies in the pool, copy positions for real, and advance the slot
records as the device does).  The fuzzer (tests/host_fuzz/fuzz_protocol.cpp)
makes random calls -- begins, ends, decode steps, explicit events, fast
forwards of every sequence or of one, a request preempted (its rows read,
its slot ended) and resumed in a free slot (begun again, forwarded by its
steps, its rows written back), row and position reads and writes, entering
and leaving graph mode, calls inside an open step, bad arguments -- and
prints every slot's
mirror after each.  Here the same calls are replayed on the oracle's
SequenceReplay (the length, step and event count of every sequence after
every call, Eq. 1 with the periodic trigger), the statuses are checked
against what the header promises, and the pool's accounting against the
slots: regions disjoint inside the pool (contiguous layouts), ceil(len /
page_rows) page groups per sequence between steps, no group in two tables
(paged).  In graph mode the calls that need the host mirror must be refused
and the mirror must stay that of the entry while the oracle advances; the
records read back on leaving must be the oracle's again.  Any sanitizer
report fails the run.
"""

import json
import os
import shutil
import subprocess

import pytest

from oracle.evict import POLICY_RANDOM, SequenceReplay, keep_count

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_03430_amd", "csrc")
FUZZ = os.path.join(ROOT, "tests", "host_fuzz")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"

OK, INVALID, CAPACITY, BUDGET, UNSUPPORTED, STATE = 0, -1, -2, -3, -4, -6
EXTERNAL = 4
SEEDS = range(1, 61)
OPS = 300

pytestmark = pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)),
                                reason="hipcc / clang++ not available")


@pytest.fixture(scope="module")
def fuzzer(tmp_path_factory):
    d = tmp_path_factory.mktemp("host_fuzz")
    common = ["-O1", "-g", "-std=c++17", "-I" + os.path.join(ROOT, "include")]
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    # HIP sources for the host pass only; each sanitizer flag for the host
    # launches of per-head kernels cut into chunks of one slot (3 heads at
    # most), so that the chunked launch loops run under the sanitizers too
    hip = [HIPCC, "-x", "hip", "--cuda-host-only", "-I" + CSRC,
           "-DRA_MAX_HEADS_PER_LAUNCH=3"] + common + [
        "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
        "-fno-sanitize-recover=all"]
    objs = []
    for src, obj in ((os.path.join(CSRC, "api.cpp"), "api.o"),
                     (os.path.join(FUZZ, "stub_launchers.cpp"), "stub.o")):
        subprocess.run(hip + ["-c", src, "-o", str(d / obj)], check=True,
                       capture_output=True)
        objs.append(str(d / obj))
    subprocess.run([CLANG] + common + san + ["-c", os.path.join(FUZZ, "fuzz_protocol.cpp"),
                                             "-o", str(d / "main.o")],
                   check=True, capture_output=True)
    exe = str(d / "fuzz_protocol")
    subprocess.run([CLANG] + san + objs + [str(d / "main.o"), "-o", exe], check=True,
                   capture_output=True)
    return exe


def _run(exe, seed):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, str(seed), str(OPS)], capture_output=True, text=True,
                       env=env, timeout=120)
    assert r.returncode == 0, "seed %d: exit %d\n%s" % (seed, r.returncode, r.stderr[-3000:])
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr[-3000:]
    return [json.loads(line) for line in r.stdout.splitlines()]


class Replay:
    """The oracle's view of every slot, driven by the fuzzer's calls."""

    def __init__(self, cfg):
        (self.L, self.Hq, self.Hkv, self.K, self.r, self.every, self.mode, self.dtype,
         self.max_seqs, self.attn_split, self.layout, self.policy, self.block,
         self.page_rows, self.max_prompt_len, self.max_lp) = cfg
        self.reps = {}
        self.graph = False
        self.entry = None

    def begin(self, s, lp, seed, rid):
        pol = POLICY_RANDOM if self.policy == EXTERNAL else self.policy
        self.reps[s] = SequenceReplay(lp, keep_count(self.K, lp, self.mode), self.r,
                                      self.every, seed, rid, [(0, 0)], pol, self.block)

    def advance_one(self, s, n):
        """n positions-only steps of the sequence in slot s."""
        rep = self.reps[s]
        if self.policy == EXTERNAL:
            for _ in range(n):
                rep.append()
        elif n == 1:
            rep.append()
            rep.end_step()
        else:
            rep.advance(n)

    def steps(self, n):
        """n decode steps of every sequence; the number of sequences that
        evicted at the last one."""
        evicted = 0
        for rep in self.reps.values():
            if self.policy == EXTERNAL:        # no end-of-step eviction
                for _ in range(n):
                    rep.append()
            elif n == 1:
                rep.append()
                evicted += rep.end_step()
            else:
                rep.advance(n)
        return evicted


def _check_pool(rp, line, pool_rows, between_steps):
    used, free = line["pool"]
    assert used + free == pool_rows
    act = [(s, x) for s, x in enumerate(line["s"]) if x[0]]
    heads = rp.L * rp.Hkv
    if rp.layout == 2:
        assert line["tables"] == 0, line          # valid groups, none shared
        group = heads * rp.page_rows
        if between_steps:
            for s, x in act:
                assert x[4] == -(-x[1] // rp.page_rows) * rp.page_rows, (s, x)
            assert used == sum(x[4] // rp.page_rows for _, x in act) * group
    else:
        spans = sorted((x[5], x[5] + heads * x[4]) for _, x in act)
        assert used == sum(b - a for a, b in spans)
        for (a0, b0), (a1, b1) in zip(spans, spans[1:]):
            assert b0 <= a1                       # regions disjoint
        assert all(0 <= a and b <= pool_rows for a, b in spans)


def _check_slots(rp, line, fields=(1, 2, 3, 7)):
    for s, x in enumerate(line["s"]):
        rep = rp.reps.get(s)
        assert bool(x[0]) == (rep is not None), (s, line["op"], line["a"])
        if rep is None:
            continue
        want = {1: len(rep.P[(0, 0)]), 2: rep.step, 3: rep.event, 7: rep.k_keep}
        for f in fields:
            assert x[f] == want[f], (s, f, x, want, line["op"], line["a"])


@pytest.mark.parametrize("seed", SEEDS)
def test_protocol_fuzz_matches_oracle(fuzzer, seed):
    lines = _run(fuzzer, seed)
    head = lines[0]
    assert head["create"] == OK
    rp = Replay(head["config"])
    pool_rows = head["pool_rows"]
    prev = lines[1]
    for line in lines[1:]:
        op, st, a = line["op"], line.get("st"), line.get("a", [])
        if op == "destroy":
            assert st == OK
            break
        was_active = [x[0] for x in prev["s"]]
        between = True
        refused_in_graph = rp.graph and op in ("begin", "end", "evict_now", "fast_forward",
                                               "seq_fast_forward", "read", "write", "resume")
        if refused_in_graph:
            assert st == STATE, line
            if op in ("read", "write"):
                assert line["x"] == STATE, line
            if op == "resume":
                assert a[6:] == [STATE] * 4, line
        elif op == "graph":
            if a[0] == 1:
                if rp.layout == 2 or rp.policy == EXTERNAL:
                    assert st == UNSUPPORTED, line
                else:
                    assert st == OK, line
                    rp.graph, rp.entry = True, [list(x) for x in line["s"]]
            else:
                assert st == OK, line
                rp.graph = False
        elif op == "begin":
            s, lp = a[0], a[1]
            if was_active[s]:
                assert st == STATE
            elif rp.mode == 1 and lp > rp.K:
                assert st == BUDGET
            elif rp.layout == 2 and lp > rp.max_prompt_len:
                assert st == CAPACITY
            else:
                assert st in (OK, CAPACITY)
            if st == OK:
                rp.begin(s, lp, a[2], a[3])
        elif op == "end":
            assert st == (OK if was_active[a[0]] else STATE)
            if st == OK:
                del rp.reps[a[0]]
        elif op == "step":
            assert st == OK
            ev = rp.steps(1)
            assert line["x"] == (0 if rp.graph else ev), (line, ev)
        elif op == "step_refused":
            assert st == CAPACITY and a[0] == 0 and not rp.graph
            assert [x[:6] for x in line["s"]] == [x[:6] for x in prev["s"]]
        elif op == "evict_now":
            s = a[0]
            if not was_active[s]:
                assert st == STATE
            else:
                assert st == OK
                rp.reps[s].evict_now()
        elif op == "fast_forward":
            if st == CAPACITY:                    # nothing done
                # rows piling up (external policy) or too few free pages
                assert rp.policy == EXTERNAL or rp.layout == 2
                assert [x[:6] for x in line["s"]] == [x[:6] for x in prev["s"]]
            else:
                assert st == OK
                rp.steps(a[0])
        elif op == "seq_fast_forward":
            s, n = a
            if not was_active[s]:
                assert st == STATE, line
            elif st == CAPACITY:                  # nothing done
                assert rp.policy == EXTERNAL or rp.layout == 2
                assert [x[:6] for x in line["s"]] == [x[:6] for x in prev["s"]]
            else:
                assert st == OK, line
                rp.advance_one(s, n)
        elif op == "resume":
            # the request of slot s ended and begun again in slot t with the
            # same prompt length, seed and request id, forwarded by its steps:
            # the oracle's state of a fresh sequence advanced by those steps
            # (the steps' periodic events; explicit events are not replayed)
            s, t, lp, seed, rid, step, e1, e2, e3, e4 = a
            assert e1 == OK and e2 == OK and e4 == OK and st == OK, line
            assert t == s or not was_active[t], line
            del rp.reps[s]
            rp.begin(t, lp, seed, rid)
            if e3 == CAPACITY:
                # rows piling up (external policy), or the forwarded rows need
                # more pages than the request held (explicit events shortened it)
                assert rp.policy == EXTERNAL or rp.layout == 2, line
            else:
                assert e3 == OK, line
                rp.advance_one(t, step)
        elif op == "read":
            s, layer, g, cap, n_out = a
            n = line["s"][s][1]
            assert st == OK
            assert line["x"] == (OK if cap >= n else CAPACITY)
            if cap >= n:
                assert n_out == n
        elif op == "write":
            s, elems = a
            assert st == OK
            rows = rp.L * rp.Hkv * line["s"][s][1]
            assert line["x"] == (OK if elems >= rows else CAPACITY)
        elif op == "midstep":
            layer, e1, e2, e3, e4 = a
            assert e1 == STATE and e2 == STATE and e4 == STATE
            assert e3 in (STATE, INVALID)
            between = False
        elif op == "bad":
            e1, e2, e3, e4, e5, e6, e7 = a
            assert (e1, e2, e3, e5, e7) == (INVALID,) * 5
            assert e4 in (INVALID, STATE)
            # a short workspace; a step the pool cannot hold is refused first
            assert e6 in (INVALID, CAPACITY)
        if rp.graph:
            # the mirror is the entry's until graph mode ends
            assert [x[:6] + x[7:] for x in line["s"]] == [x[:6] + x[7:] for x in rp.entry], line
        else:
            _check_slots(rp, line)
        _check_pool(rp, line, pool_rows, between)
        # deferred row moves: set by an end-of-step event of every active
        # sequence at once; moved by any call that reads or writes rows or
        # plans an event; otherwise carried, never created
        pend = [bool(x[6]) for x in line["s"]]
        if op == "step" and any(pend):
            assert line["x"] > 0
            assert all(p == bool(x[0]) for p, x in zip(pend, line["s"])), line
        elif op in ("read", "write", "resume") or (op in ("evict_now", "fast_forward")
                                                   and st == OK):
            assert not any(pend), line
        elif op == "seq_fast_forward" and st == OK and prev["s"][a[0]][6]:
            assert not any(pend), line        # its own pending moves done first
        elif op == "seq_fast_forward":
            # another slot's pending moves are carried
            assert [bool(x[6]) for x in prev["s"]] == pend, line
        else:
            assert all(not p or bool(q[6]) for p, q in zip(pend, prev["s"])), line
        assert all(not p or x[0] for p, x in zip(pend, line["s"]))
        prev = line
