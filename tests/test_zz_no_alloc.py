"""The allocation-free attention entry point against the one with a workspace.

Two caches receive the same sequences and the same inputs; one is decoded
with ra_decode_attention (caller's workspace), the other with
ra_decode_attention_noalloc (the library's fixed device array).  Both run
the same kernels with the same launch plan, so outputs, kept positions and
rows must be bit-identical, and both must match the fp64 oracle within the
workloads' tolerance.  Each case is run twice in a row, the second time with
a smaller input (fewer sequences, shorter caches, fewer splits), so stale
partials left in the shared array by the first call cannot leak into the
second.  A launch whose partials would not fit the array is refused before
any launch.
"""

import numpy as np
import pytest
import torch

from gpu_harness import TOL, OracleSeq, Run, check_heads, log, max_abs
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu


def _pair(**kw):
    return Run(**kw), Run(**kw)


def _run_case(dtype, L, Hq, Hkv, K, lps, steps, check_every):
    kw = dict(L=L, Hq=Hq, Hkv=Hkv, K=K, lps=lps, r=16, every=16, dtype=dtype,
              wl_seed=77)
    ref, na = _pair(**kw)
    oracles = [OracleSeq(ref, s) for s in range(ref.n)]
    splits_seen = set()
    worst = 0.0
    for t in range(steps):
        sk, ms, _ = B.ra_attention_plan(na.h)
        splits_seen.add(ms)
        outs_ref = torch.empty(L, ref.max_seqs, Hq, 128, dtype=ref.tdtype, device="cuda")
        outs_na = torch.full_like(outs_ref, float("nan"))
        for layer in range(L):
            q, k, v = ref.step_inputs(layer)
            ref.cache.decode(layer, q, k, v, outs_ref[layer])
            na.cache.decode_noalloc(layer, q, k, v, outs_na[layer])
        ev_ref = B.ra_end_step(ref.h)
        ev_na = B.ra_end_step(na.h)
        assert ev_ref == ev_na
        ref.steps = [s + 1 for s in ref.steps]
        na.steps = [s + 1 for s in na.steps]
        torch.cuda.synchronize()
        assert torch.equal(outs_ref, outs_na), ("outputs differ", t)
        for o in oracles:
            o.rep.append()
            if t % check_every == 0 or t == steps - 1:
                for layer in range(L):
                    err = max_abs(outs_na[layer, o.slot].float().cpu(), o.attend(layer, t))
                    worst = max(worst, err)
                    assert err <= TOL[dtype], (t, o.slot, layer, err)
            o.rep.end_step()
    check_heads(na, oracles)
    for s in range(ref.n):
        for layer in range(L):
            for g in range(Hkv):
                assert np.array_equal(ref.positions(s, layer, g), na.positions(s, layer, g))
    log("  no-alloc %s L=%d Hq=%d Hkv=%d lps=%s: splits %s, worst %.3g"
        % ("bf16" if dtype == B.RA_BF16 else "f32", L, Hq, Hkv, lps,
           sorted(splits_seen), worst))
    ref.close()
    na.close()
    return splits_seen


@pytest.mark.parametrize("dtype", [B.RA_BF16, B.RA_F32])
def test_noalloc_matches_workspace_entry_point(dtype):
    log("no-alloc attention, dtype %d" % dtype)
    # first call: larger input, several splits per head
    big = _run_case(dtype, L=2, Hq=8, Hkv=2, K=600, lps=[300, 900, 57],
                    steps=40, check_every=13)
    assert max(big) > 1
    # second call, right after: a smaller input on the same device array
    small = _run_case(dtype, L=1, Hq=4, Hkv=1, K=40, lps=[9], steps=35,
                      check_every=7)
    assert max(small) < max(big)


def test_noalloc_refuses_partials_beyond_its_array():
    """fp32 with 64 sequences of 8 KV heads and G = 16: two splits per head
    need 64 * 8 * 2 * 16 * 130 * 4 bytes, more than the array holds.  The
    call is refused before any launch and the workspace entry point still
    decodes the step."""
    log("no-alloc capacity refusal")
    run = Run(L=1, Hq=128, Hkv=8, K=32, lps=[64] * 64, r=16, every=16, dtype=B.RA_F32,
              wl_seed=5)
    sk, ms, _ = B.ra_attention_plan(run.h)
    need = 64 * 8 * ms * 16 * 130 * 4
    assert ms >= 2 and need > B.RA_NOALLOC_SCRATCH_BYTES, (ms, need)
    q, k, v = run.step_inputs(0)
    out = torch.zeros(run.max_seqs, run.Hq, 128, dtype=torch.float32, device="cuda")
    with pytest.raises(B.RandAttnError) as e:
        B.ra_decode_attention_noalloc(run.h, 0, q, k, v, out)
    assert e.value.status == B.RA_ERR_CAPACITY
    torch.cuda.synchronize()
    assert float(out.abs().max()) == 0.0
    # nothing was appended: the regular entry point decodes the step
    oracles = [OracleSeq(run, s, heads=[(0, g) for g in range(8)]) for s in (0, 63)]
    run.cache.decode(0, q, k, v, out)
    B.ra_end_step(run.h)
    for o in oracles:
        o.rep.append()
        err = max_abs(out[o.slot].float().cpu(), o.attend(0, 0))
        assert err <= TOL[B.RA_F32], (o.slot, err)
    run.close()
