"""The paged layout's page accounting, refusals and page reuse.

Appendix G names what physical eviction under paging must do: rewrite each
request's surviving rows into its blocks, free the tail, keep positions
logical.  Here a sequence holds exactly the pages its rows need between
steps (ceil(len / page_rows) page groups), an eviction returns the pages
past the new length to the pool, a step that needs a page the pool does not
have is refused before any launch, and pages released by one request serve
the next one.  Outputs and kept sets stay the oracle's throughout.
"""

import numpy as np
import pytest
import torch

from gpu_harness import OracleSeq, Run, attn_err, check_heads, log
from paper_2609_03430_amd import binding as B

pytestmark = pytest.mark.gpu


def _pages(rows, page_rows):
    return -(-rows // page_rows)


def _step_and_check(run, oracles, t):
    outs, ev = run.step()
    outs = outs.float().cpu()
    for o in oracles:
        o.rep.append()
        for layer in range(run.L):
            attn_err(outs[layer, o.slot], o.attend(layer, o.rep.step - 1), B.RA_BF16,
                     (t, o.slot, layer))
        o.rep.end_step()
    return ev


@pytest.mark.parametrize("page_rows", [32, 64])
def test_pages_follow_the_rows(page_rows):
    """Between steps every sequence holds ceil(len / page_rows) page groups
    (its growth takes a group when a new row starts a page; an event gives
    back the groups past the new length), the pool's used rows are the sum
    of those groups, and ending a sequence returns all of its groups."""
    log("paged accounting page_rows=%d" % page_rows)
    L, Hkv = 2, 2
    run = Run(L=L, Hq=4, Hkv=Hkv, K=70, lps=[5, 40, 0], r=8, every=8,
              layout=B.RA_LAYOUT_PAGED, page_rows=page_rows)
    group = L * Hkv * page_rows
    used0, free0 = B.ra_pool_info(run.h)
    total = used0 + free0
    oracles = [OracleSeq(run, s) for s in range(run.n)]

    def check_pages():
        used = 0
        for s in run.active:
            info = B.ra_get_seq_info(run.h, s)
            assert info.cap == _pages(info.len, page_rows) * page_rows, (s, info.len, info.cap)
            used += _pages(info.len, page_rows) * group
        u, f = B.ra_pool_info(run.h)
        assert (u, f) == (used, total - used)

    check_pages()
    events = 0
    for t in range(200):
        events += bool(_step_and_check(run, oracles, t))
        check_pages()
    assert events >= 15
    check_heads(run, oracles)
    run.end(1)
    check_pages()
    run.end(0)
    run.end(2)
    assert B.ra_pool_info(run.h) == (0, total)
    run.close()


def test_a_step_without_free_pages_is_refused():
    """A pool one page group short: the step whose new rows need the missing
    group is refused with RA_ERR_CAPACITY before any launch (nothing is
    appended, the state is unchanged); once another sequence ends, the same
    step decodes and both the survivor's outputs and sets are the oracle's."""
    log("paged capacity refusal")
    page_rows, L, Hkv = 32, 1, 2
    K, r, every = 40, 8, 8
    cfg = B.make_config(L, 4, Hkv, K, r, every, B.RA_BUDGET_EVICTABLE, B.RA_BF16, 2,
                        layout=B.RA_LAYOUT_PAGED, page_rows=page_rows, max_prompt_len=31)
    full = B.ra_seq_rows(cfg, 31)                   # the most one sequence holds
    group = L * Hkv * page_rows
    pool = 2 * full - group
    run = Run(L=L, Hq=4, Hkv=Hkv, K=K, lps=[31, 31], r=r, every=every,
              layout=B.RA_LAYOUT_PAGED, page_rows=page_rows, pool_rows=pool,
              max_prompt_len=31)
    oracles = [OracleSeq(run, s) for s in range(2)]
    refused = None
    for t in range(400):
        before = [B.ra_get_seq_info(run.h, s) for s in range(2)]
        q, k, v = run.step_inputs(0)
        out = torch.zeros(run.max_seqs, run.Hq, 128, dtype=torch.bfloat16, device="cuda")
        try:
            run.cache.decode(0, q, k, v, out)
        except B.RandAttnError as e:
            assert e.status == B.RA_ERR_CAPACITY
            refused = t
            break
        B.ra_end_step(run.h)
        run.steps = [s + 1 for s in run.steps]
        for o in oracles:
            o.rep.append()
            attn_err(out[o.slot].float().cpu(), o.attend(0, o.rep.step - 1), B.RA_BF16,
                     (t, o.slot))
            o.rep.end_step()
    assert refused is not None
    torch.cuda.synchronize()
    assert float(out.float().abs().max()) == 0.0      # nothing ran
    after = [B.ra_get_seq_info(run.h, s) for s in range(2)]
    for a, b in zip(before, after):
        assert (a.len, a.step, a.cap, a.event) == (b.len, b.step, b.cap, b.event)
    _, free = B.ra_pool_info(run.h)
    assert free == group                               # one group free, two needed
    # the refused step decodes once sequence 0 ends
    run.end(0)
    o = oracles[1]
    run.cache.decode(0, q, k, v, out)
    B.ra_end_step(run.h)
    run.steps = [s + 1 for s in run.steps]
    o.rep.append()
    attn_err(out[1].float().cpu(), o.attend(0, o.rep.step - 1), B.RA_BF16, ("after",))
    o.rep.end_step()
    for t in range(3 * every):
        _step_and_check(run, [o], t)
    check_heads(run, [o])
    run.close()


def test_freed_pages_serve_the_next_request():
    """Requests admitted one after another into a pool that holds two at
    their largest: each new request takes page groups that earlier requests
    wrote and released, so stale rows would show in its outputs; every
    request decodes as the oracle says."""
    log("paged page reuse")
    page_rows, L, Hkv = 32, 2, 2
    K, r, every = 60, 16, 16
    cfg = B.make_config(L, 4, Hkv, K, r, every, B.RA_BUDGET_EVICTABLE, B.RA_BF16, 2,
                        layout=B.RA_LAYOUT_PAGED, page_rows=page_rows, max_prompt_len=50)
    pool = 2 * B.ra_seq_rows(cfg, 50)
    run = Run(L=L, Hq=4, Hkv=Hkv, K=K, lps=[50, 7], r=r, every=every,
              layout=B.RA_LAYOUT_PAGED, page_rows=page_rows, pool_rows=pool,
              max_prompt_len=50, seeds=[11, 12], rids=[100, 101])
    oracles = {s: OracleSeq(run, s) for s in range(2)}
    rng = np.random.default_rng(3)
    next_rid = 102
    for round_ in range(6):
        for t in range(int(rng.integers(20, 120))):
            _step_and_check(run, list(oracles.values()), t)
        check_heads(run, list(oracles.values()))
        slot = round_ % 2
        run.end(slot)
        run.lps[slot] = int(rng.integers(0, 51))
        run.seeds[slot], run.rids[slot] = 1000 + next_rid, next_rid
        next_rid += 1
        run.begin(slot)
        oracles[slot] = OracleSeq(run, slot)
    run.close()
