"""The C-ABI library on the CPU: it loads, exports every declared entry
point, and rejects bad arguments on the host before touching the GPU."""

import ctypes
import os
import re

import pytest

from paper_2609_03430_amd import binding as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "randattn.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ra_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(B.library_path())
    names = _declared()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(B.EXPORTS) == names


def test_config_validation():
    ok = B.make_config(40, 40, 8, 8192, max_seqs=32)
    assert B.ra_config_check(ok) == B.RA_OK
    bad = [
        dict(num_q_heads=41), dict(num_layers=0), dict(budget_k=-1),
        dict(recent_r=-1), dict(evict_every=0), dict(max_seqs=0),
        dict(attn_split=33), dict(budget_mode=7), dict(dtype=9), dict(layout=3),
        dict(policy=5), dict(policy=-1), dict(policy=2, policy_block=0),
        # paged layout: pages a power of two in [32, 1024], a prompt bound >= 0
        # that a TOTAL budget can hold
        dict(layout=2, page_rows=48), dict(layout=2, page_rows=16),
        dict(layout=2, page_rows=2048), dict(layout=2, max_prompt_len=-1),
        dict(layout=2, budget_mode=1, max_prompt_len=8193),
    ]
    for kw in bad:
        c = B.make_config(40, 40, 8, 8192, max_seqs=32)
        for k, v in kw.items():
            setattr(c, k, v)
        assert B.ra_config_check(c) == B.RA_ERR_INVALID_ARG, kw
    unsupported = [dict(head_dim=64), dict(num_q_heads=136, num_kv_heads=8),
                   dict(evict_every=2048), dict(budget_k=40000),
                   dict(num_layers=4096, num_q_heads=32, num_kv_heads=32)]   # L * Hkv > 65536
    for kw in unsupported:
        c = B.make_config(40, 40, 8, 8192, max_seqs=32)
        for k, v in kw.items():
            setattr(c, k, v)
        assert B.ra_config_check(c) == B.RA_ERR_UNSUPPORTED, kw


def test_region_sizes():
    c = B.make_config(40, 40, 8, 8192, max_seqs=32)
    assert B.ra_region_rows(c, 1024) == 1024 + 8192 + 64 + 64
    assert B.ra_seq_rows(c, 1024) == 40 * 8 * 9344
    assert B.ra_region_rows(c, 1) % 32 == 0
    t = B.make_config(1, 4, 2, 256, budget_mode=B.RA_BUDGET_TOTAL)
    assert B.ra_region_rows(t, 200) == 384               # 200 + 56 + 64 + 64
    assert B.ra_region_rows(t, 257) == B.RA_ERR_BUDGET
    assert B.ra_region_rows(t, -1) == B.RA_ERR_INVALID_ARG
    assert B.ra_required_slots(c, [1024, 1, 0]) == sum(B.ra_seq_rows(c, lp) for lp in (1024, 1, 0))
    assert B.ra_required_slots(c, []) == 0
    assert B.ra_required_slots(t, [200, 257]) == B.RA_ERR_BUDGET
    assert B.ra_required_slots(t, [200, -1]) == B.RA_ERR_INVALID_ARG
    assert B.ra_meta_bytes(c) >= 64 * 32
    assert B.ra_workspace_bytes(c) >= 32 * 8 * 64 * 5 * 130 * 4


def test_paged_sizes():
    """Paged layout: a head's most rows round up to whole pages; the metadata
    buffer holds a block table of ceil((max prompt + K + r + R) / page_rows)
    entries per slot (and the attention's split counters, one per slot and
    KV head); a prompt longer than the bound is refused."""
    c = B.make_config(40, 40, 8, 8192, max_seqs=32, layout=B.RA_LAYOUT_PAGED,
                      page_rows=64, max_prompt_len=2048)
    assert B.ra_config_check(c) == B.RA_OK
    assert B.ra_region_rows(c, 1024) == 9344            # 1024 + 8192 + 128, 146 pages
    assert B.ra_region_rows(c, 1000) == 9344            # 9320 rounded up to a page
    assert B.ra_seq_rows(c, 1000) == 40 * 8 * 9344      # whole page groups
    assert B.ra_region_rows(c, 2049) == B.RA_ERR_CAPACITY
    pages = -(-(2048 + 8192 + 64 + 64) // 64)
    records = -(-(64 * 32) // 256) * 256
    arrivals = -(-(4 * 32 * 8) // 256) * 256           # split counters per (slot, KV head)
    assert B.ra_meta_bytes(c) == records + -(-(4 * 32 * pages) // 256) * 256 + arrivals
    t = B.make_config(2, 4, 2, 300, budget_mode=B.RA_BUDGET_TOTAL, max_seqs=3,
                      layout=B.RA_LAYOUT_PAGED, page_rows=32, max_prompt_len=300)
    assert B.ra_region_rows(t, 100) == 448              # 300 + 64 + 64 = 428 -> 14 pages
    assert B.ra_region_rows(t, 301) == B.RA_ERR_BUDGET


def test_create_rejects_null_buffers_without_gpu():
    c = B.make_config(2, 4, 2, 64, max_seqs=2)
    out = ctypes.c_void_p()
    lib = B._lib()
    st = lib.ra_cache_create(ctypes.byref(c), None, None, None, 1024, None, 0, None,
                             ctypes.byref(out))
    assert st == B.RA_ERR_INVALID_ARG
    # misaligned pool pointers are refused too
    st = lib.ra_cache_create(ctypes.byref(c), ctypes.c_void_p(8), ctypes.c_void_p(16),
                             ctypes.c_void_p(16), 1024, ctypes.c_void_p(16), 4096,
                             None, ctypes.byref(out))
    assert st == B.RA_ERR_INVALID_ARG
    # pool rows must be a multiple of 32
    st = lib.ra_cache_create(ctypes.byref(c), ctypes.c_void_p(16), ctypes.c_void_p(16),
                             ctypes.c_void_p(16), 1000, ctypes.c_void_p(16), 4096,
                             None, ctypes.byref(out))
    assert st == B.RA_ERR_INVALID_ARG
    # paged: of a whole number of page groups (L * Hkv * page_rows = 256 rows)
    p = B.make_config(2, 4, 2, 64, max_seqs=2, layout=B.RA_LAYOUT_PAGED, page_rows=64,
                      max_prompt_len=16)
    st = lib.ra_cache_create(ctypes.byref(p), ctypes.c_void_p(16), ctypes.c_void_p(16),
                             ctypes.c_void_p(16), 1024 + 32, ctypes.c_void_p(16), 4096,
                             None, ctypes.byref(out))
    assert st == B.RA_ERR_INVALID_ARG


def test_null_handle_calls_fail_cleanly():
    lib = B._lib()
    assert lib.ra_cache_destroy(None) == B.RA_ERR_INVALID_ARG
    assert lib.ra_end_step(None, None, None) == B.RA_ERR_INVALID_ARG
    assert lib.ra_fast_forward(None, 1, None) == B.RA_ERR_INVALID_ARG
    assert lib.ra_seq_fast_forward(None, 0, 1, None) == B.RA_ERR_INVALID_ARG
    assert lib.ra_decode_attention(None, 0, None, None, None, None, None, 0, None) \
        == B.RA_ERR_INVALID_ARG
    for code in range(-6, 1):
        assert B.ra_status_string(code) != "unknown status"


def test_meta_bytes_hold_drop_lists_up_to_a_cap():
    """bf16 chronological caches keep a drop list of evict_every slots per
    (slot, layer, KV head) for deferred row moves, unless the lists would
    pass 256 MiB (then moves are not deferred and no lists are kept)."""
    def records(n):
        return -(-(64 * n) // 256) * 256

    def arrivals(n, hkv):
        return -(-(4 * n * hkv) // 256) * 256
    c = B.make_config(40, 40, 8, 8192, max_seqs=32)
    drops = 4 * 32 * 40 * 8 * 64
    assert B.ra_meta_bytes(c) == records(32) + drops + arrivals(32, 8)
    f = B.make_config(40, 40, 8, 8192, max_seqs=32, dtype=B.RA_F32)
    assert B.ra_meta_bytes(f) == records(32) + arrivals(32, 8)
    big = B.make_config(64, 64, 16, 8192, 64, 1024, max_seqs=65536)
    assert B.ra_meta_bytes(big) == records(65536) + arrivals(65536, 16)
