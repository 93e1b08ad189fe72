"""Thin ctypes binding of the C ABI in ``include/randattn.h``.

Argument marshalling only: every function below has the name and argument
order of the C entry point it wraps, takes torch tensors where the C call
takes device pointers, takes ``stream=None`` for the current torch stream,
and raises ``RandAttnError`` on a non-zero status.  All work runs in the HIP
kernels of ``lib/librandattn.so``; there is no fallback, and a missing or
unloadable library raises immediately.

``Cache`` is a convenience owner: it sizes and allocates the pools, the
metadata buffer and the workspace as torch CUDA tensors and keeps them alive
for the lifetime of the C handle.
"""

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib",
                         "librandattn.so")

RA_OK = 0
RA_ERR_INVALID_ARG = -1
RA_ERR_CAPACITY = -2
RA_ERR_BUDGET = -3
RA_ERR_UNSUPPORTED = -4
RA_ERR_HIP = -5
RA_ERR_STATE = -6
RA_F32, RA_BF16 = 0, 1
RA_BUDGET_EVICTABLE, RA_BUDGET_TOTAL = 0, 1
RA_LAYOUT_CHRONOLOGICAL, RA_LAYOUT_HOLE_FILL, RA_LAYOUT_PAGED = 0, 1, 2
RA_POLICY_RANDOM, RA_POLICY_SHARED, RA_POLICY_BLOCK, RA_POLICY_RECENCY = 0, 1, 2, 3
RA_POLICY_EXTERNAL = 4
RA_SCORER_SNAPKV, RA_SCORER_RKV, RA_SCORER_VASE = 0, 1, 2
RA_NOALLOC_SCRATCH_BYTES = 8 << 20

# Every entry point declared in include/randattn.h.
EXPORTS = (
    "ra_config_check", "ra_region_rows", "ra_seq_rows", "ra_required_slots",
    "ra_meta_bytes",
    "ra_workspace_bytes", "ra_cache_create", "ra_cache_destroy",
    "ra_pool_info", "ra_seq_begin", "ra_seq_end", "ra_get_seq_info", "ra_decode_attention",
    "ra_decode_attention_noalloc",
    "ra_end_step", "ra_graph_mode", "ra_evict_now", "ra_fast_forward", "ra_seq_fast_forward",
    "ra_export_positions",
    "ra_write_rows", "ra_read_rows", "ra_read_positions", "ra_status_string",
    "ra_last_hip_error", "ra_attention_plan", "ra_window_select",
    "ra_scored_scratch_bytes", "ra_scored_evict",
)


class RandAttnError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = "%s failed: %s (%d)" % (where, status_string(status), status)
        if status == RA_ERR_HIP:
            msg += ", hipError %d" % _lib().ra_last_hip_error()
        super().__init__(msg)


class ra_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_layers", "num_q_heads", "num_kv_heads", "head_dim", "budget_k",
        "recent_r", "evict_every", "budget_mode", "dtype", "max_seqs",
        "attn_split", "layout", "policy", "policy_block", "page_rows",
        "max_prompt_len")]


class ra_scorer_params(ctypes.Structure):
    _fields_ = [("scorer", ctypes.c_int32), ("rkv_lambda", ctypes.c_float),
                ("rkv_threshold", ctypes.c_float), ("rkv_recent_dups", ctypes.c_int32),
                ("vase_n_large", ctypes.c_int32), ("vase_seed", ctypes.c_uint64)]


def make_scorer(scorer, rkv_lambda=0.1, rkv_threshold=0.9, rkv_recent_dups=1,
                vase_n_large=-1, vase_seed=0):
    return ra_scorer_params(scorer, rkv_lambda, rkv_threshold, rkv_recent_dups,
                            vase_n_large, vase_seed)


class ra_seq_info(ctypes.Structure):
    _fields_ = [("active", ctypes.c_int32), ("prompt_len", ctypes.c_int32),
                ("len", ctypes.c_int32), ("step", ctypes.c_int32),
                ("event", ctypes.c_int32), ("k_keep", ctypes.c_int32),
                ("cap", ctypes.c_int32), ("base", ctypes.c_int64),
                ("move_pending", ctypes.c_int32)]


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_U64 = ctypes.c_uint64
_SZ = ctypes.c_size_t
_CFG = ctypes.POINTER(ra_config)
_SIGS = {
    "ra_config_check": (_I32, [_CFG]),
    "ra_region_rows": (_I64, [_CFG, _I32]),
    "ra_seq_rows": (_I64, [_CFG, _I32]),
    "ra_required_slots": (_I64, [_CFG, ctypes.POINTER(ctypes.c_int32), _I32]),
    "ra_meta_bytes": (_SZ, [_CFG]),
    "ra_workspace_bytes": (_SZ, [_CFG]),
    "ra_cache_create": (_I32, [_CFG, _P, _P, _P, _I64, _P, _SZ, _P,
                               ctypes.POINTER(_P)]),
    "ra_cache_destroy": (_I32, [_P]),
    "ra_pool_info": (_I32, [_P, ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "ra_seq_begin": (_I32, [_P, _I32, _I32, _U64, _U64, _P, _P, _P]),
    "ra_seq_end": (_I32, [_P, _I32, _P]),
    "ra_get_seq_info": (_I32, [_P, _I32, ctypes.POINTER(ra_seq_info)]),
    "ra_decode_attention": (_I32, [_P, _I32, _P, _P, _P, _P, _P, _SZ, _P]),
    "ra_decode_attention_noalloc": (_I32, [_P, _I32, _P, _P, _P, _P, _P]),
    "ra_end_step": (_I32, [_P, _P, ctypes.POINTER(_I32)]),
    "ra_graph_mode": (_I32, [_P, _I32, _P]),
    "ra_evict_now": (_I32, [_P, _I32, _P]),
    "ra_fast_forward": (_I32, [_P, _I32, _P]),
    "ra_seq_fast_forward": (_I32, [_P, _I32, _I32, _P]),
    "ra_export_positions": (_I32, [_P, _I32, _P, _I64, _P]),
    "ra_write_rows": (_I32, [_P, _I32, _P, _P, _P]),
    "ra_read_rows": (_I32, [_P, _I32, _I32, _I32, _P, _P, _P]),
    "ra_read_positions": (_I32, [_P, _I32, _I32, _I32, _P, _I32,
                                 ctypes.POINTER(_I32), _P]),
    "ra_status_string": (ctypes.c_char_p, [_I32]),
    "ra_last_hip_error": (_I32, []),
    "ra_attention_plan": (_I32, [_P, ctypes.POINTER(_I32), ctypes.POINTER(_I32),
                                 ctypes.POINTER(_I32)]),
    "ra_window_select": (_I32, [_P, _I32, _I32, _P, _P, _I32, _P, _P]),
    "ra_scored_scratch_bytes": (ctypes.c_size_t, [_P, _I32]),
    "ra_scored_evict": (_I32, [_P, _I32, _I32, _P, _P, _P, ctypes.c_size_t, _P]),
}

_handle = None


def library_path():
    return _LIB_PATH


def _lib():
    """Load the shared library once; raise if it is missing."""
    global _handle
    if _handle is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError("%s is not built; run python -m "
                              "paper_2609_03430_amd.build" % _LIB_PATH)
        lib = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _handle = lib
    return _handle


def _check(status, where):
    if status != RA_OK:
        raise RandAttnError(status, where)


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


# Config of every live handle, for the tensor checks below (the C ABI takes
# bare pointers and cannot see a buffer's size, dtype or layout).
_CONFIGS = {}


def _cfg_of(handle):
    return _CONFIGS.get(getattr(handle, "value", handle))


def _cache_dtype(cfg):
    return torch.bfloat16 if cfg.dtype == RA_BF16 else torch.float32


def _arg(t, where, name, dtype=None, numel=0):
    """Refuse, before its pointer crosses the ABI, a tensor that the call
    would read or write out of bounds or misread: not a contiguous device
    tensor, another dtype than the call's, or fewer elements than it uses."""
    if t is None:
        return
    why = None
    if not isinstance(t, torch.Tensor):
        why = "not a tensor"
    elif not t.is_cuda:
        why = "not on the GPU"
    elif not t.is_contiguous():
        why = "not contiguous"
    elif dtype is not None and t.dtype != dtype:
        why = "dtype %s, expected %s" % (t.dtype, dtype)
    elif t.numel() < numel:
        why = "%d elements, needs %d" % (t.numel(), numel)
    if why:
        raise RandAttnError(RA_ERR_INVALID_ARG, "%s (%s: %s)" % (where, name, why))


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def make_config(num_layers, num_q_heads, num_kv_heads, budget_k, recent_r=64,
                evict_every=64, budget_mode=RA_BUDGET_EVICTABLE, dtype=RA_BF16,
                max_seqs=1, head_dim=128, attn_split=0,
                layout=RA_LAYOUT_CHRONOLOGICAL, policy=RA_POLICY_RANDOM,
                policy_block=1, page_rows=64, max_prompt_len=0):
    """page_rows and max_prompt_len apply to RA_LAYOUT_PAGED only."""
    return ra_config(num_layers, num_q_heads, num_kv_heads, head_dim, budget_k,
                     recent_r, evict_every, budget_mode, dtype, max_seqs,
                     attn_split, layout, policy, policy_block, page_rows,
                     max_prompt_len)


# ---- one wrapper per C entry point ------------------------------------------

def status_string(status):
    return _lib().ra_status_string(int(status)).decode()


def ra_status_string(status):
    return status_string(status)


def ra_last_hip_error():
    return _lib().ra_last_hip_error()


def ra_config_check(cfg):
    return _lib().ra_config_check(ctypes.byref(cfg))


def ra_region_rows(cfg, prompt_len):
    return _lib().ra_region_rows(ctypes.byref(cfg), int(prompt_len))


def ra_seq_rows(cfg, prompt_len):
    return _lib().ra_seq_rows(ctypes.byref(cfg), int(prompt_len))


def ra_required_slots(cfg, prompt_lens):
    """Pool rows for a batch with these prompt lengths (a host list)."""
    arr = (ctypes.c_int32 * len(prompt_lens))(*[int(x) for x in prompt_lens])
    return _lib().ra_required_slots(ctypes.byref(cfg), arr, len(prompt_lens))


def ra_meta_bytes(cfg):
    return _lib().ra_meta_bytes(ctypes.byref(cfg))


def ra_workspace_bytes(cfg):
    return _lib().ra_workspace_bytes(ctypes.byref(cfg))


def ra_cache_create(cfg, k_pool, v_pool, pos_pool, pool_rows, meta, stream=None):
    where = "ra_cache_create"
    if ra_config_check(cfg) == RA_OK:
        rows = int(pool_rows) * cfg.head_dim
        _arg(k_pool, where, "k_pool", _cache_dtype(cfg), rows)
        _arg(v_pool, where, "v_pool", _cache_dtype(cfg), rows)
        _arg(pos_pool, where, "pos_pool", torch.int32, int(pool_rows))
        _arg(meta, where, "meta")
    out = ctypes.c_void_p()
    _check(_lib().ra_cache_create(ctypes.byref(cfg), _ptr(k_pool), _ptr(v_pool),
                                  _ptr(pos_pool), int(pool_rows), _ptr(meta),
                                  meta.numel() * meta.element_size(),
                                  _stream(stream), ctypes.byref(out)),
           "ra_cache_create")
    _CONFIGS[out.value] = ra_config.from_buffer_copy(cfg)
    return out


def ra_cache_destroy(handle):
    _check(_lib().ra_cache_destroy(handle), "ra_cache_destroy")
    _CONFIGS.pop(getattr(handle, "value", handle), None)


def ra_pool_info(handle):
    """(used_rows, free_rows) of the cache's pool (host mirror)."""
    used, free = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(_lib().ra_pool_info(handle, ctypes.byref(used), ctypes.byref(free)),
           "ra_pool_info")
    return used.value, free.value


def ra_seq_begin(handle, seq, prompt_len, seed, request_id, k_prompt=None,
                 v_prompt=None, stream=None):
    cfg = _cfg_of(handle)
    if cfg is not None:
        n = cfg.num_layers * cfg.num_kv_heads * max(0, int(prompt_len)) * cfg.head_dim
        _arg(k_prompt, "ra_seq_begin", "k_prompt", _cache_dtype(cfg), n)
        _arg(v_prompt, "ra_seq_begin", "v_prompt", _cache_dtype(cfg), n)
    _check(_lib().ra_seq_begin(handle, int(seq), int(prompt_len), int(seed),
                               int(request_id), _ptr(k_prompt), _ptr(v_prompt),
                               _stream(stream)), "ra_seq_begin")


def ra_seq_end(handle, seq, stream=None):
    _check(_lib().ra_seq_end(handle, int(seq), _stream(stream)), "ra_seq_end")


def ra_get_seq_info(handle, seq):
    info = ra_seq_info()
    _check(_lib().ra_get_seq_info(handle, int(seq), ctypes.byref(info)),
           "ra_get_seq_info")
    return info


def _decode_args(handle, where, q, k_new, v_new, out):
    cfg = _cfg_of(handle)
    if cfg is None:
        return
    dt, n, d = _cache_dtype(cfg), cfg.max_seqs, cfg.head_dim
    _arg(q, where, "q", dt, n * cfg.num_q_heads * d)
    _arg(k_new, where, "k_new", dt, n * cfg.num_kv_heads * d)
    _arg(v_new, where, "v_new", dt, n * cfg.num_kv_heads * d)
    _arg(out, where, "out", dt, n * cfg.num_q_heads * d)


def ra_decode_attention(handle, layer, q, k_new, v_new, out, workspace,
                        stream=None):
    _decode_args(handle, "ra_decode_attention", q, k_new, v_new, out)
    _arg(workspace, "ra_decode_attention", "workspace")
    _check(_lib().ra_decode_attention(handle, int(layer), _ptr(q), _ptr(k_new),
                                      _ptr(v_new), _ptr(out), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(),
                                      _stream(stream)), "ra_decode_attention")


def ra_decode_attention_noalloc(handle, layer, q, k_new, v_new, out, stream=None):
    """ra_decode_attention with the split partials in the library's fixed
    device array (no workspace; see the header for its limit)."""
    _decode_args(handle, "ra_decode_attention_noalloc", q, k_new, v_new, out)
    _check(_lib().ra_decode_attention_noalloc(handle, int(layer), _ptr(q), _ptr(k_new),
                                              _ptr(v_new), _ptr(out), _stream(stream)),
           "ra_decode_attention_noalloc")


def ra_end_step(handle, stream=None):
    n = ctypes.c_int32(0)
    _check(_lib().ra_end_step(handle, _stream(stream), ctypes.byref(n)),
           "ra_end_step")
    return n.value


def ra_graph_mode(handle, on, stream=None):
    _check(_lib().ra_graph_mode(handle, 1 if on else 0, _stream(stream)), "ra_graph_mode")


def ra_evict_now(handle, seq, stream=None):
    _check(_lib().ra_evict_now(handle, int(seq), _stream(stream)), "ra_evict_now")


def ra_fast_forward(handle, n_steps, stream=None):
    _check(_lib().ra_fast_forward(handle, int(n_steps), _stream(stream)),
           "ra_fast_forward")


def ra_seq_fast_forward(handle, seq, n_steps, stream=None):
    _check(_lib().ra_seq_fast_forward(handle, int(seq), int(n_steps), _stream(stream)),
           "ra_seq_fast_forward")


def ra_export_positions(handle, seq, out, stream=None):
    _arg(out, "ra_export_positions", "out", torch.int32)
    _check(_lib().ra_export_positions(handle, int(seq), _ptr(out), out.numel(),
                                      _stream(stream)), "ra_export_positions")


def _rows_needed(handle, seq, per_head):
    """(dtype, elements) of a row array of slot `seq`: all its heads, or one."""
    cfg = _cfg_of(handle)
    if cfg is None:
        return None, 0
    info = ra_seq_info()
    if _lib().ra_get_seq_info(handle, int(seq), ctypes.byref(info)) != RA_OK:
        return _cache_dtype(cfg), 0
    heads = 1 if per_head else cfg.num_layers * cfg.num_kv_heads
    return _cache_dtype(cfg), heads * info.len * cfg.head_dim


def ra_write_rows(handle, seq, k_rows, v_rows, stream=None):
    dt, n = _rows_needed(handle, seq, False)
    _arg(k_rows, "ra_write_rows", "k_rows", dt, n)
    _arg(v_rows, "ra_write_rows", "v_rows", dt, n)
    _check(_lib().ra_write_rows(handle, int(seq), _ptr(k_rows), _ptr(v_rows),
                                _stream(stream)), "ra_write_rows")


def ra_read_rows(handle, seq, layer, kv_head, k_out=None, v_out=None,
                 stream=None):
    dt, n = _rows_needed(handle, seq, True)
    _arg(k_out, "ra_read_rows", "k_out", dt, n)
    _arg(v_out, "ra_read_rows", "v_out", dt, n)
    _check(_lib().ra_read_rows(handle, int(seq), int(layer), int(kv_head),
                               _ptr(k_out), _ptr(v_out), _stream(stream)),
           "ra_read_rows")


def ra_read_positions(handle, seq, layer, kv_head, cap, stream=None):
    """Synchronous; returns a numpy int32 array of the head's positions."""
    import numpy as np
    buf = (ctypes.c_int32 * max(1, int(cap)))()
    n = ctypes.c_int32(0)
    _check(_lib().ra_read_positions(handle, int(seq), int(layer), int(kv_head),
                                    ctypes.cast(buf, ctypes.c_void_p), int(cap),
                                    ctypes.byref(n), _stream(stream)),
           "ra_read_positions")
    return np.frombuffer(buf, dtype=np.int32, count=n.value).copy()


def ra_window_select(handle, seq_lo, seq_hi, q_window, scores=None, scores_stride=0,
                     drops=None, stream=None):
    """Measurement only: the observation-window scoring pass (see the header)."""
    cfg = _cfg_of(handle)
    if cfg is not None:
        heads = max(0, int(seq_hi) - int(seq_lo)) * cfg.num_layers * cfg.num_kv_heads
        _arg(q_window, "ra_window_select", "q_window", torch.bfloat16,
             cfg.max_seqs * cfg.num_layers * cfg.num_q_heads * 64 * cfg.head_dim)
        _arg(scores, "ra_window_select", "scores", torch.float32, heads * int(scores_stride))
        _arg(drops, "ra_window_select", "drops", torch.int32, heads * cfg.evict_every)
    _check(_lib().ra_window_select(handle, int(seq_lo), int(seq_hi), _ptr(q_window),
                                   _ptr(scores), int(scores_stride), _ptr(drops),
                                   _stream(stream)), "ra_window_select")


def ra_scored_scratch_bytes(cfg, max_prompt_len):
    return int(_lib().ra_scored_scratch_bytes(ctypes.byref(cfg), int(max_prompt_len)))


def ra_scored_evict(handle, seq_lo, seq_hi, params, q_window, scratch, stream=None):
    """Measurement only: one score-based eviction round (see the header)."""
    cfg = _cfg_of(handle)
    if cfg is not None:
        _arg(q_window, "ra_scored_evict", "q_window", torch.bfloat16,
             cfg.max_seqs * cfg.num_layers * cfg.num_q_heads * 64 * cfg.head_dim)
    _arg(scratch, "ra_scored_evict", "scratch")
    nbytes = scratch.numel() * scratch.element_size()
    _check(_lib().ra_scored_evict(handle, int(seq_lo), int(seq_hi), ctypes.byref(params),
                                  _ptr(q_window), _ptr(scratch), ctypes.c_size_t(nbytes),
                                  _stream(stream)), "ra_scored_evict")


def ra_attention_plan(handle):
    """(split_keys, max_splits, waves) of the next attention launch."""
    sk, ms, w = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(0)
    _check(_lib().ra_attention_plan(handle, ctypes.byref(sk), ctypes.byref(ms),
                                    ctypes.byref(w)), "ra_attention_plan")
    return sk.value, ms.value, w.value


# ---- owner of the device buffers ----------------------------------------------

class Cache:
    """Allocates pools, metadata and workspace with torch and owns the handle.

    pool_rows: total rows (sum of ra_seq_rows over the sequences it will hold).
    """

    def __init__(self, cfg, pool_rows, device="cuda", stream=None):
        self.cfg = cfg
        self.device = torch.device(device)
        _check(ra_config_check(cfg), "ra_config_check")
        self.dtype = torch.bfloat16 if cfg.dtype == RA_BF16 else torch.float32
        pool_rows = int(pool_rows)
        pool_rows += (-pool_rows) % 32
        self.pool_rows = pool_rows
        d = cfg.head_dim
        self.k_pool = torch.zeros(pool_rows, d, dtype=self.dtype, device=self.device)
        self.v_pool = torch.zeros(pool_rows, d, dtype=self.dtype, device=self.device)
        self.pos_pool = torch.zeros(pool_rows, dtype=torch.int32, device=self.device)
        self.meta = torch.zeros(ra_meta_bytes(cfg), dtype=torch.uint8, device=self.device)
        self.workspace = torch.empty(ra_workspace_bytes(cfg), dtype=torch.uint8,
                                     device=self.device)
        self.handle = ra_cache_create(cfg, self.k_pool, self.v_pool, self.pos_pool,
                                      pool_rows, self.meta, stream)

    def close(self):
        if self.handle is not None:
            ra_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def decode(self, layer, q, k_new, v_new, out, stream=None):
        ra_decode_attention(self.handle, layer, q, k_new, v_new, out,
                            self.workspace, stream)

    def decode_noalloc(self, layer, q, k_new, v_new, out, stream=None):
        ra_decode_attention_noalloc(self.handle, layer, q, k_new, v_new, out, stream)
