// Host-only stand-ins for the device side of the library, so that the host
// library (api.cpp) runs on the CPU under AddressSanitizer and
// UndefinedBehaviorSanitizer.  Test infrastructure: compiled only by the
// sanitizer test, never into the library.
//
// The stand-ins do no attention or eviction arithmetic.  They keep what the
// host code hands to the device honest:
//   * the per-slot records and the block tables live in the caller's
//     metadata buffer (ordinary host memory here), written as the device
//     kernels would write them, so every slot and table index is checked
//     against that buffer's allocation;
//   * every launch that touches one sequence's rows checks that those rows
//     lie inside the pool (contiguous regions) or map to valid page groups
//     (block tables), and touches the caller's row buffers at the lengths the
//     library passes;
//   * hipMemcpyAsync copies (host to host), so position reads are checked
//     against the position pool and the caller's output;
//   * the end-of-step and plan launches advance the slot records as the
//     device does (the trigger and plan rule restated below), so that the
//     records read back when graph mode ends are the ones the GPU would
//     hold.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "ra_internal.h"

namespace {

int64_t g_pool_rows = 0;     // rows of the K / V / position pools
int64_t g_n_groups = 0;      // paged: page groups in the pool
int g_max_seqs = 0;
int g_page_rows = 0;
const int32_t* g_tables = nullptr;
int g_pps = 0;               // paged: table entries per sequence

// the allocation-free entry point's partials array (its real size)
std::vector<char>& scratch_array() {
  static std::vector<char> a(ra::kNoAllocScratchBytes);
  return a;
}

[[noreturn]] void fail(const char* what, long long a, long long b) {
  std::fprintf(stderr, "stub check failed: %s (%lld, %lld)\n", what, a, b);
  std::fflush(stderr);
  std::abort();
}

size_t elem_bytes(const ra::Shape& sh) { return sh.dtype == 1 ? 2 : 4; }

// The plan rule of an end-of-step trigger: a due sequence drops to
// prompt + k_keep + r rows and counts an event.
void plan(ra::SeqMeta& M, int r, bool at_trigger) {
  M.due = 0;
  if (at_trigger && M.len - M.prompt_len - r > M.k_keep) {
    M.due = 1;
    M.plan_len = M.len;
    M.plan_event = M.event;
    M.len = M.prompt_len + M.k_keep + r;
    M.event += 1;
  }
}

// Rows [0, len) of every head of slot `slot` lie in the pool.
void check_rows(const ra::Shape& sh, const ra::SeqMeta& M, int slot, int len) {
  if (slot < 0 || slot >= g_max_seqs) fail("slot", slot, g_max_seqs);
  if (len < 0 || len > M.cap) fail("len beyond capacity", len, M.cap);
  const int64_t heads = static_cast<int64_t>(sh.L) * sh.Hkv;
  if (sh.layout != 2) {
    if (M.base < 0 || M.base + heads * M.cap > g_pool_rows)
      fail("region outside the pool", M.base, heads * M.cap);
    return;
  }
  if (!sh.pg.tables || sh.pg.tables != g_tables) fail("block tables", 0, 0);
  const int pages = (len + g_page_rows - 1) / g_page_rows;
  if (pages > sh.pg.pages_per_seq) fail("pages beyond the table", pages, sh.pg.pages_per_seq);
  for (int k = 0; k < pages; ++k) {
    const int32_t grp = g_tables[static_cast<int64_t>(slot) * g_pps + k];
    if (grp < 0 || grp >= g_n_groups) fail("page group", grp, g_n_groups);
  }
}

// Touch n bytes of a caller buffer (reads: a checksum the sanitizer sees).
void touch_read(const void* p, size_t n) {
  if (!p || !n) return;
  volatile unsigned char sink = 0;
  const unsigned char* b = static_cast<const unsigned char*>(p);
  sink = sink + b[0] + b[n - 1];
  (void)sink;
}

void touch_write(void* p, size_t n) {
  if (p && n) std::memset(p, 0, n);
}

}  // namespace

extern "C" void stub_configure(int64_t pool_rows, int64_t n_groups, int max_seqs,
                               int page_rows) {
  g_pool_rows = pool_rows;
  g_n_groups = n_groups;
  g_max_seqs = max_seqs;
  g_page_rows = page_rows;
  g_tables = nullptr;
  g_pps = 0;
}

// Paged: the active sequences' first `caps[s] / page_rows` table entries are
// valid page groups and no group belongs to two of them.  Returns 0 if so.
extern "C" int stub_check_tables(const int* active, const int* caps, int n) {
  if (!g_tables) return 0;
  std::vector<int> owner(static_cast<size_t>(g_n_groups), -1);
  for (int s = 0; s < n; ++s) {
    if (!active[s]) continue;
    if (caps[s] % g_page_rows) return 1;
    for (int k = 0; k < caps[s] / g_page_rows; ++k) {
      const int32_t grp = g_tables[static_cast<int64_t>(s) * g_pps + k];
      if (grp < 0 || grp >= g_n_groups) return 2;
      if (owner[grp] != -1) return 3;
      owner[grp] = s;
    }
  }
  return 0;
}

extern "C" hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes,
                                     hipMemcpyKind, hipStream_t) {
  if (bytes) std::memcpy(dst, src, bytes);
  return hipSuccess;
}

extern "C" hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }

namespace ra {

hipError_t launch_zero_words(uint32_t* p, int64_t n_words, hipStream_t) {
  std::memset(p, 0, static_cast<size_t>(n_words) * 4);
  return hipSuccess;
}

hipError_t launch_seq_set(SeqMeta* meta, int slot, const SeqMeta& v, hipStream_t) {
  if (slot < 0 || slot >= g_max_seqs) fail("seq_set slot", slot, g_max_seqs);
  meta[slot] = v;
  return hipSuccess;
}

hipError_t launch_advance(SeqMeta* meta, int slot_lo, int slot_hi, int n_steps, int r, int every,
                          hipStream_t) {
  if (slot_lo < 0 || slot_hi > g_max_seqs || slot_lo > slot_hi) fail("advance range", slot_lo, slot_hi);
  for (int s = slot_lo; s < slot_hi; ++s) {
    SeqMeta& M = meta[s];
    if (!M.active) continue;
    M.step += n_steps;
    M.len += n_steps;
    plan(M, r, every > 0 && M.step % every == 0);
  }
  return hipSuccess;
}

hipError_t launch_plan_now(SeqMeta* meta, int slot, int r, hipStream_t) {
  if (slot < 0 || slot >= g_max_seqs) fail("plan_now slot", slot, g_max_seqs);
  if (meta[slot].active) plan(meta[slot], r, true);
  return hipSuccess;
}

hipError_t launch_append_positions(const Shape&, const SeqMeta* meta, int32_t*, int slot_lo,
                                   int slot_hi, int run, hipStream_t) {
  if (slot_lo < 0 || slot_hi > g_max_seqs || run < 0) fail("append range", slot_lo, slot_hi);
  touch_read(meta + slot_lo, sizeof(SeqMeta) * (slot_hi - slot_lo));
  return hipSuccess;
}

// The test build cuts per-head launches into chunks of at most 3 heads, or
// one slot where a slot has more (RA_MAX_HEADS_PER_LAUNCH=3).
void check_chunk(const Shape& sh, int slot_lo, int slot_hi, const char* what) {
  if (slot_hi - slot_lo > 1 && (slot_hi - slot_lo) * sh.L * sh.Hkv > 3)
    fail(what, slot_lo, slot_hi);
}

hipError_t launch_evict(const Shape& sh, const SeqMeta* meta, void*, void*, int32_t*, int slot_lo,
                        int slot_hi, int max_candidates, bool, hipStream_t, int32_t* drops_out,
                        int drop_stride) {
  if (slot_lo < 0 || slot_hi > g_max_seqs || slot_lo >= slot_hi) fail("evict range", slot_lo, slot_hi);
  check_chunk(sh, slot_lo, slot_hi, "evict launch over the per-launch bound");
  if (max_candidates < 0 || max_candidates > kMaxCandidates) fail("candidates", max_candidates, 0);
  if (drops_out && (drop_stride < 1 || drop_stride > kMaxEvery)) fail("drop stride", drop_stride, 0);
  touch_read(meta + slot_lo, sizeof(SeqMeta) * (slot_hi - slot_lo));
  return hipSuccess;
}

hipError_t launch_mark_pending(SeqMeta* meta, int slot_lo, int slot_hi, hipStream_t) {
  if (slot_lo < 0 || slot_hi > g_max_seqs) fail("mark range", slot_lo, slot_hi);
  for (int s = slot_lo; s < slot_hi; ++s)
    if (meta[s].active && meta[s].due == 1) meta[s].due = kDueMovePending;
  return hipSuccess;
}

hipError_t launch_clear_pending(SeqMeta* meta, int slot_lo, int slot_hi, hipStream_t) {
  if (slot_lo < 0 || slot_hi > g_max_seqs) fail("clear range", slot_lo, slot_hi);
  for (int s = slot_lo; s < slot_hi; ++s)
    if (meta[s].due == kDueMovePending) meta[s].due = 0;
  return hipSuccess;
}

hipError_t launch_flush_pending(const Shape& sh, SeqMeta* meta, void*, void*, const int32_t* drops,
                                int drop_stride, int slot_lo, int slot_hi, hipStream_t) {
  if (slot_lo < 0 || slot_hi > g_max_seqs || !drops || drop_stride < 1)
    fail("flush", slot_lo, drop_stride);
  check_chunk(sh, slot_lo, slot_hi, "flush launch over the per-launch bound");
  return launch_clear_pending(meta, slot_lo, slot_hi, nullptr);   // as the device's does
}

hipError_t launch_write_rows(const Shape& sh, const SeqMeta& M, int slot, int len,
                             const void* k_src, const void* v_src, const int32_t* pos_src,
                             void*, void*, int32_t*, hipStream_t) {
  check_rows(sh, M, slot, len);
  const size_t n = static_cast<size_t>(sh.L) * sh.Hkv * len;
  touch_read(k_src, n * kHeadDim * elem_bytes(sh));
  touch_read(v_src, n * kHeadDim * elem_bytes(sh));
  touch_read(pos_src, n * sizeof(int32_t));
  return hipSuccess;
}

hipError_t launch_read_rows(const Shape& sh, const SeqMeta& M, int slot, int lg, int len,
                            const void*, const void*, void* k_out, void* v_out, hipStream_t) {
  check_rows(sh, M, slot, len);
  if (lg < 0 || lg >= sh.L * sh.Hkv) fail("read_rows head", lg, sh.L * sh.Hkv);
  touch_write(k_out, static_cast<size_t>(len) * kHeadDim * elem_bytes(sh));
  touch_write(v_out, static_cast<size_t>(len) * kHeadDim * elem_bytes(sh));
  return hipSuccess;
}

hipError_t launch_export_positions(const Shape& sh, const SeqMeta& M, int slot, int len,
                                   const int32_t*, int32_t* out, hipStream_t) {
  check_rows(sh, M, slot, len);
  touch_write(out, static_cast<size_t>(sh.L) * sh.Hkv * len * sizeof(int32_t));
  return hipSuccess;
}

hipError_t launch_table_set(const Shape& sh, const TableEntry* entries, int n, hipStream_t) {
  if (!sh.pg.tables) fail("tables", 0, 0);
  g_tables = sh.pg.tables;
  g_pps = sh.pg.pages_per_seq;
  int32_t* t = const_cast<int32_t*>(sh.pg.tables);
  for (int i = 0; i < n; ++i) {
    const TableEntry& e = entries[i];
    if (e.slot < 0 || e.slot >= g_max_seqs) fail("table slot", e.slot, g_max_seqs);
    if (e.index < 0 || e.index >= g_pps) fail("table index", e.index, g_pps);
    if (e.group < 0 || e.group >= g_n_groups) fail("table group", e.group, g_n_groups);
    t[static_cast<int64_t>(e.slot) * g_pps + e.index] = e.group;
  }
  return hipSuccess;
}

hipError_t launch_attention(const Shape& sh, const AttnLaunch& a, hipStream_t) {
  if (a.layer < 0 || a.layer >= sh.L) fail("attention layer", a.layer, sh.L);
  // the launched slots: [0, slot_hi) of the active range
  if (a.max_seqs < 1 || a.max_seqs > g_max_seqs) fail("attention slots", a.max_seqs, g_max_seqs);
  if (a.max_splits < 1 || a.max_splits > a.split_stride || a.max_splits > kMaxSplits)
    fail("attention splits", a.max_splits, a.split_stride);
  if (a.split_keys < 32 || a.split_keys % 32) fail("attention split keys", a.split_keys, 0);
  if (a.move && (!a.drops || a.drop_stride < 1 || a.max_splits != 1 || sh.dtype != 1 ||
                 sh.layout != 0))
    fail("attention move", a.max_splits, a.drop_stride);
  const size_t e = elem_bytes(sh);
  touch_read(a.q, static_cast<size_t>(a.max_seqs) * sh.Hq * kHeadDim * e);
  touch_read(a.k_new, static_cast<size_t>(a.max_seqs) * sh.Hkv * kHeadDim * e);
  touch_read(a.v_new, static_cast<size_t>(a.max_seqs) * sh.Hkv * kHeadDim * e);
  touch_write(a.out, static_cast<size_t>(a.max_seqs) * sh.Hq * kHeadDim * e);
  if (a.max_splits > 1) {
    const size_t heads = static_cast<size_t>(a.max_seqs) * sh.Hkv * a.split_stride;
    touch_write(a.ws_o, heads * sh.G * kHeadDim * sizeof(float));
    touch_write(a.ws_ml, heads * sh.G * 2 * sizeof(float));
  }
  return hipSuccess;
}

hipError_t scratch_address(void** out) {
  *out = scratch_array().data();
  return hipSuccess;
}

hipError_t launch_compact_drops(const Shape& sh, const SeqMeta*, void*, void*, int32_t*,
                                const int32_t*, int, int slot_lo, int slot_hi, hipStream_t) {
  check_chunk(sh, slot_lo, slot_hi, "compaction launch over the per-launch bound");
  return hipSuccess;
}

hipError_t launch_plan_range(SeqMeta*, int, int, int, hipStream_t) { return hipSuccess; }

hipError_t launch_scored_select(const Shape&, int, const SeqMeta*, const void*, const void*,
                                const int32_t*, const float*, float*, int, int32_t*, int, int,
                                int, float, float, int, int, uint64_t, hipStream_t) {
  return hipSuccess;
}

hipError_t launch_window_score(const Shape&, const SeqMeta*, const void*, const int32_t*,
                               const void*, float*, int32_t*, int, int, int, int, hipStream_t) {
  return hipSuccess;
}

}  // namespace ra
