// Device-side sequence state and row transfer kernels.
//
// The per-slot metadata lives in device memory so that a decode step's
// kernels need no host round trip: the end-of-step kernel advances the step
// counter and applies the periodic trigger (Appendix F: every evict_every
// steps, once the evictable rows exceed the budget) by writing an eviction
// plan that the eviction kernel consumes.  The host library replays the
// same integer rules on its mirror to decide which launches to issue.
#include "ra_internal.h"

namespace ra {
namespace {

using u32x4 = uint32_t __attribute__((ext_vector_type(4)));

__global__ void zero_words_kernel(uint32_t* p, int64_t n) {
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * blockDim.x)
    p[i] = 0u;
}

__global__ void seq_set_kernel(SeqMeta* meta, int slot, SeqMeta v) {
  if (threadIdx.x == 0) meta[slot] = v;
}

// Applies the trigger rule to a sequence that has just completed `n_steps`
// more steps (n_steps never crosses a multiple of `every` before its end).
__device__ __forceinline__ void plan(SeqMeta& M, int r, bool at_trigger) {
  M.due = 0;
  if (at_trigger && M.len - M.prompt_len - r > M.k_keep) {
    M.due = 1;
    M.plan_len = M.len;
    M.plan_event = M.event;
    M.len = M.prompt_len + M.k_keep + r;
    M.event += 1;
  }
}

__global__ void advance_kernel(SeqMeta* meta, int lo, int hi, int n_steps,
                               int r, int every) {
  const int s = lo + blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= hi) return;
  SeqMeta M = meta[s];
  if (!M.active) return;
  M.step += n_steps;
  M.len += n_steps;
  plan(M, r, every > 0 && M.step % every == 0);   // every = 0: never triggers
  meta[s] = M;
}

// The plan rule applied now to every active slot of [lo, hi).
__global__ void plan_range_kernel(SeqMeta* meta, int lo, int hi, int r) {
  const int s = lo + blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= hi) return;
  SeqMeta M = meta[s];
  if (!M.active) return;
  plan(M, r, true);
  meta[s] = M;
}

__global__ void plan_now_kernel(SeqMeta* meta, int slot, int r) {
  if (threadIdx.x != 0) return;
  SeqMeta M = meta[slot];
  if (!M.active) return;
  plan(M, r, true);
  meta[slot] = M;
}

__global__ void mark_pending_kernel(SeqMeta* meta, int lo, int hi) {
  const int s = lo + blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= hi) return;
  if (meta[s].active && meta[s].due == 1) meta[s].due = kDueMovePending;
}

__global__ void clear_pending_kernel(SeqMeta* meta, int lo, int hi) {
  const int s = lo + blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= hi) return;
  if (meta[s].due == kDueMovePending) meta[s].due = 0;
}

// Positions lp+step .. lp+step+run-1 into rows len .. len+run-1 of every
// head of every active slot (rows themselves are not touched).
// Grid: (slots, L * Hkv).
template <bool PAGED>
__global__ void append_positions_kernel(const SeqMeta* meta, int32_t* pos, int lo,
                                        int run, Paging pg) {
  const int slot = lo + blockIdx.x;
  const SeqMeta& M = meta[slot];
  if (!M.active) return;
  const RowMap rm = row_map(M, slot, blockIdx.y, pg);
  for (int i = threadIdx.x; i < run; i += blockDim.x)
    pos[pool_row<PAGED>(rm, M.len + i)] = M.prompt_len + M.step + i;
}

// Row-major source rows [L*Hkv][len][128] into the cache layout of rows
// [0, len) of each head; rows of a partly filled last value tile are
// zeroed.  Grid: (ceil(len/64), L*Hkv).  A 64-row chunk may straddle two
// pages of 32 rows, so rows are mapped one by one (value tiles of 8 rows
// never straddle a page).
template <typename E, bool PAGED>
__global__ void write_rows_kernel(SeqMeta M, int slot, int len, Paging pg,
                                  const E* __restrict__ k_src,
                                  const E* __restrict__ v_src,
                                  const int32_t* __restrict__ pos_src,
                                  E* __restrict__ kpool, E* __restrict__ vpool,
                                  int32_t* __restrict__ pos) {
  constexpr int kEpu = 16 / sizeof(E);
  const int lg = blockIdx.y;
  const int j0 = blockIdx.x * 64;
  const RowMap rm = row_map(M, slot, lg, pg);
  const int64_t src0 = static_cast<int64_t>(lg) * len;
  if (pos) {
    for (int i = threadIdx.x; i < 64; i += blockDim.x) {
      const int j = j0 + i;
      if (j < len) pos[pool_row<PAGED>(rm, j)] = pos_src ? pos_src[src0 + j] : j;
    }
  }
  if (!k_src) return;
  constexpr int kUnitsRow = kHeadDim / kEpu;
  for (int u = threadIdx.x; u < 64 * kUnitsRow; u += blockDim.x) {
    const int j = j0 + u / kUnitsRow, col = u % kUnitsRow;
    if (j < len)
      *reinterpret_cast<u32x4*>(kpool + pool_row<PAGED>(rm, j) * kHeadDim + col * kEpu) =
          *reinterpret_cast<const u32x4*>(k_src + (src0 + j) * kHeadDim + col * kEpu);
  }
  // values: each output 16-byte unit holds kEpu consecutive rows of one channel
  constexpr int kUnitsCh = 8 / kEpu;
  for (int u = threadIdx.x; u < 8 * kHeadDim * kUnitsCh; u += blockDim.x) {
    const int tile = u / (kHeadDim * kUnitsCh);
    const int rem = u % (kHeadDim * kUnitsCh);
    const int ch = rem / kUnitsCh, part = rem % kUnitsCh;
    const int jt = j0 + tile * 8;
    if (jt >= len) continue;
    E e[kEpu];
#pragma unroll
    for (int x = 0; x < kEpu; ++x) {
      const int j = jt + part * kEpu + x;
      e[x] = j < len ? v_src[(src0 + j) * kHeadDim + ch] : E(0);
    }
    u32x4 w;
    __builtin_memcpy(&w, e, 16);
    *reinterpret_cast<u32x4*>(vpool + pool_row<PAGED>(rm, jt) * kHeadDim + ch * 8 +
                              part * kEpu) = w;
  }
}

// Rows [0, len) of one head to row-major outputs.  Grid: ceil(len/64).
template <typename E, bool PAGED>
__global__ void read_rows_kernel(SeqMeta M, int slot, int lg, int len, Paging pg,
                                 const E* __restrict__ kpool,
                                 const E* __restrict__ vpool,
                                 E* __restrict__ k_out, E* __restrict__ v_out) {
  const RowMap rm = row_map(M, slot, lg, pg);
  const int j0 = blockIdx.x * 64;
  for (int u = threadIdx.x; u < 64 * kHeadDim; u += blockDim.x) {
    const int j = j0 + u / kHeadDim, ch = u % kHeadDim;
    if (j >= len) continue;
    const int64_t row = pool_row<PAGED>(rm, j);
    if (k_out) k_out[static_cast<int64_t>(j) * kHeadDim + ch] = kpool[row * kHeadDim + ch];
    if (v_out)
      v_out[static_cast<int64_t>(j) * kHeadDim + ch] =
          vpool[(row & ~int64_t(7)) * kHeadDim + ch * 8 + (row & 7)];
  }
}

template <bool PAGED>
__global__ void export_positions_kernel(SeqMeta M, int slot, int len, Paging pg,
                                        const int32_t* __restrict__ pos,
                                        int32_t* __restrict__ out) {
  const int lg = blockIdx.y;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const RowMap rm = row_map(M, slot, lg, pg);
  if (j < len) out[static_cast<int64_t>(lg) * len + j] = pos[pool_row<PAGED>(rm, j)];
}

struct TableBatch {
  TableEntry e[kTableBatch];
};

// Block-table entries chosen by the host's page allocator.
__global__ void table_set_kernel(int32_t* tables, int pages_per_seq, TableBatch b, int n) {
  const int i = threadIdx.x;
  if (i < n)
    tables[static_cast<int64_t>(b.e[i].slot) * pages_per_seq + b.e[i].index] = b.e[i].group;
}

}  // namespace

hipError_t launch_zero_words(uint32_t* p, int64_t n_words, hipStream_t s) {
  if (n_words <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n_words + 255) / 256, 4096);
  hipLaunchKernelGGL(zero_words_kernel, dim3(blocks), dim3(256), 0, s, p, n_words);
  return hipGetLastError();
}

hipError_t launch_seq_set(SeqMeta* meta, int slot, const SeqMeta& v, hipStream_t s) {
  hipLaunchKernelGGL(seq_set_kernel, dim3(1), dim3(64), 0, s, meta, slot, v);
  return hipGetLastError();
}

hipError_t launch_advance(SeqMeta* meta, int slot_lo, int slot_hi, int n_steps,
                          int r, int every, hipStream_t s) {
  const int n = slot_hi - slot_lo;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(advance_kernel, dim3((n + 255) / 256), dim3(256), 0, s,
                     meta, slot_lo, slot_hi, n_steps, r, every);
  return hipGetLastError();
}

hipError_t launch_plan_now(SeqMeta* meta, int slot, int r, hipStream_t s) {
  hipLaunchKernelGGL(plan_now_kernel, dim3(1), dim3(64), 0, s, meta, slot, r);
  return hipGetLastError();
}

hipError_t launch_plan_range(SeqMeta* meta, int slot_lo, int slot_hi, int r, hipStream_t s) {
  if (slot_hi <= slot_lo) return hipSuccess;
  const int n = slot_hi - slot_lo;
  hipLaunchKernelGGL(plan_range_kernel, dim3((n + 255) / 256), dim3(256), 0, s, meta,
                     slot_lo, slot_hi, r);
  return hipGetLastError();
}

hipError_t launch_append_positions(const Shape& sh, const SeqMeta* meta, int32_t* pos,
                                   int slot_lo, int slot_hi, int run, hipStream_t s) {
  if (slot_hi <= slot_lo || run <= 0) return hipSuccess;
  const dim3 grid(slot_hi - slot_lo, sh.L * sh.Hkv);
  if (sh.pg.tables)
    hipLaunchKernelGGL(append_positions_kernel<true>, grid, dim3(256), 0, s, meta, pos,
                       slot_lo, run, sh.pg);
  else
    hipLaunchKernelGGL(append_positions_kernel<false>, grid, dim3(256), 0, s, meta, pos,
                       slot_lo, run, sh.pg);
  return hipGetLastError();
}

template <typename E>
void write_rows_t(const Shape& sh, const SeqMeta& M, int slot, int len, const void* k_src,
                  const void* v_src, const int32_t* pos_src, void* kpool, void* vpool,
                  int32_t* pos, hipStream_t s) {
  const dim3 grid((len + 63) / 64, sh.L * sh.Hkv);
  const E* k = static_cast<const E*>(k_src);
  const E* v = static_cast<const E*>(v_src);
  if (sh.pg.tables)
    hipLaunchKernelGGL((write_rows_kernel<E, true>), grid, dim3(256), 0, s, M, slot, len,
                       sh.pg, k, v, pos_src, static_cast<E*>(kpool), static_cast<E*>(vpool),
                       pos);
  else
    hipLaunchKernelGGL((write_rows_kernel<E, false>), grid, dim3(256), 0, s, M, slot, len,
                       sh.pg, k, v, pos_src, static_cast<E*>(kpool), static_cast<E*>(vpool),
                       pos);
}

hipError_t launch_write_rows(const Shape& sh, const SeqMeta& M, int slot, int len,
                             const void* k_src, const void* v_src,
                             const int32_t* pos_src, void* kpool, void* vpool,
                             int32_t* pos, hipStream_t s) {
  if (len <= 0) return hipSuccess;
  if (sh.dtype == 1)
    write_rows_t<uint16_t>(sh, M, slot, len, k_src, v_src, pos_src, kpool, vpool, pos, s);
  else
    write_rows_t<float>(sh, M, slot, len, k_src, v_src, pos_src, kpool, vpool, pos, s);
  return hipGetLastError();
}

template <typename E>
void read_rows_t(const Shape& sh, const SeqMeta& M, int slot, int lg, int len,
                 const void* kpool, const void* vpool, void* k_out, void* v_out,
                 hipStream_t s) {
  const dim3 grid((len + 63) / 64);
  const E* k = static_cast<const E*>(kpool);
  const E* v = static_cast<const E*>(vpool);
  if (sh.pg.tables)
    hipLaunchKernelGGL((read_rows_kernel<E, true>), grid, dim3(256), 0, s, M, slot, lg, len,
                       sh.pg, k, v, static_cast<E*>(k_out), static_cast<E*>(v_out));
  else
    hipLaunchKernelGGL((read_rows_kernel<E, false>), grid, dim3(256), 0, s, M, slot, lg, len,
                       sh.pg, k, v, static_cast<E*>(k_out), static_cast<E*>(v_out));
}

hipError_t launch_read_rows(const Shape& sh, const SeqMeta& M, int slot, int lg, int len,
                            const void* kpool, const void* vpool, void* k_out,
                            void* v_out, hipStream_t s) {
  if (len <= 0) return hipSuccess;
  if (sh.dtype == 1)
    read_rows_t<uint16_t>(sh, M, slot, lg, len, kpool, vpool, k_out, v_out, s);
  else
    read_rows_t<float>(sh, M, slot, lg, len, kpool, vpool, k_out, v_out, s);
  return hipGetLastError();
}

hipError_t launch_export_positions(const Shape& sh, const SeqMeta& M, int slot, int len,
                                   const int32_t* pos, int32_t* out, hipStream_t s) {
  if (len <= 0) return hipSuccess;
  const dim3 grid((len + 255) / 256, sh.L * sh.Hkv);
  if (sh.pg.tables)
    hipLaunchKernelGGL(export_positions_kernel<true>, grid, dim3(256), 0, s, M, slot, len,
                       sh.pg, pos, out);
  else
    hipLaunchKernelGGL(export_positions_kernel<false>, grid, dim3(256), 0, s, M, slot, len,
                       sh.pg, pos, out);
  return hipGetLastError();
}

hipError_t launch_mark_pending(SeqMeta* meta, int slot_lo, int slot_hi, hipStream_t s) {
  if (slot_hi <= slot_lo) return hipSuccess;
  const int n = slot_hi - slot_lo;
  hipLaunchKernelGGL(mark_pending_kernel, dim3((n + 255) / 256), dim3(256), 0, s, meta,
                     slot_lo, slot_hi);
  return hipGetLastError();
}

hipError_t launch_clear_pending(SeqMeta* meta, int slot_lo, int slot_hi, hipStream_t s) {
  if (slot_hi <= slot_lo) return hipSuccess;
  const int n = slot_hi - slot_lo;
  hipLaunchKernelGGL(clear_pending_kernel, dim3((n + 255) / 256), dim3(256), 0, s, meta,
                     slot_lo, slot_hi);
  return hipGetLastError();
}

hipError_t launch_table_set(const Shape& sh, const TableEntry* entries, int n,
                            hipStream_t s) {
  for (int i0 = 0; i0 < n; i0 += kTableBatch) {
    TableBatch b{};
    const int k = std::min(kTableBatch, n - i0);
    for (int i = 0; i < k; ++i) b.e[i] = entries[i0 + i];
    hipLaunchKernelGGL(table_set_kernel, dim3(1), dim3(kTableBatch), 0, s,
                       const_cast<int32_t*>(sh.pg.tables), sh.pg.pages_per_seq, b, k);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace ra
