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

// Positions lp+step .. lp+step+run-1 into rows len .. len+run-1 of every
// region of every active slot (rows themselves are not touched).
__global__ void append_positions_kernel(const SeqMeta* meta, int32_t* pos,
                                        int lo, int run) {
  const SeqMeta& M = meta[lo + blockIdx.x];
  if (!M.active) return;
  const int64_t region = M.base + static_cast<int64_t>(blockIdx.y) * M.cap;
  for (int i = threadIdx.x; i < run; i += blockDim.x)
    pos[region + M.len + i] = M.prompt_len + M.step + i;
}

// Row-major source rows [L*Hkv][len][128] into the cache layout of rows
// [0, len) of each region; rows of a partly filled last value tile are
// zeroed.  Grid: (ceil(len/64), L*Hkv).
template <typename E>
__global__ void write_rows_kernel(int64_t base, int cap, int len,
                                  const E* __restrict__ k_src,
                                  const E* __restrict__ v_src,
                                  const int32_t* __restrict__ pos_src,
                                  E* __restrict__ kpool, E* __restrict__ vpool,
                                  int32_t* __restrict__ pos) {
  constexpr int kEpu = 16 / sizeof(E);
  const int lg = blockIdx.y;
  const int j0 = blockIdx.x * 64;
  const int64_t region = base + static_cast<int64_t>(lg) * cap;
  const int64_t src0 = static_cast<int64_t>(lg) * len;
  if (pos) {
    for (int i = threadIdx.x; i < 64; i += blockDim.x) {
      const int j = j0 + i;
      if (j < len) pos[region + j] = pos_src ? pos_src[src0 + j] : j;
    }
  }
  if (!k_src) return;
  constexpr int kUnitsRow = kHeadDim / kEpu;
  for (int u = threadIdx.x; u < 64 * kUnitsRow; u += blockDim.x) {
    const int j = j0 + u / kUnitsRow, col = u % kUnitsRow;
    if (j < len)
      *reinterpret_cast<u32x4*>(kpool + (region + j) * kHeadDim + col * kEpu) =
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
    *reinterpret_cast<u32x4*>(vpool + (region + jt) * kHeadDim + ch * 8 + part * kEpu) = w;
  }
}

// Rows [0, len) of one region to row-major outputs.  Grid: ceil(len/64).
template <typename E>
__global__ void read_rows_kernel(int64_t region, int len,
                                 const E* __restrict__ kpool,
                                 const E* __restrict__ vpool,
                                 E* __restrict__ k_out, E* __restrict__ v_out) {
  const int j0 = blockIdx.x * 64;
  for (int u = threadIdx.x; u < 64 * kHeadDim; u += blockDim.x) {
    const int j = j0 + u / kHeadDim, ch = u % kHeadDim;
    if (j >= len) continue;
    const int64_t row = region + j;
    if (k_out) k_out[static_cast<int64_t>(j) * kHeadDim + ch] = kpool[row * kHeadDim + ch];
    if (v_out)
      v_out[static_cast<int64_t>(j) * kHeadDim + ch] =
          vpool[(row & ~int64_t(7)) * kHeadDim + ch * 8 + (row & 7)];
  }
}

__global__ void export_positions_kernel(int64_t base, int cap, int len,
                                        const int32_t* __restrict__ pos,
                                        int32_t* __restrict__ out) {
  const int lg = blockIdx.y;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < len)
    out[static_cast<int64_t>(lg) * len + j] = pos[base + static_cast<int64_t>(lg) * cap + j];
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

hipError_t launch_append_positions(const SeqMeta* meta, int32_t* pos, int slot_lo,
                                   int slot_hi, int L, int Hkv, int run,
                                   hipStream_t s) {
  if (slot_hi <= slot_lo || run <= 0) return hipSuccess;
  hipLaunchKernelGGL(append_positions_kernel, dim3(slot_hi - slot_lo, L * Hkv),
                     dim3(256), 0, s, meta, pos, slot_lo, run);
  return hipGetLastError();
}

hipError_t launch_write_rows(const Shape& sh, int64_t base, int cap, int len,
                             const void* k_src, const void* v_src,
                             const int32_t* pos_src, void* kpool, void* vpool,
                             int32_t* pos, hipStream_t s) {
  if (len <= 0) return hipSuccess;
  const dim3 grid((len + 63) / 64, sh.L * sh.Hkv);
  if (sh.dtype == 1) {
    hipLaunchKernelGGL(write_rows_kernel<uint16_t>, grid, dim3(256), 0, s, base,
                       cap, len, static_cast<const uint16_t*>(k_src),
                       static_cast<const uint16_t*>(v_src), pos_src,
                       static_cast<uint16_t*>(kpool), static_cast<uint16_t*>(vpool), pos);
  } else {
    hipLaunchKernelGGL(write_rows_kernel<float>, grid, dim3(256), 0, s, base, cap,
                       len, static_cast<const float*>(k_src),
                       static_cast<const float*>(v_src), pos_src,
                       static_cast<float*>(kpool), static_cast<float*>(vpool), pos);
  }
  return hipGetLastError();
}

hipError_t launch_read_rows(const Shape& sh, int64_t region_row, int len,
                            const void* kpool, const void* vpool, void* k_out,
                            void* v_out, hipStream_t s) {
  if (len <= 0) return hipSuccess;
  const dim3 grid((len + 63) / 64);
  if (sh.dtype == 1) {
    hipLaunchKernelGGL(read_rows_kernel<uint16_t>, grid, dim3(256), 0, s,
                       region_row, len, static_cast<const uint16_t*>(kpool),
                       static_cast<const uint16_t*>(vpool),
                       static_cast<uint16_t*>(k_out), static_cast<uint16_t*>(v_out));
  } else {
    hipLaunchKernelGGL(read_rows_kernel<float>, grid, dim3(256), 0, s, region_row,
                       len, static_cast<const float*>(kpool),
                       static_cast<const float*>(vpool), static_cast<float*>(k_out),
                       static_cast<float*>(v_out));
  }
  return hipGetLastError();
}

hipError_t launch_export_positions(const Shape& sh, int64_t base, int cap,
                                   int len, const int32_t* pos, int32_t* out,
                                   hipStream_t s) {
  if (len <= 0) return hipSuccess;
  hipLaunchKernelGGL(export_positions_kernel, dim3((len + 255) / 256, sh.L * sh.Hkv),
                     dim3(256), 0, s, base, cap, len, pos, out);
  return hipGetLastError();
}

}  // namespace ra
