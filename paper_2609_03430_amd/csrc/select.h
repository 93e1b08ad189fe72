// Block-wide selection of the m smallest candidates, shared by the eviction
// kernel (64-bit random scores) and the observation-window scorer (32-bit
// score bits).  Each thread holds KPT candidates in registers; the order is
// the composite (key, tie) with a distinct 32-bit tie per candidate (the
// token position, or the row), so the result is unique even with equal keys.
// MSB-first radix select, 8 bits per pass, 256-bin LDS histogram; a pass
// ends the selection as soon as the whole bucket holding the m-th smallest is
// dropped (usually after two passes for uniform keys).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ra {

struct SelectShared {
  int hist[256];
  int sel[3];
  int wave_tot[16];
};

__device__ __forceinline__ int wave_inclusive_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

template <int KEY_BITS>
__device__ __forceinline__ int select_digit(int level, uint64_t key, uint32_t tie) {
  constexpr int kKeyLevels = KEY_BITS / 8;
  if (level < kKeyLevels)
    return static_cast<int>((key >> (KEY_BITS - 8 - 8 * level)) & 0xFF);
  return static_cast<int>((tie >> (24 - 8 * (level - kKeyLevels))) & 0xFF);
}

// Returns this thread's drop mask (bit i: its candidate i is among the m
// smallest (key, tie)).  `valid` marks the thread's real candidates.  All
// threads of the block must call it.
template <int NT, int KPT, int KEY_BITS>
__device__ __forceinline__ uint32_t select_smallest(const uint64_t (&key)[KPT],
                                                   const uint32_t (&tie)[KPT],
                                                   uint32_t valid, int m,
                                                   SelectShared& sh) {
  static_assert(KPT <= 32, "one 32-bit mask per thread");
  const int t = threadIdx.x;
  uint32_t undecided = valid, drop = 0;
  int remaining = m;
  if (m <= 0) return 0;
  for (int level = 0; level < KEY_BITS / 8 + 4; ++level) {
    for (int i = t; i < 256; i += NT) sh.hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < KPT; ++i)
      if ((undecided >> i) & 1)
        atomicAdd(&sh.hist[select_digit<KEY_BITS>(level, key[i], tie[i])], 1);
    __syncthreads();
    if (t < 64) {
      const int h0 = sh.hist[4 * t], h1 = sh.hist[4 * t + 1];
      const int h2 = sh.hist[4 * t + 2], h3 = sh.hist[4 * t + 3];
      const int s = h0 + h1 + h2 + h3;
      int cum = wave_inclusive_scan(s) - s;
      const int hs[4] = {h0, h1, h2, h3};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (cum < remaining && remaining <= cum + hs[j]) {
          sh.sel[0] = 4 * t + j;
          sh.sel[1] = cum;
          sh.sel[2] = hs[j];
        }
        cum += hs[j];
      }
    }
    __syncthreads();
    const int v = sh.sel[0], below = sh.sel[1], cnt = sh.sel[2];
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      if ((undecided >> i) & 1) {
        const int dg = select_digit<KEY_BITS>(level, key[i], tie[i]);
        if (dg < v) {
          drop |= 1u << i;
          undecided &= ~(1u << i);
        } else if (dg > v) {
          undecided &= ~(1u << i);
        }
      }
    }
    remaining -= below;
    if (cnt == remaining) {       // the whole bucket goes: selection complete
      drop |= undecided;
      break;
    }
    __syncthreads();
  }
  return drop;
}

// Writes the dropped candidates' slots, ascending, as f[k] = slot_k - k
// (slot = slot0 + candidate index).  Ends with a barrier.  Returns the
// number of dropped candidates held by lower threads.
template <int NT, int KPT>
__device__ __forceinline__ int drop_list(uint32_t drop, int slot0, int* f, SelectShared& sh) {
  const int t = threadIdx.x;
  const int mine = __popc(drop);
  const int incl = wave_inclusive_scan(mine);
  if ((t & 63) == 63) sh.wave_tot[t >> 6] = incl;
  __syncthreads();
  int k = incl - mine;
  for (int w = 0; w < (t >> 6); ++w) k += sh.wave_tot[w];
  const int before = k;
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    if ((drop >> i) & 1) {
      f[k] = slot0 + t * KPT + i - k;
      ++k;
    }
  }
  __syncthreads();
  return before;
}

}  // namespace ra
