// Philox4x64-10 on the device, from its published definition (Salmon,
// Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3",
// SC'11): a keyed bijection on four 64-bit words; each of the 10 rounds
// multiplies words 0 and 2 by fixed odd constants, swaps the 128-bit
// product halves into the other words mixed with the key, and the key is
// advanced by Weyl constants between rounds.
//
// It supplies Random Attention's i.i.d. uniform score of every candidate,
// drawn per KV head at every eviction (Section 3) and reproducible from the
// per-request seed (Appendix H, "Statistics and randomness"): the score of
// position p at event e of (layer l, KV head g) is word p mod 4 of the block
// at counter (p / 4, e, l, g) with key (seed, request id).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ra {

// Full 128-bit product of two 64-bit words from four 32 x 32 -> 64-bit
// multiply-adds (schoolbook, 32-bit limbs; no partial sum exceeds 64 bits:
// each is at most (2^32 - 1)^2 + 2 (2^32 - 1) = 2^64 - 1).
__device__ __forceinline__ void mul_64x64(uint64_t a, uint64_t b, uint64_t& hi,
                                          uint64_t& lo) {
  const uint64_t a0 = static_cast<uint32_t>(a), a1 = a >> 32;
  const uint64_t b0 = static_cast<uint32_t>(b), b1 = b >> 32;
  const uint64_t t = a0 * b0;
  const uint64_t u = a1 * b0 + (t >> 32);
  const uint64_t v = a0 * b1 + (u & 0xffffffffull);
  hi = a1 * b1 + (u >> 32) + (v >> 32);
  lo = (v << 32) | (t & 0xffffffffull);
}

__device__ __forceinline__ uint64_t philox_score(uint64_t p, uint64_t e,
                                                 uint64_t l, uint64_t g,
                                                 uint64_t seed, uint64_t rid) {
  constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull;
  constexpr uint64_t kM1 = 0xCA5A826395121157ull;
  constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull;
  constexpr uint64_t kW1 = 0xBB67AE8584CAA73Bull;
  uint64_t c0 = p >> 2, c1 = e, c2 = l, c3 = g;
  uint64_t k0 = seed, k1 = rid;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += kW0;
      k1 += kW1;
    }
    uint64_t hi0, lo0, hi1, lo1;
    mul_64x64(kM0, c0, hi0, lo0);
    mul_64x64(kM1, c2, hi1, lo1);
    const uint64_t n0 = hi1 ^ c1 ^ k0;
    const uint64_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  const uint32_t w = static_cast<uint32_t>(p & 3);
  return w == 0 ? c0 : (w == 1 ? c1 : (w == 2 ? c2 : c3));
}

// N blocks at counters (b[j], e, l, g), key (seed, rid), evaluated in
// lockstep so that their independent rounds interleave; w[j][i] is word i of
// block j (the scores of positions 4 b[j] .. 4 b[j] + 3).
template <int N>
__device__ __forceinline__ void philox_blocks(const uint64_t (&b)[N], uint64_t e, uint64_t l,
                                              uint64_t g, uint64_t seed, uint64_t rid,
                                              uint64_t (&w)[N][4]) {
  constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull;
  constexpr uint64_t kM1 = 0xCA5A826395121157ull;
  constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull;
  constexpr uint64_t kW1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int j = 0; j < N; ++j) {
    w[j][0] = b[j];
    w[j][1] = e;
    w[j][2] = l;
    w[j][3] = g;
  }
  uint64_t k0 = seed, k1 = rid;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += kW0;
      k1 += kW1;
    }
#pragma unroll
    for (int j = 0; j < N; ++j) {
      uint64_t hi0, lo0, hi1, lo1;
      mul_64x64(kM0, w[j][0], hi0, lo0);
      mul_64x64(kM1, w[j][2], hi1, lo1);
      const uint64_t n0 = hi1 ^ w[j][1] ^ k0;
      const uint64_t n2 = hi0 ^ w[j][3] ^ k1;
      w[j][0] = n0;
      w[j][1] = lo1;
      w[j][2] = n2;
      w[j][3] = lo0;
    }
  }
}

}  // namespace ra
