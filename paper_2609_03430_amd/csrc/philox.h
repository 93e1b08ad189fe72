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
    const uint64_t hi0 = __umul64hi(kM0, c0), lo0 = kM0 * c0;
    const uint64_t hi1 = __umul64hi(kM1, c2), lo1 = kM1 * c2;
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

}  // namespace ra
