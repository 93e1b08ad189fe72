// Observation-window scorer: the scoring pass of a score-based evictor,
// built only to measure what Random Attention saves (not used by the method).
//
// Section 2 ("Baselines as choices of s") defines SnapKV's score of a cached
// position as the sum of the attention weights of the last w queries,
// max-pooled over neighbouring positions; Eq. 1 keeps the top-scoring
// candidates (cached rows outside the r most recent).  Per (sequence, layer,
// KV head), one 512-thread workgroup:
//   pass 1: for every window query (G heads x 64 steps) the log-sum-exp of
//           q.k/sqrt(d) over the cached rows at or before its position;
//   pass 2: the same logits again, weights 2^(s - lse) summed over queries
//           into a per-row score held in LDS;
//   then max-pool over 7 rows, and the m lowest candidates (the same m as
//   Random Attention drops at this event) by the shared radix select.
// Keys stream through LDS in 64-row blocks (prefetched into registers while
// the previous block is used); both logit passes run on
// v_mfma_f32_16x16x32_bf16 with 16 queries x 16 keys per tile.
#include <type_traits>

#include "ra_internal.h"
#include "select.h"

namespace ra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kNT = 512;
constexpr int kWin = 64;          // window queries per query head
constexpr int kBlk = 64;          // key rows per LDS block
constexpr int kRowStride = 136;   // bf16 elements per LDS row (256 B + 16 B pad)
constexpr int kPoolHalf = 3;      // max-pool over 7 rows
constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  bf16x8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

struct KBlock {
  u32x4 u[2];   // this thread's two 16-byte pieces of a 64-row block
  int p;        // position of row t (threads < 64)
};

__device__ __forceinline__ void fetch_block(KBlock& b, const uint16_t* Kr,
                                            const int32_t* P, int kb, int len) {
  const int t = threadIdx.x;
  const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int piece = t + q * kNT;          // 1024 pieces of 16 bytes
    const int row = piece >> 4, col = piece & 15;
    b.u[q] = (kb + row < len)
        ? *reinterpret_cast<const u32x4*>(Kr + static_cast<int64_t>(kb + row) * kHeadDim + col * 8)
        : z;
  }
  b.p = (t < kBlk && kb + t < len) ? P[kb + t] : 0x7fffffff;
}

__device__ __forceinline__ void store_block(const KBlock& b, uint16_t* lk, int* lpos) {
  const int t = threadIdx.x;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int piece = t + q * kNT;
    const int row = piece >> 4, col = piece & 15;
    *reinterpret_cast<u32x4*>(lk + row * kRowStride + col * 8) = b.u[q];
  }
  if (t < kBlk) lpos[t] = b.p;
}

// Waves of the workgroup; query tile j of wave w is tile j * kWaves + w
// (round robin, so the tiles of G heads spread evenly over the four SIMDs).
constexpr int kWaves = kNT / 64;

// Stream the head's cached rows through LDS in 64-row blocks (the next
// block prefetched into registers while the current one is used) and call
// body(b, keys, positions) once per block, with the whole workgroup.
template <typename Body>
__device__ __forceinline__ void stream_blocks(const uint16_t* Kr, const int32_t* P, int len,
                                              uint16_t (&lk)[2][kBlk * kRowStride],
                                              int (&lpos)[2][kBlk], Body body) {
  const int nblk = (len + kBlk - 1) / kBlk;
  KBlock nb;
  fetch_block(nb, Kr, P, 0, len);
  __syncthreads();                 // the previous user of lk is done with it
  store_block(nb, lk[0], lpos[0]);
  __syncthreads();
  for (int b = 0; b < nblk; ++b) {
    const int cur = b & 1;
    if (b + 1 < nblk) fetch_block(nb, Kr, P, (b + 1) * kBlk, len);
    body(b, lk[cur], lpos[cur]);
    // the other buffer was last read before the previous barrier
    if (b + 1 < nblk) store_block(nb, lk[cur ^ 1], lpos[cur ^ 1]);
    __syncthreads();
  }
}

// Key operand of subtile kt (keys kt*16 .. kt*16+15 of the block): lane
// (qi, grp) holds key kt*16 + qi, channels 32s + 8grp .. + 7 at k-step s.
__device__ __forceinline__ void load_kop(bf16x8 (&kop)[4], const uint16_t* lkb, int kt,
                                         int qi, int grp) {
  const uint16_t* krow = lkb + (kt * 16 + qi) * kRowStride + 8 * grp;
#pragma unroll
  for (int s = 0; s < 4; ++s) kop[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(krow + 32 * s));
}

// S^T tile: 16 window queries (rows) x 16 keys (columns); the lane holds
// rows 4*grp + i of column qi.
__device__ __forceinline__ f32x4 score_tile(const bf16x8 (&qop)[4], const bf16x8 (&kop)[4]) {
  f32x4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s)
    d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qop[s], kop[s], d, 0, 0, 0);
  return d;
}

template <int KPT, int TPW, int MINW>
__global__ __launch_bounds__(kNT, MINW) void window_score_kernel(
    const SeqMeta* __restrict__ meta, const uint16_t* __restrict__ kpool,
    const int32_t* __restrict__ pos, const uint16_t* __restrict__ qwin,
    float* __restrict__ scores_out, int32_t* __restrict__ drops_out,
    int scores_stride, int L, int Hq, int Hkv, int G, int r, int every,
    int slot_lo, float scale_log2) {
  extern __shared__ float smem[];                 // scores [cap]
  __shared__ uint16_t lk[2][kBlk * kRowStride];
  __shared__ int lpos[2][kBlk];
  __shared__ SelectShared sel_sh;
  __shared__ int f[kMaxEvery];

  const int per_seq = L * Hkv;
  const int slot = slot_lo + static_cast<int>(blockIdx.x) / per_seq;
  const int lg = static_cast<int>(blockIdx.x) % per_seq;
  const int layer = lg / Hkv, g = lg % Hkv;
  const SeqMeta& M = meta[slot];
  if (!M.active) return;
  const int len = M.len, lp = M.prompt_len;
  const int m = len - lp - r - M.k_keep;          // rows Random Attention drops
  const int n_cand = len - r;
  const int64_t region = M.base + static_cast<int64_t>(lg) * M.cap;
  const uint16_t* Kr = kpool + region * kHeadDim;
  const int32_t* P = pos + region;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int qi = lane & 15, grp = lane >> 4;
  float* score = smem;
  for (int i = t; i < len; i += kNT) score[i] = 0.f;

  // window queries: tile qt covers head qt / 4, window rows 16 * (qt % 4) ..
  // + 15; this wave's tiles are qt = j * kWaves + wave for j < ntile
  const int n_tiles = G * 4;
  // (uniform across the wave: readfirstlane lets the tile loops branch on
  // scalars instead of masking lanes)
  const int ntile = __builtin_amdgcn_readfirstlane(
      wave < n_tiles ? min(TPW, (n_tiles - wave + kWaves - 1) / kWaves) : 0);
  bf16x8 qop[TPW][4];
  const int first_pos = lp + M.step - kWin;     // position of window row 0
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    const int qt = j * kWaves + wave;
    const bool ok = j < ntile;
    const int head = g * G + (ok ? qt / 4 : 0);
    const int row = 16 * ((ok ? qt : 0) % 4) + qi;
    const uint16_t* qrow = qwin + ((static_cast<int64_t>(slot) * L + layer) * Hq + head) *
                           kWin * kHeadDim + static_cast<int64_t>(row) * kHeadDim + 8 * grp;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const u32x4 z = {0u, 0u, 0u, 0u};
      qop[j][s] = as_bf16x8(ok ? *reinterpret_cast<const u32x4*>(qrow + 32 * s) : z);
    }
  }
  // position of the lane's D-row i of tile j (its window query)
  auto qpos = [&](int j, int i) {
    return first_pos + 16 * ((j * kWaves + wave) % 4) + 4 * grp + i;
  };

  // pass 1: per (tile, D-row) running max (raw dot units) and sum of
  // 2^((x - max) * scale) over this lane's key columns; every window query
  // sees every key of a block unless the block reaches past the first window
  // position (rows beyond len carry an infinite position): only then is the
  // causal mask applied
  float lse2[TPW][4];
  {
    float mx[TPW][4], sm[TPW][4];
#pragma unroll
    for (int j = 0; j < TPW; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        mx[j][i] = kNegInf;
        sm[j][i] = 0.f;
      }
    stream_blocks(Kr, P, len, lk, lpos, [&](int b, const uint16_t* lkb, const int* lpb) {
      const bool masked = lpb[kBlk - 1] > first_pos;
      float x[TPW][4][4];                        // [tile][subtile][D-row]
#pragma unroll
      for (int kt = 0; kt < kBlk / 16; ++kt) {
        bf16x8 kop[4];
        load_kop(kop, lkb, kt, qi, grp);
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
          if (j >= ntile) break;
          const f32x4 d = score_tile(qop[j], kop);
#pragma unroll
          for (int i = 0; i < 4; ++i) x[j][kt][i] = d[i];
        }
      }
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        if (j >= ntile) break;
        if (masked) {
#pragma unroll
          for (int kt = 0; kt < kBlk / 16; ++kt) {
            const int kpos = lpb[kt * 16 + qi];
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (kpos > qpos(j, i)) x[j][kt][i] = kNegInf;
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float bm = fmaxf(fmaxf(x[j][0][i], x[j][1][i]), fmaxf(x[j][2][i], x[j][3][i]));
          const float mn = fmaxf(mx[j][i], bm);
          // nothing visible yet (mn = -inf): every term below is 2^-inf = 0
          const float off = mn == kNegInf ? 0.f : -mn * scale_log2;
          float acc = sm[j][i] * __builtin_amdgcn_exp2f(fmaf(mx[j][i], scale_log2, off));
#pragma unroll
          for (int kt = 0; kt < kBlk / 16; ++kt)
            acc += __builtin_amdgcn_exp2f(fmaf(x[j][kt][i], scale_log2, off));
          sm[j][i] = acc;
          mx[j][i] = mn;
        }
      }
    });
    // merge the 16 lanes holding the same queries, then the log2-sum-exp
#pragma unroll
    for (int j = 0; j < TPW; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a_m = mx[j][i], a_s = sm[j][i];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          const float b_m = __shfl_xor(a_m, o, 64), b_s = __shfl_xor(a_s, o, 64);
          const float mn = fmaxf(a_m, b_m);
          if (mn != kNegInf) {
            a_s = a_s * __builtin_amdgcn_exp2f((a_m - mn) * scale_log2) +
                  b_s * __builtin_amdgcn_exp2f((b_m - mn) * scale_log2);
            a_m = mn;
          }
        }
        lse2[j][i] = a_m * scale_log2 + __builtin_amdgcn_logf(a_s);
      }
  }

  // pass 2: the same logits again; the weights 2^(s - lse) of every window
  // query summed per key, one 16-key subtile at a time
  auto pass2_block = [&](int b, const uint16_t* lkb, const int* lpb, auto masked) {
#pragma unroll
    for (int kt = 0; kt < kBlk / 16; ++kt) {
      const int kpos = lpb[kt * 16 + qi];
      bf16x8 kop[4];
      load_kop(kop, lkb, kt, qi, grp);
      // every tile's MFMA chain first, so the exponentials of one tile
      // overlap the products of the next
      f32x4 d[TPW];
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        if (j >= ntile) break;
        d[j] = score_tile(qop[j], kop);
      }
      float colsum = 0.f;
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        if (j >= ntile) break;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float w = __builtin_amdgcn_exp2f(fmaf(d[j][i], scale_log2, -lse2[j][i]));
          if constexpr (decltype(masked)::value) colsum += kpos > qpos(j, i) ? 0.f : w;
          else colsum += w;
        }
      }
      colsum += __shfl_xor(colsum, 16, 64);
      colsum += __shfl_xor(colsum, 32, 64);
      const int key = b * kBlk + kt * 16 + qi;
      if (grp == 0 && key < len) atomicAdd(&score[key], colsum);
    }
  };
  stream_blocks(Kr, P, len, lk, lpos, [&](int b, const uint16_t* lkb, const int* lpb) {
    if (lpb[kBlk - 1] > first_pos) pass2_block(b, lkb, lpb, std::true_type{});
    else pass2_block(b, lkb, lpb, std::false_type{});
  });

  const int64_t head_out = static_cast<int64_t>(slot - slot_lo) * per_seq + lg;
  if (scores_out) {
    for (int i = t; i < len; i += kNT) scores_out[head_out * scores_stride + i] = score[i];
  }
  if (!drops_out || m <= 0) return;
  // max-pool and select the m lowest candidates
  uint64_t key[KPT];
  uint32_t tie[KPT];
  uint32_t valid = 0;
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int c = t * KPT + i;
    key[i] = 0;
    tie[i] = static_cast<uint32_t>(c);      // ties by row, lower first
    if (c < n_cand) {
      float mxp = 0.f;
      for (int j = max(0, c - kPoolHalf); j <= min(len - 1, c + kPoolHalf); ++j)
        mxp = fmaxf(mxp, score[j]);
      key[i] = __float_as_uint(mxp);        // non-negative: bit order = value order
      valid |= 1u << i;
    }
  }
  const uint32_t drop = select_smallest<kNT, KPT, 32>(key, tie, valid, m, sel_sh);
  drop_list<kNT, KPT>(drop, 0, f, sel_sh);
  for (int k = t; k < m; k += kNT) drops_out[head_out * every + k] = f[k] + k;
}

template <int KPT>
hipError_t launch_tpw(int tpw, dim3 grid, size_t shmem, hipStream_t s,
                      const SeqMeta* meta, const uint16_t* kpool, const int32_t* pos,
                      const uint16_t* qwin, float* scores_out, int32_t* drops_out,
                      int scores_stride, int L, int Hq, int Hkv, int G, int r, int every,
                      int slot_lo, float scale) {
  // up to two tiles per wave the build fits four waves per SIMD (two
  // workgroups per CU, whose barriers do not keep them in step); more tiles
  // need the registers of two waves per SIMD
#define RA_WS_LAUNCH(T, W)                                                                  \
  hipLaunchKernelGGL((window_score_kernel<KPT, T, W>), grid, dim3(kNT), shmem, s, meta,     \
                     kpool, pos, qwin, scores_out, drops_out, scores_stride, L, Hq, Hkv,    \
                     G, r, every, slot_lo, scale)
  if (tpw <= 1) RA_WS_LAUNCH(1, 4);
  else if (tpw <= 2) RA_WS_LAUNCH(2, 4);
  else if (tpw <= 3) RA_WS_LAUNCH(3, 2);
  else if (tpw <= 4) RA_WS_LAUNCH(4, 2);
  else RA_WS_LAUNCH(8, 1);
#undef RA_WS_LAUNCH
  return hipGetLastError();
}

}  // namespace

hipError_t launch_window_score(const Shape& sh, const SeqMeta* meta, const void* kpool,
                               const int32_t* pos, const void* qwin, float* scores_out,
                               int32_t* drops_out, int scores_stride, int slot_lo,
                               int slot_hi, int max_len, hipStream_t s) {
  if (slot_hi <= slot_lo) return hipSuccess;
  const dim3 grid((slot_hi - slot_lo) * sh.L * sh.Hkv);
  const size_t shmem = sizeof(float) * static_cast<size_t>(max_len);
  const float scale = 1.4426950408889634f / sqrtf(static_cast<float>(kHeadDim));
  const int tpw = (sh.G * 4 + kWaves - 1) / kWaves;
  const uint16_t* k = static_cast<const uint16_t*>(kpool);
  const uint16_t* q = static_cast<const uint16_t*>(qwin);
  const int n_cand = max_len;   // upper bound of len - r
  if (n_cand <= kNT * 8)
    return launch_tpw<8>(tpw, grid, shmem, s, meta, k, pos, q, scores_out, drops_out,
                         scores_stride, sh.L, sh.Hq, sh.Hkv, sh.G, sh.r, sh.every, slot_lo, scale);
  if (n_cand <= kNT * 16)
    return launch_tpw<16>(tpw, grid, shmem, s, meta, k, pos, q, scores_out, drops_out,
                          scores_stride, sh.L, sh.Hq, sh.Hkv, sh.G, sh.r, sh.every, slot_lo, scale);
  if (n_cand <= kNT * 32)
    return launch_tpw<32>(tpw, grid, shmem, s, meta, k, pos, q, scores_out, drops_out,
                          scores_stride, sh.L, sh.Hq, sh.Hkv, sh.G, sh.r, sh.every, slot_lo, scale);
  return hipErrorInvalidValue;
}

}  // namespace ra
