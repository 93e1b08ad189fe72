// Selection steps of two score-based evictors, built only to price the
// selection signal that Random Attention does without (not used by the
// method).  Section 2 ("Baselines as choices of s") defines the scores:
//   R-KV: s_i = lambda * SnapKV_i - (1 - lambda) * softmax_i(cbar), cbar_i
//         the mean cosine similarity of key i to the other cached keys, its
//         most recent near-duplicates not counted;
//   VaSE: keep the n_large rows of largest value range, fill the rest of the
//         budget by sampling without replacement in proportion to SnapKV.
// Both read the raw observation-window scores that window_score.hip wrote
// for the same state (SnapKV_i = their max over rows i-3 .. i+3), select the
// m rows to drop among the candidates (every cached row outside the r most
// recent: the prompt competes), and write the ascending drop list that the
// compaction of evict.hip consumes.  One workgroup per (sequence, layer, KV
// head); candidates live in registers, KPT consecutive rows per thread.
#include <math.h>

#include "philox.h"
#include "ra_internal.h"
#include "select.h"

namespace ra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kNT = 512;
constexpr int kPoolHalf = 3;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  bf16x8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) {
  return __uint_as_float(h << 16);
}

// Order-preserving maps of floating-point values onto unsigned integers.
__device__ __forceinline__ uint64_t order_key_f64(double x) {
  const uint64_t b = static_cast<uint64_t>(__double_as_longlong(x));
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}
__device__ __forceinline__ uint64_t order_key_f32(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b >> 31) ? static_cast<uint64_t>(~b) : static_cast<uint64_t>(b | 0x80000000u);
}

// SnapKV score of candidate c: the raw window score max-pooled over 7 rows.
__device__ __forceinline__ float pooled_score(const float* raw, int c, int len) {
  float mx = 0.f;
  for (int j = max(0, c - kPoolHalf); j <= min(len - 1, c + kPoolHalf); ++j)
    mx = fmaxf(mx, raw[j]);
  return mx;
}

struct Head {
  int slot, lg, layer, g, len, lp, m, n_cand, budget;
  int64_t region;
  bool active;
};

__device__ __forceinline__ Head locate_head(const SeqMeta* meta, int L, int Hkv, int r,
                                            int slot_lo) {
  Head h;
  const int per_seq = L * Hkv;
  h.slot = slot_lo + static_cast<int>(blockIdx.x) / per_seq;
  h.lg = static_cast<int>(blockIdx.x) % per_seq;
  h.layer = h.lg / Hkv;
  h.g = h.lg % Hkv;
  const SeqMeta& M = meta[h.slot];
  h.len = M.len;
  h.lp = M.prompt_len;
  h.budget = M.prompt_len + M.k_keep;
  h.n_cand = M.len - r;
  h.m = h.n_cand - h.budget;
  h.region = M.base + static_cast<int64_t>(h.lg) * M.cap;
  h.active = M.active && h.m > 0;
  return h;
}

// ---------------------------------------------------------------------------
// VaSE
// ---------------------------------------------------------------------------

template <int KPT>
__global__ __launch_bounds__(kNT) void vase_kernel(
    const SeqMeta* __restrict__ meta, const uint16_t* __restrict__ vpool,
    const int32_t* __restrict__ pos, const float* __restrict__ raw_scores, int score_stride,
    int32_t* __restrict__ drops, int every, int L, int Hkv, int r, int slot_lo,
    int n_large_cfg, uint64_t seed) {
  extern __shared__ uint32_t vmm[];             // per row: bf16 max (hi) | bf16 min (lo)
  __shared__ SelectShared sel_sh;
  __shared__ int f[kMaxEvery];
  const Head h = locate_head(meta, L, Hkv, r, slot_lo);
  if (!h.active) return;
  const SeqMeta& M = meta[h.slot];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int32_t* P = pos + h.region;
  const float* raw = raw_scores + static_cast<int64_t>(blockIdx.x) * score_stride;

  // 1. value range of every candidate row: a wavefront takes an 8-row value
  // tile (128 channels x 8 rows, transposed); lane l reads channels 2l and
  // 2l + 1 (16 bytes each) and the wavefront reduces max and min per row
  const int n_tiles = (h.n_cand + 7) / 8;
  for (int tile = wave; tile < n_tiles; tile += kNT / 64) {
    const uint16_t* base = vpool + (h.region + 8 * tile) * kHeadDim;
    float mx[8], mn[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mx[e] = -__builtin_huge_valf();
      mn[e] = __builtin_huge_valf();
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(base + (2 * lane + c) * 8);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = bf16_bits_to_f32((w[e >> 1] >> (16 * (e & 1))) & 0xFFFF);
        mx[e] = fmaxf(mx[e], x);
        mn[e] = fminf(mn[e], x);
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], o, 64));
        mn[e] = fminf(mn[e], __shfl_xor(mn[e], o, 64));
      }
    }
    if (lane < 8) {
      float a = mx[0], b = mn[0];
#pragma unroll
      for (int e = 1; e < 8; ++e)
        if (lane == e) {
          a = mx[e];
          b = mn[e];
        }
      const int row = 8 * tile + lane;
      // bf16 values: the upper 16 bits of their float are exact
      if (row < h.n_cand) vmm[row] = (__float_as_uint(a) & 0xFFFF0000u) | (__float_as_uint(b) >> 16);
    }
  }
  __syncthreads();

  // 2. the large set: the n_large largest (range, position); the other
  // candidates are the n_cand - n_large smallest
  const int n_large = n_large_cfg < 0 ? h.budget / 2 : min(n_large_cfg, h.budget);
  uint64_t key[KPT];
  uint32_t tie[KPT];
  uint32_t valid = 0;
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int c = t * KPT + i;
    key[i] = 0;
    tie[i] = 0;
    if (c < h.n_cand) {
      const uint32_t mm = vmm[c];
      const double rg = static_cast<double>(bf16_bits_to_f32(mm >> 16)) -
                        static_cast<double>(bf16_bits_to_f32(mm & 0xFFFF));
      key[i] = static_cast<uint64_t>(__double_as_longlong(rg));   // >= 0: bits are ordered
      tie[i] = static_cast<uint32_t>(P[c]);
      valid |= 1u << i;
    }
  }
  const uint32_t small = n_large > 0
      ? select_smallest<kNT, KPT, 64>(key, tie, valid, h.n_cand - n_large, sel_sh)
      : valid;
  __syncthreads();

  // 3. proportional fill among the others: Efraimidis-Spirakis keys
  // log(u) / w (the largest kept), u in (0, 1] from the Philox word of the
  // position, w the SnapKV score; the m smallest are dropped
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    if ((small >> i) & 1) {
      const int c = t * KPT + i;
      const int p = P[c];
      const uint64_t x = philox_score(static_cast<uint64_t>(p), static_cast<uint64_t>(M.event),
                                      static_cast<uint64_t>(h.layer), static_cast<uint64_t>(h.g),
                                      seed, M.rid);
      const double u = static_cast<double>((x >> 11) + 1) * 0x1.0p-53;
      const float w = pooled_score(raw, c, h.len);
      const double e = w > 0.f ? log(u) / static_cast<double>(w) : -__builtin_huge_val();
      key[i] = order_key_f64(e);
    }
  }
  const uint32_t drop = select_smallest<kNT, KPT, 64>(key, tie, small, h.m, sel_sh);
  drop_list<kNT, KPT>(drop, 0, f, sel_sh);
  int32_t* out = drops + static_cast<int64_t>(blockIdx.x) * every;
  for (int k = t; k < h.m; k += kNT) out[k] = f[k] + k;
}

// ---------------------------------------------------------------------------
// R-KV
// ---------------------------------------------------------------------------

constexpr int kRowTiles = 4;                          // 16-row tiles per wavefront
constexpr int kChunkRows = (kNT / 64) * kRowTiles * 16;   // rows per workgroup: 512

// Sum of squares of this lane's 32 channels of an operand row (8 per k-step).
__device__ __forceinline__ float sumsq(const bf16x8 (&v)[4]) {
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = static_cast<float>(v[k][e]);
      s = fmaf(x, x, s);
    }
  return s;
}

__device__ __forceinline__ void load_operand(bf16x8 (&v)[4], const uint16_t* Kr, int row,
                                             int grp) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
    v[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(
        Kr + static_cast<int64_t>(row) * kHeadDim + 32 * s + 8 * grp));
}

// cbar of the candidate rows [chunk * 512, chunk * 512 + 512) of one head.
// D = K_rows . K_cols^T on v_mfma_f32_16x16x32_bf16: lane l holds rows
// 4*(l/16) + i of a row tile and column l % 16 of a column tile; the four
// lane groups hold a row's (or column's) channels in four parts of 32, so a
// norm is a lane sum plus two shuffles.  Column tiles are swept from the
// most recent (highest slot = highest position in the chronological layout)
// down, so the first `recent_dups` near-duplicates a row meets are the ones
// not counted; a ballot gives each row its near-duplicate columns in a tile.
__global__ __launch_bounds__(kNT) void rkv_cbar_kernel(
    const SeqMeta* __restrict__ meta, const uint16_t* __restrict__ kpool,
    float* __restrict__ cbar_out, int stride, int n_chunks, int L, int Hkv, int r,
    int slot_lo, float threshold, int recent_dups) {
  const int head_idx = static_cast<int>(blockIdx.x) / n_chunks;
  const int chunk = static_cast<int>(blockIdx.x) % n_chunks;
  const int per_seq = L * Hkv;
  const int slot = slot_lo + head_idx / per_seq;
  const int lg = head_idx % per_seq;
  const SeqMeta& M = meta[slot];
  const int len = M.len, n_cand = M.len - r;
  if (!M.active || n_cand - (M.prompt_len + M.k_keep) <= 0) return;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int qi = lane & 15, grp = lane >> 4;
  const int rt0 = (chunk * kChunkRows) / 16 + wave * kRowTiles;
  if (rt0 * 16 >= n_cand) return;
  const uint16_t* Kr = kpool + (M.base + static_cast<int64_t>(lg) * M.cap) * kHeadDim;

  bf16x8 a[kRowTiles][4];
  float sum[kRowTiles][4], dup[kRowTiles][4], invr[kRowTiles][4];
  int found[kRowTiles][4];
#pragma unroll
  for (int q = 0; q < kRowTiles; ++q) {
    load_operand(a[q], Kr, min((rt0 + q) * 16 + qi, len - 1), grp);
    float ss = sumsq(a[q]);
    ss += __shfl_xor(ss, 16, 64);
    ss += __shfl_xor(ss, 32, 64);
    const float inv = ss > 0.f ? 1.f / sqrtf(ss) : 0.f;      // row qi of the tile
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sum[q][i] = 0.f;
      dup[q][i] = 0.f;
      found[q][i] = 0;
      invr[q][i] = __shfl(inv, 4 * grp + i, 64);             // D-row 4*grp + i
    }
  }
  const int n_ct = (len + 15) / 16;
  bf16x8 b[4], bn[4];
  load_operand(b, Kr, min((n_ct - 1) * 16 + qi, len - 1), grp);
  for (int ct = n_ct - 1; ct >= 0; --ct) {
    if (ct > 0) load_operand(bn, Kr, (ct - 1) * 16 + qi, grp);   // next tile in flight
    const int col = ct * 16 + qi;
    float ss = sumsq(b);
    ss += __shfl_xor(ss, 16, 64);
    ss += __shfl_xor(ss, 32, 64);
    const float invc = ss > 0.f ? 1.f / sqrtf(ss) : 0.f;
    float c[kRowTiles][4];
    bool near = false;
#pragma unroll
    for (int q = 0; q < kRowTiles; ++q) {
      f32x4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[q][s], b[s], d, 0, 0, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        c[q][i] = d[i] * invr[q][i] * invc;
        near |= c[q][i] > threshold;
      }
    }
    // the last (ragged) column tile, the tiles holding a row's own column,
    // and tiles with a near-duplicate take the full bookkeeping; the rest
    // (nearly all) only accumulate
    const bool edge = ct == n_ct - 1 || (ct >= rt0 && ct < rt0 + kRowTiles);
    if (!edge && !__ballot(near)) {
#pragma unroll
      for (int q = 0; q < kRowTiles; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) sum[q][i] += c[q][i];
    } else {
#pragma unroll
      for (int q = 0; q < kRowTiles; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = (rt0 + q) * 16 + 4 * grp + i;
          const bool ok = col < len && col != row;
          if (ok) sum[q][i] += c[q][i];
          const uint64_t bal = __ballot(ok && c[q][i] > threshold);
          const uint32_t bits = static_cast<uint32_t>(bal >> (16 * grp)) & 0xFFFFu;
          const int need = recent_dups - found[q][i];
          if (need > 0 && bits) {
            if (((bits >> qi) & 1u) && __popc(bits >> (qi + 1)) < need) dup[q][i] += c[q][i];
            found[q][i] += min(need, __popc(bits));
          }
        }
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) b[s] = bn[s];
  }
  float* out = cbar_out + static_cast<int64_t>(head_idx) * stride;
#pragma unroll
  for (int q = 0; q < kRowTiles; ++q)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = sum[q][i] - dup[q][i];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
      const int row = (rt0 + q) * 16 + 4 * grp + i;
      if (qi == 0 && row < n_cand) out[row] = v / static_cast<float>(len - 1);
    }
}

// softmax of cbar over the candidates, the mix with SnapKV, and the m lowest.
template <int KPT>
__global__ __launch_bounds__(kNT) void rkv_select_kernel(
    const SeqMeta* __restrict__ meta, const int32_t* __restrict__ pos,
    const float* __restrict__ raw_scores, const float* __restrict__ cbar_in, int stride,
    int32_t* __restrict__ drops, int every, int L, int Hkv, int r, int slot_lo,
    float lambda) {
  __shared__ SelectShared sel_sh;
  __shared__ int f[kMaxEvery];
  __shared__ float red[kNT / 64];
  const Head h = locate_head(meta, L, Hkv, r, slot_lo);
  if (!h.active) return;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int32_t* P = pos + h.region;
  const float* raw = raw_scores + static_cast<int64_t>(blockIdx.x) * stride;
  const float* cbar = cbar_in + static_cast<int64_t>(blockIdx.x) * stride;

  float cb[KPT];
  float mx = -__builtin_huge_valf();
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int c = t * KPT + i;
    cb[i] = c < h.n_cand ? cbar[c] : -__builtin_huge_valf();
    mx = fmaxf(mx, cb[i]);
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = red[0];
#pragma unroll
  for (int w = 1; w < kNT / 64; ++w) mx = fmaxf(mx, red[w]);
  __syncthreads();
  float sm = 0.f;
#pragma unroll
  for (int i = 0; i < KPT; ++i)
    if (t * KPT + i < h.n_cand) sm += expf(cb[i] - mx);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) sm += __shfl_xor(sm, o, 64);
  if (lane == 0) red[wave] = sm;
  __syncthreads();
  sm = 0.f;
#pragma unroll
  for (int w = 0; w < kNT / 64; ++w) sm += red[w];

  uint64_t key[KPT];
  uint32_t tie[KPT];
  uint32_t valid = 0;
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int c = t * KPT + i;
    key[i] = 0;
    tie[i] = 0;
    if (c < h.n_cand) {
      const float s = lambda * pooled_score(raw, c, h.len) -
                      (1.f - lambda) * (expf(cb[i] - mx) / sm);
      key[i] = order_key_f32(s);
      tie[i] = static_cast<uint32_t>(P[c]);
      valid |= 1u << i;
    }
  }
  const uint32_t drop = select_smallest<kNT, KPT, 32>(key, tie, valid, h.m, sel_sh);
  drop_list<kNT, KPT>(drop, 0, f, sel_sh);
  int32_t* out = drops + static_cast<int64_t>(blockIdx.x) * every;
  for (int k = t; k < h.m; k += kNT) out[k] = f[k] + k;
}

template <int KPT>
hipError_t launch_kpt(int scorer, dim3 grid, size_t lds_rows, hipStream_t s,
                      const SeqMeta* meta, const void* vpool, const int32_t* pos,
                      const float* raw, const float* cbar, int stride, int32_t* drops,
                      int every, int L, int Hkv, int r, int slot_lo, float lambda,
                      int n_large, uint64_t seed) {
  if (scorer == 2) {
    hipLaunchKernelGGL((vase_kernel<KPT>), grid, dim3(kNT), lds_rows * sizeof(uint32_t), s,
                       meta, static_cast<const uint16_t*>(vpool), pos, raw, stride, drops,
                       every, L, Hkv, r, slot_lo, n_large, seed);
  } else {
    hipLaunchKernelGGL((rkv_select_kernel<KPT>), grid, dim3(kNT), 0, s, meta, pos, raw,
                       cbar, stride, drops, every, L, Hkv, r, slot_lo, lambda);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_scored_select(const Shape& sh, int scorer, const SeqMeta* meta,
                                const void* kpool, const void* vpool, const int32_t* pos,
                                const float* raw_scores, float* cbar_scratch,
                                int score_stride, int32_t* drops, int slot_lo, int slot_hi,
                                int max_len, float lambda, float threshold, int recent_dups,
                                int n_large, uint64_t seed, hipStream_t s) {
  if (slot_hi <= slot_lo) return hipSuccess;
  const int heads = (slot_hi - slot_lo) * sh.L * sh.Hkv;
  const dim3 grid(heads);
  const int n_cand = max_len;   // upper bound of len - r
  if (scorer == 1) {
    const int n_chunks = (n_cand + kChunkRows - 1) / kChunkRows;
    hipLaunchKernelGGL(rkv_cbar_kernel, dim3(heads * n_chunks), dim3(kNT), 0, s, meta,
                       static_cast<const uint16_t*>(kpool), cbar_scratch, score_stride,
                       n_chunks, sh.L, sh.Hkv, sh.r, slot_lo, threshold, recent_dups);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const size_t rows = static_cast<size_t>(max_len);
#define RA_SC_LAUNCH(K)                                                                  \
  launch_kpt<K>(scorer, grid, rows, s, meta, vpool, pos, raw_scores, cbar_scratch,       \
                score_stride, drops, sh.every, sh.L, sh.Hkv, sh.r, slot_lo, lambda,      \
                n_large, seed)
  if (n_cand <= kNT * 4) return RA_SC_LAUNCH(4);
  if (n_cand <= kNT * 8) return RA_SC_LAUNCH(8);
  if (n_cand <= kNT * 16) return RA_SC_LAUNCH(16);
  if (n_cand <= kNT * 32) return RA_SC_LAUNCH(32);
#undef RA_SC_LAUNCH
  return hipErrorInvalidValue;
}

}  // namespace ra
