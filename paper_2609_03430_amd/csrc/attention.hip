// Grouped-query decode attention over the compressed per-KV-head cache, with
// the step's append fused in (Section 2, "Notation": o = sum_i alpha_i v_i,
// alpha = softmax_i(q . k_i / sqrt(d)); Appendix F: the G query heads of a
// group read their KV head's cache).
//
// Work decomposition: one workgroup of W wavefronts per (sequence, KV head,
// split of `split_keys` keys); wavefront v streams the v-th W-th of the
// split.  Each wavefront reads its keys and values exactly once for all G
// query heads of the group and keeps an online softmax (running max and sum,
// combined across lanes with wavefront shuffles); the W states merge in LDS.
// A head with one split writes its normalised output directly; otherwise
// every split writes an unnormalised partial and a small second kernel
// merges them.  The step's new key/value is read from the input buffers by
// the wavefront that owns the last key, which also stores it into the cache
// after its reads, so no wavefront of the launch reads a row that is being
// written.  Value tiles are read with nontemporal loads, key rows with
// ordinary ones.
//
// bf16 path (MFMA, v_mfma_f32_16x16x32_bf16, 16x16 output tiles):
//   S^T[key][query] = K . Q^T   A = 16 key rows x 32 channels, B = Q^T with
//                               the group's G queries on the N side (padded
//                               to 16 with zeros);
//   O^T[ch][query] += V^T . P^T A = 16 channels x 32 keys from the
//                               transposed value tiles, B = P^T split into
//                               two bf16 parts (hi + lo) for precision.
// A lane's 8 operand elements come from one 16-byte global load: key rows
// are row-major and value rows are stored as transposed 8-row tiles.  The
// key rows are assigned to the two 16-row S tiles so that each lane's
// 8 softmax weights are exactly the 8 keys its P^T operand needs (tile t
// row 4a+i holds key 8a+4t+i), so no data moves between lanes except the
// two shuffles of the row maximum.
// fp32 path (VALU): lanes own keys for the scores and channels for P.V.
#include <mutex>

#include "ra_internal.h"

namespace ra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  bf16x8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

__device__ __forceinline__ u32x4 ld16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// Streaming load (nontemporal): the cached rows are read once per launch, so
// they are fetched without being kept in the caches.  Used where a load
// instruction covers whole 128-byte lines (the value tiles); a key load
// covers half lines of 16 rows, whose other halves the next load reads.
__device__ __forceinline__ u32x4 ld16_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
  __bf16 b = static_cast<__bf16>(x);   // round to nearest even
  uint16_t h;
  __builtin_memcpy(&h, &b, 2);
  return h;
}

struct Work {
  int slot, g, split;
  int len, n_keys, k0, k1, nsplit;
  RowMap rm;       // where the rows of the (slot, layer, g) cache live
  bool valid;
};

__device__ __forceinline__ Work locate(const SeqMeta* meta, int layer, int Hkv,
                                       int split_keys, const Paging& pg) {
  Work w;
  w.split = blockIdx.x;
  w.g = blockIdx.y;
  w.slot = blockIdx.z;
  const SeqMeta& M = meta[w.slot];
  w.valid = false;
  if (!M.active) return w;
  w.len = M.len;
  w.n_keys = w.len + 1;
  w.k0 = w.split * split_keys;
  if (w.k0 >= w.n_keys) return w;
  w.k1 = min(w.k0 + split_keys, w.n_keys);
  w.nsplit = (w.n_keys + split_keys - 1) / split_keys;
  w.rm = row_map(M, w.slot, layer * Hkv + w.g, pg);
  w.valid = true;
  return w;
}

// Store the step's new pair into the cache (row `len` of the head).
template <typename E, bool PAGED>
__device__ __forceinline__ void append_row(const Work& w, const SeqMeta* meta,
                                           int Hkv, const E* k_new,
                                           const E* v_new, E* kpool, E* vpool,
                                           int32_t* pos) {
  const int lane = threadIdx.x & 63;   // called by one whole wavefront
  const int64_t src = (static_cast<int64_t>(w.slot) * Hkv + w.g) * kHeadDim;
  const int64_t row = pool_row<PAGED>(w.rm, w.len);
  for (int c = lane; c < kHeadDim; c += 64) {
    kpool[row * kHeadDim + c] = k_new[src + c];
    vpool[(row & ~int64_t(7)) * kHeadDim + c * 8 + (row & 7)] = v_new[src + c];
  }
  if (lane == 0) pos[row] = meta[w.slot].prompt_len + meta[w.slot].step;
}

// Merge the split partials of one (sequence, KV head) into the output: the
// fp32 path (its kernel writes partials for every head) and the 12-wavefront
// contiguous bf16 build (heads of one split write their output themselves).
// One workgroup per head, launched after the attention kernel (the kernel
// boundary makes every partial visible).  Partial layout:
//   ws_o[((head * split_stride + split) * G + q) * 128 + c]  numerator / 2^m
//   ws_ml[((head * split_stride + split) * G + q) * 2 + {0,1}] = (m, l)
// with m the running max of the scores in log2 units and l the sum of
// 2^(s - m) over the split's keys.
template <typename E>
__global__ __launch_bounds__(256) void combine_kernel(AttnLaunch a, int G, int Hq, int Hkv,
                                                      bool skip_single) {
  __shared__ float sm[kMaxSplits * kMaxGroup];   // split maxima, then weights
  __shared__ float sl[kMaxSplits * kMaxGroup];   // split sums
  __shared__ float inv_l[kMaxGroup];
  const int g = blockIdx.x, slot = blockIdx.y;
  const SeqMeta& M = a.meta[slot];
  if (!M.active) return;
  const int t = threadIdx.x;
  const int n_keys = M.len + 1;
  const int nsplit = (n_keys + a.split_keys - 1) / a.split_keys;
  if (skip_single && nsplit == 1) return;
  const int head = slot * Hkv + g;
  const float* ml = a.ws_ml + static_cast<int64_t>(head) * a.split_stride * G * 2;
  const float* po = a.ws_o + static_cast<int64_t>(head) * a.split_stride * G * kHeadDim;
  for (int i = t; i < nsplit * G; i += blockDim.x) {
    sm[i] = ml[2 * i];
    sl[i] = ml[2 * i + 1];
  }
  __syncthreads();
  // per query: global max, split weights 2^(m_s - max) and the total sum
  if (t < G) {
    float mx = kNegInf;
    for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, sm[s * G + t]);
    float lsum = 0.f;
    for (int s = 0; s < nsplit; ++s) {
      const float w = exp2f(sm[s * G + t] - mx);
      sm[s * G + t] = w;
      lsum += w * sl[s * G + t];
    }
    inv_l[t] = 1.f / lsum;
  }
  __syncthreads();
  E* out = static_cast<E*>(a.out);
  // one thread per (query, 4 channels)
  for (int item = t; item < G * (kHeadDim / 4); item += blockDim.x) {
    const int q = item / (kHeadDim / 4), c4 = (item % (kHeadDim / 4)) * 4;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int s = 0; s < nsplit; ++s) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(
          po + static_cast<int64_t>(s * G + q) * kHeadDim + c4);
      acc += v * sm[s * G + q];
    }
    acc *= inv_l[q];
    const int64_t orow = (static_cast<int64_t>(slot) * Hq + g * G + q) * kHeadDim + c4;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (sizeof(E) == 2) out[orow + j] = f32_to_bf16(acc[j]);
      else out[orow + j] = acc[j];
    }
  }
}

// Partials of a head merged inside the attention kernel travel through
// device-coherent accesses (agent-scope relaxed atomics: stores written
// through to the level the chip's dies share, loads served from it), so the
// merge needs no whole-cache write-back or invalidation, which would stall
// every workgroup still streaming on the same die.
__device__ __forceinline__ void store_shared_level(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_shared_level(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The split partials of one head merged by the last of its splits to finish
// (outputs of element type E: bf16 bits or float).  Every split stores its partials with store_shared_level
// and waits until they are written; then one thread counts the split on the
// head's arrival counter.  The split that brings the count to nsplit reads
// every split's partials with load_shared_level, merges them as
// combine_kernel does and resets the counter for the next launch.  Nothing
// waits on another workgroup: the other splits simply end.  Called by every
// thread of the workgroup after its partials are stored; the head and its
// split count are taken afresh from the grid position and the slot record
// (kept from before the key loop, they would take registers the loop needs).
template <typename E>
__device__ void merge_if_last(const AttnLaunch& a, int G, int Hq, int Hkv) {
  __shared__ float sm[kMaxSplits * kMaxGroup];   // split maxima, then weights
  __shared__ float sl[kMaxSplits * kMaxGroup];   // split sums
  __shared__ float inv_l[kMaxGroup];
  __shared__ int last;
  const int slot = blockIdx.z, g = blockIdx.y, head = slot * Hkv + g;
  const int nsplit = (a.meta[slot].len + 1 + a.split_keys - 1) / a.split_keys;
  // This thread's partial stores are written before the workgroup counts
  // itself: the wait is issued as an asm statement that clobbers memory, so
  // the compiler cannot move the stores (relaxed atomics) past it either.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) {
    const int prev = __hip_atomic_fetch_add(a.arrivals + head, 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    last = prev == nsplit - 1;
    if (last)
      __hip_atomic_store(a.arrivals + head, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!last) return;
  const int t = threadIdx.x, nt = blockDim.x;
  const float* ml = a.ws_ml + static_cast<int64_t>(head) * a.split_stride * G * 2;
  const float* po = a.ws_o + static_cast<int64_t>(head) * a.split_stride * G * kHeadDim;
  // up to four splits and two outputs per thread: the numerators are loaded
  // together with the maxima and sums (one round trip to the shared level
  // instead of two)
  constexpr int kFastSplits = 4, kFastItems = 2;
  const bool fast = nsplit <= kFastSplits && G * kHeadDim <= kFastItems * nt;
  float pv[kFastItems][kFastSplits];
  if (fast) {
#pragma unroll
    for (int j = 0; j < kFastItems; ++j) {
      const int idx = t + j * nt;
#pragma unroll
      for (int s = 0; s < kFastSplits; ++s)
        pv[j][s] = s < nsplit && idx < G * kHeadDim
                       ? load_shared_level(po + (s * G) * kHeadDim + idx) : 0.f;
    }
  }
  for (int i = t; i < nsplit * G; i += nt) {
    sm[i] = load_shared_level(ml + 2 * i);
    sl[i] = load_shared_level(ml + 2 * i + 1);
  }
  __syncthreads();
  if (t < G) {
    float mx = kNegInf;
    for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, sm[s * G + t]);
    float lsum = 0.f;
    for (int s = 0; s < nsplit; ++s) {
      const float wt = exp2f(sm[s * G + t] - mx);
      sm[s * G + t] = wt;
      lsum += wt * sl[s * G + t];
    }
    inv_l[t] = 1.f / lsum;
  }
  __syncthreads();
  E* out = static_cast<E*>(a.out) + (static_cast<int64_t>(slot) * Hq + g * G) * kHeadDim;
  const auto put = [&](int idx, float o) {
    if constexpr (sizeof(E) == 2) out[idx] = f32_to_bf16(o);
    else out[idx] = o;
  };
  if (fast) {
#pragma unroll
    for (int j = 0; j < kFastItems; ++j) {
      const int idx = t + j * nt;
      if (idx >= G * kHeadDim) break;
      const int q = idx / kHeadDim;
      float o = 0.f;
#pragma unroll
      for (int s = 0; s < kFastSplits; ++s)
        if (s < nsplit) o += pv[j][s] * sm[s * G + q];
      put(idx, o * inv_l[q]);
    }
    return;
  }
  for (int idx = t; idx < G * kHeadDim; idx += nt) {
    const int q = idx / kHeadDim;
    float o = 0.f;
    for (int s = 0; s < nsplit; ++s)
      o += load_shared_level(po + (s * G) * kHeadDim + idx) * sm[s * G + q];
    put(idx, o * inv_l[q]);
  }
}

// ---------------------------------------------------------------------------
// bf16, MFMA
// ---------------------------------------------------------------------------

struct BlockRegs {
  u32x4 k[2][4];  // [S tile][k-step]
  u32x4 v[8];     // [16-channel tile]
};

// Offsets (in elements) of this lane's operand loads within a 32-key block.
struct LaneMap {
  int krow[2];   // key row within the block for S tile 0 / 1
  int kcol;      // first channel of the lane's 16-byte chunk at k-step 0
  int vrow;      // first key row of the lane's value tile
  int vch;       // channel within each 16-channel tile
};

__device__ __forceinline__ LaneMap lane_map() {
  const int lane = threadIdx.x & 63, r = lane & 15, grp = lane >> 4;
  LaneMap m;
  m.krow[0] = 8 * (r >> 2) + (r & 3);
  m.krow[1] = 8 * (r >> 2) + 4 + (r & 3);
  m.kcol = 8 * grp;
  m.vrow = 8 * grp;
  m.vch = r;
  return m;
}

// Rows kb .. kb+31 from the key rows at Kr and the value tiles at Vr (the
// head's region; in the paged layout the block's page, with kb = 0).
__device__ __forceinline__ void load_block(BlockRegs& b, const uint16_t* Kr,
                                           const uint16_t* Vr, int kb,
                                           const LaneMap& lm) {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const uint16_t* row = Kr + static_cast<int64_t>(kb + lm.krow[t]) * kHeadDim + lm.kcol;
#pragma unroll
    for (int s = 0; s < 4; ++s) b.k[t][s] = ld16(row + 32 * s);
  }
  const uint16_t* vt = Vr + static_cast<int64_t>(kb + lm.vrow) * kHeadDim + lm.vch * 8;
#pragma unroll
  for (int u = 0; u < 8; ++u) b.v[u] = ld16_stream(vt + 16 * 8 * u);
}

struct Softmax {
  float m;      // running max of the scaled scores (log2 units), per query
  float l;      // this lane's share of the running sum
  f32x4 acc[8]; // O^T tile u: channels 16u + 4*grp + i, query lane & 15
};

// One 32-key block.  `limit`: keys with index >= limit (block-relative) are
// masked out (32 for a full block); with MASKED, so are the keys whose bit is
// set in `dropped`.
template <bool MASKED = false>
__device__ __forceinline__ void compute_block(Softmax& st, const BlockRegs& b,
                                              const bf16x8 (&qop)[4],
                                              float scale_log2, int limit,
                                              uint32_t dropped = 0) {
  f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(b.k[0][s]), qop[s], s0, 0, 0, 0);
    s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(b.k[1][s]), qop[s], s1, 0, 0, 0);
  }
  const int grp = (threadIdx.x & 63) >> 4;
  float x[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[i] = s0[i] * scale_log2;
    x[4 + i] = s1[i] * scale_log2;
  }
  if (limit < 32) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (8 * grp + e >= limit) x[e] = kNegInf;
  }
  if constexpr (MASKED) {
    if (dropped) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if ((dropped >> (8 * grp + e)) & 1u) x[e] = kNegInf;
    }
  }
  float bm = x[0];
#pragma unroll
  for (int e = 1; e < 8; ++e) bm = fmaxf(bm, x[e]);
  bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
  bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
  const float mn = fmaxf(st.m, bm);
  // With MASKED, every key of a block can be masked while the state is still
  // empty (a wavefront whose first rows were all dropped): the weights and
  // the rescale are then taken against 0 instead of mn = -inf, which would
  // make them NaN; they come out 0 and the state stays empty.  Unmasked
  // blocks always hold a valid key.
  const float mr = MASKED && mn == kNegInf ? 0.f : mn;
  const float alpha = exp2f(st.m - mr);
  // P = hi + lo, both bf16, so the weights keep ~16 significant bits through
  // the bf16 MFMA (the remainder of a bf16 rounding is exact in fp32)
  bf16x8 p_hi, p_lo;
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float pf = exp2f(x[e] - mr);
    const __bf16 hi = static_cast<__bf16>(pf);
    p_hi[e] = hi;
    p_lo[e] = static_cast<__bf16>(pf - static_cast<float>(hi));
    psum += pf;
  }
  st.l = st.l * alpha + psum;
  st.m = mn;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    st.acc[u] *= alpha;
    st.acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(b.v[u]), p_hi, st.acc[u], 0, 0, 0);
    st.acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(b.v[u]), p_lo, st.acc[u], 0, 0, 0);
  }
}

// W wavefronts per workgroup share one (sequence, KV head, split) work item:
// wavefront v takes the v-th W-th of the split's keys, and the wavefronts
// merge their online-softmax states in LDS at the end.  When the
// head needs a single split, the workgroup writes the normalised output
// itself and no merge kernel runs.  MINW is the number of wavefronts per
// SIMD the build must allow (1 lets the accumulators live in the
// accumulation registers, 2 keeps each wavefront within 256 registers).
template <int W, int MINW, bool PAGED>
__global__ __launch_bounds__(64 * W, MINW) void attn_bf16_kernel(
    AttnLaunch a, Paging pg, int G, int Hq, int Hkv, float scale_log2) {
  constexpr int kNBuf = 2;   // register buffers (3 or 4 measured no faster)
  // heads of several splits merged by their last split (merge_if_last); the
  // contiguous 12-wavefront build has no registers to spare for it, and its
  // multi-split heads are merged by combine_kernel
  constexpr bool kFusedMerge = W != 12 || PAGED;
  __shared__ float s_m[W][kMaxGroup];
  __shared__ float s_l[W][kMaxGroup];
  __shared__ float s_o[W > 1 ? W : 1][kMaxGroup][kHeadDim];
  const Work w = locate(a.meta, a.layer, Hkv, a.split_keys, pg);
  if (!w.valid) return;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63, qi = lane & 15, grp = lane >> 4;
  const LaneMap lm = lane_map();
  const uint16_t* kpool = static_cast<const uint16_t*>(a.kpool);
  const uint16_t* vpool = static_cast<const uint16_t*>(a.vpool);
  const uint16_t* Kr = kpool + w.rm.region * kHeadDim;
  const uint16_t* Vr = vpool + w.rm.region * kHeadDim;
  // key block kb (a multiple of 32): its 32 rows lie in one page of the paged
  // layout, found through the block table; contiguous layouts index the region
  auto load = [&](BlockRegs& b, int kb) {
    if constexpr (PAGED) {
      const int64_t br = pool_row<true>(w.rm, kb);
      load_block(b, kpool + br * kHeadDim, vpool + br * kHeadDim, 0, lm);
    } else {
      load_block(b, Kr, Vr, kb, lm);
    }
  };
  const uint16_t* kn = static_cast<const uint16_t*>(a.k_new) +
                       (static_cast<int64_t>(w.slot) * Hkv + w.g) * kHeadDim;
  const uint16_t* vn = static_cast<const uint16_t*>(a.v_new) +
                       (static_cast<int64_t>(w.slot) * Hkv + w.g) * kHeadDim;

  // Q^T operand: query qi of the group, channels 32*s + 8*grp + [0, 8) at
  // k-step s (the key operand uses the same channel order, so a row's four
  // lane groups read 64 contiguous bytes per load)
  bf16x8 qop[4];
  {
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) +
        (static_cast<int64_t>(w.slot) * Hq + w.g * G + qi) * kHeadDim + 8 * grp;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const u32x4 z = {0u, 0u, 0u, 0u};
      qop[s] = as_bf16x8(qi < G ? ld16(qrow + 32 * s) : z);
    }
  }

  Softmax st;
  st.m = kNegInf;
  st.l = 0.f;
#pragma unroll
  for (int u = 0; u < 8; ++u) st.acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};

  // this wavefront's keys: [k0, k1) within the split (a multiple of 32 long
  // except where it ends at the new key)
  const int kpw = a.split_keys / W;
  // the same in every lane of the wavefront; in the paged builds of up to 8
  // wavefronts, made scalar, so that block-table entries are scalar loads
  // and block bases scalar sums (the 12-wavefront build has no registers to
  // spare for it and looks the table up per lane)
  constexpr bool kScalarTable = PAGED && W <= 8;
  const int k0 = kScalarTable ? __builtin_amdgcn_readfirstlane(w.k0 + wave * kpw)
                              : w.k0 + wave * kpw;
  const int k1 = min(k0 + kpw, w.k1);
  const bool has = k0 < k1;
  const bool owns_last = has && k1 == w.n_keys;
  const int nfull = !has ? 0 : (owns_last ? (w.len - k0) / 32 : (k1 - k0) / 32);
  if (nfull > 0) {
    // register buffers in rotation; every prefetch is unconditional (clamped
    // to the last block, whose repeated loads hit in cache) and the loop body
    // has no conditional code, so the loads it issues are consumed by the
    // next iteration and the compiler can neither sink them nor make the wait
    // before a block's compute also wait for later blocks' loads
    const int last = nfull - 1;
    BlockRegs buf[kNBuf];
#pragma unroll
    for (int j = 0; j < kNBuf; ++j) load(buf[j], k0 + 32 * min(j, last));
    int i = 0;
    for (; i + kNBuf - 1 < nfull; i += kNBuf) {
#pragma unroll
      for (int j = 0; j < kNBuf; ++j) {
        compute_block(st, buf[j], qop, scale_log2, 32);
        load(buf[j], k0 + 32 * min(i + kNBuf + j, last));
      }
    }
#pragma unroll
    for (int j = 0; j < kNBuf - 1; ++j)
      if (i + j < nfull) compute_block(st, buf[j], qop, scale_log2, 32);
  }
  if (owns_last) {
    // tail block: cached rows below len, the new pair at len, masked above
    const int kb = k0 + 32 * nfull;
    const int limit = w.n_keys - kb;       // 1..32 valid keys
    // rows of this block below len lie in one page of the paged layout (only
    // rows below len are read from the pools: the page of row len may not be
    // in the table yet when len is a multiple of 32)
    const uint16_t* Kb = Kr + static_cast<int64_t>(kb) * kHeadDim;
    const uint16_t* Vb = Vr + static_cast<int64_t>(kb) * kHeadDim;
    if constexpr (PAGED) {
      const int64_t br = kb < w.len ? pool_row<true>(w.rm, kb) : 0;
      Kb = kpool + br * kHeadDim;
      Vb = vpool + br * kHeadDim;
    }
    BlockRegs b;
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int key = kb + lm.krow[t];
      const uint16_t* row = key < w.len ? Kb + lm.krow[t] * kHeadDim : kn;
#pragma unroll
      for (int s = 0; s < 4; ++s)
        b.k[t][s] = key <= w.len ? ld16(row + lm.kcol + 32 * s) : z;
    }
    const int key0 = kb + lm.vrow;         // first key of this lane's tile
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int ch = 16 * u + lm.vch;
      u32x4 v = key0 < w.len ? ld16(Vb + lm.vrow * kHeadDim + ch * 8) : z;
      uint16_t e8[8];
      __builtin_memcpy(e8, &v, 16);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (key0 + e == w.len) e8[e] = vn[ch];
        else if (key0 + e > w.len) e8[e] = 0;
      }
      __builtin_memcpy(&v, e8, 16);
      b.v[u] = v;
    }
    compute_block(st, b, qop, scale_log2, limit);
  }

  // lane sums of the same query -> the wavefront's sum
  st.l += __shfl_xor(st.l, 16, 64);
  st.l += __shfl_xor(st.l, 32, 64);

  if (owns_last)
    append_row<uint16_t, PAGED>(w, a.meta, Hkv, static_cast<const uint16_t*>(a.k_new),
                         static_cast<const uint16_t*>(a.v_new),
                         static_cast<uint16_t*>(a.kpool),
                         static_cast<uint16_t*>(a.vpool), a.pos);

  const int head = w.slot * Hkv + w.g;
  const int64_t item = static_cast<int64_t>(head) * a.split_stride + w.split;
  uint16_t* out = static_cast<uint16_t*>(a.out);
  if constexpr (W == 1) {
    if (qi < G) {
      if (w.nsplit == 1) {
        const float inv = 1.f / st.l;
        const int64_t orow = (static_cast<int64_t>(w.slot) * Hq + w.g * G + qi) * kHeadDim;
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            out[orow + 16 * u + 4 * grp + i] = f32_to_bf16(st.acc[u][i] * inv);
      } else {
        float* po = a.ws_o + (item * G + qi) * kHeadDim;
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int i = 0; i < 4; ++i) store_shared_level(po + 16 * u + 4 * grp + i, st.acc[u][i]);
        if (grp == 0) {
          store_shared_level(a.ws_ml + (item * G + qi) * 2, st.m);
          store_shared_level(a.ws_ml + (item * G + qi) * 2 + 1, st.l);
        }
      }
    }
  } else {
    // merge the W wavefronts in LDS
    if (qi < G) {
#pragma unroll
      for (int u = 0; u < 8; ++u)
        *reinterpret_cast<f32x4*>(&s_o[wave][qi][16 * u + 4 * grp]) = st.acc[u];
      if (grp == 0) {
        s_m[wave][qi] = st.m;
        s_l[wave][qi] = st.l;
      }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < G * kHeadDim; idx += 64 * W) {
      const int q = idx / kHeadDim, c = idx % kHeadDim;
      float mx = kNegInf;
#pragma unroll
      for (int v = 0; v < W; ++v) mx = fmaxf(mx, s_m[v][q]);
      float lsum = 0.f, o = 0.f;
#pragma unroll
      for (int v = 0; v < W; ++v) {
        const float sc = s_m[v][q] == kNegInf ? 0.f : exp2f(s_m[v][q] - mx);
        lsum += s_l[v][q] * sc;
        o += s_o[v][q][c] * sc;
      }
      if (w.nsplit == 1) {
        out[(static_cast<int64_t>(w.slot) * Hq + w.g * G + q) * kHeadDim + c] =
            f32_to_bf16(o / lsum);
      } else if constexpr (kFusedMerge) {
        store_shared_level(a.ws_o + (item * G + q) * kHeadDim + c, o);
        if (c == 0) {
          store_shared_level(a.ws_ml + (item * G + q) * 2, mx);
          store_shared_level(a.ws_ml + (item * G + q) * 2 + 1, lsum);
        }
      } else {
        a.ws_o[(item * G + q) * kHeadDim + c] = o;
        if (c == 0) {
          a.ws_ml[(item * G + q) * 2] = mx;
          a.ws_ml[(item * G + q) * 2 + 1] = lsum;
        }
      }
    }
  }
  if constexpr (kFusedMerge) {
    if (w.nsplit > 1) merge_if_last<uint16_t>(a, G, Hq, Hkv);
  }
}

// ---------------------------------------------------------------------------
// bf16, MFMA, moving the rows of a deferred eviction on the way
// ---------------------------------------------------------------------------

// The last block of a head's source rows, kb .. kb+31, reaching past the
// cached rows: it is loaded as a full block (rows past the region's end read
// its row 0, so every lane issues the same sixteen loads as for any block and
// the loads in flight stay countable) and, once the data has arrived, row
// n_rows becomes the step's new pair (staged in LDS: nk, nv) and the rows
// above it zero.
__device__ __forceinline__ void load_block_clamped(BlockRegs& b, const uint16_t* Kr,
                                                   const uint16_t* Vr, int kb, int n_rows,
                                                   const LaneMap& lm) {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int key = kb + lm.krow[t];
    const uint16_t* row = Kr + static_cast<int64_t>(key < n_rows ? key : 0) * kHeadDim + lm.kcol;
#pragma unroll
    for (int s = 0; s < 4; ++s) b.k[t][s] = ld16(row + 32 * s);
  }
  const int key0 = kb + lm.vrow;                      // a tile's first row (8-aligned)
  const uint16_t* vt = Vr + static_cast<int64_t>(key0 < n_rows ? key0 : 0) * kHeadDim + lm.vch * 8;
#pragma unroll
  for (int u = 0; u < 8; ++u) b.v[u] = ld16_stream(vt + 16 * 8 * u);
}

__device__ __forceinline__ void patch_block_tail(BlockRegs& b, const uint16_t* nk,
                                                 const uint16_t* nv, int kb, int n_rows,
                                                 const LaneMap& lm) {
  const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int key = kb + lm.krow[t];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (key == n_rows) b.k[t][s] = *reinterpret_cast<const u32x4*>(nk + lm.kcol + 32 * s);
      else if (key > n_rows) b.k[t][s] = z;
    }
  }
  const int key0 = kb + lm.vrow;
  if (key0 + 8 > n_rows) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      uint16_t e8[8];
      __builtin_memcpy(e8, &b.v[u], 16);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (key0 + e == n_rows) e8[e] = nv[16 * u + lm.vch];
        else if (key0 + e > n_rows) e8[e] = 0;
      }
      __builtin_memcpy(&b.v[u], e8, 16);
    }
  }
}

// Decode attention for the step after a deferred eviction (contiguous
// chronological layout, bf16, one workgroup of W wavefronts per (sequence,
// KV head), the whole head).  A sequence whose event deferred its row moves
// (due == kDueMovePending) holds its key/value rows in the order before the
// event, rows [0, plan_len), and the event's drop slots; its positions are
// already compacted and len = plan_len - m.  Attention runs over the
// surviving rows and the step's new pair (the dropped rows are masked), and
// every surviving row j after the first drop moves down to its compacted
// slot j - #{drops below j}, so the rows end as a full event would leave
// them, without reading them a second time.  The blocks are dealt in rounds,
// block r * W + v to wavefront v; every wavefront's loads of a round have
// returned (the round's softmax consumed them) before the barrier that
// precedes the round's moves.  A row moves only down, into a block of its
// own round or of an earlier one, which was read before that barrier, and
// no round reads a row that an earlier round wrote; the next round's loads,
// issued before the barrier, read only rows above every destination of the
// round, except that loads of blocks past the last key, and of tail rows
// past the cached ones, read the region's row 0 (which a round may be
// writing when the prompt is empty): those values are never used, being
// replaced by the new pair or zero, or belonging to no block.  The new pair
// is stored at len after the last round.  Sequences with nothing to move
// take the same path without moves.
template <int W>
__global__ __launch_bounds__(64 * W, 1) void attn_bf16_move_kernel(
    AttnLaunch a, int L, int G, int Hq, int Hkv, float scale_log2) {
  __shared__ float s_m[W][kMaxGroup];
  __shared__ float s_l[W][kMaxGroup];
  __shared__ float s_o[W][kMaxGroup][kHeadDim];
  __shared__ int s_drop[kMaxEvery];
  // a round's surviving value rows in destination order, per channel, offset
  // by the round's first destination row mod 8 so that destination tiles
  // start on 16-byte boundaries
  constexpr int kStage = W * 32 + 16;
  __shared__ __align__(16) uint16_t s_v[kHeadDim][kStage];
  __shared__ __align__(16) uint16_t s_new[2][kHeadDim];  // the step's key, value
  const int g = blockIdx.y, slot = blockIdx.z;
  const SeqMeta& M = a.meta[slot];
  if (!M.active) return;
  const bool moving = M.due == kDueMovePending;
  const int len = M.len;                              // rows once compacted
  const int n_rows = moving ? M.plan_len : len;       // rows in the region now
  const int m = min(n_rows - len, kMaxEvery);        // <= evict_every (host)
  const int lg = a.layer * Hkv + g;
  const int64_t region = M.base + static_cast<int64_t>(lg) * M.cap;
  // wavefront-uniform (the block indices and the drop scans below are scalar)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, qi = lane & 15, grp = lane >> 4;
  if (moving) {
    const int32_t* d = a.drops + (static_cast<int64_t>(slot) * L * Hkv + lg) * a.drop_stride;
    for (int k = threadIdx.x; k < min(m, kMaxEvery); k += 64 * W) s_drop[k] = d[k];
  }
  {
    const uint16_t* src = threadIdx.x < kHeadDim ? static_cast<const uint16_t*>(a.k_new)
                                                 : static_cast<const uint16_t*>(a.v_new);
    if (threadIdx.x < 2 * kHeadDim)
      (&s_new[0][0])[threadIdx.x] =
          src[(static_cast<int64_t>(slot) * Hkv + g) * kHeadDim + (threadIdx.x & (kHeadDim - 1))];
  }
  __syncthreads();
  const LaneMap lm = lane_map();
  uint16_t* kpool = static_cast<uint16_t*>(a.kpool);
  uint16_t* vpool = static_cast<uint16_t*>(a.vpool);
  const uint16_t* Kr = kpool + region * kHeadDim;
  const uint16_t* Vr = vpool + region * kHeadDim;

  bf16x8 qop[4];
  {
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) +
        (static_cast<int64_t>(slot) * Hq + g * G + qi) * kHeadDim + 8 * grp;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const u32x4 z = {0u, 0u, 0u, 0u};
      qop[s] = as_bf16x8(qi < G ? ld16(qrow + 32 * s) : z);
    }
  }
  Softmax st;
  st.m = kNegInf;
  st.l = 0.f;
#pragma unroll
  for (int u = 0; u < 8; ++u) st.acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int n_keys = n_rows + 1;                      // the region's rows + the new pair
  const int nblk = (n_keys + 31) / 32;
  const int rounds = (nblk + W - 1) / W;
  auto load = [&](BlockRegs& b, int blk) {
    const int kb = blk * 32;
    if (kb + 32 <= n_rows) load_block(b, Kr, Vr, kb, lm);
    else load_block_clamped(b, Kr, Vr, kb, n_rows, lm);
  };
  // two register buffers, each named (an array indexed by the round's parity
  // would live in scratch memory): the loop below runs two rounds per pass
  // every round issues its sixteen prefetch loads, also for blocks past the
  // last key (they read the region's row 0 and are never used): with a fixed
  // count of loads after each block's, the wait for a block leaves the next
  // block's loads in flight
  BlockRegs buf0, buf1;
  load(buf0, wave);
  int di = 0;                 // drops below the current block (wavefront-uniform)
  auto round = [&](int r, BlockRegs& cur, BlockRegs& nxt) {
    const int blk = r * W + wave;
    const int kb = blk * 32;
    const bool have = blk < nblk;
    load(nxt, blk + W);
    uint32_t dropped = 0;
    if (have) {
      if (kb + 32 > n_rows) patch_block_tail(cur, s_new[0], s_new[1], kb, n_rows, lm);
      while (di < m && s_drop[di] < kb) ++di;
      for (int k = di; k < m && s_drop[k] < kb + 32; ++k) dropped |= 1u << (s_drop[k] - kb);
      compute_block<true>(st, cur, qop, scale_log2, min(32, n_keys - kb), dropped);
    }
    __syncthreads();          // every load of the round has been consumed
    if (moving && have) {
      const BlockRegs& b = cur;
      // key rows: this lane's two rows, four 16-byte chunks each
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int rr = lm.krow[t], j = kb + rr;
        if (j < n_rows && !((dropped >> rr) & 1u)) {
          const int dst = j - di - __popc(__builtin_amdgcn_ubfe(dropped, 0, rr));
          if (dst != j) {
            uint16_t* row = kpool + (region + dst) * kHeadDim + lm.kcol;
#pragma unroll
            for (int s = 0; s < 4; ++s) *reinterpret_cast<u32x4*>(row + 32 * s) = b.k[t][s];
          }
        }
      }
    }
    if (moving) {
      // values: the round's survivors go to LDS in destination order, then the
      // workgroup writes whole destination tiles (16 bytes per channel); only
      // the round's first and last tiles, shared with the neighbouring rounds,
      // are written element by element
      const int r0 = r * W * 32;                                 // round's first source row
      int fr = 0;                                                // drops below r0
      while (fr < m && s_drop[fr] < r0) ++fr;
      const int r1 = min(r0 + W * 32, n_rows);                   // round's source rows [r0, r1)
      int fe = fr;
      while (fe < m && s_drop[fe] < r1) ++fe;
      const int d_lo = r0 - fr, d_hi = r1 - fe;                  // destinations [d_lo, d_hi)
      const int off = d_lo & 7;
      if (have && kb < n_rows) {
        const BlockRegs& b = cur;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int rr = lm.vrow + e, j = kb + rr;
          if (j < n_rows && !((dropped >> rr) & 1u)) {
            const int dst = j - di - __popc(__builtin_amdgcn_ubfe(dropped, 0, rr));
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              uint16_t e8[8];
              __builtin_memcpy(e8, &b.v[u], 16);
              s_v[16 * u + lm.vch][off + dst - d_lo] = e8[e];
            }
          }
        }
      }
      __syncthreads();
      if (d_hi > d_lo && r1 > s_drop[0]) {
        const int t_lo = d_lo >> 3, t_hi = (d_hi - 1) >> 3;       // destination tiles
        const int items = (t_hi - t_lo + 1) * kHeadDim;
        for (int it = threadIdx.x; it < items; it += 64 * W) {
          const int tile = t_lo + it / kHeadDim, ch = it % kHeadDim;
          const int lo = max(tile * 8, d_lo), hi = min(tile * 8 + 8, d_hi);
          const int64_t row0 = region + tile * 8;                // 8-aligned (region is)
          uint16_t* dstp = vpool + row0 * kHeadDim + ch * 8;
          const uint16_t* src = &s_v[ch][off + tile * 8 - d_lo];
          if (lo == tile * 8 && hi == tile * 8 + 8) {
            *reinterpret_cast<u32x4*>(dstp) = *reinterpret_cast<const u32x4*>(src);
          } else {
            for (int x = lo; x < hi; ++x) dstp[x - tile * 8] = src[x - tile * 8];
          }
        }
      }
    }
  };
  for (int r = 0; r < rounds; r += 2) {
    round(r, buf0, buf1);
    if (r + 1 < rounds) round(r + 1, buf1, buf0);
  }
  st.l += __shfl_xor(st.l, 16, 64);
  st.l += __shfl_xor(st.l, 32, 64);
  // lane indices taken afresh (kept from before the rounds, they would be
  // spilled: the rounds hold every register)
  const int lane_e = __lane_id(), qe = lane_e & 15, ge = lane_e >> 4;
  const int tid = wave * 64 + lane_e;
  __syncthreads();            // every move is done: the new pair goes to row len
  if (wave == 0) {
    const int64_t row = region + len;
    for (int c = lane_e; c < kHeadDim; c += 64) {
      kpool[row * kHeadDim + c] = s_new[0][c];
      vpool[(row & ~int64_t(7)) * kHeadDim + c * 8 + (row & 7)] = s_new[1][c];
    }
    if (lane_e == 0) a.pos[row] = M.prompt_len + M.step;
  }

  // merge the W wavefronts in LDS and write the normalised output
  if (qe < G) {
#pragma unroll
    for (int u = 0; u < 8; ++u)
      *reinterpret_cast<f32x4*>(&s_o[wave][qe][16 * u + 4 * ge]) = st.acc[u];
    if (ge == 0) {
      s_m[wave][qe] = st.m;
      s_l[wave][qe] = st.l;
    }
  }
  __syncthreads();
  uint16_t* out = static_cast<uint16_t*>(a.out);
  for (int idx = tid; idx < G * kHeadDim; idx += 64 * W) {
    const int q = idx / kHeadDim, c = idx % kHeadDim;
    float mx = kNegInf;
#pragma unroll
    for (int v = 0; v < W; ++v) mx = fmaxf(mx, s_m[v][q]);
    float lsum = 0.f, o = 0.f;
#pragma unroll
    for (int v = 0; v < W; ++v) {
      const float sc = s_m[v][q] == kNegInf ? 0.f : exp2f(s_m[v][q] - mx);
      lsum += s_l[v][q] * sc;
      o += s_o[v][q][c] * sc;
    }
    out[(static_cast<int64_t>(slot) * Hq + g * G + q) * kHeadDim + c] = f32_to_bf16(o / lsum);
  }
}

// ---------------------------------------------------------------------------
// fp32, VALU
// ---------------------------------------------------------------------------

// GT: the group size when fixed at compile time (1, 2, 4, 8), 0 for any G.
template <int GT, bool PAGED>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnLaunch a, Paging pg, int G_rt,
                                                      int Hq, int Hkv,
                                                      float scale_log2) {
  constexpr int kQ = GT > 0 ? GT : kMaxGroup;   // query slots in registers
  const int G = GT > 0 ? GT : G_rt;
  __shared__ float qs[kMaxGroup][kHeadDim];
  __shared__ float ps[kMaxGroup][64];
  const Work w = locate(a.meta, a.layer, Hkv, a.split_keys, pg);
  if (!w.valid) return;
  const int lane = threadIdx.x;
  const float* kpool = static_cast<const float*>(a.kpool);
  const float* vpool = static_cast<const float*>(a.vpool);
  const float* kn = static_cast<const float*>(a.k_new) +
                    (static_cast<int64_t>(w.slot) * Hkv + w.g) * kHeadDim;
  const float* vn = static_cast<const float*>(a.v_new) +
                    (static_cast<int64_t>(w.slot) * Hkv + w.g) * kHeadDim;
  const float* qg = static_cast<const float*>(a.q) +
                    (static_cast<int64_t>(w.slot) * Hq + w.g * G) * kHeadDim;
  for (int i = lane; i < G * kHeadDim; i += 64) qs[i / kHeadDim][i % kHeadDim] = qg[i];
  __syncthreads();

  float m[kQ], l[kQ], acc[kQ][2];
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    m[q] = kNegInf;
    l[q] = 0.f;
    acc[q][0] = acc[q][1] = 0.f;
  }
  const float vn0 = vn[lane], vn1 = vn[lane + 64];
  for (int kb = w.k0; kb < w.k1; kb += 64) {
    // scores: lanes own keys
    const int key = kb + lane;
    const bool valid = key < w.k1;
    const float* krow = key < w.len ? kpool + pool_row<PAGED>(w.rm, key) * kHeadDim : kn;
    float s[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q) s[q] = 0.f;
    if (valid) {
      for (int c = 0; c < kHeadDim; c += 4) {
        const float4 kv = *reinterpret_cast<const float4*>(krow + c);
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
          if (GT > 0 || q < G)
            s[q] += kv.x * qs[q][c] + kv.y * qs[q][c + 1] + kv.z * qs[q][c + 2] +
                    kv.w * qs[q][c + 3];
        }
      }
    }
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      if (GT > 0 || q < G) {
        const float x = valid ? s[q] * scale_log2 : kNegInf;
        const float mn = fmaxf(m[q], wave_max(x));
        const float alpha = exp2f(m[q] - mn);
        const float p = exp2f(x - mn);
        l[q] = l[q] * alpha + wave_sum(p);
        acc[q][0] *= alpha;
        acc[q][1] *= alpha;
        m[q] = mn;
        ps[q][lane] = p;
      }
    }
    __syncthreads();
    // P.V: lanes own channels lane and lane + 64; a value tile holds the 8
    // keys of a channel in 32 contiguous bytes, so a lane reads 8 keys with
    // two 16-byte loads and the wavefront's reads are contiguous.  The
    // chunk's tiles are all issued before any is used.  Rows at or past len
    // are selected, not multiplied: the new value at len, zero above it.
    const int nk = min(64, w.k1 - kb);
    const int ntile = (nk + 7) >> 3;
    float vv[8][2][8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      if (t < ntile) {
        const int kt = kb + 8 * t;
        // a tile of 8 rows lies in one page; only tiles holding a row below
        // len are read from the pool (the others hold the new value or zero)
        const float* base = vpool + (kt < w.len ? pool_row<PAGED>(w.rm, kt) : 0) * kHeadDim;
        const float4* s0 = reinterpret_cast<const float4*>(base + lane * 8);
        const float4* s1 = reinterpret_cast<const float4*>(base + (lane + 64) * 8);
        const float4 a0 = s0[0], a1 = s0[1], b0 = s1[0], b1 = s1[1];
        const float ea[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        const float eb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int kj = kt + e;
          vv[t][0][e] = kj < w.len ? ea[e] : (kj == w.len ? vn0 : 0.f);
          vv[t][1][e] = kj < w.len ? eb[e] : (kj == w.len ? vn1 : 0.f);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      if (t < ntile) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
#pragma unroll
          for (int q = 0; q < kQ; ++q) {
            if (GT > 0 || q < G) {
              const float p = ps[q][8 * t + e];
              acc[q][0] += p * vv[t][0][e];
              acc[q][1] += p * vv[t][1][e];
            }
          }
        }
      }
    }
    __syncthreads();
  }

  if (w.k1 == w.n_keys)
    append_row<float, PAGED>(w, a.meta, Hkv, static_cast<const float*>(a.k_new),
                      static_cast<const float*>(a.v_new),
                      static_cast<float*>(a.kpool),
                      static_cast<float*>(a.vpool), a.pos);

  // one split: the normalised output; several: the partials, merged by the
  // split that finishes last (merge_if_last) or, with merge_kernel, by the
  // merge kernel launched next
  const int head = w.slot * Hkv + w.g;
  if (w.nsplit == 1) {
    float* out = static_cast<float*>(a.out) +
                 (static_cast<int64_t>(w.slot) * Hq + w.g * G) * kHeadDim;
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      if (GT > 0 || q < G) {
        const float inv = 1.f / l[q];
        out[q * kHeadDim + lane] = acc[q][0] * inv;
        out[q * kHeadDim + lane + 64] = acc[q][1] * inv;
      }
    }
    return;
  }
  const int64_t item = static_cast<int64_t>(head) * a.split_stride + w.split;
  if (a.merge_kernel) {
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      if (GT > 0 || q < G) {
        float* po = a.ws_o + (item * G + q) * kHeadDim;
        po[lane] = acc[q][0];
        po[lane + 64] = acc[q][1];
        if (lane == 0) {
          a.ws_ml[(item * G + q) * 2] = m[q];
          a.ws_ml[(item * G + q) * 2 + 1] = l[q];
        }
      }
    }
    return;
  }
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    if (GT > 0 || q < G) {
      float* po = a.ws_o + (item * G + q) * kHeadDim;
      store_shared_level(po + lane, acc[q][0]);
      store_shared_level(po + lane + 64, acc[q][1]);
      if (lane == 0) {
        store_shared_level(a.ws_ml + (item * G + q) * 2, m[q]);
        store_shared_level(a.ws_ml + (item * G + q) * 2 + 1, l[q]);
      }
    }
  }
  merge_if_last<float>(a, G, Hq, Hkv);
}

template <int GT, bool PAGED>
void launch_f32(const dim3& grid, hipStream_t s, const AttnLaunch& a, const Shape& sh,
                float scale_log2) {
  hipLaunchKernelGGL((attn_f32_kernel<GT, PAGED>), grid, dim3(64), 0, s, a, sh.pg, sh.G,
                     sh.Hq, sh.Hkv, scale_log2);
}

template <bool PAGED>
hipError_t launch_attention_t(const Shape& sh, const AttnLaunch& a, hipStream_t s) {
  const dim3 grid(a.max_splits, sh.Hkv, a.max_seqs);
  // scores in log2 units: q.k / sqrt(d) * log2(e)
  const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(kHeadDim));
  const dim3 cgrid(sh.Hkv, a.max_seqs);
  if (sh.dtype == 1 && a.move) {
    // one workgroup per head (max_splits == 1), rows of deferred events moved;
    // eight wavefronts (256 registers each: two per SIMD; a four-wavefront
    // build needs more than 256 and would run one per SIMD)
    const dim3 mgrid(1, sh.Hkv, a.max_seqs);
    hipLaunchKernelGGL((attn_bf16_move_kernel<8>), mgrid, dim3(512), 0, s, a, sh.L, sh.G,
                       sh.Hq, sh.Hkv, scale_log2);
  } else if (sh.dtype == 1) {
    if (a.waves == 12)
      hipLaunchKernelGGL((attn_bf16_kernel<12, 1, PAGED>), grid, dim3(768), 0, s, a, sh.pg,
                         sh.G, sh.Hq, sh.Hkv, scale_log2);
    else if (a.waves == 8)
      hipLaunchKernelGGL((attn_bf16_kernel<8, 1, PAGED>), grid, dim3(512), 0, s, a, sh.pg,
                         sh.G, sh.Hq, sh.Hkv, scale_log2);
    else if (a.waves == 4 && a.wide_regs)
      hipLaunchKernelGGL((attn_bf16_kernel<4, 1, PAGED>), grid, dim3(256), 0, s, a, sh.pg,
                         sh.G, sh.Hq, sh.Hkv, scale_log2);
    else if (a.waves == 4)
      hipLaunchKernelGGL((attn_bf16_kernel<4, 2, PAGED>), grid, dim3(256), 0, s, a, sh.pg,
                         sh.G, sh.Hq, sh.Hkv, scale_log2);
    else if (a.waves == 1)
      hipLaunchKernelGGL((attn_bf16_kernel<1, 2, PAGED>), grid, dim3(64), 0, s, a, sh.pg,
                         sh.G, sh.Hq, sh.Hkv, scale_log2);
    else
      return hipErrorInvalidConfiguration;
    // a head with several splits is merged by its last split (merge_if_last),
    // except in the contiguous 12-wavefront build
    if (a.max_splits > 1 && a.waves == 12 && !PAGED)
      hipLaunchKernelGGL(combine_kernel<uint16_t>, cgrid, dim3(256), 0, s, a, sh.G, sh.Hq,
                         sh.Hkv, true);
  } else {
    switch (sh.G) {
      case 1: launch_f32<1, PAGED>(grid, s, a, sh, scale_log2); break;
      case 2: launch_f32<2, PAGED>(grid, s, a, sh, scale_log2); break;
      case 4: launch_f32<4, PAGED>(grid, s, a, sh, scale_log2); break;
      case 8: launch_f32<8, PAGED>(grid, s, a, sh, scale_log2); break;
      default: launch_f32<0, PAGED>(grid, s, a, sh, scale_log2); break;
    }
    if (a.merge_kernel && a.max_splits > 1)
      hipLaunchKernelGGL(combine_kernel<float>, cgrid, dim3(256), 0, s, a, sh.G, sh.Hq,
                         sh.Hkv, true);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const Shape& sh, const AttnLaunch& a, hipStream_t s) {
  return sh.pg.tables ? launch_attention_t<true>(sh, a, s) : launch_attention_t<false>(sh, a, s);
}

// Partials of the allocation-free attention entry point.  Every GPU the
// library runs on holds its own copy until the process ends.  In host code
// `scratch` names a host-side stand-in, not device memory: host code uses
// only the address scratch_address returns.
static __device__ __align__(256) float scratch[kNoAllocScratchBytes / sizeof(float)];

hipError_t scratch_address(void** out) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

}  // namespace ra
