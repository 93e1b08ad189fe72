// Random Attention eviction on gfx950: uniform per-head scores, selection of
// the dropped candidates, and the order-preserving in-place compaction.
//
// One workgroup owns one (sequence, layer, KV head) region for the whole
// event (Eq. 1 with Section 3's scores; Appendix F: per-KV-head eviction,
// keep-sets sorted chronologically, compaction by a gather):
//   1. every candidate slot (outside the prompt and the r most recent rows)
//      gets its 64-bit Philox score, held in registers (KPT per thread, in
//      slot order);
//   2. an MSB-first radix select over the composite (score, position)
//      finds the m = |C| - k_keep smallest (select.h);
//   3. a block scan turns the drop flags into the sorted drop list, stored as
//      f[k] = d_k - k, so that destination row j receives source row
//      j + #{k : f[k] <= j};
//   4. chronological layout (the paper's): the surviving rows are moved
//      down in chunks of destination rows (512 for bf16 with 1,024 threads):
//      every thread gathers its part of the chunk into registers, the block
//      waits until all loads have returned and synchronises, then writes.
//      Sources are never below destinations and a chunk's writes land below
//      the next chunk's sources, so the in-place move is race-free;
//      hole-fill layout: only the surviving rows of the last m slots move,
//      into the holes below the new length (order no longer chronological;
//      the positions travel with the rows).
#include "philox.h"
#include "ra_internal.h"
#include "select.h"

namespace ra {
namespace {

using u32x4 = uint32_t __attribute__((ext_vector_type(4)));

// Destination rows moved per barrier round: as many as give every thread 8
// key units and 8 value units of 16 bytes in flight (512 rows of bf16 or 256
// of fp32 for 1,024 threads).  Each round waits for all of its loads, so the
// bytes in flight per workgroup set the move's rate (rounds of 128 rows ran
// 9% slower on a full event of the Qwen3-14B shape).
template <int NT, typename E>
constexpr int chunk_rows() {
  return NT * 8 / (kHeadDim * static_cast<int>(sizeof(E)) / 16);
}

// Number of f[k] <= x for the non-decreasing list f[0..m).
__device__ __forceinline__ int count_le(const int* f, int m, int x) {
  int lo = 0, hi = m;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (f[mid] <= x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// The key whose m smallest values an event drops (ties by position).
// Random Attention: the per-head uniform draw of position p; the diagnostic
// policies of the paper change only this key (see ra_policy).
__device__ __forceinline__ uint64_t policy_key(int policy, int block, int p, int lp,
                                               int event, int layer, int g,
                                               uint64_t seed, uint64_t rid) {
  const uint64_t e = static_cast<uint64_t>(event);
  switch (policy) {
    case 1:   // shared draw: the same positions in every (layer, KV head)
      return philox_score(static_cast<uint64_t>(p), e, 0, 0, seed, rid);
    case 2: { // block-wise: every position takes the draw of its block's first
      const int first = lp + (p - lp) / block * block;
      return philox_score(static_cast<uint64_t>(first), e, static_cast<uint64_t>(layer),
                          static_cast<uint64_t>(g), seed, rid);
    }
    case 3:   // recency: drop the oldest
      return static_cast<uint64_t>(p);
    default:
      return philox_score(static_cast<uint64_t>(p), e, static_cast<uint64_t>(layer),
                          static_cast<uint64_t>(g), seed, rid);
  }
}

// The position whose draw scores position p under `policy`: the block-wise
// policy draws once per block of `block` positions from the prompt's end.
__device__ __forceinline__ int draw_position(int policy, int block, int p, int lp) {
  return policy == 2 ? lp + (p - lp) / block * block : p;
}

// Number of drops d_k (= f[k] + k, ascending) with d_k <= x.
__device__ __forceinline__ int count_le_slot(const int* f, int m, int x) {
  int lo = 0, hi = m;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (f[mid] + mid <= x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Nontemporal 16-byte load and store for the compaction's row moves: a key
// unit is read once and every destination unit written once per event.  The
// value units stay on ordinary loads: with a shift that is not a multiple of
// 8 rows each source tile is read by two destination tiles, and the second
// read is served from the cache.
template <typename E>
__device__ __forceinline__ u32x4 load_stream(const E* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

template <typename E>
__device__ __forceinline__ void store_stream(E* p, u32x4 x) {
  __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(p));
}

__device__ __forceinline__ int64_t vt_index(int64_t row, int ch) {
  // element index of (row, channel) in the transposed 8-row value tiles
  return (row & ~int64_t(7)) * kHeadDim + ch * 8 + (row & 7);
}

// Eight consecutive bf16 elements starting at element `off` of the 16
// elements a:b (two adjacent 8-row value tiles of one channel).
template <int OFF>
__device__ __forceinline__ u32x4 funnel_at(const uint32_t (&w)[8]) {
  u32x4 r;
  if constexpr (OFF % 2 == 0) {
    r.x = w[OFF / 2];
    r.y = w[OFF / 2 + 1];
    r.z = w[OFF / 2 + 2];
    r.w = w[OFF / 2 + 3];
  } else {
    constexpr int i = OFF / 2;
    r.x = __builtin_amdgcn_alignbyte(w[i + 1], w[i], 2);
    r.y = __builtin_amdgcn_alignbyte(w[i + 2], w[i + 1], 2);
    r.z = __builtin_amdgcn_alignbyte(w[i + 3], w[i + 2], 2);
    r.w = __builtin_amdgcn_alignbyte(w[i + 4], w[i + 3], 2);
  }
  return r;
}

__device__ __forceinline__ u32x4 funnel8(u32x4 a, u32x4 b, int off) {
  const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  switch (off) {
    case 0: return a;
    case 1: return funnel_at<1>(w);
    case 2: return funnel_at<2>(w);
    case 3: return funnel_at<3>(w);
    case 4: return funnel_at<4>(w);
    case 5: return funnel_at<5>(w);
    case 6: return funnel_at<6>(w);
    default: return funnel_at<7>(w);
  }
}

// Pool row of row j of the head being compacted: a contiguous region, or
// pages found through the sequence's block table, copied to LDS.
// Positions are indexed by pos_row(j) from the base the caller passes: the
// region's first position for a contiguous region, the pool's otherwise.
struct RegionRows {
  static constexpr bool kPaged = false;
  int64_t region;
  __device__ __forceinline__ int64_t operator()(int j) const { return region + j; }
  __device__ __forceinline__ int pos_row(int j) const { return j; }
  // region + a + b, added in that order (the 64-bit sum first keeps the
  // compaction within its 128 registers)
  __device__ __forceinline__ int64_t plus(int a, int b) const { return region + a + b; }
};

struct PagedRows {
  static constexpr bool kPaged = true;
  const int* table;        // LDS copy of the sequence's block table
  int64_t group_rows, head_off;
  int shift;
  __device__ __forceinline__ int64_t operator()(int j) const {
    return static_cast<int64_t>(table[j >> shift]) * group_rows + head_off +
           (j & ((1 << shift) - 1));
  }
  __device__ __forceinline__ int64_t pos_row(int j) const { return (*this)(j); }
  __device__ __forceinline__ int64_t plus(int a, int b) const { return (*this)(a + b); }
};

// Order-preserving in-place compaction of one head's region: destination
// row j < new_len (from the first drop d0 on) receives source row
// j + #{k : f[k] <= j}, where f[k] = d_k - k for the ascending drop list d.
// Chunks of chunk_rows<NT, E>() destination rows: every thread gathers its
// part of the chunk into registers, the block waits until all loads have
// returned and synchronises, then writes.  Sources are never below destinations and a
// chunk's writes land below the next chunk's sources, so the move is
// race-free.  Called by every thread of the workgroup.
template <int NT, typename E, bool POS_ONLY, typename Rows, bool MOVE_POS = true>
__device__ __forceinline__ void compact_rows(const int* f, int m, int* src_of, int d0,
                                             int new_len, int old_len, const Rows& row,
                                             E* __restrict__ kpool, E* __restrict__ vpool,
                                             int32_t* __restrict__ P) {
  constexpr bool PAGED = Rows::kPaged;
  constexpr int kEpu = 16 / sizeof(E);            // elements per 16-byte unit
  constexpr int kKUnitsRow = kHeadDim / kEpu;     // 16-byte units per key row
  constexpr int kVUnitsCh = 8 / kEpu;             // units per (tile, channel)
  constexpr int kChunk = chunk_rows<NT, E>();
  static_assert(kChunk % 8 == 0 && kChunk <= NT, "a chunk is whole value tiles, one row per thread");
  constexpr int kKUnits = kChunk * kKUnitsRow;
  constexpr int kVUnits = (kChunk / 8) * kHeadDim * kVUnitsCh;
  constexpr int kKPer = (kKUnits + NT - 1) / NT;
  constexpr int kVPer = (kVUnits + NT - 1) / NT;
  const int t = threadIdx.x;
  const E zero_e = E(0);
  for (int j0 = d0 & ~7; j0 < new_len; j0 += kChunk) {
    if (t < kChunk) src_of[t] = j0 + t + count_le(f, m, j0 + t);
    __syncthreads();

    int pval = 0;
    const bool pos_mine = MOVE_POS && t < kChunk && j0 + t >= d0 && j0 + t < new_len;
    if (pos_mine) pval = P[row.pos_row(src_of[t])];
    u32x4 kbuf[POS_ONLY ? 1 : kKPer];
    E vbuf[POS_ONLY ? 1 : kVPer][kEpu];
    if constexpr (!POS_ONLY) {
#pragma unroll
      for (int q = 0; q < kKPer; ++q) {
        const int u = t + q * NT;
        const int r = u / kKUnitsRow, col = u % kKUnitsRow;
        const int j = j0 + r;
        if (u < kKUnits && j >= d0 && j < new_len) {
          const E* src = kpool + row(src_of[r]) * kHeadDim + col * kEpu;
          kbuf[q] = load_stream(src);
        }
      }
#pragma unroll
      for (int q = 0; q < kVPer; ++q) {
        const int u = t + q * NT;
        const int tile = u / (kHeadDim * kVUnitsCh);
        const int rem = u % (kHeadDim * kVUnitsCh);
        const int ch = rem / kVUnitsCh, part = rem % kVUnitsCh;
        const int jt = j0 + tile * 8 + part * kEpu;
        if (u < kVUnits && j0 + tile * 8 < new_len) {
          const int s0 = src_of[jt - j0], s_last = src_of[jt + kEpu - 1 - j0];
          if (sizeof(E) == 2 && s_last - s0 == kEpu - 1 && s_last < old_len) {
            // no drop inside this destination tile: its 8 sources are
            // consecutive rows, i.e. one or two adjacent source tiles (the
            // offset is the same for the whole wavefront, so the branch and
            // the switch in funnel8 do not diverge)
            const E* a = vpool + vt_index(row(s0 & ~7), ch);
            const u32x4 va = *reinterpret_cast<const u32x4*>(a);
            const int off = s0 & 7;
            u32x4 vb = va;
            // the next tile may lie in another page of the paged layout
            if (off)
              vb = *reinterpret_cast<const u32x4*>(
                  PAGED ? vpool + vt_index(row((s0 & ~7) + 8), ch) : a + 8 * kHeadDim);
            const u32x4 r = funnel8(va, vb, off);
            __builtin_memcpy(vbuf[q], &r, 16);
          } else {
#pragma unroll
            for (int e = 0; e < kEpu; ++e) {
              const int sj = src_of[jt + e - j0];
              vbuf[q][e] = sj < old_len ? vpool[vt_index(row(sj), ch)] : zero_e;
            }
          }
        }
      }
    }
    // every load of this chunk has returned before any thread writes
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();

    if (pos_mine) P[row.pos_row(j0 + t)] = pval;
    if constexpr (!POS_ONLY) {
#pragma unroll
      for (int q = 0; q < kKPer; ++q) {
        const int u = t + q * NT;
        const int r = u / kKUnitsRow, col = u % kKUnitsRow;
        const int j = j0 + r;
        if (u < kKUnits && j >= d0 && j < new_len) {
          E* dst = kpool + row(j) * kHeadDim + col * kEpu;
          store_stream(dst, kbuf[q]);
        }
      }
#pragma unroll
      for (int q = 0; q < kVPer; ++q) {
        const int u = t + q * NT;
        const int tile = u / (kHeadDim * kVUnitsCh);
        const int rem = u % (kHeadDim * kVUnitsCh);
        const int ch = rem / kVUnitsCh, part = rem % kVUnitsCh;
        if (u < kVUnits && j0 + tile * 8 < new_len) {
          E* dst = vpool + vt_index(row.plus(j0, tile * 8), ch) + part * kEpu;
          u32x4 w;
          __builtin_memcpy(&w, vbuf[q], 16);
          store_stream(dst, w);
        }
      }
    }
  }
}

// LAYOUT: 0 chronological, 1 hole-fill, 2 chronological in pages.
template <int NT, int KPT, typename E, bool POS_ONLY, int LAYOUT>
__global__ __launch_bounds__(NT) void evict_kernel(
    const SeqMeta* __restrict__ meta, E* __restrict__ kpool,
    E* __restrict__ vpool, int32_t* __restrict__ pos, int L, int Hkv, int r,
    int slot_lo, int policy, int block, Paging pg, int32_t* __restrict__ drops_out,
    int drop_stride) {
  constexpr bool PAGED = LAYOUT == 2;
  static_assert(KPT <= 32, "drop flags live in one 32-bit mask");
  __shared__ SelectShared sel_sh;
  __shared__ int f[kMaxEvery];

  const int per_seq = L * Hkv;
  const int slot = slot_lo + static_cast<int>(blockIdx.x) / per_seq;
  const int lg = static_cast<int>(blockIdx.x) % per_seq;
  const int layer = lg / Hkv, g = lg % Hkv;
  const SeqMeta& Mref = meta[slot];
  if (!Mref.active || !Mref.due) return;
  const int lp = Mref.prompt_len, old_len = Mref.plan_len;
  const int event = Mref.plan_event;
  const uint64_t seed = Mref.seed, rid = Mref.rid;
  const int C = old_len - lp - r;          // candidates: every cached position
  const int m = C - Mref.k_keep;           // outside the prompt and the r most
  if (m <= 0) return;                      // recent ones (positions < thr)
  const int thr = lp + Mref.step - r;
  const int new_len = old_len - m;
  // slots that can hold candidates: all of them in the chronological layouts
  // are [lp, old_len - r); after hole-fill events the recent rows may sit
  // anywhere above the prompt, so every slot from lp is examined
  const int span = LAYOUT == 1 ? old_len - lp : C;
  const int64_t region = Mref.base + static_cast<int64_t>(lg) * Mref.cap;
  int32_t* P = pos + region;     // contiguous layouts
  const int t = threadIdx.x;
  // paged: the sequence's block table, read once into LDS
  __shared__ int tbl[PAGED ? kMaxPagesLds : 1];
  PagedRows prow{};
  if constexpr (PAGED) {
    const int32_t* table = pg.tables + static_cast<int64_t>(slot) * pg.pages_per_seq;
    const int n_pages = (old_len + (1 << pg.page_shift) - 1) >> pg.page_shift;
    for (int i = t; i < n_pages; i += NT) tbl[i] = table[i];
    __syncthreads();
    prow = PagedRows{tbl, pg.group_rows, static_cast<int64_t>(lg) << pg.page_shift,
                     pg.page_shift};
  }

  // 1. scores of this thread's KPT consecutive slots; ties by position
  uint64_t score[KPT];
  uint32_t tie[KPT];
  uint32_t valid = 0;
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int c = t * KPT + i;
    score[i] = 0;
    tie[i] = 0;
    if (c < span) {
      int p;
      if constexpr (PAGED) p = pos[prow(lp + c)];
      else p = P[lp + c];
      // every slot's position is kept (not only the candidates'): the
      // positions-only compaction below writes the survivors from here
      tie[i] = static_cast<uint32_t>(p);
      if (p < thr) {
        // the largest builds draw per candidate as it is read
        if (KPT > 9) score[i] = policy_key(policy, block, p, lp, event, layer, g, seed, rid);
        valid |= 1u << i;
      }
    }
  }
  if (KPT <= 9) {
    // The keys of every slot (a slot that is no candidate keeps a zero key,
    // which the selection ignores), three Philox blocks in lockstep: their
    // independent rounds interleave, where one conditional draw per candidate
    // runs each 10-round chain of dependent multiplies on its own.  The
    // policy is the same for the whole workgroup.
    if (policy == 3) {
#pragma unroll
      for (int i = 0; i < KPT; ++i)
        score[i] = (valid >> i) & 1 ? policy_key(3, block, static_cast<int>(tie[i]), lp, event,
                                                 layer, g, seed, rid)
                                    : 0;
    } else {
      int q[KPT];
#pragma unroll
      for (int i = 0; i < KPT; ++i) q[i] = static_cast<int>(tie[i]);
      if (policy == 2) {
#pragma unroll
        for (int i = 0; i < KPT; ++i) q[i] = draw_position(2, block, q[i], lp);
      }
      const uint64_t dl = policy == 1 ? 0 : static_cast<uint64_t>(layer);
      const uint64_t dg = policy == 1 ? 0 : static_cast<uint64_t>(g);
      constexpr int kWays = 3;
#pragma unroll
      for (int i0 = 0; i0 < KPT; i0 += kWays) {
        uint64_t b[kWays], w[kWays][4];
#pragma unroll
        for (int j = 0; j < kWays; ++j)
          b[j] = i0 + j < KPT ? static_cast<uint64_t>(q[i0 + j] >> 2) : 0;
        philox_blocks<kWays>(b, static_cast<uint64_t>(event), dl, dg, seed, rid, w);
#pragma unroll
        for (int j = 0; j < kWays; ++j) {
          if (i0 + j < KPT) {
            // word k of the block, by masks (a select chain becomes branches)
            const int i = i0 + j, k = q[i] & 3;
            uint64_t x = 0;
#pragma unroll
            for (int n = 0; n < 4; ++n) x |= w[j][n] & (0ull - static_cast<uint64_t>(k == n));
            score[i] = x & (0ull - static_cast<uint64_t>((valid >> i) & 1));
          }
        }
      }
    }
  }

  // 2. radix select of the m smallest (score, position); 3. drop list
  const uint32_t drop = select_smallest<NT, KPT, 64>(score, tie, valid, m, sel_sh);
  const int drops_below = drop_list<NT, KPT>(drop, lp, f, sel_sh);
  const int d0 = f[0];
  // deferred row moves: this head's drop slots, ascending, for the next
  // step's attention (rows are left in place by a positions-only event)
  if (drops_out) {
    int32_t* dst = drops_out + (static_cast<int64_t>(slot) * per_seq + lg) * drop_stride;
    for (int k = t; k < m; k += NT) dst[k] = f[k] + k;
  }

  if constexpr (LAYOUT == 1) {
    // hole-fill: the h holes below new_len take the h surviving rows of the
    // tail [new_len, old_len), in ascending order; nothing else moves
    __shared__ int mv_src[kMaxEvery];
    __shared__ int mv_dst[kMaxEvery];
    __shared__ int n_holes;
    if (t == 0) n_holes = count_le_slot(f, m, new_len - 1);
    __syncthreads();
    const int h = n_holes;
    for (int i = t; i < m; i += NT) {
      const int s = new_len + i;                 // tail slot
      const int before = count_le_slot(f, m, s - 1) - h;   // tail drops below s
      const bool dropped = h + before < m && f[h + before] + h + before == s;
      if (!dropped) {
        const int j = i - before;                // rank among tail survivors
        mv_src[j] = s;
        mv_dst[j] = f[j] + j;
      }
    }
    __syncthreads();
    for (int j = t; j < h; j += NT) P[mv_dst[j]] = P[mv_src[j]];
    if constexpr (!POS_ONLY) {
      constexpr int kUnitsRow = kHeadDim * sizeof(E) / 16;
      for (int idx = t; idx < h * kUnitsRow; idx += NT) {
        const int j = idx / kUnitsRow, col = idx % kUnitsRow;
        *reinterpret_cast<u32x4*>(kpool + (region + mv_dst[j]) * kHeadDim + col * (16 / sizeof(E))) =
            *reinterpret_cast<const u32x4*>(kpool + (region + mv_src[j]) * kHeadDim +
                                            col * (16 / sizeof(E)));
      }
      for (int idx = t; idx < h * kHeadDim; idx += NT) {
        const int j = idx / kHeadDim, ch = idx % kHeadDim;
        vpool[vt_index(region + mv_dst[j], ch)] = vpool[vt_index(region + mv_src[j], ch)];
      }
    }
    return;
  }

  // 4. order-preserving in-place compaction of positions, keys and values
  __shared__ int src_of[chunk_rows<NT, E>()];
  if constexpr (POS_ONLY) {
    // Positions only: every slot below old_len - r was read into tie[] before
    // the selection's barriers, so each survivor among them goes straight to
    // its compacted slot (its slot less the drops below it), with no read of
    // the region after those barriers.  Only the r most recent rows, above
    // every candidate, take the chunked move: their sources lie above every
    // destination written here.
    int k = drops_below;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = t * KPT + i;
      if (c < span) {
        if ((drop >> i) & 1) {
          ++k;
        } else if (k) {
          if constexpr (PAGED) pos[prow(lp + c - k)] = static_cast<int32_t>(tie[i]);
          else P[lp + c - k] = static_cast<int32_t>(tie[i]);
        }
      }
    }
    if (r > 0) {
      if constexpr (PAGED)
        compact_rows<NT, E, true>(f, m, src_of, new_len - r, new_len, old_len, prow, kpool,
                                  vpool, pos);
      else
        compact_rows<NT, E, true>(f, m, src_of, new_len - r, new_len, old_len,
                                  RegionRows{region}, kpool, vpool, P);
    }
    return;
  }
  if constexpr (PAGED)
    compact_rows<NT, E, POS_ONLY>(f, m, src_of, d0, new_len, old_len, prow, kpool, vpool, pos);
  else
    compact_rows<NT, E, POS_ONLY>(f, m, src_of, d0, new_len, old_len, RegionRows{region},
                                  kpool, vpool, P);
}

// Compaction of a score-based round: each due head's drop list comes from
// `drops` (ascending slot indices, `stride` per head, head index =
// (slot - slot_lo) * L * Hkv + layer * Hkv + g); the state kernels have
// already set len to the new length and plan_len to the old one.
template <int NT, typename E>
__global__ __launch_bounds__(NT) void compact_drops_kernel(
    const SeqMeta* __restrict__ meta, E* __restrict__ kpool, E* __restrict__ vpool,
    int32_t* __restrict__ pos, const int32_t* __restrict__ drops, int stride, int L,
    int Hkv, int slot_lo) {
  __shared__ int f[kMaxEvery];
  __shared__ int src_of[chunk_rows<NT, E>()];
  const int per_seq = L * Hkv;
  const int slot = slot_lo + static_cast<int>(blockIdx.x) / per_seq;
  const int lg = static_cast<int>(blockIdx.x) % per_seq;
  const SeqMeta& M = meta[slot];
  if (!M.active || !M.due) return;
  const int old_len = M.plan_len, new_len = M.len, m = old_len - new_len;
  if (m <= 0 || m > stride) return;
  const int32_t* d = drops + static_cast<int64_t>(blockIdx.x) * stride;
  for (int k = threadIdx.x; k < m; k += NT) f[k] = d[k] - k;
  __syncthreads();
  const int64_t region = M.base + static_cast<int64_t>(lg) * M.cap;
  compact_rows<NT, E, false>(f, m, src_of, f[0], new_len, old_len, RegionRows{region}, kpool,
                             vpool, pos + region);
}

// Key/value rows of a deferred event (contiguous chronological layout): the
// event compacted the positions and recorded each head's drop slots; the
// rows move here, for sequences whose next attention did not move them.
template <int NT, typename E>
__global__ __launch_bounds__(NT) void move_pending_kernel(
    const SeqMeta* __restrict__ meta, E* __restrict__ kpool, E* __restrict__ vpool,
    const int32_t* __restrict__ drops, int stride, int L, int Hkv, int slot_lo) {
  __shared__ int f[kMaxEvery];
  __shared__ int src_of[chunk_rows<NT, E>()];
  const int per_seq = L * Hkv;
  const int slot = slot_lo + static_cast<int>(blockIdx.x) / per_seq;
  const int lg = static_cast<int>(blockIdx.x) % per_seq;
  const SeqMeta& M = meta[slot];
  if (!M.active || M.due != kDueMovePending) return;
  const int old_len = M.plan_len, new_len = M.len, m = old_len - new_len;
  if (m <= 0 || m > stride) return;
  const int32_t* d = drops + (static_cast<int64_t>(slot) * per_seq + lg) * stride;
  for (int k = threadIdx.x; k < m; k += NT) f[k] = d[k] - k;
  __syncthreads();
  const int64_t region = M.base + static_cast<int64_t>(lg) * M.cap;
  compact_rows<NT, E, false, RegionRows, false>(f, m, src_of, f[0], new_len, old_len,
                                                RegionRows{region}, kpool, vpool, nullptr);
}

template <int NT, int KPT, bool POS_ONLY, int LAYOUT>
hipError_t launch_layout(const Shape& sh, const SeqMeta* meta, void* kpool,
                         void* vpool, int32_t* pos, int slot_lo, int slot_hi,
                         hipStream_t s, int32_t* drops_out, int drop_stride) {
  const dim3 grid((slot_hi - slot_lo) * sh.L * sh.Hkv);
  if (sh.dtype == 1) {
    hipLaunchKernelGGL((evict_kernel<NT, KPT, uint16_t, POS_ONLY, LAYOUT>), grid,
                       dim3(NT), 0, s, meta, static_cast<uint16_t*>(kpool),
                       static_cast<uint16_t*>(vpool), pos, sh.L, sh.Hkv, sh.r,
                       slot_lo, sh.policy, sh.block, sh.pg, drops_out, drop_stride);
  } else {
    hipLaunchKernelGGL((evict_kernel<NT, KPT, float, POS_ONLY, LAYOUT>), grid,
                       dim3(NT), 0, s, meta, static_cast<float*>(kpool),
                       static_cast<float*>(vpool), pos, sh.L, sh.Hkv, sh.r,
                       slot_lo, sh.policy, sh.block, sh.pg, drops_out, drop_stride);
  }
  return hipGetLastError();
}

template <int NT, int KPT, bool POS_ONLY>
hipError_t launch_kpt(const Shape& sh, const SeqMeta* meta, void* kpool,
                      void* vpool, int32_t* pos, int slot_lo, int slot_hi,
                      hipStream_t s, int32_t* drops_out, int drop_stride) {
  if (sh.layout == 1)
    return launch_layout<NT, KPT, POS_ONLY, 1>(sh, meta, kpool, vpool, pos, slot_lo,
                                               slot_hi, s, drops_out, drop_stride);
  if (sh.layout == 2)
    return launch_layout<NT, KPT, POS_ONLY, 2>(sh, meta, kpool, vpool, pos, slot_lo,
                                               slot_hi, s, drops_out, drop_stride);
  return launch_layout<NT, KPT, POS_ONLY, 0>(sh, meta, kpool, vpool, pos, slot_lo,
                                             slot_hi, s, drops_out, drop_stride);
}

template <bool POS_ONLY>
hipError_t launch_mode(const Shape& sh, const SeqMeta* meta, void* kpool,
                       void* vpool, int32_t* pos, int slot_lo, int slot_hi,
                       int max_candidates, hipStream_t s, int32_t* drops_out,
                       int drop_stride) {
  // 1,024 threads, KPT scores each: the smallest KPT that holds the
  // candidates (C = K + 64 at the usual budgets: K = 1,024 -> 2, 2,048 -> 3,
  // 4,096 -> 5, 8,192 -> 9).  More than 16 scores per thread is kept for the
  // largest budgets only: 32 unrolled Philox evaluations exceed the
  // compiler's unroll budget and the score array then lives in scratch memory.
  if (max_candidates <= 1024 * 1)
    return launch_kpt<1024, 1, POS_ONLY>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi, s, drops_out, drop_stride);
  if (max_candidates <= 1024 * 2)
    return launch_kpt<1024, 2, POS_ONLY>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi, s, drops_out, drop_stride);
  if (max_candidates <= 1024 * 3)
    return launch_kpt<1024, 3, POS_ONLY>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi, s, drops_out, drop_stride);
  if (max_candidates <= 1024 * 5)
    return launch_kpt<1024, 5, POS_ONLY>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi, s, drops_out, drop_stride);
  if (max_candidates <= 1024 * 9)
    return launch_kpt<1024, 9, POS_ONLY>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi, s, drops_out, drop_stride);
  if (max_candidates <= 1024 * 16)
    return launch_kpt<1024, 16, POS_ONLY>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi, s, drops_out, drop_stride);
  if (max_candidates <= kMaxCandidates)
    return launch_kpt<1024, 32, POS_ONLY>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi, s, drops_out, drop_stride);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_compact_drops(const Shape& sh, const SeqMeta* meta, void* kpool,
                                void* vpool, int32_t* pos, const int32_t* drops,
                                int stride, int slot_lo, int slot_hi, hipStream_t s) {
  if (slot_hi <= slot_lo) return hipSuccess;
  const dim3 grid((slot_hi - slot_lo) * sh.L * sh.Hkv);
  if (sh.dtype == 1)
    hipLaunchKernelGGL((compact_drops_kernel<1024, uint16_t>), grid, dim3(1024), 0, s, meta,
                       static_cast<uint16_t*>(kpool), static_cast<uint16_t*>(vpool), pos,
                       drops, stride, sh.L, sh.Hkv, slot_lo);
  else
    hipLaunchKernelGGL((compact_drops_kernel<1024, float>), grid, dim3(1024), 0, s, meta,
                       static_cast<float*>(kpool), static_cast<float*>(vpool), pos,
                       drops, stride, sh.L, sh.Hkv, slot_lo);
  return hipGetLastError();
}

hipError_t launch_evict(const Shape& sh, const SeqMeta* meta, void* kpool,
                        void* vpool, int32_t* pos, int slot_lo, int slot_hi,
                        int max_candidates, bool positions_only,
                        hipStream_t s, int32_t* drops_out, int drop_stride) {
  if (slot_hi <= slot_lo) return hipSuccess;
  if (positions_only)
    return launch_mode<true>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi,
                             max_candidates, s, drops_out, drop_stride);
  return launch_mode<false>(sh, meta, kpool, vpool, pos, slot_lo, slot_hi,
                            max_candidates, s, drops_out, drop_stride);
}

hipError_t launch_flush_pending(const Shape& sh, SeqMeta* meta, void* kpool, void* vpool,
                                const int32_t* drops, int drop_stride, int slot_lo,
                                int slot_hi, hipStream_t s) {
  if (slot_hi <= slot_lo) return hipSuccess;
  const dim3 grid((slot_hi - slot_lo) * sh.L * sh.Hkv);
  if (sh.dtype == 1)
    hipLaunchKernelGGL((move_pending_kernel<1024, uint16_t>), grid, dim3(1024), 0, s, meta,
                       static_cast<uint16_t*>(kpool), static_cast<uint16_t*>(vpool), drops,
                       drop_stride, sh.L, sh.Hkv, slot_lo);
  else
    hipLaunchKernelGGL((move_pending_kernel<1024, float>), grid, dim3(1024), 0, s, meta,
                       static_cast<float*>(kpool), static_cast<float*>(vpool), drops,
                       drop_stride, sh.L, sh.Hkv, slot_lo);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_clear_pending(meta, slot_lo, slot_hi, s);
}

}  // namespace ra
