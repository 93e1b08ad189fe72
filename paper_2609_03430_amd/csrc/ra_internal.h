// Internal definitions shared by the host library and the HIP kernels.
//
// HBM layout (one ra_cache):
//   K pool  [pool_rows][128]          row-major rows, dtype E
//   V pool  [pool_rows / 8][128][8]   tiles of 8 rows stored transposed, so a
//                                     16-byte load holds 8 consecutive rows of
//                                     one channel (the MFMA operand shape of
//                                     the P.V product)
//   pos     [pool_rows]               int32 token position of each row
// Contiguous layouts: a sequence owns L * Hkv consecutive regions of `cap`
// rows (cap a multiple of 32); region (l, g) starts at row base + (l * Hkv +
// g) * cap.  Rows [0, len) of a region are cached, in chronological order
// (or, in the hole-fill layout, in no particular order).
// Paged layout: the pool is a sequence of page groups of L * Hkv pages of
// page_rows rows each (page (l, g) of group p starts at row (p * L * Hkv +
// l * Hkv + g) * page_rows).  A sequence's block table lists its groups in
// order; row j of its head (l, g) lives in page (l, g) of group table[j /
// page_rows], at offset j mod page_rows.  Every head of a sequence holds the
// same number of rows, so one table serves all of them.  Rows stay in
// chronological order across the pages.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ra {

constexpr int kHeadDim = 128;
constexpr int kMaxGroup = 16;       // query heads per KV head (MFMA N tile)
constexpr int kMaxSplits = 64;      // attention work items per head
constexpr int kMaxEvery = 1024;     // evict_every limit: drops per event <= this
constexpr int kMaxCandidates = 32768;
constexpr int kRegionAlign = 32;    // region rows rounded to the key block
constexpr int kMaxPagesLds = 4096;  // paged layout: block-table entries per sequence

// Per-slot device state, 64 bytes.  The hot-path kernels read it; the
// end-of-step and plan kernels update it; the host keeps an identical mirror.
struct SeqMeta {
  int64_t base;        // first pool row of the sequence's regions
  int32_t cap;         // rows per (layer, KV head) region
  int32_t prompt_len;  // lp
  int32_t len;         // cached rows per region between steps
  int32_t step;        // completed decode steps
  int32_t event;       // eviction events performed
  int32_t k_keep;      // evictable rows kept per head
  uint64_t seed;       // Philox key word 0
  uint64_t rid;        // Philox key word 1 (request id)
  int32_t active;
  int32_t due;         // 1: an eviction is planned for this sequence;
                       // kDueMovePending: its positions are compacted and the
                       // next step's attention moves its key/value rows
  int32_t plan_len;    // rows per region before the planned eviction
  int32_t plan_event;  // event index of the planned eviction
};
static_assert(sizeof(SeqMeta) == 64, "SeqMeta must stay 64 bytes");
constexpr int kDueMovePending = 2;

// Block tables of the paged layout (null tables: a contiguous layout).
struct Paging {
  const int32_t* tables = nullptr;  // [max_seqs][pages_per_seq] page groups
  int pages_per_seq = 0;            // table entries per sequence
  int page_shift = 0;               // log2(page_rows)
  int64_t group_rows = 0;           // rows of one page group: L * Hkv * page_rows
};

struct Shape {
  int L, Hq, Hkv, G, r, every, dtype;  // dtype: 0 f32, 1 bf16
  int layout;                          // 0 chronological, 1 hole-fill, 2 paged
  int policy;                          // ra_policy
  int block;                           // tokens per block (block policy)
  Paging pg;                           // the paged layout's tables
};

// Pool row of row j of one (sequence, layer, KV head) cache.
struct RowMap {
  int64_t region;          // contiguous: first pool row of the head's region
  const int32_t* table;    // paged: the sequence's block table
  int64_t group_rows;      // paged: rows of one page group
  int64_t head_off;        // paged: (layer * Hkv + g) * page_rows
  int page_shift;          // paged: log2(page_rows)
};

__device__ __host__ inline RowMap row_map(const SeqMeta& M, int slot, int lg, const Paging& pg) {
  RowMap m;
  m.region = M.base + static_cast<int64_t>(lg) * M.cap;
  m.table = pg.tables ? pg.tables + static_cast<int64_t>(slot) * pg.pages_per_seq : nullptr;
  m.group_rows = pg.group_rows;
  m.head_off = static_cast<int64_t>(lg) << pg.page_shift;
  m.page_shift = pg.page_shift;
  return m;
}

template <bool PAGED>
__device__ __forceinline__ int64_t pool_row(const RowMap& m, int j) {
  if constexpr (PAGED) {
    const int64_t page = m.table[j >> m.page_shift];
    return page * m.group_rows + m.head_off + (j & ((1 << m.page_shift) - 1));
  } else {
    return m.region + j;
  }
}

// ---- launch wrappers (defined in the .hip files) ----------------------------

hipError_t launch_zero_words(uint32_t* p, int64_t n_words, hipStream_t s);
hipError_t launch_seq_set(SeqMeta* meta, int slot, const SeqMeta& v, hipStream_t s);
hipError_t launch_advance(SeqMeta* meta, int slot_lo, int slot_hi, int n_steps,
                          int r, int every, hipStream_t s);
hipError_t launch_plan_now(SeqMeta* meta, int slot, int r, hipStream_t s);
hipError_t launch_append_positions(const Shape& sh, const SeqMeta* meta, int32_t* pos,
                                   int slot_lo, int slot_hi, int run, hipStream_t s);
hipError_t launch_evict(const Shape& sh, const SeqMeta* meta, void* kpool,
                        void* vpool, int32_t* pos, int slot_lo, int slot_hi,
                        int max_candidates, bool positions_only, hipStream_t s,
                        int32_t* drops_out = nullptr, int drop_stride = 0);
// Deferred row moves: the drop lists of the last event, [max_seqs][L][Hkv]
// [drop_stride] int32 (ascending slots), written by a positions-only event.
// launch_mark_pending turns due == 1 into kDueMovePending for the active
// slots of [lo, hi); launch_flush_pending moves the key/value rows of every
// pending sequence (positions are already in place) and clears the flag.
hipError_t launch_mark_pending(SeqMeta* meta, int slot_lo, int slot_hi, hipStream_t s);
hipError_t launch_clear_pending(SeqMeta* meta, int slot_lo, int slot_hi, hipStream_t s);
hipError_t launch_flush_pending(const Shape& sh, SeqMeta* meta, void* kpool, void* vpool,
                                const int32_t* drops, int drop_stride, int slot_lo,
                                int slot_hi, hipStream_t s);
// Rows [0, len) of every head of slot `slot` (host mirror M) from row-major
// sources [L * Hkv][len][128] (positions: pos_src, or 0..len-1 if null).
hipError_t launch_write_rows(const Shape& sh, const SeqMeta& M, int slot, int len,
                             const void* k_src, const void* v_src,
                             const int32_t* pos_src, void* kpool, void* vpool,
                             int32_t* pos, hipStream_t s);
// Rows [0, len) of head lg = layer * Hkv + g of slot `slot` to row-major outputs.
hipError_t launch_read_rows(const Shape& sh, const SeqMeta& M, int slot, int lg, int len,
                            const void* kpool, const void* vpool, void* k_out,
                            void* v_out, hipStream_t s);
// Positions of rows [0, len) of every head of slot `slot`: [L * Hkv][len].
hipError_t launch_export_positions(const Shape& sh, const SeqMeta& M, int slot, int len,
                                   const int32_t* pos, int32_t* out, hipStream_t s);

// Paged layout: table entries set by the host (slot, index, page group).
struct TableEntry {
  int32_t slot, index, group;
};
constexpr int kTableBatch = 64;   // entries per table-update launch
hipError_t launch_table_set(const Shape& sh, const TableEntry* entries, int n,
                            hipStream_t s);

struct AttnLaunch {
  const SeqMeta* meta;
  void* kpool;
  void* vpool;
  int32_t* pos;
  const void* q;
  const void* k_new;
  const void* v_new;
  void* out;
  float* ws_o;         // [heads][split_stride][G][128] partial numerators
  float* ws_ml;        // [heads][split_stride][G][2]  running max (log2), sum
  int split_stride;    // partial slots per head (>= max_splits)
  int layer;
  int max_seqs;
  int split_keys;
  int max_splits;
  int waves;           // wavefronts per work item (bf16 path: 1, 4, 8 or 12)
  int wide_regs;       // bf16, 4 wavefronts: the build for one wavefront per SIMD
  // some sequence has a deferred row move (bf16, one split per head): the
  // launch runs the kernel that moves rows while it attends
  int move;
  // fp32: heads of several splits are merged by a merge kernel launched after
  // the attention (1) instead of by their last split (0)
  int merge_kernel;
  const int32_t* drops;  // the deferred drop lists (see launch_evict)
  int drop_stride;
  // bf16: per (slot, KV head) count of the splits done this launch, zero
  // between launches (the last split resets it after merging)
  int* arrivals;
};
hipError_t launch_attention(const Shape& sh, const AttnLaunch& a, hipStream_t s);

// The allocation-free attention's partials: a file-scope device array of
// kNoAllocScratchBytes (attention.hip).  scratch_address returns its device
// address on the current device, looked up once per device.
constexpr size_t kNoAllocScratchBytes = size_t(8) << 20;
hipError_t scratch_address(void** out);

// Score-based rounds (measurement only): compaction from given drop lists,
// and the plan rule applied to a slot range.
hipError_t launch_compact_drops(const Shape& sh, const SeqMeta* meta, void* kpool,
                                void* vpool, int32_t* pos, const int32_t* drops,
                                int stride, int slot_lo, int slot_hi, hipStream_t s);
hipError_t launch_plan_range(SeqMeta* meta, int slot_lo, int slot_hi, int r, hipStream_t s);
// R-KV (scorer 1) or VaSE (scorer 2) selection from raw window scores (scored.hip).
hipError_t launch_scored_select(const Shape& sh, int scorer, const SeqMeta* meta,
                                const void* kpool, const void* vpool, const int32_t* pos,
                                const float* raw_scores, float* cbar_scratch,
                                int score_stride, int32_t* drops, int slot_lo, int slot_hi,
                                int max_len, float lambda, float threshold, int recent_dups,
                                int n_large, uint64_t seed, hipStream_t s);

// Observation-window scorer (measurement only, window_score.hip).
hipError_t launch_window_score(const Shape& sh, const SeqMeta* meta, const void* kpool,
                               const int32_t* pos, const void* qwin, float* scores_out,
                               int32_t* drops_out, int scores_stride, int slot_lo,
                               int slot_hi, int max_len, hipStream_t s);

}  // namespace ra
