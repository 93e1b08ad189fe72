/*
 * randattn.h -- C ABI of the Random Attention decode hot path on MI355X.
 *
 * Random Attention (Section 3 of the paper) keeps, per KV head, the prompt
 * and the r most recent pairs, and evicts the other cached pairs uniformly
 * at random down to a budget, with no scoring pass.  This library holds the
 * compressed per-KV-head cache in caller-owned device memory and exposes the
 * three operations of the problem statement:
 *   - append one key/value pair per decode step (Section 2, periodic
 *     eviction paragraph: each decode step appends one pair);
 *   - evict per KV head to the budget, reproducibly from a per-request seed
 *     (Eq. 1; Section 3; Appendix F; Appendix H "Statistics and randomness");
 *   - grouped-query decode attention over the kept pairs (Section 2,
 *     "Notation"; Appendix F: query groups share their KV head's keep-set).
 *
 * Conventions for every call
 * --------------------------
 * - Pointers named dev_* / pools / q / out / workspace are DEVICE pointers
 *   (hipMalloc or torch CUDA tensors, 16-byte aligned); pointers named
 *   host_* are host memory.  `stream` is a hipStream_t passed as void*
 *   (NULL = the null stream).  All calls are asynchronous on `stream` unless
 *   marked synchronous.
 * - The library never allocates device memory.  The caller owns the pools,
 *   the metadata buffer and the workspace and must keep them alive until
 *   ra_cache_destroy.  (The one fixed device array the library holds, that
 *   of ra_decode_attention_noalloc, comes with its code object.)  One
 *   ra_cache must be driven from one stream (calls are stream-ordered); it
 *   is not thread-safe.
 * - Every call returns an ra_status.  Shapes, capacities, budgets and the
 *   step protocol are validated on the host mirror BEFORE any launch, so an
 *   error leaves device state untouched.  A failed launch returns
 *   RA_ERR_HIP (ra_last_hip_error gives the hipError_t); after RA_ERR_HIP
 *   from a call that launches several kernels (ra_seq_begin, a paged or
 *   move-carrying ra_decode_attention, ra_end_step, ra_evict_now,
 *   ra_fast_forward, ra_seq_fast_forward, ra_scored_evict) the host mirror
 *   and the device state may disagree, and the cache should be destroyed.
 *   Nothing throws across the ABI.
 * - head_dim must be 128; dtype f32 or bf16 (keys, values, queries and
 *   outputs all in that dtype); positions are int32.
 *
 * Eviction rule (what the kernels compute; the CPU oracle restates it)
 * -----------------------------------------------------------------
 * A sequence's prompt positions 0..lp-1 are never evicted.  Decode step t
 * (1-based) caches position lp+t-1 in every (layer, KV head).  At the end
 * of step t, if t mod evict_every == 0 and the entries outside prompt and
 * recent buffer exceed k_keep, eviction event e (0-based count per
 * sequence) runs in every (layer l, KV head g): the candidates are the
 * cached positions outside the prompt and the r most recent; each candidate
 * p gets the 64-bit uniform key = word (p mod 4) of Philox4x64-10 at counter
 * (p/4, e, l, g) with key (seed, request_id); the m = |C| - k_keep smallest
 * (key, p) pairs are dropped and the survivors are compacted in place,
 * chronological order kept.  k_keep = budget_k (RA_BUDGET_EVICTABLE) or
 * budget_k - lp (RA_BUDGET_TOTAL, the convention of Eq. 1, where the
 * prompt counts against K).  The diagnostic policies of ra_policy change
 * only the key: the shared draw uses counter (p/4, e, 0, 0); the block
 * policy uses the key of s = lp + policy_block * floor((p - lp) /
 * policy_block) in place of that of p; recency uses p itself.
 */
#ifndef RANDATTN_H
#define RANDATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RA_OK = 0,
  RA_ERR_INVALID_ARG = -1,  /* bad pointer, index, shape or config field */
  RA_ERR_CAPACITY = -2,     /* pool full, or a head region would overflow */
  RA_ERR_BUDGET = -3,       /* TOTAL mode and the prompt exceeds budget_k */
  RA_ERR_UNSUPPORTED = -4,  /* valid but not implemented (head_dim, group) */
  RA_ERR_HIP = -5,          /* a HIP call or kernel launch failed */
  RA_ERR_STATE = -6         /* call out of protocol order for this state */
} ra_status;

typedef enum { RA_F32 = 0, RA_BF16 = 1 } ra_dtype;

typedef enum {
  RA_BUDGET_EVICTABLE = 0,  /* budget_k counts kept non-prompt, non-buffer rows */
  RA_BUDGET_TOTAL = 1       /* budget_k counts the prompt too (Eq. 1) */
} ra_budget_mode;

typedef struct {
  int32_t num_layers;     /* L >= 1 */
  int32_t num_q_heads;    /* Hq, a multiple of Hkv */
  int32_t num_kv_heads;   /* Hkv >= 1; group G = Hq / Hkv, G <= 16;
                             L * Hkv <= 65536 (RA_ERR_UNSUPPORTED beyond) */
  int32_t head_dim;       /* d; must be 128 */
  int32_t budget_k;       /* K >= 0 (see budget_mode) */
  int32_t recent_r;       /* r >= 0: the buffer of most recent pairs (64) */
  int32_t evict_every;    /* R in [1, 1024]: trigger period in steps (64) */
  int32_t budget_mode;    /* ra_budget_mode */
  int32_t dtype;          /* ra_dtype */
  int32_t max_seqs;       /* sequence slots, [1, 65536] */
  int32_t attn_split;     /* keys per attention work item (multiple of 32),
                             0 = chosen by the library */
  int32_t layout;         /* ra_layout: row order kept in each region */
  int32_t policy;         /* ra_policy: which candidates an eviction keeps */
  int32_t policy_block;   /* RA_POLICY_BLOCK: tokens per block (>= 1) */
  int32_t page_rows;      /* RA_LAYOUT_PAGED: rows per page, a power of two in
                             [32, 1024] (ignored by the other layouts) */
  int32_t max_prompt_len; /* RA_LAYOUT_PAGED: longest prompt ra_seq_begin
                             accepts; sizes the block tables (ignored by the
                             other layouts) */
} ra_config;

typedef enum {
  RA_LAYOUT_CHRONOLOGICAL = 0, /* rows in position order; an eviction shifts every
                                  survivor after the first drop (Appendix F: keep
                                  sets sorted chronologically, gather compaction) */
  RA_LAYOUT_HOLE_FILL = 1,     /* an eviction moves only the surviving rows of the
                                  last m slots into the holes; rows are unordered
                                  (positions travel with them); the same kept sets */
  RA_LAYOUT_PAGED = 2          /* rows in position order in fixed pages of page_rows
                                  rows mapped by a block table per sequence (Appendix
                                  G: physical eviction under paging rewrites each
                                  request's surviving KV into its blocks, frees the
                                  tail and keeps positions logical).  The pool is a
                                  sequence of page groups of L * Hkv pages, one per
                                  (layer, KV head): every head of a sequence holds
                                  the same number of rows, so one table entry maps
                                  one group.  A group is taken from the pool's free
                                  list when an append needs a new page and returned
                                  when an eviction or ra_seq_end releases it; an
                                  event keeps the chronological order (the same
                                  shift as RA_LAYOUT_CHRONOLOGICAL through the
                                  table) and frees the pages past the new length */
} ra_layout;

typedef enum {
  RA_POLICY_RANDOM = 0,   /* Random Attention (Section 3): an independent
                             uniform draw per candidate, per KV head, per event */
  RA_POLICY_SHARED = 1,   /* shared-draw control (Section 5, Appendix D): the
                             same random positions in every head -- the draw
                             omits the layer and the KV head */
  RA_POLICY_BLOCK = 2,    /* block-wise eviction (Section 5): history kept in
                             contiguous blocks of policy_block tokens -- every
                             position takes the draw of its block's first
                             position (blocks aligned at the prompt end), so
                             policy_block = 1 is RA_POLICY_RANDOM */
  RA_POLICY_RECENCY = 3,  /* recency+prompt (Section 4.1): the prompt plus the
                             contiguous recent window -- the oldest candidates
                             are dropped, no draw */
  RA_POLICY_EXTERNAL = 4  /* no eviction at the end of a step: the caller runs
                             score-based rounds with ra_scored_evict (used to
                             price the selection signal, not by the method) */
} ra_policy;

/* Score-based evictors of Section 2 ("Baselines as choices of s"), run only
 * to measure what Random Attention saves.  Every cached row outside the r
 * most recent is a candidate (the prompt competes, as in those methods), and
 * a round keeps lp + k_keep of them. */
typedef enum {
  RA_SCORER_SNAPKV = 0,   /* sum of the attention weights of the last 64
                             queries of the group's query heads, max-pooled
                             over 7 neighbouring rows; the lowest are dropped */
  RA_SCORER_RKV = 1,      /* lambda * SnapKV - (1 - lambda) * softmax(c), c_i
                             the mean cosine similarity of key i to the other
                             cached keys, its `rkv_recent_dups` most recent
                             near-duplicates (cosine > rkv_threshold) not
                             counted */
  RA_SCORER_VASE = 2      /* keep the vase_n_large rows of largest value range
                             (max - min over channels), fill the rest of the
                             budget by sampling without replacement with
                             probability proportional to the SnapKV score */
} ra_scorer;

typedef struct {
  int32_t scorer;          /* ra_scorer */
  float rkv_lambda;        /* R-KV weight of the SnapKV term, in [0, 1] */
  float rkv_threshold;     /* R-KV near-duplicate cosine threshold */
  int32_t rkv_recent_dups; /* R-KV near-duplicates not counted (>= 0) */
  int32_t vase_n_large;    /* VaSE rows kept by value range (< 0: half the
                              kept budget) */
  uint64_t vase_seed;      /* VaSE: seed of the proportional fill's draws */
} ra_scorer_params;

typedef struct ra_cache ra_cache;   /* host-side descriptor + host mirror */

typedef struct {
  int32_t active;       /* 1 if the slot holds a sequence */
  int32_t prompt_len;   /* lp */
  int32_t len;          /* cached rows per (layer, KV head) between steps */
  int32_t step;         /* completed decode steps */
  int32_t event;        /* eviction events performed */
  int32_t k_keep;       /* evictable rows kept per head */
  int32_t cap;          /* row capacity of each (layer, KV head) region */
  int64_t base;         /* first pool row of the sequence's regions */
  int32_t move_pending; /* 1: the last event compacted the positions and the
                           next step's attention moves the key/value rows
                           (see ra_end_step) */
} ra_seq_info;

/* ---- sizing (pure host functions; no device access) --------------------- */

/* RA_OK if the config is usable. */
ra_status ra_config_check(const ra_config* cfg);

/* Row capacity of one (layer, KV head) region for a prompt of prompt_len:
 * lp + k_keep + recent_r + evict_every rounded up to a multiple of 32 (of
 * page_rows in the paged layout, where it is the most rows a head of such a
 * sequence ever holds).  Negative ra_status on error (bad config, TOTAL mode
 * with lp > K, a paged prompt longer than max_prompt_len). */
int64_t ra_region_rows(const ra_config* cfg, int32_t prompt_len);

/* Pool rows one sequence occupies: L * Hkv * ra_region_rows (in the paged
 * layout, at most: it holds pages only for the rows it has).  The K and V
 * pools hold pool_rows * head_dim elements each, the position pool
 * pool_rows int32.  Negative ra_status on error. */
int64_t ra_seq_rows(const ra_config* cfg, int32_t prompt_len);

/* Pool rows a batch of sequences occupies at once: the sum of ra_seq_rows
 * over host_prompt_lens[0..n_seqs) (host memory).  The pool of
 * ra_cache_create needs at least this many rows to hold them all.  Negative
 * ra_status on error (bad config or argument, TOTAL mode with lp > K). */
int64_t ra_required_slots(const ra_config* cfg, const int32_t* host_prompt_lens,
                          int32_t n_seqs);

/* Bytes of the persistent device metadata buffer: per-slot state; in the
 * paged layout the block tables, max_seqs * ceil((max_prompt_len + k_keep +
 * recent_r + evict_every) / page_rows) int32; in the bf16 chronological
 * layout the drop lists of deferred row moves, max_seqs * L * Hkv *
 * evict_every int32 (none, and no deferred moves, when that would exceed
 * 256 MiB); the attention's split arrival counters, max_seqs * Hkv
 * int32 (zero between calls: one cache is driven from one stream).  0 on a
 * bad config. */
size_t ra_meta_bytes(const ra_config* cfg);

/* Bytes of the attention workspace (split partial results) that
 * ra_decode_attention needs.  0 on a bad config. */
size_t ra_workspace_bytes(const ra_config* cfg);

/* ---- lifetime ----------------------------------------------------------- */

/* Create a cache over caller-owned device buffers:
 *   k_pool, v_pool: pool_rows * head_dim elements of cfg->dtype each;
 *   pos_pool:       pool_rows int32;
 *   meta:           ra_meta_bytes(cfg) bytes (zeroed here on `stream`).
 * pool_rows is a multiple of 32 (of L * Hkv * page_rows, one page group, in
 * the paged layout).  Keys are stored row-major; values in tiles of 8 rows
 * stored transposed ([row/8][head_dim][8]); positions row-major.  Contiguous
 * layouts place each sequence's regions by a first-fit allocator over the
 * pool at ra_seq_begin; the paged layout hands out page groups from a free
 * list as rows are appended. */
ra_status ra_cache_create(const ra_config* cfg, void* k_pool, void* v_pool,
                          int32_t* pos_pool, int64_t pool_rows, void* meta,
                          size_t meta_bytes, void* stream, ra_cache** out);

ra_status ra_cache_destroy(ra_cache* cache);

/* ---- sequences ----------------------------------------------------------- */

/* Pool occupancy (host mirror, no device access): rows in use by sequences
 * and rows free (contiguous layouts: the first-fit free list, whose largest
 * hole bounds the next admission; paged: free page groups * L * Hkv *
 * page_rows).  Either output may be NULL. */
ra_status ra_pool_info(const ra_cache* cache, int64_t* used_rows, int64_t* free_rows);

/* Pin a prompt into slot `seq` (Section 3: the prompt is never evicted).
 * dev_k_prompt / dev_v_prompt: [L][Hkv][prompt_len][head_dim] row-major, or
 * both NULL to leave the prompt rows unwritten (positions are still set;
 * the rows are then expected from ra_write_rows).  `seed` and `request_id`
 * key every eviction draw of this sequence.  Errors: RA_ERR_STATE if the
 * slot is active, RA_ERR_BUDGET (TOTAL mode, lp > K), RA_ERR_CAPACITY if
 * the pool has no room (paged: for the prompt's pages) or a paged prompt is
 * longer than max_prompt_len. */
ra_status ra_seq_begin(ra_cache* cache, int32_t seq, int32_t prompt_len,
                       uint64_t seed, uint64_t request_id,
                       const void* dev_k_prompt, const void* dev_v_prompt,
                       void* stream);

/* Release slot `seq` and its pool rows. */
ra_status ra_seq_end(ra_cache* cache, int32_t seq, void* stream);

/* Host mirror of a slot (no device access). */
ra_status ra_get_seq_info(const ra_cache* cache, int32_t seq, ra_seq_info* out);

/* ---- decode step --------------------------------------------------------- */

/* Append + attend for one layer of every active sequence (Section 2).
 *   q:     [max_seqs][Hq][d]   this step's queries (inactive slots ignored)
 *   k_new: [max_seqs][Hkv][d]  this step's key of each KV head
 *   v_new: [max_seqs][Hkv][d]
 *   out:   [max_seqs][Hq][d]   written for active slots only
 *   workspace: ra_workspace_bytes(cfg) bytes of scratch.
 * Each active sequence caches (k_new, v_new) at position lp + step in every
 * KV head of `layer`, and query head h attends, with softmax over
 * q.k/sqrt(d), to every cached pair of KV head h / G, the new one included.
 * Each layer must be called once per step (RA_ERR_STATE otherwise) and
 * RA_ERR_CAPACITY is returned before a region would overflow.  In the paged
 * layout the first layer of a step takes a page group for every sequence
 * whose new row starts a page; RA_ERR_CAPACITY, before any launch, if the
 * pool has too few free groups (ending a sequence frees its groups).  After
 * an event whose row moves were deferred (ra_end_step), the layer's
 * attention also moves that layer's surviving rows to their compacted slots
 * (if the step's plan splits a head into several work items, a separate
 * launch moves them first). */
ra_status ra_decode_attention(ra_cache* cache, int32_t layer, const void* q,
                              const void* k_new, const void* v_new, void* out,
                              void* workspace, size_t workspace_bytes,
                              void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * append + attention as ra_decode_attention, with the same arguments minus
 * the workspace.  The split partial results go to a file-scope device array
 * of RA_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends (its address is looked up once per device, at
 * ra_cache_create).  The call allocates nothing and calls no allocating
 * routine.  It needs (slots up to the highest active one) * Hkv * splits * G
 * * 130 * 4 bytes of that array when the launch has more than one split per
 * head (always for f32; see ra_attention_plan), and returns RA_ERR_CAPACITY,
 * before any launch, when that exceeds RA_NOALLOC_SCRATCH_BYTES.  Every call
 * on one GPU shares the array, from any cache: calls that overlap on one GPU
 * (other streams, other threads) race on it and must be serialised by the
 * caller.  Nothing in the array needs to start at zero. */
#define RA_NOALLOC_SCRATCH_BYTES (8u << 20)
ra_status ra_decode_attention_noalloc(ra_cache* cache, int32_t layer, const void* q,
                                      const void* k_new, const void* v_new, void* out,
                                      void* stream);

/* End the decode step of every active sequence: step += 1, then run the
 * periodic eviction (Eq. 1 with Random Attention's scores, Appendix F
 * trigger) on every (layer, KV head) of each sequence that is due (never
 * under RA_POLICY_EXTERNAL).  bf16, contiguous chronological layout: when
 * every active sequence is due at this step and the next step's attention
 * gives each head one work item, the event selects and compacts the
 * positions only, and that attention moves each layer's key/value rows while
 * it reads them (the kept sets are final at once; the rows are final after
 * the next step, or as soon as a call that reads or writes rows, or plans
 * another event, moves them first).
 * Requires every layer to have been appended this step (RA_ERR_STATE
 * otherwise; with no active sequence, a step with no layer appended ends as
 * a no-op).  If n_evicted is non-NULL it receives the number of sequences
 * evicted (host mirror). */
ra_status ra_end_step(ra_cache* cache, void* stream, int32_t* n_evicted);

/* For callers that capture decode steps into HIP graphs (a step's
 * ra_decode_attention calls for every layer and its ra_end_step, captured
 * once and replayed at every step).  on = 1 enters graph mode: the attention
 * plan is fixed for every state the active sequences can reach (their caches
 * never outgrow their regions), and ra_end_step launches the step's advance
 * and the eviction of every active head unconditionally; each eviction
 * workgroup reads on the device whether its sequence is due, so the launches
 * of a step depend on no host state and a captured step replays correctly at
 * any later step.  The host mirror is not advanced in graph mode:
 * ra_get_seq_info reports the state at entry, ra_end_step's n_evicted
 * receives 0, and calls that need the mirror (ra_seq_begin, ra_seq_end,
 * ra_evict_now, ra_fast_forward, row and position reads and writes, the
 * measurement-only calls) return RA_ERR_STATE.  Events do not defer their
 * row moves in graph mode (rows pending from an earlier event are moved at
 * entry).  on = 0 leaves graph mode: the stream is synchronised and the
 * device's per-slot records become the mirror again; graphs captured in
 * graph mode are to be replayed only while it lasts (replayed later, they
 * would advance the device past the mirror).  RA_ERR_STATE inside
 * an open step; RA_ERR_UNSUPPORTED for the paged layout (page groups are
 * handed out by the host) and RA_POLICY_EXTERNAL.  Entering or leaving a
 * second time is a no-op. */
ra_status ra_graph_mode(ra_cache* cache, int32_t on, void* stream);

/* Run one eviction event on slot `seq` now, whatever the step count, if
 * its evictable rows exceed k_keep (otherwise a no-op).  The event is the
 * one of Eq. 1 with Section 3's scores (i.i.d. uniform per candidate, the
 * top k_keep kept): the same keys, selection and compaction as a periodic
 * event, with the next event index.  Not allowed in
 * the middle of a step, nor with more than 1024 rows over k_keep (possible
 * only under RA_POLICY_EXTERNAL): RA_ERR_STATE; RA_ERR_UNSUPPORTED if such
 * a pile-up makes more than 32768 candidate slots.  The keys are Random
 * Attention's (or the policy's). */
ra_status ra_evict_now(ra_cache* cache, int32_t seq, void* stream);

/* ---- state transfer and audit --------------------------------------------- */

/* Advance every active sequence by n_steps decode steps touching positions
 * only: each step caches position lp + step and the periodic eviction runs
 * on the positions exactly as in a real decode, but no key/value rows are
 * written or moved (rows of newly cached positions are left stale).  Used
 * to reach a long-generation state quickly; follow with ra_write_rows.
 * RA_ERR_STATE inside an open step; RA_ERR_CAPACITY, before any launch, if
 * some sequence would outgrow its region on the way (only possible under
 * RA_POLICY_EXTERNAL, whose rows are evicted by explicit rounds only) or, in
 * the paged layout, if the pool has too few free page groups for the rows
 * the sequences hold on the way. */
ra_status ra_fast_forward(ra_cache* cache, int32_t n_steps, void* stream);

/* ra_fast_forward for the one active slot `seq`: the other slots' records,
 * positions and rows are left as they are (their deferred row moves stay
 * pending unless `seq` has one too).  Use: resuming a preempted request
 * inside a live batch (Appendix G: eviction under paging must stay correct
 * across preemption).  Its kept positions depend only on its seed, request
 * id and step, so ra_seq_begin with the same prompt length, seed and
 * request id (prompt rows optional), ra_seq_fast_forward by the steps it
 * had decoded, then ra_write_rows with its saved rows (ra_read_rows of
 * every head before ra_seq_end) restore the state it had, in any free slot.
 * Only periodic events are replayed: a request that had explicit events
 * (ra_evict_now, ra_scored_evict) resumes in another state.  Errors as
 * ra_fast_forward, and RA_ERR_STATE if the slot is not active. */
ra_status ra_seq_fast_forward(ra_cache* cache, int32_t seq, int32_t n_steps,
                              void* stream);

/* Copy slot `seq`'s cached positions, [L][Hkv][len] int32 row-major, to
 * device memory (dev_out holds at least L*Hkv*len int32; RA_ERR_CAPACITY,
 * nothing copied, if out_elems is smaller; NULL allowed when len is 0). */
ra_status ra_export_positions(ra_cache* cache, int32_t seq, int32_t* dev_out,
                              int64_t out_elems, void* stream);

/* Overwrite slot `seq`'s cached rows from row-major device arrays
 * [L][Hkv][len][d] (row j belongs to the j-th cached position, the order of
 * ra_export_positions; NULL allowed when len is 0). */
ra_status ra_write_rows(ra_cache* cache, int32_t seq, const void* dev_k,
                        const void* dev_v, void* stream);

/* Copy the cached rows of one (seq, layer, KV head) to row-major device
 * arrays [len][d] (values un-tiled).  Either output may be NULL. */
ra_status ra_read_rows(ra_cache* cache, int32_t seq, int32_t layer,
                       int32_t kv_head, void* dev_k_out, void* dev_v_out,
                       void* stream);

/* SYNCHRONOUS: copy one head's cached positions, in row order (ascending in
 * the chronological layout), to host memory; *n_out receives len.  This is
 * the keep-set of Appendix D's keep-log (the positions a head holds after
 * each event), read one head at a time.  RA_ERR_CAPACITY if host_cap < len (nothing
 * copied).  Synchronizes `stream`. */
ra_status ra_read_positions(ra_cache* cache, int32_t seq, int32_t layer,
                            int32_t kv_head, int32_t* host_out,
                            int32_t host_cap, int32_t* n_out, void* stream);

/* ---- measurement only --------------------------------------------------------- */

/* NOT PART OF RANDOM ATTENTION.  The scoring pass of a score-based evictor,
 * provided to measure the cost that Random Attention removes: Section 2
 * ("Baselines as choices of s") defines SnapKV's score of a cached position
 * as the sum of the attention weights of the last w queries, max-pooled over
 * neighbouring positions, and Eq. 1 keeps the top-scoring candidates.  For
 * every (layer, KV head) of the active slots in [seq_lo, seq_hi):
 *   score[j] = sum over the G*64 window queries of softmax(q.k/sqrt(d)) at
 *              cached row j (a query sees the rows at or before its
 *              position), then max-pooled over 7 rows;
 *   drops    = the m lowest candidates (cached rows before the r most
 *              recent; ties by row), m = the number Random Attention would
 *              drop at this state.
 * dev_q_window: [max_seqs][L][Hq][64][d] bf16, the queries of each
 * sequence's last 64 decode steps, oldest first.  dev_scores (optional):
 * [seq_hi-seq_lo][L][Hkv][scores_stride] float, the un-pooled scores of rows
 * [0, len).  dev_drops (optional): [seq_hi-seq_lo][L][Hkv][evict_every]
 * int32, the dropped rows ascending.  The cache is not modified.  bf16 and
 * the chronological layout only, and at most 2^20 (slot, layer, KV head)
 * heads per call (RA_ERR_UNSUPPORTED otherwise); RA_ERR_STATE if a slot has
 * fewer than 64 steps or more than evict_every rows to drop. */
ra_status ra_window_select(ra_cache* cache, int32_t seq_lo, int32_t seq_hi,
                           const void* dev_q_window, float* dev_scores,
                           int32_t scores_stride, int32_t* dev_drops, void* stream);

/* Bytes of device scratch ra_scored_evict needs for a cache whose longest
 * prompt is max_prompt_len (0 on an invalid config). */
size_t ra_scored_scratch_bytes(const ra_config* cfg, int32_t max_prompt_len);

/* One score-based eviction round (scoring + selection + compaction) for every
 * active sequence in [seq_lo, seq_hi) whose rows outside the r most recent
 * exceed lp + k_keep; the others are left as they are.  dev_q_window is
 * [max_seqs][L][Hq][64][128] bf16: the queries of each sequence's last 64
 * decode steps, oldest first.  The kept rows stay in chronological order;
 * len becomes lp + k_keep + r.  bf16 and the chronological layout only, at
 * most 2^20 (slot, layer, KV head) heads per call (RA_ERR_UNSUPPORTED
 * otherwise); RA_ERR_STATE inside an open step, before
 * step 64 or when a sequence has more than evict_every rows over its
 * budget; RA_ERR_INVALID_ARG on a bad parameter or a scratch smaller than
 * ra_scored_scratch_bytes.  Asynchronous on `stream`. */
ra_status ra_scored_evict(ra_cache* cache, int32_t seq_lo, int32_t seq_hi,
                          const ra_scorer_params* params, const void* dev_q_window,
                          void* dev_scratch, size_t scratch_bytes, void* stream);

/* ---- diagnostics ----------------------------------------------------------- */

const char* ra_status_string(int32_t status);

/* hipError_t of the last failed HIP call in this process (0 if none). */
int32_t ra_last_hip_error(void);

/* Keys per attention work item, work items per head and wavefronts per work
 * item that the next ra_decode_attention launch uses (host mirror; for
 * measurement and tests).  `waves` may be NULL. */
ra_status ra_attention_plan(const ra_cache* cache, int32_t* split_keys,
                            int32_t* max_splits, int32_t* waves);

#ifdef __cplusplus
}
#endif

#endif /* RANDATTN_H */
