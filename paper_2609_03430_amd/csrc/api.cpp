// Host side of the C ABI (include/randattn.h): validation, the host mirror
// of every slot's state, pool placement, and kernel launches.
//
// The host mirror replays the same integer rules as the device state
// kernels (append one row per step, the Appendix F trigger, eviction back to
// lp + k_keep + r), so every capacity and protocol error is reported before
// any launch and the eviction kernel is launched only on steps where some
// sequence is due.  The library never allocates device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <map>
#include <new>
#include <vector>

#include "randattn.h"
#include "ra_internal.h"

using ra::SeqMeta;

static_assert(RA_NOALLOC_SCRATCH_BYTES == ra::kNoAllocScratchBytes,
              "the header's no-alloc limit is the size of the device array");

namespace {

std::atomic<int32_t> g_last_hip_error{0};

ra_status hip_fail(hipError_t e) {
  if (e == hipSuccess) return RA_OK;
  g_last_hip_error.store(static_cast<int32_t>(e));
  return RA_ERR_HIP;
}

#define RA_LAUNCH(expr)                         \
  do {                                          \
    const hipError_t e_ = (expr);               \
    if (e_ != hipSuccess) return hip_fail(e_);  \
  } while (0)

int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// The per-(sequence, layer, KV head) kernels (eviction, deferred moves,
// external rounds' compaction) run one workgroup of up to 1,024 threads per
// head of the slots given; a range of slots is cut so that one launch holds
// at most 2^20 workgroups, well inside the dispatch grid's limit.
#ifndef RA_MAX_HEADS_PER_LAUNCH
#define RA_MAX_HEADS_PER_LAUNCH (1 << 20)   // smaller in the host-only test build
#endif
constexpr int64_t kMaxHeadsPerLaunch = RA_MAX_HEADS_PER_LAUNCH;

template <class F>
hipError_t by_slot_chunks(const ra_config& c, int lo, int hi, F&& launch) {
  const int64_t per = static_cast<int64_t>(c.num_layers) * c.num_kv_heads;
  const int chunk = static_cast<int>(std::max<int64_t>(1, kMaxHeadsPerLaunch / per));
  for (int a = lo; a < hi; a += chunk) {
    const hipError_t e = launch(a, std::min(hi, a + chunk));
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Trigger period of the end-of-step rule; 0 = never (external rounds only).
int trigger_every(const ra_config& c) {
  return c.policy == RA_POLICY_EXTERNAL ? 0 : c.evict_every;
}

bool at_trigger(const ra_config& c, int step) {
  const int e = trigger_every(c);
  return e > 0 && step % e == 0;
}

int64_t keep_rows(const ra_config& c, int32_t lp) {
  if (c.budget_mode == RA_BUDGET_EVICTABLE) return c.budget_k;
  return static_cast<int64_t>(c.budget_k) - lp;
}

bool paged(const ra_config& c) { return c.layout == RA_LAYOUT_PAGED; }

int log2_exact(int x) {
  int k = 0;
  while ((1 << k) < x) ++k;
  return (1 << k) == x ? k : -1;
}

// Most rows a head of the paged layout ever holds, over the prompts it
// accepts: lp + k_keep + r + R (the prompt counts against K in TOTAL mode).
int64_t paged_rows_max(const ra_config& c) {
  const int64_t held = c.budget_mode == RA_BUDGET_TOTAL
                           ? static_cast<int64_t>(c.budget_k)
                           : static_cast<int64_t>(c.max_prompt_len) + c.budget_k;
  return held + c.recent_r + c.evict_every;
}

int64_t pages_per_seq(const ra_config& c) {
  return (paged_rows_max(c) + c.page_rows - 1) / c.page_rows;
}

size_t meta_records_bytes(const ra_config& c) {
  return static_cast<size_t>(round_up(static_cast<int64_t>(sizeof(SeqMeta)) * c.max_seqs, 256));
}

size_t tables_bytes(const ra_config& c) {
  if (!paged(c)) return 0;
  return static_cast<size_t>(round_up(
      static_cast<int64_t>(sizeof(int32_t)) * c.max_seqs * pages_per_seq(c), 256));
}

// Events whose row moves the next step's attention can carry (bf16, the
// contiguous chronological layout): their drop lists, evict_every per head,
// kept in the metadata buffer.  Past 256 MiB of lists (far more slots,
// layers or drops per event than any measured shape: the Qwen3-14B batch
// needs 2.6 MB) the cache does not defer, rather than ask for that much.
constexpr int64_t kMaxDropsBytes = int64_t(256) << 20;

bool defers_moves(const ra_config& c) {
  const int64_t lists = static_cast<int64_t>(sizeof(int32_t)) * c.max_seqs * c.num_layers *
                        c.num_kv_heads * c.evict_every;
  return c.dtype == RA_BF16 && c.layout == RA_LAYOUT_CHRONOLOGICAL &&
         c.policy != RA_POLICY_EXTERNAL && lists <= kMaxDropsBytes;
}

// Split arrival counters of the bf16 attention, one per (slot, KV head).
size_t arrivals_bytes(const ra_config& c) {
  return static_cast<size_t>(
      round_up(static_cast<int64_t>(sizeof(int32_t)) * c.max_seqs * c.num_kv_heads, 256));
}

size_t drops_bytes(const ra_config& c) {
  if (!defers_moves(c)) return 0;
  return static_cast<size_t>(round_up(static_cast<int64_t>(sizeof(int32_t)) * c.max_seqs *
                                          c.num_layers * c.num_kv_heads * c.evict_every,
                                      256));
}

}  // namespace

struct ra_cache {
  ra_config cfg{};
  int G = 0;
  size_t elem = 0;
  void* kpool = nullptr;
  void* vpool = nullptr;
  int32_t* pos = nullptr;
  int64_t pool_rows = 0;
  SeqMeta* meta = nullptr;
  std::vector<SeqMeta> mirror;           // host copy of the device metadata
  std::map<int64_t, int64_t> free_rows;  // first-fit free list: base -> rows
  std::vector<uint8_t> appended;         // layers appended in the open step
  int n_appended = 0;
  int slot_lo = 0, slot_hi = 0;          // range covering the active slots
  // paged layout
  ra::Paging pg{};                       // device tables and page geometry
  int page_rows = 0;
  int64_t n_groups = 0;                  // page groups in the pool
  std::vector<int32_t> free_groups;      // stack: the next group is back()
  std::vector<std::vector<int32_t>> groups;   // per slot: its table, in order
  // deferred row moves (see ra_end_step)
  int32_t* drops = nullptr;              // drop lists of the last events
  int32_t* arrivals = nullptr;           // split arrival counters (bf16 attention)
  // graph mode (see ra_graph_mode): launches that depend on no host state
  bool graph = false;
  int graph_split_keys = 0, graph_max_splits = 0, graph_waves = 0, graph_wide_regs = 0;
  int graph_candidates = 0;              // bound on any event's candidate slots
  void* scratch = nullptr;               // device address of the no-alloc partials

  ra::Shape shape() const {
    return ra::Shape{cfg.num_layers, cfg.num_q_heads, cfg.num_kv_heads, G,
                     cfg.recent_r, cfg.evict_every, cfg.dtype, cfg.layout,
                     cfg.policy, std::max(1, cfg.policy_block), pg};
  }
  bool is_paged() const { return cfg.layout == RA_LAYOUT_PAGED; }
  bool any_pending() const {
    for (int s = slot_lo; s < slot_hi; ++s)
      if (mirror[s].active && mirror[s].due == ra::kDueMovePending) return true;
    return false;
  }
  int64_t pages_for(int64_t rows) const { return (rows + page_rows - 1) / page_rows; }
  // paged: whether `rows` rows fit the block table of one sequence (rows
  // pile up past lp + k_keep + r + R only under the external policy)
  bool fits_table(int64_t rows) const { return pages_for(rows) <= pg.pages_per_seq; }
  // paged: page groups slot `s` must add to hold `rows` rows
  int64_t groups_short(int s, int64_t rows) const {
    return std::max<int64_t>(0, pages_for(rows) - static_cast<int64_t>(groups[s].size()));
  }
  // paged: take groups from the free list until slot `s` holds `rows` rows;
  // the new table entries are appended to `out` (the caller checked that
  // enough groups are free)
  void grow(int s, int64_t rows, std::vector<ra::TableEntry>& out) {
    while (static_cast<int64_t>(groups[s].size()) < pages_for(rows)) {
      const int32_t g = free_groups.back();
      free_groups.pop_back();
      out.push_back(ra::TableEntry{s, static_cast<int32_t>(groups[s].size()), g});
      groups[s].push_back(g);
    }
    mirror[s].cap = static_cast<int32_t>(groups[s].size()) * page_rows;
  }
  // paged: return the groups past the first pages_for(rows) to the free list
  void shrink(int s, int64_t rows) {
    while (static_cast<int64_t>(groups[s].size()) > pages_for(rows)) {
      free_groups.push_back(groups[s].back());
      groups[s].pop_back();
    }
    mirror[s].cap = static_cast<int32_t>(groups[s].size()) * page_rows;
  }
  bool step_open() const { return n_appended != 0; }
  void update_range() {
    slot_lo = 0;
    slot_hi = 0;
    bool any = false;
    for (int s = 0; s < cfg.max_seqs; ++s) {
      if (!mirror[s].active) continue;
      if (!any) slot_lo = s;
      slot_hi = s + 1;
      any = true;
    }
  }
  // slots the selection examines per head (see evict.hip)
  int span(const SeqMeta& M) const {
    return M.plan_len - M.prompt_len - (cfg.layout == RA_LAYOUT_HOLE_FILL ? 0 : cfg.recent_r);
  }
  int max_candidates_due() const {
    int mx = 0;
    for (int s = slot_lo; s < slot_hi; ++s)
      if (mirror[s].active && mirror[s].due) mx = std::max(mx, span(mirror[s]));
    return mx;
  }
};

namespace {

// The host mirror of the device plan rule (state.hip).
void mirror_plan(SeqMeta& M, int r, bool at_trigger) {
  M.due = 0;
  if (at_trigger && M.len - M.prompt_len - r > M.k_keep) {
    M.due = 1;
    M.plan_len = M.len;
    M.plan_event = M.event;
    M.len = M.prompt_len + M.k_keep + r;
    M.event += 1;
  }
}

// Launch plan of the decode attention (measured on the workloads' shapes).
// A bf16 work item is one (sequence, KV head, split) on a workgroup of W
// wavefronts, each streaming a contiguous W-th of the split's keys.  The
// chip has 256 CUs: with at most 256 heads, the heads are split so that
// about 256 workgroups run, one per CU, and W is the largest of 12, 8, 4
// that leaves each wavefront a long enough run of keys (12 or 8
// wavefronts keep 3 or 2 per SIMD in flight; a short run per wavefront
// costs more in prologue than the extra wavefronts gain).  With many more
// heads than CUs the workgroups run in several waves of dispatch, and 4
// wavefronts built for one wavefront per SIMD (accumulators in the
// accumulation registers) stream best; between 256 and 768 heads the 4-
// wavefront build that fits three workgroups per CU keeps every head
// resident at once.  fp32 (VALU): one wavefront per item, about 1024 items.
struct Plan {
  int split_keys, max_splits, waves, wide_regs;
};

// The plan for `n_active` sequences whose longest cache, the new row
// included, has keys_max keys.
Plan plan_for(const ra_cache* c, int keys_max, int n_active) {
  const int heads = std::max(1, n_active * c->cfg.num_kv_heads);
  Plan p{0, 0, 1, 0};
  int splits = 1;
  if (c->cfg.dtype == RA_BF16) {
    if (heads >= 768) {
      p.waves = 4;
      p.wide_regs = 1;
    } else if (heads > 256) {
      p.waves = 4;
    } else {
      splits = std::max(1, (256 + heads / 2) / heads);
      const int keys = (keys_max + splits - 1) / splits;
      p.waves = keys >= 12 * 640 ? 12 : keys >= 8 * 256 ? 8 : keys >= 4 * 128 ? 4 : 1;
      p.wide_regs = p.waves == 4;
    }
  } else {
    splits = (1024 + heads - 1) / heads;
  }
  splits = std::min(ra::kMaxSplits, splits);
  const int unit = 32 * p.waves;
  int sk = c->cfg.attn_split > 0 ? static_cast<int>(round_up(c->cfg.attn_split, unit))
                                 : static_cast<int>(round_up((keys_max + splits - 1) / splits, unit));
  sk = std::max<int>(sk, static_cast<int>(round_up((keys_max + ra::kMaxSplits - 1) / ra::kMaxSplits, unit)));
  p.split_keys = sk;
  p.max_splits = (keys_max + sk - 1) / sk;
  return p;
}

Plan attention_plan(const ra_cache* c) {
  if (c->graph)
    return Plan{c->graph_split_keys, c->graph_max_splits, c->graph_waves, c->graph_wide_regs};
  // sized by the longest cache of this step (cached rows + the new one), so
  // that while sequences are younger than their budget no wavefront or split
  // is planned over rows that do not exist yet
  int keys_max = 32, n_active = 0;
  for (int s = c->slot_lo; s < c->slot_hi; ++s) {
    if (!c->mirror[s].active) continue;
    keys_max = std::max(keys_max, c->mirror[s].len + 1);
    ++n_active;
  }
  return plan_for(c, keys_max, n_active);
}

// Host checks shared by both attention entry points; nothing is launched.
ra_status check_decode(const ra_cache* c, int32_t layer, const void* q, const void* k_new,
                       const void* v_new, const void* out) {
  if (!c || layer < 0 || layer >= c->cfg.num_layers || !q || !k_new || !v_new || !out)
    return RA_ERR_INVALID_ARG;
  if (c->appended[layer]) return RA_ERR_STATE;
  if (c->is_paged()) {
    // the step's new rows may start pages: enough free groups for all of them
    int64_t short_groups = 0;
    for (int s = c->slot_lo; s < c->slot_hi; ++s) {
      if (!c->mirror[s].active) continue;
      if (!c->fits_table(c->mirror[s].len + 1)) return RA_ERR_CAPACITY;
      short_groups += c->groups_short(s, c->mirror[s].len + 1);
    }
    if (short_groups > static_cast<int64_t>(c->free_groups.size())) return RA_ERR_CAPACITY;
    return RA_OK;
  }
  for (int s = c->slot_lo; s < c->slot_hi; ++s)
    if (c->mirror[s].active && c->mirror[s].len + 1 > c->mirror[s].cap) return RA_ERR_CAPACITY;
  return RA_OK;
}

// Moves the key/value rows of every sequence whose last event deferred them
// (their positions are already compacted); a call that reads or writes rows,
// or plans another event, runs this first.
ra_status flush_pending(ra_cache* c, hipStream_t s) {
  if (!c->any_pending()) return RA_OK;
  RA_LAUNCH(by_slot_chunks(c->cfg, c->slot_lo, c->slot_hi, [&](int lo, int hi) {
    return ra::launch_flush_pending(c->shape(), c->meta, c->kpool, c->vpool, c->drops,
                                    c->cfg.evict_every, lo, hi, s);
  }));
  for (int i = c->slot_lo; i < c->slot_hi; ++i)
    if (c->mirror[i].due == ra::kDueMovePending) c->mirror[i].due = 0;
  return RA_OK;
}

// Marks the layer appended and launches its append + attention with the
// given partials buffers (split_stride partial slots per head).
ra_status launch_decode(ra_cache* c, int32_t layer, const void* q, const void* k_new,
                        const void* v_new, void* out, const Plan& plan, float* ws_o,
                        float* ws_ml, int split_stride, hipStream_t stream) {
  if (c->is_paged()) {
    // pages for the rows this step appends (the first layer of the step)
    std::vector<ra::TableEntry> te;
    for (int s = c->slot_lo; s < c->slot_hi; ++s)
      if (c->mirror[s].active) c->grow(s, c->mirror[s].len + 1, te);
    if (!te.empty()) {
      const hipError_t e = ra::launch_table_set(c->shape(), te.data(),
                                                static_cast<int>(te.size()), stream);
      if (e != hipSuccess) return hip_fail(e);
    }
  }
  // rows of deferred events move in this step's attention when every head is
  // one work item; otherwise they move first, on their own
  bool move = false;
  if (c->any_pending()) {
    if (plan.max_splits == 1) {
      move = true;
    } else {
      const ra_status st = flush_pending(c, stream);
      if (st != RA_OK) return st;
    }
  }
  c->appended[layer] = 1;
  ++c->n_appended;
  if (c->slot_hi <= c->slot_lo) return RA_OK;
  ra::AttnLaunch a{};
  a.meta = c->meta;
  a.kpool = c->kpool;
  a.vpool = c->vpool;
  a.pos = c->pos;
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.out = out;
  a.ws_o = ws_o;
  a.ws_ml = ws_ml;
  a.split_stride = split_stride;
  a.layer = layer;
  a.max_seqs = c->slot_hi;
  a.split_keys = plan.split_keys;
  a.max_splits = plan.max_splits;
  a.arrivals = c->arrivals;
  a.waves = plan.waves;
  a.wide_regs = plan.wide_regs;
  // fp32 heads of several splits: merged by their last split, which spares
  // a launch and its gap; in graph mode the launches follow each other with
  // no gap and the merge kernel (256 threads per head, against the 64 of a
  // split) is the faster of the two
  a.merge_kernel = c->graph ? 1 : 0;
  if (move) {
    a.move = 1;
    a.waves = 8;
    a.drops = c->drops;
    a.drop_stride = c->cfg.evict_every;
  }
  const hipError_t e = ra::launch_attention(c->shape(), a, stream);
  if (e != hipSuccess) {
    c->appended[layer] = 0;
    --c->n_appended;
    return hip_fail(e);
  }
  return RA_OK;
}

}  // namespace

extern "C" {

const char* ra_status_string(int32_t status) {
  switch (status) {
    case RA_OK: return "ok";
    case RA_ERR_INVALID_ARG: return "invalid argument";
    case RA_ERR_CAPACITY: return "capacity exceeded";
    case RA_ERR_BUDGET: return "prompt exceeds the budget (TOTAL mode)";
    case RA_ERR_UNSUPPORTED: return "unsupported configuration";
    case RA_ERR_HIP: return "HIP error";
    case RA_ERR_STATE: return "call out of protocol order";
    default: return "unknown status";
  }
}

int32_t ra_last_hip_error(void) { return g_last_hip_error.load(); }

ra_status ra_config_check(const ra_config* c) {
  if (!c) return RA_ERR_INVALID_ARG;
  if (c->num_layers < 1 || c->num_q_heads < 1 || c->num_kv_heads < 1 ||
      c->num_q_heads % c->num_kv_heads != 0 || c->budget_k < 0 ||
      c->recent_r < 0 || c->evict_every < 1 || c->max_seqs < 1 ||
      c->max_seqs > 65536 || c->attn_split < 0 || c->attn_split % 32 != 0 ||
      (c->budget_mode != RA_BUDGET_EVICTABLE && c->budget_mode != RA_BUDGET_TOTAL) ||
      (c->dtype != RA_F32 && c->dtype != RA_BF16) || c->num_layers > 4096 ||
      (c->layout != RA_LAYOUT_CHRONOLOGICAL && c->layout != RA_LAYOUT_HOLE_FILL &&
       c->layout != RA_LAYOUT_PAGED) ||
      c->policy < RA_POLICY_RANDOM || c->policy > RA_POLICY_EXTERNAL ||
      (c->policy == RA_POLICY_BLOCK && c->policy_block < 1) ||
      c->num_kv_heads > 4096)
    return RA_ERR_INVALID_ARG;
  // kernels with one grid row per (layer, KV head): at most 65,536 of them
  if (static_cast<int64_t>(c->num_layers) * c->num_kv_heads > 65536) return RA_ERR_UNSUPPORTED;
  if (paged(*c)) {
    if (c->page_rows < 32 || c->page_rows > 1024 || log2_exact(c->page_rows) < 0 ||
        c->max_prompt_len < 0 ||
        (c->budget_mode == RA_BUDGET_TOTAL && c->max_prompt_len > c->budget_k))
      return RA_ERR_INVALID_ARG;
    // the eviction kernel holds a sequence's block table in LDS
    if (pages_per_seq(*c) > ra::kMaxPagesLds) return RA_ERR_UNSUPPORTED;
  }
  if (c->head_dim != ra::kHeadDim) return RA_ERR_UNSUPPORTED;
  if (c->num_q_heads / c->num_kv_heads > ra::kMaxGroup) return RA_ERR_UNSUPPORTED;
  if (c->evict_every > ra::kMaxEvery) return RA_ERR_UNSUPPORTED;
  // the selection holds every examined slot's score in registers (hole-fill
  // examines the r most recent slots too)
  if (static_cast<int64_t>(c->budget_k) + c->evict_every +
          (c->layout == RA_LAYOUT_HOLE_FILL ? c->recent_r : 0) > ra::kMaxCandidates)
    return RA_ERR_UNSUPPORTED;
  return RA_OK;
}

int64_t ra_region_rows(const ra_config* c, int32_t prompt_len) {
  const ra_status st = ra_config_check(c);
  if (st != RA_OK) return st;
  if (prompt_len < 0) return RA_ERR_INVALID_ARG;
  const int64_t k = keep_rows(*c, prompt_len);
  if (k < 0) return RA_ERR_BUDGET;
  if (paged(*c) && prompt_len > c->max_prompt_len) return RA_ERR_CAPACITY;
  const int64_t rows = round_up(static_cast<int64_t>(prompt_len) + k + c->recent_r +
                                    c->evict_every,
                                paged(*c) ? c->page_rows : ra::kRegionAlign);
  if (rows > (int64_t(1) << 30)) return RA_ERR_UNSUPPORTED;
  return rows;
}

int64_t ra_seq_rows(const ra_config* c, int32_t prompt_len) {
  const int64_t rows = ra_region_rows(c, prompt_len);
  if (rows < 0) return rows;
  return rows * c->num_layers * c->num_kv_heads;
}

int64_t ra_required_slots(const ra_config* c, const int32_t* prompt_lens, int32_t n_seqs) {
  if (!prompt_lens || n_seqs < 0) return RA_ERR_INVALID_ARG;
  const ra_status st = ra_config_check(c);
  if (st != RA_OK) return st;
  int64_t total = 0;
  for (int32_t i = 0; i < n_seqs; ++i) {
    const int64_t rows = ra_seq_rows(c, prompt_lens[i]);
    if (rows < 0) return rows;
    total += rows;
  }
  return total;
}

size_t ra_meta_bytes(const ra_config* c) {
  if (ra_config_check(c) != RA_OK) return 0;
  return meta_records_bytes(*c) + tables_bytes(*c) + drops_bytes(*c) + arrivals_bytes(*c);
}

size_t ra_workspace_bytes(const ra_config* c) {
  if (ra_config_check(c) != RA_OK) return 0;
  const size_t G = c->num_q_heads / c->num_kv_heads;
  const size_t items = static_cast<size_t>(c->max_seqs) * c->num_kv_heads * ra::kMaxSplits;
  return items * G * (ra::kHeadDim + 2) * sizeof(float) + 256;
}

ra_status ra_cache_create(const ra_config* cfg, void* k_pool, void* v_pool,
                          int32_t* pos_pool, int64_t pool_rows, void* meta,
                          size_t meta_bytes, void* stream, ra_cache** out) {
  if (!out) return RA_ERR_INVALID_ARG;
  *out = nullptr;
  const ra_status st = ra_config_check(cfg);
  if (st != RA_OK) return st;
  if (!k_pool || !v_pool || !pos_pool || !meta || pool_rows <= 0 ||
      pool_rows % ra::kRegionAlign != 0 || meta_bytes < ra_meta_bytes(cfg))
    return RA_ERR_INVALID_ARG;
  const int64_t group_rows = paged(*cfg) ? static_cast<int64_t>(cfg->num_layers) *
                                               cfg->num_kv_heads * cfg->page_rows
                                         : 0;
  if (paged(*cfg) && (pool_rows % group_rows != 0 || pool_rows / group_rows > INT32_MAX))
    return RA_ERR_INVALID_ARG;
  const auto misaligned = [](const void* p) {
    return (reinterpret_cast<uintptr_t>(p) & 15u) != 0;
  };
  if (misaligned(k_pool) || misaligned(v_pool) || misaligned(pos_pool) || misaligned(meta))
    return RA_ERR_INVALID_ARG;
  ra_cache* c = new (std::nothrow) ra_cache();
  if (!c) return RA_ERR_CAPACITY;
  c->cfg = *cfg;
  c->G = cfg->num_q_heads / cfg->num_kv_heads;
  c->elem = cfg->dtype == RA_BF16 ? 2 : 4;
  c->kpool = k_pool;
  c->vpool = v_pool;
  c->pos = pos_pool;
  c->pool_rows = pool_rows;
  c->meta = static_cast<SeqMeta*>(meta);
  c->mirror.assign(cfg->max_seqs, SeqMeta{});
  c->free_rows[0] = pool_rows;
  c->appended.assign(cfg->num_layers, 0);
  if (paged(*cfg)) {
    c->page_rows = cfg->page_rows;
    c->n_groups = pool_rows / group_rows;
    c->pg.tables = reinterpret_cast<const int32_t*>(static_cast<char*>(meta) +
                                                    meta_records_bytes(*cfg));
    c->pg.pages_per_seq = static_cast<int>(pages_per_seq(*cfg));
    c->pg.page_shift = log2_exact(cfg->page_rows);
    c->pg.group_rows = group_rows;
    c->free_groups.resize(c->n_groups);
    for (int64_t i = 0; i < c->n_groups; ++i)
      c->free_groups[i] = static_cast<int32_t>(c->n_groups - 1 - i);   // 0 first
    c->groups.assign(cfg->max_seqs, {});
  }
  if (defers_moves(*cfg))
    c->drops = reinterpret_cast<int32_t*>(static_cast<char*>(meta) + meta_records_bytes(*cfg) +
                                          tables_bytes(*cfg));
  c->arrivals = reinterpret_cast<int32_t*>(static_cast<char*>(meta) + meta_records_bytes(*cfg) +
                                           tables_bytes(*cfg) + drops_bytes(*cfg));
  const hipError_t e = ra::launch_zero_words(static_cast<uint32_t*>(meta),
                                             static_cast<int64_t>(ra_meta_bytes(cfg) / 4),
                                             static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    delete c;
    return hip_fail(e);
  }
  // the allocation-free attention's partials: this device's copy of the
  // library's static array (looked up once per device, with it current)
  const hipError_t es = ra::scratch_address(&c->scratch);
  if (es != hipSuccess) {
    delete c;
    return hip_fail(es);
  }
  *out = c;
  return RA_OK;
}

ra_status ra_cache_destroy(ra_cache* c) {
  if (!c) return RA_ERR_INVALID_ARG;
  delete c;
  return RA_OK;
}

ra_status ra_get_seq_info(const ra_cache* c, int32_t seq, ra_seq_info* out) {
  if (!c || !out || seq < 0 || seq >= c->cfg.max_seqs) return RA_ERR_INVALID_ARG;
  const SeqMeta& M = c->mirror[seq];
  out->active = M.active;
  out->prompt_len = M.prompt_len;
  out->len = M.len;
  out->step = M.step;
  out->event = M.event;
  out->k_keep = M.k_keep;
  out->cap = M.cap;
  out->base = M.base;
  out->move_pending = M.due == ra::kDueMovePending;
  return RA_OK;
}

ra_status ra_attention_plan(const ra_cache* c, int32_t* split_keys, int32_t* max_splits,
                            int32_t* waves) {
  if (!c || !split_keys || !max_splits) return RA_ERR_INVALID_ARG;
  const Plan p = attention_plan(c);
  *split_keys = p.split_keys;
  *max_splits = p.max_splits;
  if (waves) *waves = p.waves;
  return RA_OK;
}

ra_status ra_pool_info(const ra_cache* c, int64_t* used_rows, int64_t* free_rows) {
  if (!c) return RA_ERR_INVALID_ARG;
  int64_t free = 0;
  if (c->is_paged()) {
    free = static_cast<int64_t>(c->free_groups.size()) * c->pg.group_rows;
  } else {
    for (const auto& kv : c->free_rows) free += kv.second;
  }
  if (used_rows) *used_rows = c->pool_rows - free;
  if (free_rows) *free_rows = free;
  return RA_OK;
}

ra_status ra_seq_begin(ra_cache* c, int32_t seq, int32_t prompt_len, uint64_t seed,
                       uint64_t request_id, const void* dev_k_prompt,
                       const void* dev_v_prompt, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || prompt_len < 0 ||
      (dev_k_prompt == nullptr) != (dev_v_prompt == nullptr))
    return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  if (c->mirror[seq].active) return RA_ERR_STATE;
  const int64_t cap = ra_region_rows(&c->cfg, prompt_len);
  if (cap < 0) return static_cast<ra_status>(cap);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (c->is_paged()) {
    // pages for the prompt rows; the first append takes the next page
    if (c->groups_short(seq, prompt_len) > static_cast<int64_t>(c->free_groups.size()))
      return RA_ERR_CAPACITY;
    SeqMeta M{};
    M.prompt_len = prompt_len;
    M.len = prompt_len;
    M.k_keep = static_cast<int32_t>(keep_rows(c->cfg, prompt_len));
    M.seed = seed;
    M.rid = request_id;
    M.active = 1;
    std::vector<ra::TableEntry> te;
    c->grow(seq, prompt_len, te);
    M.cap = c->mirror[seq].cap;
    hipError_t e = ra::launch_table_set(c->shape(), te.data(), static_cast<int>(te.size()), s);
    if (e == hipSuccess)
      e = ra::launch_write_rows(c->shape(), M, seq, prompt_len, dev_k_prompt, dev_v_prompt,
                                nullptr, c->kpool, c->vpool, c->pos, s);
    if (e == hipSuccess) e = ra::launch_seq_set(c->meta, seq, M, s);
    if (e != hipSuccess) {   // the slot stays inactive: its pages go back
      c->shrink(seq, 0);
      return hip_fail(e);
    }
    c->mirror[seq] = M;
    c->update_range();
    return RA_OK;
  }
  const int64_t need = cap * c->cfg.num_layers * c->cfg.num_kv_heads;
  auto it = c->free_rows.begin();
  for (; it != c->free_rows.end(); ++it)
    if (it->second >= need) break;
  if (it == c->free_rows.end()) return RA_ERR_CAPACITY;
  const int64_t base = it->first;

  SeqMeta M{};
  M.base = base;
  M.cap = static_cast<int32_t>(cap);
  M.prompt_len = prompt_len;
  M.len = prompt_len;
  M.k_keep = static_cast<int32_t>(keep_rows(c->cfg, prompt_len));
  M.seed = seed;
  M.rid = request_id;
  M.active = 1;
  // rows first, then the metadata that makes the slot active: a failed launch
  // leaves the slot inactive on the device as in the mirror
  RA_LAUNCH(ra::launch_write_rows(c->shape(), M, seq, prompt_len, dev_k_prompt,
                                  dev_v_prompt, nullptr, c->kpool, c->vpool, c->pos, s));
  RA_LAUNCH(ra::launch_seq_set(c->meta, seq, M, s));
  const int64_t rest = it->second - need;
  c->free_rows.erase(it);
  if (rest > 0) c->free_rows[base + need] = rest;
  c->mirror[seq] = M;
  c->update_range();
  return RA_OK;
}

ra_status ra_seq_end(ra_cache* c, int32_t seq, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs) return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  SeqMeta off{};
  RA_LAUNCH(ra::launch_seq_set(c->meta, seq, off, static_cast<hipStream_t>(stream)));
  if (c->is_paged()) {
    c->shrink(seq, 0);
    M = SeqMeta{};
    c->update_range();
    return RA_OK;
  }
  int64_t base = M.base;
  int64_t rows = static_cast<int64_t>(M.cap) * c->cfg.num_layers * c->cfg.num_kv_heads;
  // return the rows to the free list, merging with neighbours
  auto next = c->free_rows.lower_bound(base);
  if (next != c->free_rows.end() && base + rows == next->first) {
    rows += next->second;
    next = c->free_rows.erase(next);
  }
  if (next != c->free_rows.begin()) {
    auto prev = std::prev(next);
    if (prev->first + prev->second == base) {
      base = prev->first;
      rows += prev->second;
      c->free_rows.erase(prev);
    }
  }
  c->free_rows[base] = rows;
  M = SeqMeta{};
  c->update_range();
  return RA_OK;
}

ra_status ra_decode_attention(ra_cache* c, int32_t layer, const void* q,
                              const void* k_new, const void* v_new, void* out,
                              void* workspace, size_t workspace_bytes,
                              void* stream) {
  const ra_status st = check_decode(c, layer, q, k_new, v_new, out);
  if (st != RA_OK) return st;
  if (!workspace || workspace_bytes < ra_workspace_bytes(&c->cfg)) return RA_ERR_INVALID_ARG;
  const size_t items = static_cast<size_t>(c->cfg.max_seqs) * c->cfg.num_kv_heads * ra::kMaxSplits;
  float* ws = static_cast<float*>(workspace);
  return launch_decode(c, layer, q, k_new, v_new, out, attention_plan(c), ws,
                       ws + items * c->G * ra::kHeadDim, ra::kMaxSplits,
                       static_cast<hipStream_t>(stream));
}

ra_status ra_decode_attention_noalloc(ra_cache* c, int32_t layer, const void* q,
                                      const void* k_new, const void* v_new, void* out,
                                      void* stream) {
  const ra_status st = check_decode(c, layer, q, k_new, v_new, out);
  if (st != RA_OK) return st;
  if (!c->scratch) return RA_ERR_STATE;
  // partial slots only for the splits this launch has, packed per head
  const Plan plan = attention_plan(c);
  const size_t items = static_cast<size_t>(c->slot_hi) * c->cfg.num_kv_heads * plan.max_splits;
  const size_t floats = items * c->G * ra::kHeadDim;
  const bool partials = c->cfg.dtype == RA_F32 || plan.max_splits > 1;
  if (partials && (floats + items * c->G * 2) * sizeof(float) > ra::kNoAllocScratchBytes)
    return RA_ERR_CAPACITY;
  float* ws = static_cast<float*>(c->scratch);
  return launch_decode(c, layer, q, k_new, v_new, out, plan, ws, ws + floats,
                       std::max(1, plan.max_splits), static_cast<hipStream_t>(stream));
}

ra_status ra_end_step(ra_cache* c, void* stream, int32_t* n_evicted) {
  if (!c) return RA_ERR_INVALID_ARG;
  if (n_evicted) *n_evicted = 0;
  bool any_active = c->slot_hi > c->slot_lo;
  // a step is open once a layer is appended and must append every layer;
  // with no active sequence, ending a step nothing was appended to is a no-op
  if (c->n_appended != 0 && c->n_appended != c->cfg.num_layers) return RA_ERR_STATE;
  if (any_active && c->n_appended != c->cfg.num_layers) return RA_ERR_STATE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  std::fill(c->appended.begin(), c->appended.end(), 0);
  c->n_appended = 0;
  if (!any_active) return RA_OK;
  RA_LAUNCH(ra::launch_advance(c->meta, c->slot_lo, c->slot_hi, 1, c->cfg.recent_r,
                               trigger_every(c->cfg), s));
  if (c->graph) {
    // every head's workgroup reads on the device whether its sequence is
    // due; the mirror stays that of the entry into graph mode
    RA_LAUNCH(by_slot_chunks(c->cfg, c->slot_lo, c->slot_hi, [&](int lo, int hi) {
      return ra::launch_evict(c->shape(), c->meta, c->kpool, c->vpool, c->pos, lo, hi,
                              c->graph_candidates, false, s);
    }));
    return RA_OK;
  }
  int due = 0;
  for (int i = c->slot_lo; i < c->slot_hi; ++i) {
    SeqMeta& M = c->mirror[i];
    if (!M.active) continue;
    M.step += 1;
    M.len += 1;
    mirror_plan(M, c->cfg.recent_r, at_trigger(c->cfg, M.step));   // clears a pending move
    due += M.due;
    // the pages past the new length are free once the event (launched below,
    // ahead of any later use of them on this stream) has moved their rows
    if (M.due && c->is_paged()) c->shrink(i, M.len);
  }
  if (due) {
    // When every active sequence evicts at this step and the next step's
    // attention gives every head one work item, the event only selects
    // (positions compacted, each head's drop list kept) and that attention,
    // which reads every row anyway, moves the key/value rows
    // (attn_bf16_move_kernel): the rows are read once instead of twice.
    // Sequences evicting on staggered phases keep the event's own moves, so
    // that steps of heads with nothing to move run the streaming kernel.
    int n_active = 0;
    for (int i = c->slot_lo; i < c->slot_hi; ++i) n_active += c->mirror[i].active;
    const bool defer = c->drops && due == n_active && attention_plan(c).max_splits == 1;
    const int candidates = c->max_candidates_due();
    RA_LAUNCH(by_slot_chunks(c->cfg, c->slot_lo, c->slot_hi, [&](int lo, int hi) {
      return ra::launch_evict(c->shape(), c->meta, c->kpool, c->vpool, c->pos, lo, hi,
                              candidates, defer, s, defer ? c->drops : nullptr,
                              c->cfg.evict_every);
    }));
    if (defer) {
      RA_LAUNCH(ra::launch_mark_pending(c->meta, c->slot_lo, c->slot_hi, s));
      for (int i = c->slot_lo; i < c->slot_hi; ++i)
        if (c->mirror[i].active && c->mirror[i].due) c->mirror[i].due = ra::kDueMovePending;
    }
  }
  if (n_evicted) *n_evicted = due;
  return RA_OK;
}

ra_status ra_graph_mode(ra_cache* c, int32_t on, void* stream) {
  if (!c || (on != 0 && on != 1)) return RA_ERR_INVALID_ARG;
  if (c->step_open()) return RA_ERR_STATE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (on) {
    if (c->graph) return RA_OK;
    // page groups are handed out by the host as rows grow, and rows piling
    // up under the external policy need the host's capacity checks
    if (c->is_paged() || c->cfg.policy == RA_POLICY_EXTERNAL) return RA_ERR_UNSUPPORTED;
    int cap_max = 32, n_active = 0, candidates = 0;
    for (int i = c->slot_lo; i < c->slot_hi; ++i) {
      const SeqMeta& M = c->mirror[i];
      if (!M.active) continue;
      cap_max = std::max(cap_max, M.cap);      // no cache outgrows its region
      candidates = std::max(candidates, M.cap - M.prompt_len);
      ++n_active;
    }
    if (candidates > ra::kMaxCandidates) return RA_ERR_UNSUPPORTED;
    const ra_status fl = flush_pending(c, s);
    if (fl != RA_OK) return fl;
    const Plan p = plan_for(c, cap_max, n_active);
    c->graph_split_keys = p.split_keys;
    c->graph_max_splits = p.max_splits;
    c->graph_waves = p.waves;
    c->graph_wide_regs = p.wide_regs;
    c->graph_candidates = candidates;
    c->graph = true;
    return RA_OK;
  }
  if (!c->graph) return RA_OK;
  // the records the device advanced become the mirror again
  std::vector<SeqMeta> dev(c->cfg.max_seqs);
  RA_LAUNCH(hipMemcpyAsync(dev.data(), c->meta, sizeof(SeqMeta) * dev.size(),
                           hipMemcpyDeviceToHost, s));
  RA_LAUNCH(hipStreamSynchronize(s));
  for (int i = c->slot_lo; i < c->slot_hi; ++i) {
    if (!c->mirror[i].active) continue;
    if (!dev[i].active || dev[i].base != c->mirror[i].base || dev[i].cap != c->mirror[i].cap)
      return RA_ERR_STATE;
    c->mirror[i] = dev[i];
  }
  c->graph = false;
  return RA_OK;
}

ra_status ra_evict_now(ra_cache* c, int32_t seq, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs) return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  // the drop list of one event holds at most kMaxEvery rows (more can pile up
  // only when no end-of-step rule evicts, i.e. under the external policy)
  if (M.len - M.prompt_len - c->cfg.recent_r - M.k_keep > ra::kMaxEvery) return RA_ERR_STATE;
  // the select holds every examined slot's key in registers: more slots than
  // it supports (only reachable with rows piled up under the external policy)
  if (M.len - M.prompt_len - (c->cfg.layout == RA_LAYOUT_HOLE_FILL ? 0 : c->cfg.recent_r) >
      ra::kMaxCandidates)
    return RA_ERR_UNSUPPORTED;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const ra_status fl = flush_pending(c, s);
  if (fl != RA_OK) return fl;
  RA_LAUNCH(ra::launch_plan_now(c->meta, seq, c->cfg.recent_r, s));
  for (int i = c->slot_lo; i < c->slot_hi; ++i) c->mirror[i].due = 0;
  mirror_plan(M, c->cfg.recent_r, true);
  if (M.due) {
    if (c->is_paged()) c->shrink(seq, M.len);
    RA_LAUNCH(ra::launch_evict(c->shape(), c->meta, c->kpool, c->vpool, c->pos, seq,
                               seq + 1, c->span(M), false, s));
  }
  return RA_OK;
}

namespace {

// Positions-only advance of the active sequences of slots [lo, hi) by
// n_steps (the whole active range for ra_fast_forward, one slot for
// ra_seq_fast_forward); the other slots' records and rows are not touched
// (their deferred moves, if any, stay pending).
ra_status fast_forward_range(ra_cache* c, int lo, int hi, int32_t n_steps, hipStream_t s) {
  const int every = c->cfg.evict_every;
  bool pending = false;
  for (int i = lo; i < hi; ++i) pending = pending || c->mirror[i].due == ra::kDueMovePending;
  if (pending) {
    const ra_status fl = flush_pending(c, s);
    if (fl != RA_OK) return fl;
  }
  // Runs of steps up to the next trigger of any sequence.  The first pass
  // replays them on a copy of the mirror only, so that a capacity error (rows
  // piling up under the external policy) is reported before any launch; the
  // second pass launches and updates the mirror.
  std::vector<SeqMeta> saved = c->mirror;
  const std::vector<int32_t> saved_free = c->free_groups;
  const std::vector<std::vector<int32_t>> saved_groups = c->groups;
  auto restore = [&]() {
    c->mirror = saved;
    c->free_groups = saved_free;
    c->groups = saved_groups;
  };
  for (int pass = 0; pass < 2; ++pass) {
    const bool launch = pass == 1;
    if (launch) restore();
    int remaining = n_steps;
    while (remaining > 0 && hi > lo) {
      int run = remaining;
      for (int i = lo; i < hi; ++i)
        if (c->mirror[i].active) run = std::min(run, every - c->mirror[i].step % every);
      if (c->is_paged()) {
        // pages for the run's rows
        int64_t short_groups = 0;
        bool fits = true;
        for (int i = lo; i < hi; ++i) {
          if (!c->mirror[i].active) continue;
          fits = fits && c->fits_table(c->mirror[i].len + run);
          short_groups += c->groups_short(i, c->mirror[i].len + run);
        }
        if (!fits || short_groups > static_cast<int64_t>(c->free_groups.size())) {
          restore();
          return RA_ERR_CAPACITY;
        }
        std::vector<ra::TableEntry> te;
        for (int i = lo; i < hi; ++i)
          if (c->mirror[i].active) c->grow(i, c->mirror[i].len + run, te);
        if (launch && !te.empty())
          RA_LAUNCH(ra::launch_table_set(c->shape(), te.data(), static_cast<int>(te.size()), s));
      } else {
        for (int i = lo; i < hi; ++i) {
          const SeqMeta& M = c->mirror[i];
          if (M.active && M.len + run > M.cap) {
            restore();
            return RA_ERR_CAPACITY;
          }
        }
      }
      if (launch) {
        RA_LAUNCH(ra::launch_append_positions(c->shape(), c->meta, c->pos, lo, hi, run, s));
        RA_LAUNCH(ra::launch_advance(c->meta, lo, hi, run, c->cfg.recent_r,
                                     trigger_every(c->cfg), s));
      }
      int due = 0, candidates = 0;
      for (int i = lo; i < hi; ++i) {
        SeqMeta& M = c->mirror[i];
        if (!M.active) continue;
        M.step += run;
        M.len += run;
        mirror_plan(M, c->cfg.recent_r, at_trigger(c->cfg, M.step));
        due += M.due;
        if (M.due) candidates = std::max(candidates, c->span(M));
        if (M.due && c->is_paged()) c->shrink(i, M.len);
      }
      if (due && launch) {
        RA_LAUNCH(by_slot_chunks(c->cfg, lo, hi, [&](int a, int b) {
          return ra::launch_evict(c->shape(), c->meta, c->kpool, c->vpool, c->pos, a, b,
                                  candidates, true, s);
        }));
      }
      remaining -= run;
    }
  }
  return RA_OK;
}

}  // namespace

ra_status ra_fast_forward(ra_cache* c, int32_t n_steps, void* stream) {
  if (!c || n_steps < 0) return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  return fast_forward_range(c, c->slot_lo, c->slot_hi, n_steps,
                            static_cast<hipStream_t>(stream));
}

ra_status ra_seq_fast_forward(ra_cache* c, int32_t seq, int32_t n_steps, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || n_steps < 0) return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  if (!c->mirror[seq].active) return RA_ERR_STATE;
  return fast_forward_range(c, seq, seq + 1, n_steps, static_cast<hipStream_t>(stream));
}

ra_status ra_export_positions(ra_cache* c, int32_t seq, int32_t* dev_out,
                              int64_t out_elems, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs) return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  const SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  if (!dev_out && M.len > 0) return RA_ERR_INVALID_ARG;   // nothing to copy: may be NULL
  if (out_elems < static_cast<int64_t>(M.len) * c->cfg.num_layers * c->cfg.num_kv_heads)
    return RA_ERR_CAPACITY;
  RA_LAUNCH(ra::launch_export_positions(c->shape(), M, seq, M.len, c->pos, dev_out,
                                        static_cast<hipStream_t>(stream)));
  return RA_OK;
}

ra_status ra_write_rows(ra_cache* c, int32_t seq, const void* dev_k, const void* dev_v,
                        void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs) return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  const SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  if ((!dev_k || !dev_v) && M.len > 0) return RA_ERR_INVALID_ARG;   // NULL only if empty
  const ra_status fl = flush_pending(c, static_cast<hipStream_t>(stream));
  if (fl != RA_OK) return fl;
  // positions are left as they are: pass the region's own positions through
  RA_LAUNCH(ra::launch_write_rows(c->shape(), M, seq, M.len, dev_k, dev_v, nullptr,
                                  c->kpool, c->vpool, nullptr, static_cast<hipStream_t>(stream)));
  return RA_OK;
}

ra_status ra_read_rows(ra_cache* c, int32_t seq, int32_t layer, int32_t kv_head,
                       void* dev_k_out, void* dev_v_out, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || layer < 0 ||
      layer >= c->cfg.num_layers || kv_head < 0 || kv_head >= c->cfg.num_kv_heads)
    return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  const SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  const ra_status fl = flush_pending(c, static_cast<hipStream_t>(stream));
  if (fl != RA_OK) return fl;
  RA_LAUNCH(ra::launch_read_rows(c->shape(), M, seq, layer * c->cfg.num_kv_heads + kv_head,
                                 M.len, c->kpool, c->vpool, dev_k_out, dev_v_out,
                                 static_cast<hipStream_t>(stream)));
  return RA_OK;
}

ra_status ra_window_select(ra_cache* c, int32_t seq_lo, int32_t seq_hi,
                           const void* dev_q_window, float* dev_scores,
                           int32_t scores_stride, int32_t* dev_drops, void* stream) {
  if (!c || seq_lo < 0 || seq_hi > c->cfg.max_seqs || seq_lo >= seq_hi || !dev_q_window)
    return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->cfg.dtype != RA_BF16 || c->cfg.layout != RA_LAYOUT_CHRONOLOGICAL)
    return RA_ERR_UNSUPPORTED;
  if (static_cast<int64_t>(seq_hi - seq_lo) * c->cfg.num_layers * c->cfg.num_kv_heads >
      kMaxHeadsPerLaunch)
    return RA_ERR_UNSUPPORTED;            // one launch per call (measurement only)
  if (c->step_open()) return RA_ERR_STATE;
  int max_len = 0;
  for (int s = seq_lo; s < seq_hi; ++s) {
    const SeqMeta& M = c->mirror[s];
    if (!M.active) continue;
    if (M.step < 64) return RA_ERR_STATE;           // a full 64-query window
    if (M.len - M.prompt_len - c->cfg.recent_r - M.k_keep > c->cfg.evict_every)
      return RA_ERR_STATE;
    max_len = std::max(max_len, M.len);
  }
  if (max_len == 0) return RA_OK;
  if (dev_scores && scores_stride < max_len) return RA_ERR_INVALID_ARG;
  if (max_len - c->cfg.recent_r > 512 * 32) return RA_ERR_UNSUPPORTED;
  const ra_status fl = flush_pending(c, static_cast<hipStream_t>(stream));
  if (fl != RA_OK) return fl;
  RA_LAUNCH(ra::launch_window_score(c->shape(), c->meta, c->kpool, c->pos, dev_q_window,
                                    dev_scores, dev_drops, scores_stride, seq_lo, seq_hi,
                                    max_len, static_cast<hipStream_t>(stream)));
  return RA_OK;
}

size_t ra_scored_scratch_bytes(const ra_config* cfg, int32_t max_prompt_len) {
  if (ra_config_check(cfg) != RA_OK || max_prompt_len < 0) return 0;
  const int64_t cap = ra_region_rows(cfg, max_prompt_len);
  if (cap < 0) return 0;
  const size_t heads = static_cast<size_t>(cfg->max_seqs) * cfg->num_layers * cfg->num_kv_heads;
  return heads * (static_cast<size_t>(cfg->evict_every) + 2 * static_cast<size_t>(round_up(cap, 64))) *
         sizeof(int32_t);
}

ra_status ra_scored_evict(ra_cache* c, int32_t seq_lo, int32_t seq_hi,
                          const ra_scorer_params* prm, const void* dev_q_window,
                          void* dev_scratch, size_t scratch_bytes, void* stream) {
  if (!c || !prm || seq_lo < 0 || seq_hi > c->cfg.max_seqs || seq_lo >= seq_hi ||
      !dev_q_window || !dev_scratch)
    return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (prm->scorer < RA_SCORER_SNAPKV || prm->scorer > RA_SCORER_VASE)
    return RA_ERR_INVALID_ARG;
  if (static_cast<int64_t>(seq_hi - seq_lo) * c->cfg.num_layers * c->cfg.num_kv_heads >
      kMaxHeadsPerLaunch)
    return RA_ERR_UNSUPPORTED;            // one launch per call (measurement only)
  if (c->cfg.dtype != RA_BF16 || c->cfg.layout != RA_LAYOUT_CHRONOLOGICAL)
    return RA_ERR_UNSUPPORTED;
  if (prm->scorer == RA_SCORER_RKV &&
      (!(prm->rkv_lambda >= 0.f && prm->rkv_lambda <= 1.f) || prm->rkv_recent_dups < 0 ||
       !std::isfinite(prm->rkv_threshold)))
    return RA_ERR_INVALID_ARG;
  if (c->step_open()) return RA_ERR_STATE;
  const int r = c->cfg.recent_r, every = c->cfg.evict_every;
  int max_len = 0, max_cap = 0, due = 0;
  for (int s = seq_lo; s < seq_hi; ++s) {
    const SeqMeta& M = c->mirror[s];
    if (!M.active) continue;
    const int m = M.len - M.prompt_len - r - M.k_keep;
    if (m <= 0) continue;
    if (M.step < 64 || m > every) return RA_ERR_STATE;
    max_len = std::max(max_len, M.len);
    max_cap = std::max(max_cap, M.cap);
    ++due;
  }
  if (!due) return RA_OK;
  if (max_len - r > 512 * 32) return RA_ERR_UNSUPPORTED;

  const size_t heads = static_cast<size_t>(seq_hi - seq_lo) * c->cfg.num_layers *
                       c->cfg.num_kv_heads;
  const int score_stride = static_cast<int>(round_up(max_cap, 64));
  if (scratch_bytes < heads * (static_cast<size_t>(every) + 2 * score_stride) * sizeof(int32_t))
    return RA_ERR_INVALID_ARG;
  int32_t* drops = static_cast<int32_t*>(dev_scratch);
  float* scores = reinterpret_cast<float*>(drops + heads * every);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const ra_status fl = flush_pending(c, s);
  if (fl != RA_OK) return fl;
  // 1. score and select on the current rows; 2. the plan rule (new length,
  // event count) on device and mirror; 3. compaction from the drop lists
  if (prm->scorer == RA_SCORER_SNAPKV) {
    RA_LAUNCH(ra::launch_window_score(c->shape(), c->meta, c->kpool, c->pos, dev_q_window,
                                      nullptr, drops, score_stride, seq_lo, seq_hi, max_len, s));
  } else {
    RA_LAUNCH(ra::launch_window_score(c->shape(), c->meta, c->kpool, c->pos, dev_q_window,
                                      scores, nullptr, score_stride, seq_lo, seq_hi, max_len, s));
    RA_LAUNCH(ra::launch_scored_select(c->shape(), prm->scorer, c->meta, c->kpool, c->vpool,
                                       c->pos, scores, scores + heads * score_stride,
                                       score_stride, drops, seq_lo, seq_hi, max_len,
                                       prm->rkv_lambda, prm->rkv_threshold,
                                       prm->rkv_recent_dups, prm->vase_n_large,
                                       prm->vase_seed, s));
  }
  RA_LAUNCH(ra::launch_plan_range(c->meta, seq_lo, seq_hi, r, s));
  for (int i = c->slot_lo; i < c->slot_hi; ++i) c->mirror[i].due = 0;
  for (int i = seq_lo; i < seq_hi; ++i)
    if (c->mirror[i].active) mirror_plan(c->mirror[i], r, true);
  RA_LAUNCH(by_slot_chunks(c->cfg, seq_lo, seq_hi, [&](int lo, int hi) {
    return ra::launch_compact_drops(c->shape(), c->meta, c->kpool, c->vpool, c->pos, drops,
                                    every, lo, hi, s);
  }));
  return RA_OK;
}

ra_status ra_read_positions(ra_cache* c, int32_t seq, int32_t layer, int32_t kv_head,
                            int32_t* host_out, int32_t host_cap, int32_t* n_out,
                            void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || layer < 0 ||
      layer >= c->cfg.num_layers || kv_head < 0 || kv_head >= c->cfg.num_kv_heads ||
      !host_out || !n_out)
    return RA_ERR_INVALID_ARG;
  if (c->graph) return RA_ERR_STATE;   // needs the host mirror (ra_graph_mode)
  if (c->step_open()) return RA_ERR_STATE;
  const SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  *n_out = M.len;
  if (host_cap < M.len) return RA_ERR_CAPACITY;
  const int lg = layer * c->cfg.num_kv_heads + kv_head;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (c->is_paged()) {
    // one copy per page of the head
    for (int64_t k = 0; k * c->page_rows < M.len; ++k) {
      const int64_t first = static_cast<int64_t>(c->groups[seq][k]) * c->pg.group_rows +
                            static_cast<int64_t>(lg) * c->page_rows;
      const int64_t n = std::min<int64_t>(c->page_rows, M.len - k * c->page_rows);
      RA_LAUNCH(hipMemcpyAsync(host_out + k * c->page_rows, c->pos + first,
                               sizeof(int32_t) * n, hipMemcpyDeviceToHost, s));
    }
  } else if (M.len > 0) {
    const int64_t region = M.base + static_cast<int64_t>(lg) * M.cap;
    RA_LAUNCH(hipMemcpyAsync(host_out, c->pos + region, sizeof(int32_t) * M.len,
                             hipMemcpyDeviceToHost, s));
  }
  RA_LAUNCH(hipStreamSynchronize(s));
  return RA_OK;
}

}  // extern "C"
