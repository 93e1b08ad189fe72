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
  void* scratch = nullptr;               // device address of the no-alloc partials

  ra::Shape shape() const {
    return ra::Shape{cfg.num_layers, cfg.num_q_heads, cfg.num_kv_heads, G,
                     cfg.recent_r, cfg.evict_every, cfg.dtype, cfg.layout,
                     cfg.policy, std::max(1, cfg.policy_block)};
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

Plan attention_plan(const ra_cache* c) {
  // sized by the longest cache of this step (cached rows + the new one), so
  // that while sequences are younger than their budget no wavefront or split
  // is planned over rows that do not exist yet
  int keys_max = 32, n_active = 0;
  for (int s = c->slot_lo; s < c->slot_hi; ++s) {
    if (!c->mirror[s].active) continue;
    keys_max = std::max(keys_max, c->mirror[s].len + 1);
    ++n_active;
  }
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

// Host checks shared by both attention entry points; nothing is launched.
ra_status check_decode(const ra_cache* c, int32_t layer, const void* q, const void* k_new,
                       const void* v_new, const void* out) {
  if (!c || layer < 0 || layer >= c->cfg.num_layers || !q || !k_new || !v_new || !out)
    return RA_ERR_INVALID_ARG;
  if (c->appended[layer]) return RA_ERR_STATE;
  for (int s = c->slot_lo; s < c->slot_hi; ++s)
    if (c->mirror[s].active && c->mirror[s].len + 1 > c->mirror[s].cap) return RA_ERR_CAPACITY;
  return RA_OK;
}

// Marks the layer appended and launches its append + attention with the
// given partials buffers (split_stride partial slots per head).
ra_status launch_decode(ra_cache* c, int32_t layer, const void* q, const void* k_new,
                        const void* v_new, void* out, const Plan& plan, float* ws_o,
                        float* ws_ml, int split_stride, hipStream_t stream) {
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
  a.waves = plan.waves;
  a.wide_regs = plan.wide_regs;
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
      (c->layout != RA_LAYOUT_CHRONOLOGICAL && c->layout != RA_LAYOUT_HOLE_FILL) ||
      c->policy < RA_POLICY_RANDOM || c->policy > RA_POLICY_EXTERNAL ||
      (c->policy == RA_POLICY_BLOCK && c->policy_block < 1) ||
      c->num_kv_heads > 4096)
    return RA_ERR_INVALID_ARG;
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
  const int64_t rows = round_up(static_cast<int64_t>(prompt_len) + k + c->recent_r +
                                    c->evict_every, ra::kRegionAlign);
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
  const size_t metas = sizeof(SeqMeta) * static_cast<size_t>(c->max_seqs);
  return round_up(static_cast<int64_t>(metas), 256);
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

ra_status ra_seq_begin(ra_cache* c, int32_t seq, int32_t prompt_len, uint64_t seed,
                       uint64_t request_id, const void* dev_k_prompt,
                       const void* dev_v_prompt, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || prompt_len < 0 ||
      (dev_k_prompt == nullptr) != (dev_v_prompt == nullptr))
    return RA_ERR_INVALID_ARG;
  if (c->step_open()) return RA_ERR_STATE;
  if (c->mirror[seq].active) return RA_ERR_STATE;
  const int64_t cap = ra_region_rows(&c->cfg, prompt_len);
  if (cap < 0) return static_cast<ra_status>(cap);
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
  const hipStream_t s = static_cast<hipStream_t>(stream);
  // rows first, then the metadata that makes the slot active: a failed launch
  // leaves the slot inactive on the device as in the mirror
  RA_LAUNCH(ra::launch_write_rows(c->shape(), base, M.cap, prompt_len, dev_k_prompt,
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
  if (c->step_open()) return RA_ERR_STATE;
  SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  SeqMeta off{};
  RA_LAUNCH(ra::launch_seq_set(c->meta, seq, off, static_cast<hipStream_t>(stream)));
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
  if (any_active && c->n_appended != c->cfg.num_layers) return RA_ERR_STATE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  std::fill(c->appended.begin(), c->appended.end(), 0);
  c->n_appended = 0;
  if (!any_active) return RA_OK;
  RA_LAUNCH(ra::launch_advance(c->meta, c->slot_lo, c->slot_hi, 1, c->cfg.recent_r,
                               trigger_every(c->cfg), s));
  int due = 0;
  for (int i = c->slot_lo; i < c->slot_hi; ++i) {
    SeqMeta& M = c->mirror[i];
    if (!M.active) continue;
    M.step += 1;
    M.len += 1;
    mirror_plan(M, c->cfg.recent_r, at_trigger(c->cfg, M.step));
    due += M.due;
  }
  if (due) {
    RA_LAUNCH(ra::launch_evict(c->shape(), c->meta, c->kpool, c->vpool, c->pos,
                               c->slot_lo, c->slot_hi, c->max_candidates_due(), false, s));
  }
  if (n_evicted) *n_evicted = due;
  return RA_OK;
}

ra_status ra_evict_now(ra_cache* c, int32_t seq, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs) return RA_ERR_INVALID_ARG;
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
  RA_LAUNCH(ra::launch_plan_now(c->meta, seq, c->cfg.recent_r, s));
  for (int i = c->slot_lo; i < c->slot_hi; ++i) c->mirror[i].due = 0;
  mirror_plan(M, c->cfg.recent_r, true);
  if (M.due) {
    RA_LAUNCH(ra::launch_evict(c->shape(), c->meta, c->kpool, c->vpool, c->pos, seq,
                               seq + 1, c->span(M), false, s));
  }
  return RA_OK;
}

ra_status ra_fast_forward(ra_cache* c, int32_t n_steps, void* stream) {
  if (!c || n_steps < 0) return RA_ERR_INVALID_ARG;
  if (c->step_open()) return RA_ERR_STATE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int every = c->cfg.evict_every;
  // Runs of steps up to the next trigger of any sequence.  The first pass
  // replays them on a copy of the mirror only, so that a capacity error (rows
  // piling up under the external policy) is reported before any launch; the
  // second pass launches and updates the mirror.
  std::vector<SeqMeta> saved = c->mirror;
  for (int pass = 0; pass < 2; ++pass) {
    const bool launch = pass == 1;
    if (launch) c->mirror = saved;
    int remaining = n_steps;
    while (remaining > 0 && c->slot_hi > c->slot_lo) {
      int run = remaining;
      for (int i = c->slot_lo; i < c->slot_hi; ++i)
        if (c->mirror[i].active) run = std::min(run, every - c->mirror[i].step % every);
      for (int i = c->slot_lo; i < c->slot_hi; ++i) {
        const SeqMeta& M = c->mirror[i];
        if (M.active && M.len + run > M.cap) {
          c->mirror = saved;
          return RA_ERR_CAPACITY;
        }
      }
      if (launch) {
        RA_LAUNCH(ra::launch_append_positions(c->meta, c->pos, c->slot_lo, c->slot_hi,
                                              c->cfg.num_layers, c->cfg.num_kv_heads, run, s));
        RA_LAUNCH(ra::launch_advance(c->meta, c->slot_lo, c->slot_hi, run, c->cfg.recent_r,
                                     trigger_every(c->cfg), s));
      }
      int due = 0;
      for (int i = c->slot_lo; i < c->slot_hi; ++i) {
        SeqMeta& M = c->mirror[i];
        if (!M.active) continue;
        M.step += run;
        M.len += run;
        mirror_plan(M, c->cfg.recent_r, at_trigger(c->cfg, M.step));
        due += M.due;
      }
      if (due && launch) {
        RA_LAUNCH(ra::launch_evict(c->shape(), c->meta, c->kpool, c->vpool, c->pos,
                                   c->slot_lo, c->slot_hi, c->max_candidates_due(), true, s));
      }
      remaining -= run;
    }
  }
  return RA_OK;
}

ra_status ra_export_positions(ra_cache* c, int32_t seq, int32_t* dev_out,
                              int64_t out_elems, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || !dev_out) return RA_ERR_INVALID_ARG;
  if (c->step_open()) return RA_ERR_STATE;
  const SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  if (out_elems < static_cast<int64_t>(M.len) * c->cfg.num_layers * c->cfg.num_kv_heads)
    return RA_ERR_CAPACITY;
  RA_LAUNCH(ra::launch_export_positions(c->shape(), M.base, M.cap, M.len, c->pos, dev_out,
                                        static_cast<hipStream_t>(stream)));
  return RA_OK;
}

ra_status ra_write_rows(ra_cache* c, int32_t seq, const void* dev_k, const void* dev_v,
                        void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || !dev_k || !dev_v) return RA_ERR_INVALID_ARG;
  if (c->step_open()) return RA_ERR_STATE;
  const SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  // positions are left as they are: pass the region's own positions through
  RA_LAUNCH(ra::launch_write_rows(c->shape(), M.base, M.cap, M.len, dev_k, dev_v, nullptr,
                                  c->kpool, c->vpool, nullptr, static_cast<hipStream_t>(stream)));
  return RA_OK;
}

ra_status ra_read_rows(ra_cache* c, int32_t seq, int32_t layer, int32_t kv_head,
                       void* dev_k_out, void* dev_v_out, void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || layer < 0 ||
      layer >= c->cfg.num_layers || kv_head < 0 || kv_head >= c->cfg.num_kv_heads)
    return RA_ERR_INVALID_ARG;
  if (c->step_open()) return RA_ERR_STATE;
  const SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  const int64_t region = M.base + static_cast<int64_t>(layer * c->cfg.num_kv_heads + kv_head) * M.cap;
  RA_LAUNCH(ra::launch_read_rows(c->shape(), region, M.len, c->kpool, c->vpool, dev_k_out,
                                 dev_v_out, static_cast<hipStream_t>(stream)));
  return RA_OK;
}

ra_status ra_window_select(ra_cache* c, int32_t seq_lo, int32_t seq_hi,
                           const void* dev_q_window, float* dev_scores,
                           int32_t scores_stride, int32_t* dev_drops, void* stream) {
  if (!c || seq_lo < 0 || seq_hi > c->cfg.max_seqs || seq_lo >= seq_hi || !dev_q_window)
    return RA_ERR_INVALID_ARG;
  if (c->cfg.dtype != RA_BF16 || c->cfg.layout != RA_LAYOUT_CHRONOLOGICAL)
    return RA_ERR_UNSUPPORTED;
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
  if (prm->scorer < RA_SCORER_SNAPKV || prm->scorer > RA_SCORER_VASE)
    return RA_ERR_INVALID_ARG;
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
  RA_LAUNCH(ra::launch_compact_drops(c->shape(), c->meta, c->kpool, c->vpool, c->pos, drops,
                                     every, seq_lo, seq_hi, s));
  return RA_OK;
}

ra_status ra_read_positions(ra_cache* c, int32_t seq, int32_t layer, int32_t kv_head,
                            int32_t* host_out, int32_t host_cap, int32_t* n_out,
                            void* stream) {
  if (!c || seq < 0 || seq >= c->cfg.max_seqs || layer < 0 ||
      layer >= c->cfg.num_layers || kv_head < 0 || kv_head >= c->cfg.num_kv_heads ||
      !host_out || !n_out)
    return RA_ERR_INVALID_ARG;
  if (c->step_open()) return RA_ERR_STATE;
  const SeqMeta& M = c->mirror[seq];
  if (!M.active) return RA_ERR_STATE;
  *n_out = M.len;
  if (host_cap < M.len) return RA_ERR_CAPACITY;
  const int64_t region = M.base + static_cast<int64_t>(layer * c->cfg.num_kv_heads + kv_head) * M.cap;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (M.len > 0) {
    RA_LAUNCH(hipMemcpyAsync(host_out, c->pos + region, sizeof(int32_t) * M.len,
                             hipMemcpyDeviceToHost, s));
  }
  RA_LAUNCH(hipStreamSynchronize(s));
  return RA_OK;
}

}  // extern "C"
