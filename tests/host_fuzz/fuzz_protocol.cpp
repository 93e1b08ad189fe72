// Seeded protocol fuzzer of the host library (test infrastructure).
//
// Drives one cache through a random sequence of calls of the C ABI: sequences
// begin and end, decode steps (every layer, then the end of the step, with
// the allocation-free entry point now and then), explicit events, fast
// forwards of every sequence or of one, a request preempted and resumed in a
// free slot, row and position reads and writes, entering and leaving graph
// mode, and calls that break the protocol or pass bad arguments.  The device side is the stand-ins of
// stub_launchers.cpp, so this runs on the CPU, under AddressSanitizer and
// UndefinedBehaviorSanitizer.  After every call it prints one JSON line: the
// call, its status and every slot's host mirror (active, len, step, event,
// cap, base, move_pending, k_keep) with the pool's used and free rows; the
// test replays the same calls on the oracle's SequenceReplay and compares.
//
// Usage: fuzz_protocol SEED N_OPS
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "randattn.h"

extern "C" void stub_configure(int64_t pool_rows, int64_t n_groups, int max_seqs,
                               int page_rows);
extern "C" int stub_check_tables(const int* active, const int* caps, int n);

namespace {

uint64_t g_rng;
uint64_t next_u64() {   // splitmix64
  uint64_t z = (g_rng += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}
int rnd(int n) { return static_cast<int>(next_u64() % static_cast<uint64_t>(n)); }

struct Buf {               // a caller buffer of exactly the bytes asked for
  std::vector<unsigned char> b;
  explicit Buf(size_t n) : b(n ? n : 1) {}
  void* p() { return b.data(); }
};

ra_config g_cfg;
ra_cache* g_c = nullptr;
int g_external = 0;

struct Request {           // what began each slot
  int lp;
  uint64_t seed, rid;
};
std::vector<Request> g_req;

void print_state(const char* op, const char* args, int status, int extra) {
  std::printf("{\"op\":\"%s\",\"a\":[%s],\"st\":%d,\"x\":%d,\"s\":[", op, args, status, extra);
  std::vector<int> active(g_cfg.max_seqs), caps(g_cfg.max_seqs);
  for (int s = 0; s < g_cfg.max_seqs; ++s) {
    ra_seq_info i;
    if (ra_get_seq_info(g_c, s, &i) != RA_OK) std::abort();
    active[s] = i.active;
    caps[s] = i.cap;
    std::printf("%s[%d,%d,%d,%d,%d,%lld,%d,%d]", s ? "," : "", i.active, i.len, i.step,
                i.event, i.cap, static_cast<long long>(i.base), i.move_pending, i.k_keep);
  }
  int64_t used = -1, free_rows = -1;
  if (ra_pool_info(g_c, &used, &free_rows) != RA_OK) std::abort();
  std::printf("],\"pool\":[%lld,%lld],\"tables\":%d}\n", static_cast<long long>(used),
              static_cast<long long>(free_rows),
              stub_check_tables(active.data(), caps.data(), g_cfg.max_seqs));
}

int active_slot() {        // a random active slot, or -1
  std::vector<int> a;
  for (int s = 0; s < g_cfg.max_seqs; ++s) {
    ra_seq_info i;
    ra_get_seq_info(g_c, s, &i);
    if (i.active) a.push_back(s);
  }
  return a.empty() ? -1 : a[rnd(static_cast<int>(a.size()))];
}

int free_slot() {          // a free slot (searched from a random one), or -1
  const int n = g_cfg.max_seqs, start = rnd(n);
  for (int k = 0; k < n; ++k) {
    ra_seq_info i;
    ra_get_seq_info(g_c, (start + k) % n, &i);
    if (!i.active) return (start + k) % n;
  }
  return -1;
}

int seq_len(int s) {
  ra_seq_info i;
  ra_get_seq_info(g_c, s, &i);
  return i.len;
}

// lockstep: a configuration whose events can defer their row moves (bf16,
// the chronological layout, an end-of-step policy, one work item per head)
void random_config(bool lockstep) {
  for (;;) {
    ra_config c;
    std::memset(&c, 0, sizeof c);
    const int G[] = {1, 2, 4, 5};
    c.num_layers = 1 + rnd(3);
    c.num_kv_heads = 1 + rnd(2);
    c.num_q_heads = c.num_kv_heads * G[rnd(4)];
    c.head_dim = 128;
    c.budget_k = 8 + rnd(90);
    const int R[] = {0, 4, 8, 16};
    c.recent_r = R[rnd(4)];
    const int E[] = {1, 4, 8, 16, 32};
    c.evict_every = E[rnd(5)];
    c.budget_mode = rnd(2);
    c.dtype = rnd(3) ? RA_BF16 : RA_F32;
    c.max_seqs = 1 + rnd(5);
    c.attn_split = rnd(2) ? 0 : 32 * (1 + rnd(4));
    c.layout = rnd(3);
    c.policy = rnd(5);
    c.policy_block = c.policy == RA_POLICY_BLOCK ? 1 + rnd(4) : 1;
    c.page_rows = rnd(2) ? 32 : 64;
    c.max_prompt_len = 10 + rnd(80);
    if (lockstep) {
      c.dtype = RA_BF16;
      c.layout = RA_LAYOUT_CHRONOLOGICAL;
      c.attn_split = 0;
      if (c.policy == RA_POLICY_EXTERNAL) c.policy = RA_POLICY_RANDOM;
    }
    if (ra_config_check(&c) == RA_OK) {
      g_cfg = c;
      g_external = c.policy == RA_POLICY_EXTERNAL;
      return;
    }
  }
}

int max_prompt() {
  int lp = g_cfg.layout == RA_LAYOUT_PAGED ? g_cfg.max_prompt_len : 90;
  if (g_cfg.budget_mode == RA_BUDGET_TOTAL && lp > g_cfg.budget_k) lp = g_cfg.budget_k;
  return lp;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc < 3) return 2;
  std::setvbuf(stdout, nullptr, _IOLBF, 0);    // lines up to a sanitizer abort survive
  g_rng = std::strtoull(argv[1], nullptr, 10);
  const int n_ops = std::atoi(argv[2]);
  // a third of the runs begin every slot at once and rarely end or begin one
  // after that, so that the sequences' events fall on the same steps (the
  // events whose row moves ride on the next step's attention)
  const bool lockstep = rnd(3) == 0;
  random_config(lockstep);
  const ra_config& c = g_cfg;
  const size_t esz = c.dtype == RA_BF16 ? 2 : 4;
  const int L = c.num_layers, Hq = c.num_q_heads, Hkv = c.num_kv_heads;
  // pool: room for 1..max_seqs sequences at the longest prompt
  const int64_t per = ra_seq_rows(&c, max_prompt());
  if (per <= 0) return 3;
  int64_t pool_rows, n_groups = 0;
  if (c.layout == RA_LAYOUT_PAGED) {
    const int64_t group = static_cast<int64_t>(L) * Hkv * c.page_rows;
    n_groups = (per / group) * (1 + rnd(c.max_seqs)) - rnd(2);
    if (n_groups < 1) n_groups = 1;
    pool_rows = n_groups * group;
  } else {
    pool_rows = (per * (1 + rnd(c.max_seqs)) + 31) / 32 * 32;
  }
  stub_configure(pool_rows, n_groups, c.max_seqs, c.page_rows);
  Buf kpool(pool_rows * 128 * esz), vpool(pool_rows * 128 * esz);
  std::vector<int32_t> pos(static_cast<size_t>(pool_rows));
  const size_t meta_bytes = ra_meta_bytes(&c);
  Buf meta(meta_bytes);
  int s0 = ra_cache_create(&c, kpool.p(), vpool.p(), pos.data(), pool_rows, meta.p(),
                           meta_bytes, nullptr, &g_c);
  std::printf("{\"config\":[%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d],"
              "\"pool_rows\":%lld,\"create\":%d}\n",
              c.num_layers, c.num_q_heads, c.num_kv_heads, c.budget_k, c.recent_r,
              c.evict_every, c.budget_mode, c.dtype, c.max_seqs, c.attn_split, c.layout,
              c.policy, c.policy_block, c.page_rows, c.max_prompt_len, max_prompt(),
              static_cast<long long>(pool_rows), s0);
  if (s0 != RA_OK) return 4;
  print_state("create", "", 0, 0);

  Buf q(static_cast<size_t>(c.max_seqs) * Hq * 128 * esz);
  Buf kn(static_cast<size_t>(c.max_seqs) * Hkv * 128 * esz);
  Buf vn(static_cast<size_t>(c.max_seqs) * Hkv * 128 * esz);
  Buf out(static_cast<size_t>(c.max_seqs) * Hq * 128 * esz);
  const size_t ws_bytes = ra_workspace_bytes(&c);
  Buf ws(ws_bytes);
  char args[192];
  g_req.assign(c.max_seqs, Request{0, 0, 0});

  if (lockstep) {
    for (int s = 0; s < c.max_seqs; ++s) {
      const int lp = rnd(max_prompt() + 1);
      const uint64_t seed = next_u64() >> 1, rid = next_u64() >> 1;
      const int st = ra_seq_begin(g_c, s, lp, seed, rid, nullptr, nullptr, nullptr);
      if (st == RA_OK) g_req[s] = Request{lp, seed, rid};
      std::snprintf(args, sizeof args, "%d,%d,%llu,%llu", s, lp,
                    static_cast<unsigned long long>(seed), static_cast<unsigned long long>(rid));
      print_state("begin", args, st, 0);
    }
  }

  int in_graph = 0;
  for (int op = 0; op < n_ops; ++op) {
    int kind = rnd(100);
    if (lockstep && kind < 21 && rnd(8)) kind = 21 + rnd(45);   // mostly steps instead
    if (kind < 14) {                                   // begin (any slot)
      const int s = rnd(c.max_seqs);
      int lp = rnd(max_prompt() + 1);
      if (rnd(10) == 0) lp += c.budget_k + 1;         // too long (budget or table)
      const uint64_t seed = next_u64() >> 1, rid = next_u64() >> 1;
      const bool rows = rnd(2);
      Buf kp(rows ? static_cast<size_t>(L) * Hkv * lp * 128 * esz : 0);
      Buf vp(rows ? static_cast<size_t>(L) * Hkv * lp * 128 * esz : 0);
      const int st = ra_seq_begin(g_c, s, lp, seed, rid, rows ? kp.p() : nullptr,
                                  rows ? vp.p() : nullptr, nullptr);
      if (st == RA_OK) g_req[s] = Request{lp, seed, rid};
      std::snprintf(args, sizeof args, "%d,%d,%llu,%llu", s, lp,
                    static_cast<unsigned long long>(seed), static_cast<unsigned long long>(rid));
      print_state("begin", args, st, 0);
    } else if (kind < 21) {                            // end (any slot)
      const int s = rnd(c.max_seqs);
      const int st = ra_seq_end(g_c, s, nullptr);
      std::snprintf(args, sizeof args, "%d", s);
      print_state("end", args, st, 0);
    } else if (kind < 66) {                            // decode step
      const bool noalloc = rnd(4) == 0;
      int st = RA_OK;
      int layer = 0;
      for (; layer < L; ++layer) {
        st = noalloc ? ra_decode_attention_noalloc(g_c, layer, q.p(), kn.p(), vn.p(), out.p(),
                                                   nullptr)
                     : ra_decode_attention(g_c, layer, q.p(), kn.p(), vn.p(), out.p(), ws.p(),
                                           ws_bytes, nullptr);
        if (st != RA_OK) break;
        if (rnd(40) == 0) {                            // protocol breaks inside the step
          const int e1 = ra_decode_attention(g_c, layer, q.p(), kn.p(), vn.p(), out.p(),
                                             ws.p(), ws_bytes, nullptr);
          int32_t n;
          const int e2 = layer + 1 < L ? ra_end_step(g_c, nullptr, &n) : RA_ERR_STATE;
          const int e3 = ra_evict_now(g_c, 0, nullptr);
          const int e4 = ra_fast_forward(g_c, 1, nullptr);
          std::snprintf(args, sizeof args, "%d,%d,%d,%d,%d", layer, e1, e2, e3, e4);
          print_state("midstep", args, 0, 0);
        }
      }
      if (st != RA_OK) {
        // only a refusal before the step's first launch is expected: the
        // pool is out of pages or a region is full (rows piling up)
        std::snprintf(args, sizeof args, "%d", layer);
        print_state("step_refused", args, st, 0);
        if (layer != 0 || st != RA_ERR_CAPACITY) return 5;
        continue;
      }
      int32_t n_ev = -1;
      st = ra_end_step(g_c, nullptr, &n_ev);
      std::snprintf(args, sizeof args, "%d", noalloc ? 1 : 0);
      print_state("step", args, st, n_ev);
    } else if (kind < 72) {                            // explicit event
      const int s = rnd(c.max_seqs);
      const int st = ra_evict_now(g_c, s, nullptr);
      std::snprintf(args, sizeof args, "%d", s);
      print_state("evict_now", args, st, 0);
    } else if (kind < 77) {                            // fast forward: all, or one slot
      const int n = rnd(3 * c.evict_every + 2);
      if (rnd(2)) {
        const int st = ra_fast_forward(g_c, n, nullptr);
        std::snprintf(args, sizeof args, "%d", n);
        print_state("fast_forward", args, st, 0);
      } else {
        const int s = rnd(c.max_seqs);
        const int st = ra_seq_fast_forward(g_c, s, n, nullptr);
        std::snprintf(args, sizeof args, "%d,%d", s, n);
        print_state("seq_fast_forward", args, st, 0);
      }
    } else if (kind < 80) {                            // preempt a request, resume it
      const int s = active_slot();
      if (s < 0) continue;
      ra_seq_info was;
      ra_get_seq_info(g_c, s, &was);
      const Request q = g_req[s];
      const size_t rows = static_cast<size_t>(L) * Hkv * was.len;
      Buf ks(rows * 128 * esz), vs(rows * 128 * esz);
      for (int lg = 0; lg < L * Hkv; ++lg)             // its rows, saved head by head
        ra_read_rows(g_c, s, lg / Hkv, lg % Hkv,
                     ks.b.data() + static_cast<size_t>(lg) * was.len * 128 * esz,
                     vs.b.data() + static_cast<size_t>(lg) * was.len * 128 * esz, nullptr);
      const int e1 = ra_seq_end(g_c, s, nullptr);
      const int t = e1 == RA_OK ? free_slot() : s;
      const int e2 = ra_seq_begin(g_c, t, q.lp, q.seed, q.rid, nullptr, nullptr, nullptr);
      if (e2 == RA_OK) g_req[t] = q;
      const int e3 = ra_seq_fast_forward(g_c, t, was.step, nullptr);
      // the saved rows back (as many as the resumed head holds: explicit
      // events of its past are not replayed, so it may hold more)
      const size_t back = static_cast<size_t>(L) * Hkv * (e2 == RA_OK ? seq_len(t) : 0);
      if (back > rows) {
        ks.b.resize(back * 128 * esz);
        vs.b.resize(back * 128 * esz);
      }
      const int e4 = ra_write_rows(g_c, t, ks.p(), vs.p(), nullptr);
      std::snprintf(args, sizeof args, "%d,%d,%d,%llu,%llu,%d,%d,%d,%d,%d", s, t, q.lp,
                    static_cast<unsigned long long>(q.seed),
                    static_cast<unsigned long long>(q.rid), was.step, e1, e2, e3, e4);
      print_state("resume", args, e4, 0);
    } else if (kind < 83) {                            // read rows / positions of one head
      const int s = active_slot();
      if (s < 0) continue;
      const int layer = rnd(L), g = rnd(Hkv), len = seq_len(s);
      Buf ko(static_cast<size_t>(len) * 128 * esz), vo(static_cast<size_t>(len) * 128 * esz);
      const int st = ra_read_rows(g_c, s, layer, g, ko.p(), rnd(2) ? vo.p() : nullptr, nullptr);
      std::vector<int32_t> hp(static_cast<size_t>(len) + 1);
      const int cap = rnd(4) ? len : len - 1;
      int32_t n_out = -1;
      const int st2 = ra_read_positions(g_c, s, layer, g, hp.data(), cap, &n_out, nullptr);
      std::snprintf(args, sizeof args, "%d,%d,%d,%d,%d", s, layer, g, cap, n_out);
      print_state("read", args, st, st2);
    } else if (kind < 88) {                            // write rows, export positions
      const int s = active_slot();
      if (s < 0) continue;
      const size_t rows = static_cast<size_t>(L) * Hkv * seq_len(s);
      Buf kw(rows * 128 * esz), vw(rows * 128 * esz);
      const int st = ra_write_rows(g_c, s, kw.p(), vw.p(), nullptr);
      std::vector<int32_t> ex(rows + 1);
      const int64_t elems = rnd(4) ? static_cast<int64_t>(rows) : static_cast<int64_t>(rows) - 1;
      const int st2 = ra_export_positions(g_c, s, ex.data(), elems, nullptr);
      std::snprintf(args, sizeof args, "%d,%lld", s, static_cast<long long>(elems));
      print_state("write", args, st, st2);
    } else if (kind < 91) {                            // enter or leave graph mode
      const int st = ra_graph_mode(g_c, !in_graph, nullptr);
      std::snprintf(args, sizeof args, "%d", !in_graph);
      if (st == RA_OK) in_graph = !in_graph;
      print_state("graph", args, st, 0);
    } else {                                           // bad arguments
      ra_seq_info i;
      const int e1 = ra_get_seq_info(g_c, c.max_seqs, &i);
      const int e2 = ra_evict_now(g_c, -1, nullptr);
      const int e3 = rnd(3) == 0 ? ra_fast_forward(g_c, -1, nullptr)
                     : rnd(2)    ? ra_seq_fast_forward(g_c, 0, -1, nullptr)
                                 : ra_seq_fast_forward(g_c, c.max_seqs, 1, nullptr);
      const int e4 = ra_read_rows(g_c, 0, L, 0, nullptr, nullptr, nullptr);
      const int e5 = ra_decode_attention(g_c, L, q.p(), kn.p(), vn.p(), out.p(), ws.p(),
                                         ws_bytes, nullptr);
      const int e6 = ra_decode_attention(g_c, 0, q.p(), kn.p(), vn.p(), out.p(), ws.p(),
                                         ws_bytes / 2, nullptr);
      const int e7 = ra_seq_begin(g_c, -1, 0, 0, 0, nullptr, nullptr, nullptr);
      std::snprintf(args, sizeof args, "%d,%d,%d,%d,%d,%d,%d", e1, e2, e3, e4, e5, e6, e7);
      print_state("bad", args, 0, 0);
    }
  }
  const int st = ra_cache_destroy(g_c);
  std::printf("{\"op\":\"destroy\",\"st\":%d}\n", st);
  return st == RA_OK ? 0 : 6;
}
