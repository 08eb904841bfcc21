// host_logic_check.cpp -- drives librv's host-only planning code (rv_plan.cpp) over many
// shapes, devices and work-plan overrides.  Built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_sanitizers.py, so any out-of-bounds table
// access, signed overflow or division by zero in the planning aborts the run; the
// checks below add the invariants the kernels rely on.  Prints "host logic OK".
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <initializer_list>

#include "../../paper_2609_23286_amd/csrc/rv_plan.h"

static int g_fail = 0;
#define CHECK(c, ...)                                    \
  do {                                                   \
    if (!(c)) {                                          \
      std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      std::fprintf(stderr, __VA_ARGS__);                 \
      std::fprintf(stderr, "\n");                        \
      ++g_fail;                                          \
    }                                                    \
  } while (0)

// Every queue's iterations are covered exactly once by its chunks, in order, through the
// chunk arithmetic the kernels use.
static void check_attention(int n_tokens, int n_fkeys, int64_t mem_len, int n_heads, int n_cus, int n_queues,
                            bool forced_split) {
  const rv::AttnPlan p = rv::plan_attention(n_cus, n_queues, n_tokens, n_fkeys, mem_len, n_heads);
  const int q_tiles = (n_tokens + 127) / 128;
  const int64_t T = (mem_len + 63) / 64 + (n_fkeys + 63) / 64;
  CHECK(p.q_tiles == q_tiles && p.T == T && p.n_units == q_tiles * n_heads, "plan sizes");
  CHECK(p.U >= p.T && p.E >= 1 && p.E1 >= 1 && p.E >= p.E1, "chunk sizes E=%d E1=%d U=%d T=%d", p.E, p.E1,
        p.U, p.T);
  CHECK(p.unit_base[0] == 0 && p.unit_base[n_queues] == p.n_units, "unit ranges");
  CHECK(p.grid % n_queues == 0, "grid");
  int total = 0;
  for (int q = 0; q < n_queues; ++q) {
    CHECK(p.unit_base[q] <= p.unit_base[q + 1], "unit ranges ordered");
    const int64_t iters = (int64_t)(p.unit_base[q + 1] - p.unit_base[q]) * p.U;
    const int n = p.n_chunks[q];
    CHECK(p.chunk_base[q] == total && n >= 0 && n <= p.grid / n_queues, "chunk table");
    total += n;
    if (iters == 0) {
      CHECK(n == 0, "empty queue has chunks");
      continue;
    }
    int64_t at = 0;
    for (int c = 0; c < n; ++c) {
      int64_t s0, s1;
      rv::chunk_iters(p, c, iters, &s0, &s1);
      CHECK(s0 == at && s0 < s1 && s1 <= iters, "chunk %d of queue %d: [%lld, %lld) after %lld", c, q,
            (long long)s0, (long long)s1, (long long)at);
      CHECK(rv::chunk_holding(p, s0) == c && rv::chunk_holding(p, s1 - 1) == c, "chunk of an iteration");
      at = s1;
    }
    CHECK(at == iters, "chunks cover the queue");
  }
  CHECK(total == p.total_chunks, "total chunks");
  // the workspace rv_init allocates holds every plan that RV_ATTN_SPLIT does not force
  if (!forced_split)
    CHECK(rv::plan_partial_slots(p) <= rv::default_partial_slots(n_cus, n_queues),
          "plan needs %lld partial slots, default workspace %lld (N=%d M=%lld H=%d cus=%d q=%d)",
          (long long)rv::plan_partial_slots(p), (long long)rv::default_partial_slots(n_cus, n_queues), n_tokens,
          (long long)mem_len, n_heads, n_cus, n_queues);
}

static void check_saliency(int grid_h, int grid_w, int n_special, int stride, int n_lh, int n_cus, int max_lds) {
  const int n_tokens = grid_h * grid_w + n_special;
  rv_qsub qs{grid_h, grid_w, n_special, stride};
  CHECK(rv::qsub_problem(&qs, n_tokens) == nullptr, "valid descriptor rejected");
  CHECK(rv::qsub_problem(&qs, n_tokens + 1) != nullptr, "wrong token count accepted");
  rv::AdmitArgs a{};
  rv::set_qsub(&a, qs);
  const int rows = (grid_h + stride - 1) / stride, cols = (grid_w + stride - 1) / stride;
  CHECK(a.n_q == rows * cols, "sampled query count");
  for (int i = 0; i < a.n_q; ++i) {  // every sampled token lies on the grid
    const int qi = i / a.q_cols;
    const int tok = a.q_base + qi * a.q_row_stride + (i - qi * a.q_cols) * a.q_col_stride;
    CHECK(tok >= n_special && tok < n_tokens, "sampled token %d outside the grid", tok);
  }
  a.n_tokens = n_tokens;
  a.budget = n_tokens < 10 ? n_tokens : 10;
  a.mode = rv::kModeBoth;
  rv::plan_saliency(&a, n_lh, n_cus, max_lds);
  const int nq_pad = (a.n_q + 31) & ~31;
  CHECK(a.sal_groups >= 1, "saliency groups");
  // the groups' block ranges partition the frame's 32-key blocks, in order
  const int n_blocks = (n_tokens + 31) / 32;
  int at = 0;
  for (int g = 0; g < a.sal_groups; ++g) {
    int b0, b1;
    rv::sal_group_blocks(a, g, n_blocks, &b0, &b1);
    CHECK(b0 <= b1 && (b0 == b1 || b0 == at), "group %d blocks [%d, %d) after %d", g, b0, b1, at);
    if (b1 > b0) at = b1;
  }
  CHECK(at == n_blocks, "saliency groups cover %d of %d blocks", at, n_blocks);
  if (a.stage_queries) {
    CHECK(a.q_pass >= 32 && a.q_pass % 32 == 0, "pass size %d", a.q_pass);
    CHECK(rv::sal_lds_bytes(a) <= (size_t)rv::admit_max_dynamic_lds(max_lds), "staged rows exceed LDS");
  } else {
    CHECK(a.q_pass == nq_pad, "unstaged pass covers every sampled query");
  }
}

// The attention tiles' LDS swizzle: distinct chunks on every 8 aligned rows (the K reads
// of 8 lanes, one row each, at 128 bytes a cycle) and distinct (row parity, chunk) pairs
// on every 16 (16 lanes at 256 bytes a cycle); and every aligned group of 4 rows puts a
// 32-byte piece (an even chunk pair) on 4 disjoint chunk pairs (the transposing V reads).
static void check_tile_swizzle() {
  for (int r0 = 0; r0 < 64; r0 += 8) {
    int seen = 0;
    for (int r = r0; r < r0 + 8; ++r) seen |= 1 << rv::attn_tile_swizzle(r);
    CHECK(seen == 0xFF, "rows %d..%d: swizzle values not distinct", r0, r0 + 7);
  }
  for (int r0 = 0; r0 < 64; r0 += 16) {
    int seen = 0;
    for (int r = r0; r < r0 + 16; ++r) seen |= 1 << (rv::attn_tile_swizzle(r) + 8 * (r & 1));
    CHECK(seen == 0xFFFF, "rows %d..%d: (parity, swizzle) pairs not distinct", r0, r0 + 15);
  }
  for (int r0 = 0; r0 < 64; r0 += 4)
    for (int c = 0; c < 8; c += 2) {
      int seen = 0;
      for (int r = r0; r < r0 + 4; ++r) seen |= 3 << ((c ^ rv::attn_tile_swizzle(r)) & 6);
      CHECK(seen == 0xFF, "rows %d..%d, chunks %d,%d: pieces overlap", r0, r0 + 3, c, c + 1);
    }
}

int main() {
  check_tile_swizzle();
  static const int shapes[][4] = {  // n_tokens, n_fkeys, mem_len, n_heads
      {1041, 1041, 0, 16},   {1041, 1041, 1000, 16}, {1041, 1041, 5000, 16}, {1041, 1041, 9990, 16},
      {1041, 1041, 52000, 16}, {1041, 0, 11031, 16}, {1374, 1374, 26000, 16}, {16384, 16384, 3000, 2},
      {65, 65, 0, 1},        {333, 333, 1500, 4},    {1, 1, 0, 1},           {1, 1, 63, 3},
      {128, 128, 64, 1},     {1041, 1041, 250, 16},  {2000, 2000, 100000, 16}};
  static const int devices[][2] = {{256, 8}, {304, 8}, {80, 2}, {32, 1}, {120, 3}, {1, 1}, {512, 16}};
  struct Env {
    const char *split, *pct, *wg, *min_chunk;
  };
  static const Env envs[] = {{nullptr, nullptr, nullptr, nullptr}, {"0", nullptr, nullptr, nullptr},
                             {"3", nullptr, nullptr, nullptr},       {"1", nullptr, nullptr, nullptr},
                             {"0", "100", nullptr, nullptr},         {"0", "101", nullptr, nullptr},
                             {"0", "400", nullptr, nullptr},         {nullptr, nullptr, "1", nullptr},
                             {nullptr, nullptr, "4", "1"},           {nullptr, "250", "3", "1"},
                             {nullptr, nullptr, nullptr, "100000"},  {"0", "133", nullptr, "1"},
                             {"0", "400", "4", "1"}};
  for (const Env& e : envs) {
    auto set = [](const char* k, const char* v) {
      if (v)
        setenv(k, v, 1);
      else
        unsetenv(k);
    };
    set("RV_ATTN_SPLIT", e.split);
    set("RV_ATTN_FIRST_PCT", e.pct);
    set("RV_ATTN_WG_PER_CU", e.wg);
    set("RV_ATTN_MIN_CHUNK", e.min_chunk);
    for (const auto& d : devices)
      for (const auto& s : shapes)
        check_attention(s[0], s[1], s[2], s[3], d[0], d[1], e.split && std::atoi(e.split) > 0);
  }
  // a stream-K split (RV_ATTN_SPLIT=0) is not a forced k-way split: the bound holds
  static const int grids[][4] = {  // grid_h, grid_w, n_special, stride
      {28, 37, 5, 2}, {37, 37, 5, 2}, {8, 8, 0, 2}, {8, 8, 0, 1}, {28, 37, 5, 1}, {28, 37, 5, 3},
      {28, 37, 5, 4}, {128, 128, 0, 2}, {1, 1041, 0, 2}, {0, 5, 7, 2}, {5, 0, 7, 2}, {0, 0, 1, 1},
      {3, 3, 0, 5}, {1, 1, 0, 1}};
  static const int lds_limits[] = {65536, 163840, 16384, 4096};
  for (const auto& g : grids)
    for (int n_lh : {1, 16, 384})
      for (int n_cus : {1, 80, 256})
        for (int lds : lds_limits) check_saliency(g[0], g[1], g[2], g[3], n_lh, n_cus, lds);
  rv_qsub bad{-1, 2, 0, 2};
  CHECK(rv::qsub_problem(&bad, 0) != nullptr, "negative grid accepted");
  bad = rv_qsub{2, 2, 0, 0};
  CHECK(rv::qsub_problem(&bad, 4) != nullptr, "stride 0 accepted");
  CHECK(rv::qsub_problem(nullptr, 4) != nullptr, "NULL descriptor accepted");
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("host logic OK\n");
  return 0;
}
