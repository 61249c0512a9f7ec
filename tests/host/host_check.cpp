// Exercises the HIP-free host part of the library (paper_2609_14237_amd/csrc/
// ods_host.cpp: allocator, sizing, validation, launch planning) on the CPU, for
// a build under AddressSanitizer and UndefinedBehaviorSanitizer. No device
// memory is touched: every device pointer is an aligned address that is never
// dereferenced. Usage: host_check <workloads.txt>; prints "host_check OK".
//
// workloads.txt: one block per line,
//   name batch max_pages n_layers  then per layer:
//   hidden n_q n_kv head_dim ffn n_experts top_k moe_ffn window
#include <assert.h>
#include <stddef.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <random>
#include <set>
#include <string>
#include <vector>

#include "../../paper_2609_14237_amd/csrc/plan.hpp"

using namespace ods;

static int g_checks = 0;
#define CHECK(c)                                                                    \
  do {                                                                              \
    ++g_checks;                                                                     \
    if (!(c)) {                                                                     \
      fprintf(stderr, "CHECK failed at %s:%d: %s (%s)\n", __FILE__, __LINE__, #c,    \
              ods_last_error());                                                    \
      exit(1);                                                                      \
    }                                                                               \
  } while (0)

static void *const kFake = (void *)0x100000;  // aligned, never dereferenced

struct Work {
  std::string name;
  int batch, max_pages;
  std::vector<ods_layer> layers;
};

// Offsets of every pointer member of ods_state (set through memcpy, so each
// member keeps its own pointer type).
static const size_t kStatePtrs[] = {
    offsetof(ods_state, resid), offsetof(ods_state, xn), offsetof(ods_state, qkv), offsetof(ods_state, o),
    offsetof(ods_state, hn), offsetof(ods_state, gu), offsetof(ods_state, act), offsetof(ods_state, logits),
    offsetof(ods_state, topk_w), offsetof(ods_state, topk_ids), offsetof(ods_state, perm),
    offsetof(ods_state, slot_pos), offsetof(ods_state, expert_off), offsetof(ods_state, xp),
    offsetof(ods_state, gu_p), offsetof(ods_state, act_p), offsetof(ods_state, yp), offsetof(ods_state, ws)};
constexpr size_t kNumStatePtrs = sizeof(kStatePtrs) / sizeof(kStatePtrs[0]);

static void set_ptr(ods_state &s, size_t i, void *v) { memcpy((char *)&s + kStatePtrs[i], &v, sizeof(v)); }

static ods_state fake_state(size_t ws_bytes) {
  ods_state s;
  memset(&s, 0, sizeof(s));
  for (size_t i = 0; i < kNumStatePtrs; ++i) set_ptr(s, i, kFake);
  s.ws_bytes = ws_bytes;
  return s;
}

static void check_allocator() {
  // the specification's worked example (tests/golden/kv_alloc_worked_example.txt)
  const int32_t ctx[4] = {20, 16, 1, 33};
  int32_t table[4 * 3];
  CHECK(ods_kv_alloc(10, ctx, 4, 0, 3, table) == ODS_OK);
  const int32_t want[12] = {6, 3, -1, 2, -1, -1, 9, -1, -1, 8, 1, 4};
  CHECK(memcmp(table, want, sizeof(want)) == 0);
  CHECK(ods_kv_alloc(5, ctx, 4, 0, 3, table) == ODS_ENOMEM);
  CHECK(ods_kv_alloc(10, ctx, 4, 0, 2, table) == ODS_ERANGE);
  CHECK(ods_kv_alloc(10, nullptr, 4, 0, 3, table) == ODS_EINVAL);
  CHECK(ods_kv_alloc(10, ctx, 4, 0, 3, nullptr) == ODS_EINVAL);
  CHECK(ods_kv_alloc(0, ctx, 4, 0, 3, table) == ODS_EINVAL);
  CHECK(ods_kv_alloc(10, ctx, 0, 0, 3, table) == ODS_OK);  // empty batch
  // random batches: every page used at most once, ceil(ctx / 16) per sequence
  std::mt19937_64 rng(5);
  for (int rep = 0; rep < 200; ++rep) {
    const int B = 1 + (int)(rng() % 40), mp = 1 + (int)(rng() % 12);
    std::vector<int32_t> c(B), t((size_t)B * mp);
    int64_t need = 0;
    for (int b = 0; b < B; ++b) {
      c[b] = 1 + (int)(rng() % (16 * mp));
      need += (c[b] + 15) / 16;
    }
    const int64_t P = need + (int64_t)(rng() % 9);
    CHECK(ods_kv_alloc(P, c.data(), B, rng(), mp, t.data()) == ODS_OK);
    std::set<int32_t> seen;
    for (int b = 0; b < B; ++b)
      for (int j = 0; j < mp; ++j) {
        const int32_t v = t[(size_t)b * mp + j];
        if (j < (c[b] + 15) / 16) {
          CHECK(v >= 0 && v < P && seen.insert(v).second);
        } else {
          CHECK(v == -1);
        }
      }
  }
}

// Every range of the block: validation passes with a large enough workspace,
// and the planned launches tile the range exactly with sane shapes.
static void check_block_ranges(const Work &w, int cus) {
  const ods_block blk{(int32_t)w.layers.size(), w.layers.data()};
  const int n = ods_block_num_ops(&blk);
  CHECK(n > 0);
  const ods_batch batch{w.batch, w.max_pages, (const int32_t *)kFake, (const int32_t *)kFake, 0, 0, nullptr};
  const size_t ws = block_ws_bytes(&blk, &batch, cus);
  CHECK(ws >= 256);
  for (int a = 0; a < n; ++a)
    for (int b = a + 1; b <= n; ++b) {
      CHECK(range_ws_bytes(&blk, a, b, &batch, cus) <= ws);
      ods_state st = fake_state(ws);
      CHECK(validate_range(&blk, a, b, &batch, &st, cus) == ODS_OK);
      int covered = 0;
      for (int i = 0; i < b - a;) {
        Launch L;
        plan_launch(&blk, a, b, i, &batch, &st, cus, &L);
        CHECK(L.n_ops >= 1 && L.n_ops <= 3 && i + L.n_ops <= b - a);
        CHECK(L.layer == op_at(&blk, a + i).layer && L.what != nullptr);
        if (L.kind == LK_GEMM || L.kind == LK_QKV_ROPE) {
          const GemmArgs &g = L.gemm;
          CHECK(g.M == w.batch || g.group_off != nullptr);
          CHECK(g.splits == 1 || g.splits == 2 || g.splits == 4 || g.splits == 8 || g.splits == 16);
          if (g.splits > 1)
            CHECK((size_t)g.splits * g.M * g.N * (g.epi == EPI_SILU ? 2 : 1) * sizeof(float) <= ws);
          CHECK(g.N > 0 && g.K > 0);
        }
        if (L.kind == LK_ATTENTION) {
          CHECK(L.attn.plan.grid >= 1 && L.attn.plan.grid <= (cus > 0 ? cus : 1));
          CHECK(attn_ws_bytes(w.batch, L.attn.n_q, L.attn.n_kv, L.attn.D, L.attn.plan) <= ws);
        }
        i += L.n_ops;
        covered += L.n_ops;
      }
      CHECK(covered == b - a);
    }
  // stage wrappers and names
  for (int g = 0; g < n; ++g) CHECK(ods_op_name(&blk, g) != nullptr);
  CHECK(ods_op_name(&blk, n) == nullptr && ods_op_name(&blk, -1) == nullptr);
  // every live buffer a range needs: null and misaligned pointers are rejected
  for (int a = 0; a < n; ++a) {
    ods_state st = fake_state(ws);
    for (size_t k = 0; k < kNumStatePtrs; ++k) {
      set_ptr(st, k, nullptr);
      const ods_status r1 = validate_range(&blk, a, a + 1, &batch, &st, cus);
      set_ptr(st, k, (char *)kFake + 2);
      const ods_status r2 = validate_range(&blk, a, a + 1, &batch, &st, cus);
      set_ptr(st, k, kFake);
      CHECK(r1 == ODS_OK || r1 == ODS_EINVAL);
      CHECK(r2 == r1);  // a pointer the operator uses fails both ways, an unused one neither
    }
  }
  // sizing over batch sizes and device sizes
  for (int B : {0, 1, 7, 64, 255, 1024, 4096})
    for (int i = 0; i < ODS_BUF_COUNT; ++i) (void)ods_live_bytes(&blk, B, (ods_buffer)i);
  ods_state st = fake_state(ws);
  CHECK(validate_range(&blk, 0, n, &batch, &st, cus) == ODS_OK);
  st.ws_bytes = 0;
  CHECK(validate_range(&blk, 0, n, &batch, &st, cus) == ODS_ENOMEM);
  CHECK(validate_range(&blk, 0, n + 1, &batch, &st, cus) == ODS_ERANGE);
  CHECK(validate_range(&blk, 3, 3, &batch, &st, cus) == ODS_ERANGE);
  CHECK(validate_range(&blk, 0, n, nullptr, &st, cus) == ODS_EINVAL);
  const ods_batch empty{0, w.max_pages, nullptr, nullptr, 0, 0, nullptr};
  ods_state none;
  memset(&none, 0, sizeof(none));
  CHECK(validate_range(&blk, 0, n, &empty, &none, cus) == ODS_OK);  // empty batch reads no pointer
}

static void check_bad_configs() {
  ods_layer L;
  memset(&L, 0, sizeof(L));
  L.cfg = ods_layer_cfg{256, 4, 2, 64, 688, 0, 0, 0, 0, 10000.f, 1e-6f};
  const ods_block blk{1, &L};
  CHECK(check_block(&blk) == ODS_OK);
  auto bad = [&](void (*mut)(ods_layer_cfg &), ods_status want) {
    ods_layer M = L;
    mut(M.cfg);
    const ods_block b2{1, &M};
    CHECK(check_block(&b2) == want);
    CHECK(ods_kv_pool_bytes(&M.cfg, 10) == 0);
  };
  bad([](ods_layer_cfg &c) { c.head_dim = 96; }, ODS_EUNSUPPORTED);
  bad([](ods_layer_cfg &c) { c.n_q = 5; }, ODS_EUNSUPPORTED);
  bad([](ods_layer_cfg &c) { c.n_q = 64; c.n_kv = 2; }, ODS_EUNSUPPORTED);
  bad([](ods_layer_cfg &c) { c.ffn = 690; }, ODS_EUNSUPPORTED);
  bad([](ods_layer_cfg &c) { c.hidden = -1; }, ODS_EINVAL);
  bad([](ods_layer_cfg &c) { c.rms_eps = -1.f; }, ODS_EINVAL);
  bad([](ods_layer_cfg &c) { c.n_experts = 128; c.top_k = 65; c.moe_ffn = 64; }, ODS_EUNSUPPORTED);
  CHECK(check_block(nullptr) == ODS_EINVAL);
  CHECK(ods_block_num_ops(nullptr) == -1);
  CHECK(ods_tiled_weight_bytes(128, 100, 0, 1) == 0 && ods_tiled_weight_bytes(128, 128, 2, 1) == 0);
  CHECK(ods_tiled_weight_bytes(14336, 4096, 1, 1) == (size_t)14336 / 64 * 64 * 128 * 64 * 2);
}

static std::vector<Work> read_works(const char *path) {
  std::vector<Work> out;
  FILE *f = fopen(path, "r");
  CHECK(f != nullptr);
  char name[128];
  int batch, mp, nl;
  while (fscanf(f, "%127s %d %d %d", name, &batch, &mp, &nl) == 4) {
    Work w{name, batch, mp, {}};
    for (int l = 0; l < nl; ++l) {
      ods_layer L;
      memset(&L, 0, sizeof(L));
      ods_layer_cfg &c = L.cfg;
      CHECK(fscanf(f, "%d %d %d %d %d %d %d %d %d", &c.hidden, &c.n_q, &c.n_kv, &c.head_dim, &c.ffn, &c.n_experts,
                   &c.top_k, &c.moe_ffn, &c.window) == 9);
      c.rope_theta = 10000.f;
      c.rms_eps = 1e-6f;
      L.g_attn = L.w_qkv = L.w_o = L.g_ffn = L.w_gate_up = L.w_down = L.w_router = kFake;
      L.kv_pool = kFake;
      L.pool_pages = 1000;
      w.layers.push_back(L);
    }
    out.push_back(w);
  }
  fclose(f);
  return out;
}

// Block rows and split-K of the dense streaming GEMM at the shapes the
// tile rule was measured on: the 8B-shaped layer at 256 rows keeps the
// 256-row tile, one GPU's 8-way tensor-parallel share of it takes 64-row
// tiles, and up to 64 rows every GEMM takes 64-row tiles.
static void check_stream_tiles() {
  struct Case {
    int M, N, K, epi, rows, splits;
  };
  const Case cases[] = {
      {256, 14336, 4096, EPI_SILU, 256, 1}, {256, 4096, 14336, EPI_RESID, 256, 8},
      {256, 6144, 4096, EPI_BF16, 256, 4},  {256, 4096, 4096, EPI_RESID, 256, 8},
      {256, 1792, 4096, EPI_SILU, 256, 8},   {256, 4096, 1792, EPI_RESID, 64, 2},
      {256, 768, 4096, EPI_BF16, 64, 8},    {256, 4096, 512, EPI_RESID, 64, 1},
      {64, 14336, 4096, EPI_SILU, 64, 1},   {64, 4096, 4096, EPI_RESID, 64, 8},
      {512, 4096, 4096, EPI_RESID, 256, 4}, {512, 5120, 4096, EPI_BF16, 256, 2},
      {200, 9000, 512, EPI_SILU, 256, 1},   {200, 896, 640, EPI_BF16, 64, 1},
  };
  for (const Case &c : cases) {
    CHECK(gemm_stream_rows(c.M, c.N, c.K, c.epi) == c.rows);
    CHECK(gemm_stream_splits(c.M, c.N, c.K, c.epi) == c.splits);
  }
}

// Random layer shapes the library accepts (dense and MoE, full and sliding-
// window attention, row-major and tiled weights, batches 1 to 700): every
// operator range validates and plans as above, and the streaming GEMM's tile
// and split choices stay inside what its launcher takes.
static void check_random_shapes() {
  std::mt19937_64 rng(11);
  auto pick = [&](std::initializer_list<int> v) { return *(v.begin() + rng() % v.size()); };
  for (int rep = 0; rep < 60; ++rep) {
    const int D = pick({64, 128}), group = pick({1, 2, 4, 8, 16}), n_kv = pick({1, 2, 4, 8});
    const bool moe = rng() % 3 == 0;
    ods_layer L;
    memset(&L, 0, sizeof(L));
    ods_layer_cfg &c = L.cfg;
    c.hidden = 64 * (2 + (int)(rng() % 40)) + (rng() % 4 == 0 ? 8 * (int)(1 + rng() % 7) : 0);
    c.n_q = group * n_kv;
    c.n_kv = n_kv;
    c.head_dim = D;
    c.window = rng() % 3 == 0 ? 16 * (int)(1 + rng() % 64) + (int)(rng() % 16) : 0;
    if (moe) {
      c.n_experts = pick({8, 16, 64, 128});
      c.top_k = 1 + (int)(rng() % std::min(8, c.n_experts));
      c.moe_ffn = 64 * (1 + (int)(rng() % 24)) + (rng() % 4 == 0 ? 8 : 0);
    } else {
      c.ffn = 64 * (1 + (int)(rng() % 200)) + (rng() % 4 == 0 ? 8 * (int)(1 + rng() % 7) : 0);
    }
    c.rope_theta = 10000.f;
    c.rms_eps = 1e-6f;
    L.g_attn = L.w_qkv = L.w_o = L.g_ffn = L.w_gate_up = L.w_down = L.w_router = kFake;
    L.kv_pool = kFake;
    L.pool_pages = 1000;
    Work w{"random", 1 + (int)(rng() % 700), 1 + (int)(rng() % 300), {L}};
    for (int tiled = 0; tiled < 2; ++tiled) {
      w.layers[0].weight_layout = tiled ? ODS_WEIGHTS_TILED : ODS_WEIGHTS_ROWS;
      const ods_block blk{1, w.layers.data()};
      CHECK(check_block(&blk) == ODS_OK || (tiled && check_block(&blk) == ODS_EUNSUPPORTED));
      if (check_block(&blk) != ODS_OK) continue;
      check_block_ranges(w, 256);
    }
  }
  for (int rep = 0; rep < 20000; ++rep) {
    const int M = 1 + (int)(rng() % 4096), N = 8 * (1 + (int)(rng() % 4096)), K = 64 * (1 + (int)(rng() % 256));
    const int epi = (int)(rng() % 4);
    const int rows = gemm_stream_rows(M, N, K, epi), s = gemm_stream_splits(M, N, K, epi);
    CHECK(rows == 64 || rows == 256);
    CHECK(M > 64 || rows == 64);
    CHECK(s == 1 || s == 2 || s == 4 || s == 8);
    CHECK(s == 1 || K / 64 / s >= 8);  // every split keeps at least 8 K steps
    const int tiles = (M + rows - 1) / rows * (epi == EPI_SILU ? (N + 63) / 64 : (N + 127) / 128);
    CHECK(s == 1 || tiles * s <= 256);  // split-K never spills into a second wave
  }
}

int main(int argc, char **argv) {
  if (argc < 2) {
    fprintf(stderr, "usage: host_check workloads.txt\n");
    return 2;
  }
  check_allocator();
  check_bad_configs();
  check_stream_tiles();
  check_random_shapes();
  for (Work &w : read_works(argv[1])) {
    for (int tiled = 0; tiled < 2; ++tiled) {
      for (ods_layer &L : w.layers) L.weight_layout = tiled ? ODS_WEIGHTS_TILED : ODS_WEIGHTS_ROWS;
      const ods_block blk{(int32_t)w.layers.size(), w.layers.data()};
      if (check_block(&blk) != ODS_OK) continue;  // a shape the tiled layout does not take
      for (int cus : {1, 80, 256, 304}) check_block_ranges(w, cus);
    }
  }
  printf("host_check OK (%d checks)\n", g_checks);
  return 0;
}
