// Host side of the ODS decode library that needs no GPU: operator tables,
// argument validation, the KV page allocator, buffer and workspace sizing,
// the kernels' launch-shape choices, and the planner that turns an operator
// range into launch descriptions (one native submission per stage; Section 6,
// "Single native submission"). Plain C++: it builds with a host compiler
// alone, so the CPU sanitizers can run it. Nothing here allocates device
// memory or calls the HIP runtime; the validation and planning paths allocate
// no host memory either.
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <vector>

#include "plan.hpp"

namespace ods {

namespace {

thread_local char g_err[512] = "";

const OpKind kDenseOps[10] = {K_ATTN_NORM, K_QKV, K_ROPE, K_KV_APPEND, K_ATTN_CORE,
                              K_O_PROJ, K_FFN_NORM, K_GATE_UP, K_SILU, K_DOWN};
const OpKind kMoeOps[14] = {K_ATTN_NORM, K_QKV, K_ROPE, K_KV_APPEND, K_ATTN_CORE, K_O_PROJ, K_FFN_NORM,
                            K_ROUTER, K_TOPK, K_PERMUTE, K_EXP_GATE_UP, K_EXP_SILU, K_EXP_DOWN, K_COMBINE};
const char *const kNames[] = {"attn_norm", "qkv_proj", "rope", "kv_append", "attn_core", "o_proj_residual",
                              "ffn_norm", "gate_up", "silu_mul", "down_residual", "router", "topk_softmax",
                              "moe_permute", "expert_gate_up", "silu_mul", "expert_down",
                              "moe_combine_residual"};

bool is_moe(const ods_layer_cfg &c) { return c.n_experts > 0; }
int qkv_dim(const ods_layer_cfg &c) { return (c.n_q + 2 * c.n_kv) * c.head_dim; }
bool tiled(const ods_layer &L) { return L.weight_layout == ODS_WEIGHTS_TILED; }
size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }
bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

ods_status check_cfg(const ods_layer_cfg &c, int layer) {
  if (c.hidden <= 0 || c.n_q <= 0 || c.n_kv <= 0 || c.head_dim <= 0 || c.window < 0 || c.n_experts < 0)
    return set_error(ODS_EINVAL, "layer %d: non-positive dimension or negative window", layer);
  if (c.head_dim != 64 && c.head_dim != 128)
    return set_error(ODS_EUNSUPPORTED, "layer %d: head_dim %d (supported: 64, 128)", layer, c.head_dim);
  if (c.n_q % c.n_kv != 0 || c.n_q / c.n_kv > 16)
    return set_error(ODS_EUNSUPPORTED, "layer %d: n_q %d / n_kv %d must be an integer <= 16", layer, c.n_q,
                     c.n_kv);
  if (c.hidden % 8 != 0) return set_error(ODS_EUNSUPPORTED, "layer %d: hidden %% 8 != 0", layer);
  if (!(c.rms_eps >= 0.f) || !(c.rope_theta > 0.f))
    return set_error(ODS_EINVAL, "layer %d: rms_eps must be >= 0 and rope_theta > 0", layer);
  if (is_moe(c)) {
    if (c.n_experts > 256 || c.top_k < 1 || c.top_k > c.n_experts || c.top_k > 64)
      return set_error(ODS_EUNSUPPORTED, "layer %d: n_experts %d / top_k %d (need 1 <= k <= min(E, 64), E <= 256)",
                       layer, c.n_experts, c.top_k);
    if (c.moe_ffn <= 0 || c.moe_ffn % 8 != 0)
      return set_error(ODS_EUNSUPPORTED, "layer %d: moe_ffn must be a positive multiple of 8", layer);
  } else if (c.ffn <= 0 || c.ffn % 8 != 0) {
    return set_error(ODS_EUNSUPPORTED, "layer %d: ffn must be a positive multiple of 8", layer);
  }
  return ODS_OK;
}

// Page table a layer's KV operators use: the window-only ring for a sliding-
// window layer when the batch carries one, the full page table otherwise.
struct KvMap {
  const int32_t *table;
  int cols;  // table columns
  int ring;  // > 0: logical page lp lives in column lp % ring
};

KvMap kv_map(const ods_layer_cfg &c, const ods_batch *b) {
  if (c.window > 0 && b->ring_pages > 0) return KvMap{b->ring_table, b->ring_pages, b->ring_pages};
  return KvMap{b->page_table, b->max_pages, 0};
}

AttnPlan plan_for(const ods_layer_cfg &c, const ods_batch *b, int cus) {
  return attn_plan(b->batch, c.n_kv, c.head_dim, kv_map(c, b).cols, c.window, b->split_pages, cus);
}

size_t layer_ws_bytes(const ods_layer &L, const ods_batch *b, int cus) {
  const ods_layer_cfg &c = L.cfg;
  const int B = b->batch;
  const bool t = tiled(L);
  size_t w = align_up(attn_ws_bytes(B, c.n_q, c.n_kv, c.head_dim, plan_for(c, b, cus)));
  auto g = [&](int N, int K, int epi, bool bt) { w = std::max(w, align_up(gemm_partial_bytes(B, N, K, epi, bt))); };
  g(qkv_dim(c), c.hidden, EPI_BF16, t);
  g(c.hidden, c.n_q * c.head_dim, EPI_RESID, t);
  if (is_moe(c)) {
    g(c.n_experts, c.hidden, EPI_F32, false);  // the router stays row-major
  } else {
    g(c.ffn, c.hidden, EPI_SILU, t);
    g(2 * c.ffn, c.hidden, EPI_BF16, t);
    g(c.hidden, c.ffn, EPI_RESID, t);
  }
  return w;
}

bool uses_ws(OpKind k) {
  return k == K_ATTN_CORE || k == K_QKV || k == K_O_PROJ || k == K_GATE_UP || k == K_DOWN || k == K_ROUTER;
}

struct Need {
  const void *p;
  const char *name;
};

}  // namespace

// ---------------------------------------------------------------- error state

ods_status set_error(ods_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}
void clear_error() { g_err[0] = 0; }
const char *error_text() { return g_err; }

// ---------------------------------------------------------------- launch shapes

// Large-M tiles pay off when the output is wide enough to fill 128-column
// tiles; a narrow output (the router's expert logits) stays on 64-row tiles.
bool use_big(int M, int N) { return M > kDecodeBM && N > 128; }

// Output tile width: 32 columns for narrow outputs (more blocks), 64 otherwise.
// SiLU-gated outputs count gate and up rows, so their tile is half as wide.
// A long-K narrow output (K >= 2N, the down projection) takes 64 columns: every
// block re-reads the activation rows of its K range, and at 32 columns those
// re-reads cost twice the weight bytes (down at M = 64: 38.4 -> 31.3 us with
// 8-way split-K restoring the block count).
bool long_k(int N, int K, int epi) { return epi != EPI_SILU && N > 128 && K >= 2 * N; }
int tile_n(int N, int K, int epi) {
  if (long_k(N, K, epi)) return 64;
  return (epi == EPI_SILU ? 2 * N : N) <= 8192 ? 32 : (epi == EPI_SILU ? 32 : 64);
}

// Dense GEMMs past 128 rows, and those of 33 to 64 rows except the SiLU-gated
// one (64-row tiles: at 64 rows qkv 20.2 -> 18.0 us, o_proj 16.4 -> 15.9 us and
// down 31.8 -> 29.2 us on the 8B-shaped layer, gate_up level at 53 us and
// slower below 48 rows; at 32 rows and fewer the gains are under 1 us).
bool gemm_use_stream(int M, int N, int K, int epi) {
  if (N <= 128 || K % 64 != 0) return false;
  return M > 128 || (M > 32 && M <= 64 && epi != EPI_SILU);
}

namespace {

// Split K (1, 2, 4 or 8 ways, at least 8 steps per split) while the blocks
// still fit one wave over the 256 compute units (the 256-row tile runs one
// block per CU, so 257 to 511 blocks would leave a mostly idle second wave:
// the MoE layer's qkv projection at 512 rows, 80 tiles, took 53 us with 4
// splits against 40 us with 2, reduce included).
int stream_splits(int tiles, int steps) {
  int s = 1;
  while (tiles * s * 2 <= 256 && s < 8 && steps / (s * 2) >= 8) s *= 2;
  return s;
}

int stream_n_tiles(int N, int epi) { return epi == EPI_SILU ? (N + 63) / 64 : (N + 127) / 128; }

}  // namespace

// Past 64 rows a dense GEMM takes the 256-row tile unless that grid, split-K
// included, would occupy fewer than half of the 256 compute units (small
// weights: a tensor-parallel share of a layer, a narrow model). Then 64-row
// tiles give it ceil(M / 64) times the blocks, and the blocks of one N tile
// read its weights through one XCD's L2. Measured at M = 256 on one GPU's
// share of the 8B-shaped layer under 8-way tensor parallelism (lab, tiled
// weights, reduce included; 256-row -> 64-row tile): qkv (N 768, 48 -> 192
// blocks) 13.0 -> 8.3 us, o_proj (K 512, 32 -> 128 blocks) 12.9 -> 7.9 us,
// down (K 1792, 64 -> 256 blocks) 23.7 -> 17.2 us; gate_up + SiLU (N 1792)
// keeps 224 256-row blocks (24.3 us; 22.9 us as 64-row tiles). With 192 or
// more 256-row blocks the 256-row tile stays ahead (the 8B-shaped layer's
// GEMMs at M = 256: gate_up 81 against 113 us, down 48-51 against 62-64 us
// as 64-row tiles).
int gemm_stream_rows(int M, int N, int K, int epi) {
  if (M <= 64) return 64;
  const int tiles = (M + 255) / 256 * stream_n_tiles(N, epi);
  const int s = N % 4 != 0 ? 1 : stream_splits(tiles, K / 64);
  return tiles * s < 128 ? 64 : 256;
}

// The reduce works on 4-column groups: other widths run unsplit.
int gemm_stream_splits(int M, int N, int K, int epi) {
  if (N % 4 != 0) return 1;
  const int rows = gemm_stream_rows(M, N, K, epi);
  return stream_splits((M + rows - 1) / rows * stream_n_tiles(N, epi), K / 64);
}

int gemm_splits(int M, int N, int K, int epi, bool b_tiled) {
  if (b_tiled || gemm_use_stream(M, N, K, epi)) return gemm_stream_splits(M, N, K, epi);
  if (N % 4 != 0) return 1;  // the reduce works on 4-column groups
  if (use_big(M, N)) {
    // Large-M tiles: one 512-thread block per compute unit; split K (up to 8
    // ways, at least 8 steps of 64 per block) until ~192 blocks are in flight.
    const int bm = M > 128 ? 256 : 128, bn = epi == EPI_SILU ? 64 : 128;
    const int tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    const int steps = (K + 63) / 64;
    int s = 1;
    while (tiles * s < 192 && s < 8 && steps / (s * 2) >= 8) s *= 2;
    return s;
  }
  const int bn = tile_n(N, K, epi);
  const int tiles = ((M + kDecodeBM - 1) / kDecodeBM) * ((N + bn - 1) / bn);
  const int steps = (K + kDecodeBK - 1) / kDecodeBK;
  int s = 1;
  // Too few tiles leaves HBM idle: split K up to 4 ways (8 for long K) until
  // there are about two blocks per compute unit, keeping at least 8 K steps
  // per block. The SiLU-gated GEMM is wide enough at decode batches and skips
  // the extra pass. A narrow output has few tiles at any batch: split it up to
  // 16 ways, down to 2 K steps per block.
  const int want = epi == EPI_SILU ? 256 : 512;
  const bool narrow = N <= 128;
  const int max_s = narrow ? 16 : long_k(N, K, epi) ? 8 : 4, min_steps = narrow ? 2 : 8;
  while (tiles * s < want && s < max_s && steps / (s * 2) >= min_steps) s *= 2;
  return s;
}

size_t gemm_partial_bytes(int M, int N, int K, int epi, bool b_tiled) {
  const int s = gemm_splits(M, N, K, epi, b_tiled);
  if (s <= 1) return 0;
  return (size_t)s * M * N * (epi == EPI_SILU ? 2 : 1) * sizeof(float);
}

int64_t tiled_weight_elems(int out, int in, bool gated, int groups) {
  const int64_t tiles = gated ? (out + 63) / 64 : (out + 127) / 128;
  return (int64_t)groups * tiles * (in / 64) * (128 * 64);
}

// Grid of the attention kernel: one 4-wave block per compute unit, fewer when
// the batch cannot fill them with ranges of at least 8 pages. Fewer waves in
// flight stream the pool faster: measured on one MI355X, B = 64 x U[512, 4096]
// 122.7 -> 115.6 us, B = 256 x 8192 1444 -> 1376 us, MoE B = 512 1593 ->
// 1563 us from three blocks per unit to one (two was in between). The kernel
// is built for at most two waves per SIMD (256 VGPRs), which leaves its 170
// registers unspilled.
int attn_grid(int B, int n_kv, int span, int cus) {
  const int64_t max_units = (int64_t)B * n_kv * span;
  return (int)std::max<int64_t>(1, std::min<int64_t>(std::max(cus, 1), (max_units + 31) / 32));
}

int attn_span(int max_pages, int window) {
  int span = max_pages;
  if (window > 0) span = std::min(max_pages, (window + ODS_PAGE_TOKENS - 1) / ODS_PAGE_TOKENS + 1);
  return std::max(span, 1);
}

AttnPlan attn_plan(int B, int n_kv, int D, int max_pages, int window, int split_pages_req, int cus) {
  (void)D;
  const int span = attn_span(max_pages, window);
  AttnPlan plan;
  plan.seg_pages = split_pages_req;
  plan.grid = attn_grid(B, n_kv, span, cus);
  // Records r + seq with r a range index: ranges <= waves when S is chosen
  // from the total, else <= ceil(max units / S).
  const int64_t seqs = (int64_t)B * n_kv;
  const int64_t ranges = split_pages_req > 0 ? (seqs * span + split_pages_req - 1) / split_pages_req
                                             : (int64_t)plan.grid * 4;
  plan.records = ranges + seqs;
  plan.units_ok = seqs * span < (int64_t)1 << 30;
  return plan;
}

size_t attn_ws_bytes(int B, int n_q, int n_kv, int D, const AttnPlan &plan) {
  const size_t group = n_q / n_kv;
  return (size_t)B * n_kv * 2 * sizeof(int32_t) + (size_t)plan.records * group * (D + 2) * sizeof(float);
}

// ---------------------------------------------------------------- blocks and ranges

const char *op_kind_name(OpKind k) { return kNames[k]; }
int layer_num_ops(const ods_layer_cfg &c) { return is_moe(c) ? 14 : 10; }

ods_status check_block(const ods_block *blk) {
  if (!blk || !blk->layers || blk->n_layers <= 0) return set_error(ODS_EINVAL, "null or empty block");
  for (int l = 0; l < blk->n_layers; ++l) {
    const ods_layer &L = blk->layers[l];
    ods_status st = check_cfg(L.cfg, l);
    if (st != ODS_OK) return st;
    if (L.weight_layout != ODS_WEIGHTS_ROWS && L.weight_layout != ODS_WEIGHTS_TILED)
      return set_error(ODS_EINVAL, "layer %d: weight_layout %d", l, L.weight_layout);
    if (tiled(L)) {
      const ods_layer_cfg &c = L.cfg;
      const int f = is_moe(c) ? c.moe_ffn : c.ffn;
      if (c.hidden % 64 != 0 || (c.n_q * c.head_dim) % 64 != 0 || f % 64 != 0)
        return set_error(ODS_EUNSUPPORTED, "layer %d: tiled weights need hidden, n_q * head_dim and the FFN width "
                         "to be multiples of 64", l);
    }
  }
  return ODS_OK;
}

int num_ops(const ods_block *blk) {
  int n = 0;
  for (int l = 0; l < blk->n_layers; ++l) n += layer_num_ops(blk->layers[l].cfg);
  return n;
}

OpRef op_at(const ods_block *blk, int g) {
  if (g < 0) return OpRef{-1, K_ATTN_NORM};
  for (int l = 0; l < blk->n_layers; ++l) {
    const ods_layer_cfg &c = blk->layers[l].cfg;
    const int n = layer_num_ops(c);
    if (g < n) return OpRef{l, is_moe(c) ? kMoeOps[g] : kDenseOps[g]};
    g -= n;
  }
  return OpRef{-1, K_ATTN_NORM};
}

int layer_offset(const ods_block *blk, int layer) {
  int n = 0;
  for (int l = 0; l < layer; ++l) n += layer_num_ops(blk->layers[l].cfg);
  return n;
}

size_t range_ws_bytes(const ods_block *blk, int op_begin, int op_end, const ods_batch *batch, int cus) {
  size_t w = 0;
  int last = -1;
  for (int g = op_begin; g < op_end; ++g) {
    const int l = op_at(blk, g).layer;
    if (l != last) w = std::max(w, layer_ws_bytes(blk->layers[l], batch, cus));
    last = l;
  }
  return w;
}

size_t block_ws_bytes(const ods_block *blk, const ods_batch *batch, int cus) {
  size_t w = 256;
  for (int l = 0; l < blk->n_layers; ++l) w = std::max(w, layer_ws_bytes(blk->layers[l], batch, cus));
  return w;
}

namespace {

// Same layer, next operator inside the range?
bool next_is(const ods_block *blk, int g, int op_end, OpKind k) {
  if (g + 1 >= op_end) return false;
  const OpRef a = op_at(blk, g), b = op_at(blk, g + 1);
  return a.layer == b.layer && b.kind == k;
}

// The expert gate_up GEMM reads its rows of hn through perm (no xp copy)
// when moe_permute precedes it in the same range and the streaming kernel
// runs it (K % 64 == 0).
bool gather_fused(const ods_block *blk, int g_permute, int op_end) {
  const OpRef op = op_at(blk, g_permute);
  return op.kind == K_PERMUTE && next_is(blk, g_permute, op_end, K_EXP_GATE_UP) &&
         blk->layers[op.layer].cfg.hidden % 64 == 0;
}

}  // namespace

ods_status validate_range(const ods_block *blk, int op_begin, int op_end, const ods_batch *batch,
                          const ods_state *st, int cus) {
  ods_status rc = check_block(blk);
  if (rc != ODS_OK) return rc;
  if (!batch || !st) return set_error(ODS_EINVAL, "null batch or state");
  const int n_ops = num_ops(blk);
  if (op_begin < 0 || op_end > n_ops || op_begin >= op_end)
    return set_error(ODS_ERANGE, "operator range [%d, %d) outside [0, %d) or empty", op_begin, op_end, n_ops);
  const int B = batch->batch;
  if (B < 0) return set_error(ODS_EINVAL, "negative batch");
  if (batch->split_pages < 0) return set_error(ODS_EINVAL, "negative split_pages");
  if (batch->ring_pages < 0) return set_error(ODS_EINVAL, "negative ring_pages");
  if (B == 0) return ODS_OK;  // nothing to read or write: the batch-sized pointers may be null

  bool need_ws = false;
  for (int g = op_begin; g < op_end; ++g) {
    const OpRef op = op_at(blk, g);
    const ods_layer &L = blk->layers[op.layer];
    const ods_layer_cfg &c = L.cfg;
    const OpKind k = op.kind;
    const bool fuse_silu = (k == K_GATE_UP && next_is(blk, g, op_end, K_SILU)) ||
                           (k == K_EXP_GATE_UP && next_is(blk, g, op_end, K_EXP_SILU));
    Need need[8];
    int n = 0;
    auto add = [&](const void *p, const char *name) { need[n++] = Need{p, name}; };
    bool paged = false;
    need_ws = need_ws || uses_ws(k);
    switch (k) {
      case K_ATTN_NORM: add(st->resid, "resid"); add(st->xn, "xn"); add(L.g_attn, "g_attn"); break;
      case K_QKV: add(st->xn, "xn"); add(st->qkv, "qkv"); add(L.w_qkv, "w_qkv"); break;
      case K_ROPE: add(st->qkv, "qkv"); add(batch->ctx_lens, "ctx_lens"); paged = true; break;
      case K_KV_APPEND:
      case K_ATTN_CORE: {
        const KvMap m = kv_map(c, batch);
        add(st->qkv, "qkv");
        add(batch->ctx_lens, "ctx_lens");
        add(m.table, m.ring ? "ring_table" : "page_table");
        add(L.kv_pool, "kv_pool");
        if (k == K_ATTN_CORE) {
          add(st->o, "o");
          add(st->ws, "ws");
          if (B > kMaxAttnBatch)
            return set_error(ODS_EUNSUPPORTED, "layer %d: attn_core supports batch <= %d, got %d", op.layer,
                             kMaxAttnBatch, B);
          if (!plan_for(c, batch, cus).units_ok)
            return set_error(ODS_EUNSUPPORTED, "layer %d: batch * n_kv * window pages exceeds 2^30", op.layer);
        }
        paged = true;
        break;
      }
      case K_O_PROJ: add(st->o, "o"); add(st->resid, "resid"); add(L.w_o, "w_o"); break;
      case K_FFN_NORM: add(st->resid, "resid"); add(st->hn, "hn"); add(L.g_ffn, "g_ffn"); break;
      case K_GATE_UP:
        add(st->hn, "hn");
        add(L.w_gate_up, "w_gate_up");
        if (fuse_silu) add(st->act, "act"); else add(st->gu, "gu");
        break;
      case K_SILU: add(st->gu, "gu"); add(st->act, "act"); break;
      case K_DOWN: add(st->act, "act"); add(st->resid, "resid"); add(L.w_down, "w_down"); break;
      case K_ROUTER: add(st->hn, "hn"); add(L.w_router, "w_router"); add(st->logits, "logits"); break;
      case K_TOPK: add(st->logits, "logits"); add(st->topk_ids, "topk_ids"); add(st->topk_w, "topk_w"); break;
      case K_PERMUTE:
        add(st->topk_ids, "topk_ids"); add(st->hn, "hn"); add(st->perm, "perm"); add(st->slot_pos, "slot_pos");
        add(st->expert_off, "expert_off"); add(st->xp, "xp");
        break;
      case K_EXP_GATE_UP:
        if (g > op_begin && gather_fused(blk, g - 1, op_end)) {
          add(st->hn, "hn");
          add(st->perm, "perm");
        } else {
          add(st->xp, "xp");
        }
        add(st->expert_off, "expert_off");
        add(L.w_gate_up, "w_gate_up");
        if (fuse_silu) add(st->act_p, "act_p"); else add(st->gu_p, "gu_p");
        break;
      case K_EXP_SILU: add(st->gu_p, "gu_p"); add(st->act_p, "act_p"); break;
      case K_EXP_DOWN:
        add(st->act_p, "act_p"); add(st->expert_off, "expert_off"); add(L.w_down, "w_down"); add(st->yp, "yp");
        break;
      case K_COMBINE:
        add(st->yp, "yp"); add(st->topk_w, "topk_w"); add(st->slot_pos, "slot_pos"); add(st->resid, "resid");
        break;
    }
    for (int i = 0; i < n; ++i) {
      if (!need[i].p)
        return set_error(ODS_EINVAL, "op %s (layer %d): %s is null", kNames[k], op.layer, need[i].name);
      if (!aligned16(need[i].p))
        return set_error(ODS_EINVAL, "op %s (layer %d): %s is not 16-byte aligned", kNames[k], op.layer,
                         need[i].name);
    }
    if (paged) {
      if (batch->max_pages <= 0) return set_error(ODS_EINVAL, "max_pages must be positive");
      if ((int64_t)batch->max_pages * ODS_PAGE_TOKENS > INT32_MAX) return set_error(ODS_ERANGE, "max_pages too large");
      if (k != K_ROPE && L.pool_pages <= 0) return set_error(ODS_EINVAL, "layer %d: pool_pages <= 0", op.layer);
      const KvMap m = kv_map(c, batch);
      if (m.ring > 0) {
        const int64_t need_pages = ((int64_t)c.window + ODS_PAGE_TOKENS - 1) / ODS_PAGE_TOKENS + 1;
        if (m.ring < need_pages)
          return set_error(ODS_EINVAL, "layer %d: ring_pages %d < ceil(window / 16) + 1 = %lld", op.layer, m.ring,
                           (long long)need_pages);
      }
    }
    if (is_moe(c) && (int64_t)B * c.top_k > INT32_MAX / 2) return set_error(ODS_ERANGE, "batch * top_k too large");
  }
  if (need_ws) {
    const size_t ws_need = range_ws_bytes(blk, op_begin, op_end, batch, cus);
    if (!st->ws) return set_error(ODS_EINVAL, "ws is null");
    if (!aligned16(st->ws)) return set_error(ODS_EINVAL, "ws is not 16-byte aligned");
    if (st->ws_bytes < ws_need)
      return set_error(ODS_ENOMEM, "workspace %zu bytes < required %zu", st->ws_bytes, ws_need);
  }
  return ODS_OK;
}

void plan_launch(const ods_block *blk, int op_begin, int op_end, int i, const ods_batch *batch, const ods_state *st,
                 int cus, Launch *out) {
  const int g = op_begin + i;
  const OpRef op = op_at(blk, g);
  const ods_layer &L = blk->layers[op.layer];
  const ods_layer_cfg &c = L.cfg;
  const int B = batch->batch, H = c.hidden, D = c.head_dim;
  const bool wt = tiled(L);  // projection weights in tile order (the router never is)
  Launch &o = *out;
  o = Launch{};
  o.layer = op.layer;
  o.n_ops = 1;
  o.what = kNames[op.kind];
  auto U = [](const void *p) { return (uint16_t *)p; };
  auto dense_gemm = [&](const void *A, const void *Bw, void *C, int N, int K, int epi, int n_up, int ldc,
                        bool defer_reduce, bool b_tiled) {
    GemmArgs &ga = o.gemm;
    ga.A = (const uint16_t *)A; ga.lda = K;
    ga.B = (const uint16_t *)Bw; ga.ldb = K; ga.b_group_stride = 0;
    ga.C = C; ga.ldc = ldc;
    ga.M = B; ga.N = N; ga.K = K; ga.n_up = n_up; ga.epi = epi;
    ga.group_off = nullptr; ga.groups = 0;
    ga.b_tiled = b_tiled ? 1 : 0;
    ga.splits = gemm_splits(B, N, K, epi, b_tiled);
    ga.partial = (float *)st->ws;
    ga.defer_reduce = defer_reduce ? 1 : 0;
    o.kind = LK_GEMM;
  };
  auto rope = [&](bool do_rope, bool do_append) {
    const KvMap m = kv_map(c, batch);
    RopeArgs &r = o.rope;
    r.qkv = U(st->qkv); r.B = B; r.n_q = c.n_q; r.n_kv = c.n_kv; r.D = D; r.theta = c.rope_theta;
    r.ctx_lens = batch->ctx_lens; r.table = m.table; r.cols = m.cols; r.ring = m.ring;
    r.pool = U(L.kv_pool); r.pool_pages = L.pool_pages;
    r.do_rope = do_rope; r.do_append = do_append;
    r.partial = nullptr; r.splits = 1;
  };
  switch (op.kind) {
    case K_ATTN_NORM:
    case K_FFN_NORM:
      o.kind = LK_RMSNORM;
      o.x = U(st->resid);
      o.gain = U(op.kind == K_ATTN_NORM ? L.g_attn : L.g_ffn);
      o.out = U(op.kind == K_ATTN_NORM ? st->xn : st->hn);
      o.rows = B; o.width = H; o.eps = c.rms_eps;
      break;
    case K_QKV: {
      // With split-K and RoPE next in the range, the RoPE / KV-append kernel
      // sums the partials itself (same order and rounding as the reduce).
      const bool fuse = next_is(blk, g, op_end, K_ROPE) && gemm_splits(B, qkv_dim(c), H, EPI_BF16, wt) > 1;
      dense_gemm(st->xn, L.w_qkv, st->qkv, qkv_dim(c), H, EPI_BF16, 0, qkv_dim(c), fuse, wt);
      if (fuse) {
        const bool app = g + 2 < op_end && op_at(blk, g + 2).layer == op.layer && op_at(blk, g + 2).kind == K_KV_APPEND;
        rope(true, app);
        o.rope.partial = (const float *)st->ws;
        o.rope.splits = o.gemm.splits;
        o.kind = LK_QKV_ROPE;
        o.what = app ? "qkv_proj+rope+kv_append" : "qkv_proj+rope";
        o.n_ops = app ? 3 : 2;
      }
      break;
    }
    case K_ROPE:
    case K_KV_APPEND: {
      const bool both = op.kind == K_ROPE && next_is(blk, g, op_end, K_KV_APPEND);
      rope(op.kind == K_ROPE, both || op.kind == K_KV_APPEND);
      o.kind = LK_ROPE_APPEND;
      if (both) {
        o.what = "rope+kv_append";
        o.n_ops = 2;
      }
      break;
    }
    case K_ATTN_CORE: {
      const KvMap m = kv_map(c, batch);
      AttnArgs &a = o.attn;
      a.qkv = U(st->qkv); a.B = B; a.n_q = c.n_q; a.n_kv = c.n_kv; a.D = D; a.window = c.window;
      a.ctx_lens = batch->ctx_lens; a.table = m.table; a.cols = m.cols; a.ring = m.ring;
      a.pool = U(L.kv_pool); a.pool_pages = L.pool_pages;
      a.plan = plan_for(c, batch, cus);
      a.ws = (float *)st->ws;
      a.o = U(st->o);
      o.kind = LK_ATTENTION;
      break;
    }
    case K_O_PROJ: dense_gemm(st->o, L.w_o, st->resid, H, c.n_q * D, EPI_RESID, 0, H, false, wt); break;
    case K_GATE_UP:
      if (next_is(blk, g, op_end, K_SILU)) {
        dense_gemm(st->hn, L.w_gate_up, st->act, c.ffn, H, EPI_SILU, c.ffn, c.ffn, false, wt);
        o.what = "gate_up+silu_mul";
        o.n_ops = 2;
      } else {
        // tiled gate_up pairs gate and up rows per tile: n_up tells the plain epilogue where the up half goes
        dense_gemm(st->hn, L.w_gate_up, st->gu, 2 * c.ffn, H, EPI_BF16, wt ? c.ffn : 0, 2 * c.ffn, false, wt);
      }
      break;
    case K_SILU:
    case K_EXP_SILU:
      o.kind = LK_SILU;
      o.x = U(op.kind == K_SILU ? st->gu : st->gu_p);
      o.out = U(op.kind == K_SILU ? st->act : st->act_p);
      o.rows = op.kind == K_SILU ? B : B * c.top_k;
      o.width = op.kind == K_SILU ? c.ffn : c.moe_ffn;
      break;
    case K_DOWN: dense_gemm(st->act, L.w_down, st->resid, H, c.ffn, EPI_RESID, 0, H, false, wt); break;
    case K_ROUTER: {
      // With split-K and top-k next in the range, the top-k kernel sums the
      // partials itself (same order as the reduce) and writes the logits.
      const bool fuse = next_is(blk, g, op_end, K_TOPK) && gemm_splits(B, c.n_experts, H, EPI_F32, false) > 1;
      dense_gemm(st->hn, L.w_router, st->logits, c.n_experts, H, EPI_F32, 0, c.n_experts, fuse, false);
      if (fuse) {
        o.kind = LK_ROUTER_TOPK;
        o.rows = B; o.E = c.n_experts; o.k = c.top_k; o.ids = st->topk_ids; o.weights = st->topk_w;
        o.logits_out = st->logits; o.topk_partial = (const float *)st->ws; o.topk_splits = o.gemm.splits;
        o.what = "router+topk_softmax";
        o.n_ops = 2;
      }
      break;
    }
    case K_TOPK:
      o.kind = LK_TOPK;
      o.logits = st->logits; o.rows = B; o.E = c.n_experts; o.k = c.top_k; o.ids = st->topk_ids; o.weights = st->topk_w;
      break;
    case K_PERMUTE:
      o.kind = LK_PERMUTE;
      o.ids = st->topk_ids; o.rows = B; o.k = c.top_k; o.E = c.n_experts; o.perm = st->perm;
      o.slot_pos = st->slot_pos; o.expert_off = st->expert_off; o.x = U(st->hn); o.width = H;
      o.xp = gather_fused(blk, g, op_end) ? nullptr : U(st->xp);  // null: the expert GEMM gathers
      break;
    case K_EXP_GATE_UP:
    case K_EXP_DOWN: {
      const bool fuse = op.kind == K_EXP_GATE_UP && next_is(blk, g, op_end, K_EXP_SILU);
      const int I = c.moe_ffn;
      GemmArgs &ga = o.gemm;
      ga.M = B * c.top_k;
      ga.group_off = st->expert_off;
      ga.groups = c.n_experts;
      ga.splits = 1;
      ga.partial = nullptr;
      ga.b_tiled = wt ? 1 : 0;
      if (op.kind == K_EXP_GATE_UP) {
        ga.A = U(st->xp); ga.lda = H; ga.K = H;
        if (g > op_begin && gather_fused(blk, g - 1, op_end)) {
          ga.A = U(st->hn);
          ga.a_gather = st->perm; ga.a_gather_div = c.top_k; ga.a_gather_rows = B;
          o.what = fuse ? "expert_gate_up+silu_mul (rows gathered by perm)" : "expert_gate_up (rows gathered by perm)";
        }
        ga.B = U(L.w_gate_up); ga.ldb = H;
        ga.b_group_stride = wt ? tiled_weight_elems(I, H, true, 1) : (int64_t)2 * I * H;
        if (fuse) {
          ga.C = st->act_p; ga.ldc = I; ga.N = I; ga.n_up = I; ga.epi = EPI_SILU;
          if (!ga.a_gather) o.what = "expert_gate_up+silu_mul";
          o.n_ops = 2;
        } else {
          ga.C = st->gu_p; ga.ldc = 2 * I; ga.N = 2 * I; ga.n_up = wt ? I : 0; ga.epi = EPI_BF16;
        }
      } else {
        ga.A = U(st->act_p); ga.lda = I; ga.K = I;
        ga.B = U(L.w_down); ga.ldb = I;
        ga.b_group_stride = wt ? tiled_weight_elems(H, I, false, 1) : (int64_t)H * I;
        ga.C = st->yp; ga.ldc = H; ga.N = H; ga.n_up = 0; ga.epi = EPI_BF16;
      }
      o.kind = LK_GEMM;
      break;
    }
    case K_COMBINE:
      o.kind = LK_COMBINE;
      o.x = U(st->yp); o.weights = st->topk_w; o.slot_pos = st->slot_pos; o.rows = B; o.k = c.top_k; o.width = H;
      o.out = U(st->resid);
      break;
  }
}

}  // namespace ods

// ---------------------------------------------------------------- C ABI (host-only entry points)

using namespace ods;

extern "C" {

const char *ods_last_error(void) { return error_text(); }

ods_status ods_kv_alloc(int64_t pool_pages, const int32_t *ctx_lens_host, int32_t batch, uint64_t seed,
                        int32_t max_pages, int32_t *page_table_host) {
  if (!ctx_lens_host || !page_table_host) return set_error(ODS_EINVAL, "ods_kv_alloc: null pointer");
  if (batch < 0 || max_pages <= 0 || pool_pages <= 0)
    return set_error(ODS_EINVAL, "ods_kv_alloc: batch %d, max_pages %d, pool_pages %lld", batch, max_pages,
                     (long long)pool_pages);
  int64_t need = 0;
  for (int b = 0; b < batch; ++b) {
    if (ctx_lens_host[b] <= 0)
      return set_error(ODS_EINVAL, "ods_kv_alloc: ctx_lens[%d] = %d", b, ctx_lens_host[b]);
    const int64_t n = ((int64_t)ctx_lens_host[b] + ODS_PAGE_TOKENS - 1) / ODS_PAGE_TOKENS;
    if (n > max_pages)
      return set_error(ODS_ERANGE, "ods_kv_alloc: sequence %d needs %lld pages > max_pages %d", b, (long long)n,
                       max_pages);
    need += n;
  }
  if (need > pool_pages)
    return set_error(ODS_ENOMEM, "ods_kv_alloc: batch needs %lld pages, pool has %lld", (long long)need,
                     (long long)pool_pages);
  if (pool_pages > INT32_MAX) return set_error(ODS_ERANGE, "ods_kv_alloc: pool_pages exceeds int32 page ids");
  std::vector<int32_t> ids((size_t)pool_pages);
  for (int64_t i = 0; i < pool_pages; ++i) ids[(size_t)i] = (int32_t)i;
  uint64_t state = seed;
  for (int64_t i = pool_pages - 1; i >= 1; --i) {
    state += 0x9E3779B97F4A7C15ull;  // splitmix64 (Steele, Lea, Flood 2014)
    uint64_t z = state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    const int64_t j = (int64_t)(z % (uint64_t)(i + 1));
    std::swap(ids[(size_t)i], ids[(size_t)j]);
  }
  size_t next = 0;
  for (int b = 0; b < batch; ++b) {
    const int n = (ctx_lens_host[b] + ODS_PAGE_TOKENS - 1) / ODS_PAGE_TOKENS;
    int32_t *row = page_table_host + (int64_t)b * max_pages;
    for (int j = 0; j < max_pages; ++j) row[j] = j < n ? ids[next + j] : -1;
    next += n;
  }
  clear_error();
  return ODS_OK;
}

size_t ods_kv_pool_bytes(const ods_layer_cfg *cfg, int64_t pool_pages) {
  if (!cfg || pool_pages < 0 || check_cfg(*cfg, 0) != ODS_OK) return 0;
  return (size_t)pool_pages * 2 * cfg->n_kv * ODS_PAGE_TOKENS * cfg->head_dim * 2;
}

size_t ods_live_bytes(const ods_block *blk, int32_t batch, ods_buffer which) {
  if (check_block(blk) != ODS_OK || batch < 0) return 0;
  size_t best = 0;
  const size_t B = (size_t)batch;
  for (int l = 0; l < blk->n_layers; ++l) {
    const ods_layer_cfg &c = blk->layers[l].cfg;
    const size_t H = c.hidden, E = c.n_experts, k = c.top_k, I = c.moe_ffn, F = c.ffn;
    size_t s = 0;
    switch (which) {
      case ODS_BUF_RESID: case ODS_BUF_XN: case ODS_BUF_HN: s = B * H * 2; break;
      case ODS_BUF_QKV: s = B * qkv_dim(c) * 2; break;
      case ODS_BUF_O: s = B * c.n_q * c.head_dim * 2; break;
      case ODS_BUF_GU: s = is_moe(c) ? 0 : B * 2 * F * 2; break;
      case ODS_BUF_ACT: s = is_moe(c) ? 0 : B * F * 2; break;
      case ODS_BUF_LOGITS: s = B * E * 4; break;
      case ODS_BUF_TOPK_W: case ODS_BUF_TOPK_IDS: case ODS_BUF_PERM: case ODS_BUF_SLOT_POS: s = B * k * 4; break;
      case ODS_BUF_EXPERT_OFF: s = is_moe(c) ? (E + 1) * 4 : 0; break;
      case ODS_BUF_XP: case ODS_BUF_YP: s = B * k * H * 2; break;
      case ODS_BUF_GU_P: s = B * k * 2 * I * 2; break;
      case ODS_BUF_ACT_P: s = B * k * I * 2; break;
      default: return 0;
    }
    best = std::max(best, s);
  }
  return best;
}

int32_t ods_block_num_ops(const ods_block *blk) {
  if (check_block(blk) != ODS_OK) return -1;
  return num_ops(blk);
}

const char *ods_op_name(const ods_block *blk, int32_t op) {
  if (check_block(blk) != ODS_OK || op < 0 || op >= num_ops(blk)) return nullptr;
  return kNames[op_at(blk, op).kind];
}

size_t ods_tiled_weight_bytes(int32_t out, int32_t in, int32_t gated, int32_t groups) {
  if (out < 1 || in < 64 || in % 64 != 0 || groups < 1 || (gated != 0 && gated != 1)) return 0;
  return (size_t)tiled_weight_elems(out, in, gated != 0, groups) * 2;
}

}  // extern "C"
