// Host side of the ODS decode library: argument validation, the KV page
// allocator, buffer sizing, and the operator-range dispatcher that turns a
// stage [op_begin, op_end) of a partition block into kernel launches on one
// stream (one native submission per stage, no allocation, no synchronisation).
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/ods.h"
#include "kernels.hpp"

using namespace ods;

namespace {

thread_local char g_err[512] = "";

ods_status fail(ods_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

enum OpKind {
  K_ATTN_NORM, K_QKV, K_ROPE, K_KV_APPEND, K_ATTN_CORE, K_O_PROJ, K_FFN_NORM,
  K_GATE_UP, K_SILU, K_DOWN,
  K_ROUTER, K_TOPK, K_PERMUTE, K_EXP_GATE_UP, K_EXP_SILU, K_EXP_DOWN, K_COMBINE
};

const OpKind kDenseOps[10] = {K_ATTN_NORM, K_QKV, K_ROPE, K_KV_APPEND, K_ATTN_CORE,
                              K_O_PROJ, K_FFN_NORM, K_GATE_UP, K_SILU, K_DOWN};
const OpKind kMoeOps[14] = {K_ATTN_NORM, K_QKV, K_ROPE, K_KV_APPEND, K_ATTN_CORE, K_O_PROJ, K_FFN_NORM,
                            K_ROUTER, K_TOPK, K_PERMUTE, K_EXP_GATE_UP, K_EXP_SILU, K_EXP_DOWN, K_COMBINE};
const char *kNames[] = {"attn_norm", "qkv_proj", "rope", "kv_append", "attn_core", "o_proj_residual",
                        "ffn_norm", "gate_up", "silu_mul", "down_residual", "router", "topk_softmax",
                        "moe_permute", "expert_gate_up", "silu_mul", "expert_down",
                        "moe_combine_residual"};

bool is_moe(const ods_layer_cfg &c) { return c.n_experts > 0; }
int layer_ops(const ods_layer_cfg &c) { return is_moe(c) ? 14 : 10; }
int qkv_dim(const ods_layer_cfg &c) { return (c.n_q + 2 * c.n_kv) * c.head_dim; }

struct OpRef {
  int layer;
  OpKind kind;
};

ods_status check_cfg(const ods_layer_cfg &c, int layer) {
  if (c.hidden <= 0 || c.n_q <= 0 || c.n_kv <= 0 || c.head_dim <= 0 || c.window < 0 || c.n_experts < 0)
    return fail(ODS_EINVAL, "layer %d: non-positive dimension or negative window", layer);
  if (c.head_dim != 64 && c.head_dim != 128)
    return fail(ODS_EUNSUPPORTED, "layer %d: head_dim %d (supported: 64, 128)", layer, c.head_dim);
  if (c.n_q % c.n_kv != 0 || c.n_q / c.n_kv > 16)
    return fail(ODS_EUNSUPPORTED, "layer %d: n_q %d / n_kv %d must be an integer <= 16", layer, c.n_q, c.n_kv);
  if (c.hidden % 8 != 0) return fail(ODS_EUNSUPPORTED, "layer %d: hidden %% 8 != 0", layer);
  if (!(c.rms_eps >= 0.f) || !(c.rope_theta > 0.f))
    return fail(ODS_EINVAL, "layer %d: rms_eps must be >= 0 and rope_theta > 0", layer);
  if (is_moe(c)) {
    if (c.n_experts > 256 || c.top_k < 1 || c.top_k > c.n_experts || c.top_k > 64)
      return fail(ODS_EUNSUPPORTED, "layer %d: n_experts %d / top_k %d (need 1 <= k <= min(E, 64), E <= 256)",
                  layer, c.n_experts, c.top_k);
    if (c.moe_ffn <= 0 || c.moe_ffn % 8 != 0)
      return fail(ODS_EUNSUPPORTED, "layer %d: moe_ffn must be a positive multiple of 8", layer);
  } else if (c.ffn <= 0 || c.ffn % 8 != 0) {
    return fail(ODS_EUNSUPPORTED, "layer %d: ffn must be a positive multiple of 8", layer);
  }
  return ODS_OK;
}

bool tiled(const ods_layer &L) { return L.weight_layout == ODS_WEIGHTS_TILED; }

ods_status check_block(const ods_block *blk) {
  if (!blk || !blk->layers || blk->n_layers <= 0) return fail(ODS_EINVAL, "null or empty block");
  for (int l = 0; l < blk->n_layers; ++l) {
    const ods_layer &L = blk->layers[l];
    ods_status st = check_cfg(L.cfg, l);
    if (st != ODS_OK) return st;
    if (L.weight_layout != ODS_WEIGHTS_ROWS && L.weight_layout != ODS_WEIGHTS_TILED)
      return fail(ODS_EINVAL, "layer %d: weight_layout %d", l, L.weight_layout);
    if (tiled(L)) {
      const ods_layer_cfg &c = L.cfg;
      const int f = is_moe(c) ? c.moe_ffn : c.ffn;
      if (c.hidden % 64 != 0 || (c.n_q * c.head_dim) % 64 != 0 || f % 64 != 0)
        return fail(ODS_EUNSUPPORTED, "layer %d: tiled weights need hidden, n_q * head_dim and the FFN width "
                    "to be multiples of 64", l);
    }
  }
  return ODS_OK;
}

int num_ops(const ods_block *blk) {
  int n = 0;
  for (int l = 0; l < blk->n_layers; ++l) n += layer_ops(blk->layers[l].cfg);
  return n;
}

OpRef op_at(const ods_block *blk, int g) {
  for (int l = 0; l < blk->n_layers; ++l) {
    const ods_layer_cfg &c = blk->layers[l].cfg;
    const int n = layer_ops(c);
    if (g < n) return OpRef{l, is_moe(c) ? kMoeOps[g] : kDenseOps[g]};
    g -= n;
  }
  return OpRef{-1, K_ATTN_NORM};
}

int layer_offset(const ods_block *blk, int layer) {
  int n = 0;
  for (int l = 0; l < layer; ++l) n += layer_ops(blk->layers[l].cfg);
  return n;
}

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

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

AttnPlan plan_for(const ods_layer_cfg &c, const ods_batch *b) {
  return attn_plan(b->batch, c.n_kv, c.head_dim, kv_map(c, b).cols, c.window, b->split_pages);
}

size_t layer_ws_bytes(const ods_layer &L, const ods_batch *b) {
  const ods_layer_cfg &c = L.cfg;
  const int B = b->batch;
  const bool t = tiled(L);
  size_t w = align_up(attn_ws_bytes(B, c.n_q, c.n_kv, c.head_dim, plan_for(c, b)));
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

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

bool trace_on() {
  const char *e = getenv("ODS_TRACE");
  return e && e[0] && e[0] != '0';
}

size_t range_ws_bytes(const ods_block *blk, int op_begin, int op_end, const ods_batch *batch) {
  size_t w = 0;
  for (int g = op_begin; g < op_end; ++g) w = std::max(w, layer_ws_bytes(blk->layers[op_at(blk, g).layer], batch));
  return w;
}

}  // namespace

// Workspace held by the library for callers that cannot allocate device
// memory (ods_run_partition_scratch). Each device the library runs on holds
// its own copy, zero-filled at load, until the process ends. In host code
// this name is a host-side stand-in, never a device address: the address is
// resolved per device with hipGetSymbolAddress and only that pointer is
// passed to kernels.
static __device__ __align__(256) uint8_t scratch[ODS_SCRATCH_BYTES];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of `scratch` on the current device, resolved on the first
// call per device (with that device current) and cached.
ods_status scratch_ptr(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(ODS_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(ODS_EUNSUPPORTED, "device %d: the library scratch supports device ids below %d", dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(ODS_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ODS_OK;
}

}  // namespace

extern "C" {

const char *ods_last_error(void) { return g_err; }

ods_status ods_kv_alloc(int64_t pool_pages, const int32_t *ctx_lens_host, int32_t batch, uint64_t seed,
                        int32_t max_pages, int32_t *page_table_host) {
  if (!ctx_lens_host || !page_table_host) return fail(ODS_EINVAL, "ods_kv_alloc: null pointer");
  if (batch < 0 || max_pages <= 0 || pool_pages <= 0)
    return fail(ODS_EINVAL, "ods_kv_alloc: batch %d, max_pages %d, pool_pages %lld", batch, max_pages,
                (long long)pool_pages);
  int64_t need = 0;
  for (int b = 0; b < batch; ++b) {
    if (ctx_lens_host[b] <= 0) return fail(ODS_EINVAL, "ods_kv_alloc: ctx_lens[%d] = %d", b, ctx_lens_host[b]);
    const int64_t n = ((int64_t)ctx_lens_host[b] + ODS_PAGE_TOKENS - 1) / ODS_PAGE_TOKENS;
    if (n > max_pages)
      return fail(ODS_ERANGE, "ods_kv_alloc: sequence %d needs %lld pages > max_pages %d", b, (long long)n,
                  max_pages);
    need += n;
  }
  if (need > pool_pages)
    return fail(ODS_ENOMEM, "ods_kv_alloc: batch needs %lld pages, pool has %lld", (long long)need,
                (long long)pool_pages);
  if (pool_pages > INT32_MAX) return fail(ODS_ERANGE, "ods_kv_alloc: pool_pages exceeds int32 page ids");
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
  g_err[0] = 0;
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

size_t ods_workspace_bytes(const ods_block *blk, const ods_batch *batch) {
  if (check_block(blk) != ODS_OK || !batch || batch->batch < 0 || batch->max_pages <= 0) return 0;
  size_t w = 256;
  for (int l = 0; l < blk->n_layers; ++l) w = std::max(w, layer_ws_bytes(blk->layers[l], batch));
  return w;
}

int32_t ods_block_num_ops(const ods_block *blk) {
  if (check_block(blk) != ODS_OK) return -1;
  return num_ops(blk);
}

const char *ods_op_name(const ods_block *blk, int32_t op) {
  if (check_block(blk) != ODS_OK || op < 0 || op >= num_ops(blk)) return nullptr;
  return kNames[op_at(blk, op).kind];
}

ods_status ods_run_partition(const ods_block *blk, int32_t op_begin, int32_t op_end, const ods_batch *batch,
                             ods_state *st, hipStream_t stream) {
  ods_status rc = check_block(blk);
  if (rc != ODS_OK) return rc;
  if (!batch || !st) return fail(ODS_EINVAL, "null batch or state");
  const int n_ops = num_ops(blk);
  if (op_begin < 0 || op_end > n_ops || op_begin >= op_end)
    return fail(ODS_ERANGE, "operator range [%d, %d) outside [0, %d) or empty", op_begin, op_end, n_ops);
  const int B = batch->batch;
  if (B < 0) return fail(ODS_EINVAL, "negative batch");
  if (batch->split_pages < 0) return fail(ODS_EINVAL, "negative split_pages");
  if (batch->ring_pages < 0) return fail(ODS_EINVAL, "negative ring_pages");
  if (B == 0) {  // nothing to read or write: the batch-sized pointers may be null
    g_err[0] = 0;
    return ODS_OK;
  }

  // ---- validation pass: every pointer an operator in the range touches ----
  std::vector<OpRef> ops;
  for (int g = op_begin; g < op_end; ++g) ops.push_back(op_at(blk, g));
  for (size_t i = 0; i < ops.size(); ++i) {
    const ods_layer &L = blk->layers[ops[i].layer];
    const ods_layer_cfg &c = L.cfg;
    const OpKind k = ops[i].kind;
    const bool fuse_next_silu = (i + 1 < ops.size()) && ops[i + 1].layer == ops[i].layer &&
                                ((k == K_GATE_UP && ops[i + 1].kind == K_SILU) ||
                                 (k == K_EXP_GATE_UP && ops[i + 1].kind == K_EXP_SILU));
    std::vector<std::pair<const void *, const char *>> need;
    bool paged = false;
    switch (k) {
      case K_ATTN_NORM: need = {{st->resid, "resid"}, {st->xn, "xn"}, {L.g_attn, "g_attn"}}; break;
      case K_QKV: need = {{st->xn, "xn"}, {st->qkv, "qkv"}, {L.w_qkv, "w_qkv"}}; break;
      case K_ROPE: need = {{st->qkv, "qkv"}, {batch->ctx_lens, "ctx_lens"}}; paged = true; break;
      case K_KV_APPEND:
      case K_ATTN_CORE:
        need = {{st->qkv, "qkv"}, {batch->ctx_lens, "ctx_lens"},
                {kv_map(c, batch).table, kv_map(c, batch).ring ? "ring_table" : "page_table"},
                {L.kv_pool, "kv_pool"}};
        if (k == K_ATTN_CORE) {
          need.push_back({st->o, "o"});
          need.push_back({st->ws, "ws"});
          if (B > kMaxAttnBatch)
            return fail(ODS_EUNSUPPORTED, "layer %d: attn_core supports batch <= %d, got %d", ops[i].layer,
                        kMaxAttnBatch, B);
          if (!plan_for(c, batch).units_ok)
            return fail(ODS_EUNSUPPORTED, "layer %d: batch * n_kv * window pages exceeds 2^30", ops[i].layer);
        }
        paged = true;
        break;
      case K_O_PROJ: need = {{st->o, "o"}, {st->resid, "resid"}, {L.w_o, "w_o"}}; break;
      case K_FFN_NORM: need = {{st->resid, "resid"}, {st->hn, "hn"}, {L.g_ffn, "g_ffn"}}; break;
      case K_GATE_UP:
        need = {{st->hn, "hn"}, {L.w_gate_up, "w_gate_up"}};
        need.push_back(fuse_next_silu ? std::make_pair((const void *)st->act, "act")
                                      : std::make_pair((const void *)st->gu, "gu"));
        break;
      case K_SILU: need = {{st->gu, "gu"}, {st->act, "act"}}; break;
      case K_DOWN: need = {{st->act, "act"}, {st->resid, "resid"}, {L.w_down, "w_down"}}; break;
      case K_ROUTER: need = {{st->hn, "hn"}, {L.w_router, "w_router"}, {st->logits, "logits"}}; break;
      case K_TOPK: need = {{st->logits, "logits"}, {st->topk_ids, "topk_ids"}, {st->topk_w, "topk_w"}}; break;
      case K_PERMUTE:
        need = {{st->topk_ids, "topk_ids"}, {st->hn, "hn"}, {st->perm, "perm"}, {st->slot_pos, "slot_pos"},
                {st->expert_off, "expert_off"}, {st->xp, "xp"}};
        break;
      case K_EXP_GATE_UP:
        need = {{st->xp, "xp"}, {st->expert_off, "expert_off"}, {L.w_gate_up, "w_gate_up"}};
        need.push_back(fuse_next_silu ? std::make_pair((const void *)st->act_p, "act_p")
                                      : std::make_pair((const void *)st->gu_p, "gu_p"));
        break;
      case K_EXP_SILU: need = {{st->gu_p, "gu_p"}, {st->act_p, "act_p"}}; break;
      case K_EXP_DOWN:
        need = {{st->act_p, "act_p"}, {st->expert_off, "expert_off"}, {L.w_down, "w_down"}, {st->yp, "yp"}};
        break;
      case K_COMBINE:
        need = {{st->yp, "yp"}, {st->topk_w, "topk_w"}, {st->slot_pos, "slot_pos"}, {st->resid, "resid"}};
        break;
    }
    for (auto &pn : need) {
      if (!pn.first) return fail(ODS_EINVAL, "op %s (layer %d): %s is null", kNames[k], ops[i].layer, pn.second);
      if (!aligned16(pn.first))
        return fail(ODS_EINVAL, "op %s (layer %d): %s is not 16-byte aligned", kNames[k], ops[i].layer, pn.second);
    }
    if (paged) {
      if (batch->max_pages <= 0) return fail(ODS_EINVAL, "max_pages must be positive");
      if ((int64_t)batch->max_pages * ODS_PAGE_TOKENS > INT32_MAX) return fail(ODS_ERANGE, "max_pages too large");
      if (k != K_ROPE && L.pool_pages <= 0) return fail(ODS_EINVAL, "layer %d: pool_pages <= 0", ops[i].layer);
      const KvMap m = kv_map(c, batch);
      if (m.ring > 0) {
        const int64_t need_pages = ((int64_t)c.window + ODS_PAGE_TOKENS - 1) / ODS_PAGE_TOKENS + 1;
        if (m.ring < need_pages)
          return fail(ODS_EINVAL, "layer %d: ring_pages %d < ceil(window / 16) + 1 = %lld", ops[i].layer, m.ring,
                      (long long)need_pages);
      }
    }
    if (is_moe(c) && (int64_t)B * c.top_k > INT32_MAX / 2) return fail(ODS_ERANGE, "batch * top_k too large");
  }
  const size_t ws_need = range_ws_bytes(blk, op_begin, op_end, batch);
  bool uses_ws = false;
  for (auto &o : ops)
    if (o.kind == K_ATTN_CORE || o.kind == K_QKV || o.kind == K_O_PROJ || o.kind == K_GATE_UP ||
        o.kind == K_DOWN || o.kind == K_ROUTER)
      uses_ws = true;
  if (uses_ws) {
    if (!st->ws) return fail(ODS_EINVAL, "ws is null");
    if (st->ws_bytes < ws_need)
      return fail(ODS_ENOMEM, "workspace %zu bytes < required %zu", st->ws_bytes, ws_need);
  }
  // ---- dispatch ----
  const bool trace = trace_on();
  auto U = [](const void *p) { return (uint16_t *)p; };
  for (size_t i = 0; i < ops.size(); ++i) {
    const ods_layer &L = blk->layers[ops[i].layer];
    const ods_layer_cfg &c = L.cfg;
    const OpKind k = ops[i].kind;
    const bool next_same_layer = i + 1 < ops.size() && ops[i + 1].layer == ops[i].layer;
    const int H = c.hidden, D = c.head_dim;
    hipError_t e = hipSuccess;
    const char *what = kNames[k];
    GemmArgs ga{};
    const bool wt = tiled(L);  // projection weights in tile order (the router never is)
    auto dense_gemm = [&](const void *A, const void *Bw, void *C, int N, int K, int epi, int n_up, int ldc,
                          bool defer_reduce = false, bool b_tiled = false) {
      ga.A = (const uint16_t *)A; ga.lda = K;
      ga.B = (const uint16_t *)Bw; ga.ldb = K; ga.b_group_stride = 0;
      ga.C = C; ga.ldc = ldc;
      ga.M = B; ga.N = N; ga.K = K; ga.n_up = n_up; ga.epi = epi;
      ga.group_off = nullptr; ga.groups = 0;
      ga.b_tiled = b_tiled ? 1 : 0;
      ga.splits = gemm_splits(B, N, K, epi, b_tiled);
      ga.partial = (float *)st->ws;
      ga.defer_reduce = defer_reduce ? 1 : 0;
      return launch_gemm(ga, stream);
    };
    switch (k) {
      case K_ATTN_NORM: e = launch_rmsnorm(U(st->resid), U(L.g_attn), U(st->xn), B, H, c.rms_eps, stream); break;
      case K_FFN_NORM: e = launch_rmsnorm(U(st->resid), U(L.g_ffn), U(st->hn), B, H, c.rms_eps, stream); break;
      case K_QKV: {
        // With split-K and RoPE next in the range, the RoPE / KV-append kernel
        // sums the partials itself (same order and rounding as the reduce).
        const bool fuse =
            next_same_layer && ops[i + 1].kind == K_ROPE && gemm_splits(B, qkv_dim(c), H, EPI_BF16, wt) > 1;
        e = dense_gemm(st->xn, L.w_qkv, st->qkv, qkv_dim(c), H, EPI_BF16, 0, qkv_dim(c), fuse, wt);
        if (fuse && e == hipSuccess) {
          const bool app = i + 2 < ops.size() && ops[i + 2].layer == ops[i].layer && ops[i + 2].kind == K_KV_APPEND;
          const KvMap m = kv_map(c, batch);
          e = launch_rope_append(U(st->qkv), B, c.n_q, c.n_kv, D, c.rope_theta, batch->ctx_lens, m.table, m.cols,
                                 m.ring, U(L.kv_pool), L.pool_pages, true, app, stream, (const float *)st->ws,
                                 ga.splits);
          what = app ? "qkv_proj+rope+kv_append" : "qkv_proj+rope";
          i += app ? 2 : 1;
        }
        break;
      }
      case K_ROPE:
      case K_KV_APPEND: {
        const bool both = k == K_ROPE && next_same_layer && ops[i + 1].kind == K_KV_APPEND;
        const KvMap m = kv_map(c, batch);
        e = launch_rope_append(U(st->qkv), B, c.n_q, c.n_kv, D, c.rope_theta, batch->ctx_lens, m.table, m.cols,
                               m.ring, U(L.kv_pool), L.pool_pages, k == K_ROPE, both || k == K_KV_APPEND, stream);
        if (both) {
          what = "rope+kv_append";
          ++i;
        }
        break;
      }
      case K_ATTN_CORE:
      {
        const KvMap m = kv_map(c, batch);
        e = launch_attention(U(st->qkv), B, c.n_q, c.n_kv, D, c.window, batch->ctx_lens, m.table, m.cols, m.ring,
                             U(L.kv_pool), L.pool_pages, plan_for(c, batch), (float *)st->ws, U(st->o), stream);
        break;
      }
      case K_O_PROJ: e = dense_gemm(st->o, L.w_o, st->resid, H, c.n_q * D, EPI_RESID, 0, H, false, wt); break;
      case K_GATE_UP:
        if (next_same_layer && ops[i + 1].kind == K_SILU) {
          e = dense_gemm(st->hn, L.w_gate_up, st->act, c.ffn, H, EPI_SILU, c.ffn, c.ffn, false, wt);
          what = "gate_up+silu_mul";
          ++i;
        } else {
          // tiled gate_up pairs gate and up rows per tile: n_up tells the plain epilogue where the up half goes
          e = dense_gemm(st->hn, L.w_gate_up, st->gu, 2 * c.ffn, H, EPI_BF16, wt ? c.ffn : 0, 2 * c.ffn, false, wt);
        }
        break;
      case K_SILU: e = launch_silu_mul(U(st->gu), U(st->act), B, c.ffn, stream); break;
      case K_DOWN: e = dense_gemm(st->act, L.w_down, st->resid, H, c.ffn, EPI_RESID, 0, H, false, wt); break;
      case K_ROUTER: e = dense_gemm(st->hn, L.w_router, st->logits, c.n_experts, H, EPI_F32, 0, c.n_experts); break;
      case K_TOPK: e = launch_topk(st->logits, B, c.n_experts, c.top_k, st->topk_ids, st->topk_w, stream); break;
      case K_PERMUTE:
        e = launch_permute(st->topk_ids, B, c.top_k, c.n_experts, st->perm, st->slot_pos, st->expert_off, stream);
        if (e == hipSuccess)
          e = launch_gather_rows(U(st->hn), st->perm, st->expert_off + c.n_experts, B * c.top_k, c.top_k, H,
                                 U(st->xp), stream);
        break;
      case K_EXP_GATE_UP:
      case K_EXP_DOWN: {
        const bool fuse = k == K_EXP_GATE_UP && next_same_layer && ops[i + 1].kind == K_EXP_SILU;
        const int I = c.moe_ffn;
        const int rows = B * c.top_k;
        ga.M = rows;
        ga.group_off = st->expert_off;
        ga.groups = c.n_experts;
        ga.splits = 1;
        ga.partial = nullptr;
        ga.b_tiled = wt ? 1 : 0;
        if (k == K_EXP_GATE_UP) {
          ga.A = U(st->xp); ga.lda = H; ga.K = H;
          ga.B = U(L.w_gate_up); ga.ldb = H;
          ga.b_group_stride = wt ? tiled_weight_elems(I, H, true, 1) : (int64_t)2 * I * H;
          if (fuse) {
            ga.C = st->act_p; ga.ldc = I; ga.N = I; ga.n_up = I; ga.epi = EPI_SILU;
            what = "expert_gate_up+silu_mul";
            ++i;
          } else {
            ga.C = st->gu_p; ga.ldc = 2 * I; ga.N = 2 * I; ga.n_up = wt ? I : 0; ga.epi = EPI_BF16;
          }
        } else {
          ga.A = U(st->act_p); ga.lda = I; ga.K = I;
          ga.B = U(L.w_down); ga.ldb = I;
          ga.b_group_stride = wt ? tiled_weight_elems(H, I, false, 1) : (int64_t)H * I;
          ga.C = st->yp; ga.ldc = H; ga.N = H; ga.n_up = 0; ga.epi = EPI_BF16;
        }
        e = launch_gemm(ga, stream);
        break;
      }
      case K_EXP_SILU: e = launch_silu_mul(U(st->gu_p), U(st->act_p), B * c.top_k, c.moe_ffn, stream); break;
      case K_COMBINE:
        e = launch_moe_combine(U(st->yp), st->topk_w, st->slot_pos, B, c.top_k, H, U(st->resid), stream);
        break;
    }
    if (trace) fprintf(stderr, "[ods] layer %d %s B=%d -> %s\n", ops[i].layer, what, B, hipGetErrorString(e));
    if (e != hipSuccess) return fail(ODS_EHIP, "launch of %s (layer %d) failed: %s", what, ops[i].layer,
                                     hipGetErrorString(e));
  }
  g_err[0] = 0;
  return ODS_OK;
}

ods_status ods_run_partition_scratch(const ods_block *blk, int32_t op_begin, int32_t op_end,
                                     const ods_batch *batch, ods_state *state, hipStream_t stream) {
  ods_status rc = check_block(blk);
  if (rc != ODS_OK) return rc;
  if (!batch || !state) return fail(ODS_EINVAL, "null batch or state");
  const int n_ops = num_ops(blk);
  if (op_begin < 0 || op_end > n_ops || op_begin >= op_end)
    return fail(ODS_ERANGE, "operator range [%d, %d) outside [0, %d) or empty", op_begin, op_end, n_ops);
  if (batch->batch < 0 || batch->split_pages < 0 || batch->ring_pages < 0)
    return fail(ODS_EINVAL, "negative batch, split_pages or ring_pages");
  ods_state st = *state;
  st.ws = nullptr;
  st.ws_bytes = 0;
  if (batch->batch == 0) return ods_run_partition(blk, op_begin, op_end, batch, &st, stream);
  const size_t need = range_ws_bytes(blk, op_begin, op_end, batch);
  if (need > ODS_SCRATCH_BYTES)
    return fail(ODS_ENOMEM, "operators [%d, %d) need %zu bytes of workspace; the library scratch holds %zu",
                op_begin, op_end, need, (size_t)ODS_SCRATCH_BYTES);
  rc = scratch_ptr(&st.ws);
  if (rc != ODS_OK) return rc;
  st.ws_bytes = ODS_SCRATCH_BYTES;
  return ods_run_partition(blk, op_begin, op_end, batch, &st, stream);
}

size_t ods_tiled_weight_bytes(int32_t out, int32_t in, int32_t gated, int32_t groups) {
  if (out < 1 || in < 64 || in % 64 != 0 || groups < 1 || (gated != 0 && gated != 1)) return 0;
  return (size_t)tiled_weight_elems(out, in, gated != 0, groups) * 2;
}

ods_status ods_tile_weight(const void *src, void *dst, int32_t out, int32_t in, int32_t gated, int32_t groups,
                           hipStream_t stream) {
  const size_t bytes = ods_tiled_weight_bytes(out, in, gated, groups);
  if (!bytes) return fail(ODS_EINVAL, "ods_tile_weight: out %d, in %d, gated %d, groups %d", out, in, gated, groups);
  if (!src || !dst) return fail(ODS_EINVAL, "ods_tile_weight: null pointer");
  if (!aligned16(src) || !aligned16(dst)) return fail(ODS_EINVAL, "ods_tile_weight: pointers must be 16-byte aligned");
  const size_t src_bytes = (size_t)groups * (gated ? 2 : 1) * out * in * 2;
  const uintptr_t s0 = (uintptr_t)src, d0 = (uintptr_t)dst;
  if (s0 < d0 + bytes && d0 < s0 + src_bytes) return fail(ODS_EINVAL, "ods_tile_weight: src and dst overlap");
  const hipError_t e = launch_tile_weight((const uint16_t *)src, (uint16_t *)dst, out, in, gated != 0, groups, stream);
  if (e != hipSuccess) return fail(ODS_EHIP, "ods_tile_weight: %s", hipGetErrorString(e));
  g_err[0] = 0;
  return ODS_OK;
}

ods_status ods_attn_stage(const ods_block *blk, int32_t layer, const ods_batch *batch, ods_state *state,
                          hipStream_t stream) {
  ods_status rc = check_block(blk);
  if (rc != ODS_OK) return rc;
  if (layer < 0 || layer >= blk->n_layers) return fail(ODS_ERANGE, "layer %d outside [0, %d)", layer, blk->n_layers);
  const int off = layer_offset(blk, layer);
  return ods_run_partition(blk, off, off + 6, batch, state, stream);
}

ods_status ods_ffn_stage(const ods_block *blk, int32_t layer, const ods_batch *batch, ods_state *state,
                         hipStream_t stream) {
  ods_status rc = check_block(blk);
  if (rc != ODS_OK) return rc;
  if (layer < 0 || layer >= blk->n_layers) return fail(ODS_ERANGE, "layer %d outside [0, %d)", layer, blk->n_layers);
  const int off = layer_offset(blk, layer);
  return ods_run_partition(blk, off + 6, off + layer_ops(blk->layers[layer].cfg), batch, state, stream);
}

ods_status ods_partition_graph(const ods_block *blk, int32_t op_begin, int32_t op_end, const ods_batch *batch,
                               ods_state *state, hipGraphExec_t *exec) {
  if (!exec) return fail(ODS_EINVAL, "exec is null");
  *exec = nullptr;
  hipStream_t s = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
  if (e != hipSuccess) return fail(ODS_EHIP, "hipStreamCreate: %s", hipGetErrorString(e));
  e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) {
    hipStreamDestroy(s);
    return fail(ODS_EHIP, "hipStreamBeginCapture: %s", hipGetErrorString(e));
  }
  const ods_status rc = ods_run_partition(blk, op_begin, op_end, batch, state, s);
  std::string msg = rc == ODS_OK ? "" : g_err;
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(s, &graph);
  hipStreamDestroy(s);
  if (rc != ODS_OK) {
    if (graph) hipGraphDestroy(graph);
    return fail(rc, "%s", msg.c_str());
  }
  if (e != hipSuccess || !graph) return fail(ODS_EHIP, "hipStreamEndCapture: %s", hipGetErrorString(e));
  e = hipGraphInstantiate(exec, graph, nullptr, nullptr, 0);
  hipGraphDestroy(graph);
  if (e != hipSuccess) {
    *exec = nullptr;
    return fail(ODS_EHIP, "hipGraphInstantiate: %s", hipGetErrorString(e));
  }
  g_err[0] = 0;
  return ODS_OK;
}

ods_status ods_graph_launch(hipGraphExec_t exec, hipStream_t stream) {
  if (!exec) return fail(ODS_EINVAL, "exec is null");
  const hipError_t e = hipGraphLaunch(exec, stream);
  if (e != hipSuccess) return fail(ODS_EHIP, "hipGraphLaunch: %s", hipGetErrorString(e));
  g_err[0] = 0;
  return ODS_OK;
}

ods_status ods_graph_destroy(hipGraphExec_t exec) {
  if (!exec) return ODS_OK;
  const hipError_t e = hipGraphExecDestroy(exec);
  if (e != hipSuccess) return fail(ODS_EHIP, "hipGraphExecDestroy: %s", hipGetErrorString(e));
  g_err[0] = 0;
  return ODS_OK;
}

}  // extern "C"
