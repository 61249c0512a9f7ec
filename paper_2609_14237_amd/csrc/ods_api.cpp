// HIP side of the ODS decode library: the operator-range dispatcher that
// enqueues the launches ods_host.cpp plans for a stage [op_begin, op_end) of a
// partition block on one stream (one native submission per stage, no
// allocation, no synchronisation), graph capture of a stage, the on-device
// weight tiling, and the library-held workspace of the scratch entry point.
// Validation, sizing, the allocator and every launch-shape choice are in the
// HIP-free ods_host.cpp.
#include <stdlib.h>
#include <stdio.h>

#include <mutex>
#include <string>

#include "../../include/ods.h"
#include "kernels.hpp"

using namespace ods;

namespace {

bool trace_on() {
  const char *e = getenv("ODS_TRACE");
  return e && e[0] && e[0] != '0';
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

hipError_t execute(const Launch &L, hipStream_t s) {
  switch (L.kind) {
    case LK_RMSNORM: return launch_rmsnorm(L.x, L.gain, L.out, L.rows, L.width, L.eps, s);
    case LK_GEMM: return launch_gemm(L.gemm, s);
    case LK_QKV_ROPE:
    case LK_ROPE_APPEND: {
      if (L.kind == LK_QKV_ROPE) {
        const hipError_t e = launch_gemm(L.gemm, s);
        if (e != hipSuccess) return e;
      }
      const RopeArgs &r = L.rope;
      return launch_rope_append(r.qkv, r.B, r.n_q, r.n_kv, r.D, r.theta, r.ctx_lens, r.table, r.cols, r.ring, r.pool,
                                r.pool_pages, r.do_rope, r.do_append, s, r.partial, r.splits);
    }
    case LK_ATTENTION: {
      const AttnArgs &a = L.attn;
      return launch_attention(a.qkv, a.B, a.n_q, a.n_kv, a.D, a.window, a.ctx_lens, a.table, a.cols, a.ring, a.pool,
                              a.pool_pages, a.plan, a.ws, a.o, s);
    }
    case LK_SILU: return launch_silu_mul(L.x, L.out, L.rows, L.width, s);
    case LK_TOPK: return launch_topk(L.logits, L.rows, L.E, L.k, L.ids, L.weights, s);
    case LK_ROUTER_TOPK: {
      const hipError_t e = launch_gemm(L.gemm, s);
      if (e != hipSuccess) return e;
      return launch_topk(nullptr, L.rows, L.E, L.k, L.ids, L.weights, s, L.topk_partial, L.topk_splits, L.logits_out);
    }
    case LK_PERMUTE: {
      const hipError_t e = launch_permute(L.ids, L.rows, L.k, L.E, L.perm, L.slot_pos, L.expert_off, s);
      if (e != hipSuccess || !L.xp) return e;  // no xp: the expert GEMM that follows gathers its rows
      return launch_gather_rows(L.x, L.perm, L.expert_off + L.E, L.rows * L.k, L.k, L.width, L.xp, s);
    }
    case LK_COMBINE: return launch_moe_combine(L.x, L.weights, L.slot_pos, L.rows, L.k, L.width, L.out, s);
  }
  return hipErrorInvalidValue;
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
  if (e != hipSuccess) return set_error(ODS_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices)
    return set_error(ODS_EUNSUPPORTED, "device %d: the library scratch supports device ids below %d", dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(ODS_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ODS_OK;
}

}  // namespace

extern "C" {

size_t ods_workspace_bytes(const ods_block *blk, const ods_batch *batch) {
  if (check_block(blk) != ODS_OK || !batch || batch->batch < 0 || batch->max_pages <= 0) return 0;
  return block_ws_bytes(blk, batch, num_cus());
}

ods_status ods_run_partition(const ods_block *blk, int32_t op_begin, int32_t op_end, const ods_batch *batch,
                             ods_state *st, hipStream_t stream) {
  const int cus = num_cus();
  const ods_status rc = validate_range(blk, op_begin, op_end, batch, st, cus);
  if (rc != ODS_OK) return rc;
  if (batch->batch == 0) {
    clear_error();
    return ODS_OK;
  }
  const bool trace = trace_on();
  for (int i = 0; i < op_end - op_begin;) {
    Launch L;
    plan_launch(blk, op_begin, op_end, i, batch, st, cus, &L);
    const hipError_t e = execute(L, stream);
    if (trace) fprintf(stderr, "[ods] layer %d %s B=%d -> %s\n", L.layer, L.what, batch->batch, hipGetErrorString(e));
    if (e != hipSuccess)
      return set_error(ODS_EHIP, "launch of %s (layer %d) failed: %s", L.what, L.layer, hipGetErrorString(e));
    i += L.n_ops;
  }
  clear_error();
  return ODS_OK;
}

ods_status ods_run_partition_scratch(const ods_block *blk, int32_t op_begin, int32_t op_end,
                                     const ods_batch *batch, ods_state *state, hipStream_t stream) {
  ods_status rc = check_block(blk);
  if (rc != ODS_OK) return rc;
  if (!batch || !state) return set_error(ODS_EINVAL, "null batch or state");
  const int n_ops = num_ops(blk);
  if (op_begin < 0 || op_end > n_ops || op_begin >= op_end)
    return set_error(ODS_ERANGE, "operator range [%d, %d) outside [0, %d) or empty", op_begin, op_end, n_ops);
  if (batch->batch < 0 || batch->split_pages < 0 || batch->ring_pages < 0)
    return set_error(ODS_EINVAL, "negative batch, split_pages or ring_pages");
  ods_state st = *state;
  st.ws = nullptr;
  st.ws_bytes = 0;
  if (batch->batch == 0) return ods_run_partition(blk, op_begin, op_end, batch, &st, stream);
  const size_t need = range_ws_bytes(blk, op_begin, op_end, batch, num_cus());
  if (need > ODS_SCRATCH_BYTES)
    return set_error(ODS_ENOMEM, "operators [%d, %d) need %zu bytes of workspace; the library scratch holds %zu",
                     op_begin, op_end, need, (size_t)ODS_SCRATCH_BYTES);
  rc = scratch_ptr(&st.ws);
  if (rc != ODS_OK) return rc;
  st.ws_bytes = ODS_SCRATCH_BYTES;
  return ods_run_partition(blk, op_begin, op_end, batch, &st, stream);
}

ods_status ods_tile_weight(const void *src, void *dst, int32_t out, int32_t in, int32_t gated, int32_t groups,
                           hipStream_t stream) {
  const size_t bytes = ods_tiled_weight_bytes(out, in, gated, groups);
  if (!bytes) return set_error(ODS_EINVAL, "ods_tile_weight: out %d, in %d, gated %d, groups %d", out, in, gated, groups);
  if (!src || !dst) return set_error(ODS_EINVAL, "ods_tile_weight: null pointer");
  if (!aligned16(src) || !aligned16(dst)) return set_error(ODS_EINVAL, "ods_tile_weight: pointers must be 16-byte aligned");
  const size_t src_bytes = (size_t)groups * (gated ? 2 : 1) * out * in * 2;
  const uintptr_t s0 = (uintptr_t)src, d0 = (uintptr_t)dst;
  if (s0 < d0 + bytes && d0 < s0 + src_bytes) return set_error(ODS_EINVAL, "ods_tile_weight: src and dst overlap");
  const hipError_t e = launch_tile_weight((const uint16_t *)src, (uint16_t *)dst, out, in, gated != 0, groups, stream);
  if (e != hipSuccess) return set_error(ODS_EHIP, "ods_tile_weight: %s", hipGetErrorString(e));
  clear_error();
  return ODS_OK;
}

ods_status ods_attn_stage(const ods_block *blk, int32_t layer, const ods_batch *batch, ods_state *state,
                          hipStream_t stream) {
  ods_status rc = check_block(blk);
  if (rc != ODS_OK) return rc;
  if (layer < 0 || layer >= blk->n_layers) return set_error(ODS_ERANGE, "layer %d outside [0, %d)", layer, blk->n_layers);
  const int off = layer_offset(blk, layer);
  return ods_run_partition(blk, off, off + 6, batch, state, stream);
}

ods_status ods_ffn_stage(const ods_block *blk, int32_t layer, const ods_batch *batch, ods_state *state,
                         hipStream_t stream) {
  ods_status rc = check_block(blk);
  if (rc != ODS_OK) return rc;
  if (layer < 0 || layer >= blk->n_layers) return set_error(ODS_ERANGE, "layer %d outside [0, %d)", layer, blk->n_layers);
  const int off = layer_offset(blk, layer);
  return ods_run_partition(blk, off + 6, off + layer_num_ops(blk->layers[layer].cfg), batch, state, stream);
}

ods_status ods_partition_graph(const ods_block *blk, int32_t op_begin, int32_t op_end, const ods_batch *batch,
                               ods_state *state, hipGraphExec_t *exec) {
  if (!exec) return set_error(ODS_EINVAL, "exec is null");
  *exec = nullptr;
  hipStream_t s = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
  if (e != hipSuccess) return set_error(ODS_EHIP, "hipStreamCreate: %s", hipGetErrorString(e));
  e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) {
    hipStreamDestroy(s);
    return set_error(ODS_EHIP, "hipStreamBeginCapture: %s", hipGetErrorString(e));
  }
  const ods_status rc = ods_run_partition(blk, op_begin, op_end, batch, state, s);
  std::string msg = rc == ODS_OK ? "" : error_text();
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(s, &graph);
  hipStreamDestroy(s);
  if (rc != ODS_OK) {
    if (graph) hipGraphDestroy(graph);
    return set_error(rc, "%s", msg.c_str());
  }
  if (e != hipSuccess || !graph) return set_error(ODS_EHIP, "hipStreamEndCapture: %s", hipGetErrorString(e));
  e = hipGraphInstantiate(exec, graph, nullptr, nullptr, 0);
  hipGraphDestroy(graph);
  if (e != hipSuccess) {
    *exec = nullptr;
    return set_error(ODS_EHIP, "hipGraphInstantiate: %s", hipGetErrorString(e));
  }
  clear_error();
  return ODS_OK;
}

ods_status ods_graph_launch(hipGraphExec_t exec, hipStream_t stream) {
  if (!exec) return set_error(ODS_EINVAL, "exec is null");
  const hipError_t e = hipGraphLaunch(exec, stream);
  if (e != hipSuccess) return set_error(ODS_EHIP, "hipGraphLaunch: %s", hipGetErrorString(e));
  clear_error();
  return ODS_OK;
}

ods_status ods_graph_destroy(hipGraphExec_t exec) {
  if (!exec) return ODS_OK;
  const hipError_t e = hipGraphExecDestroy(exec);
  if (e != hipSuccess) return set_error(ODS_EHIP, "hipGraphExecDestroy: %s", hipGetErrorString(e));
  clear_error();
  return ODS_OK;
}

}  // extern "C"
