// Internal launch interface between the host dispatcher and the gfx950 kernels.
// The launch-shape choices themselves (split-K counts, tiles, the attention
// work split) live in plan.hpp, free of HIP.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.hpp"

namespace ods {

hipError_t launch_tile_weight(const uint16_t *src, uint16_t *dst, int out, int in, bool gated, int groups,
                              hipStream_t s);

// Compute units of the current device (queried once per process and device).
int num_cus();

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s);
// Sum of split-K partials plus the epilogue (after a partial-writing launch).
hipError_t launch_splitk_reduce(const GemmArgs &a, hipStream_t s);
// Weight-streaming kernel (K % 64 == 0): dense GEMMs past 128 rows, of 33 to
// 64 rows but the SiLU-gated one, grouped GEMMs, and every GEMM on tiled weights.
hipError_t launch_gemm_stream(const GemmArgs &a, hipStream_t s);

hipError_t launch_rmsnorm(const uint16_t *x, const uint16_t *gain, uint16_t *out, int rows, int H,
                          float eps, hipStream_t s);

// In-place RoPE of the q and k heads of qkv and/or append of k, v to the KV pool.
// With splits > 1, each qkv row is first summed from the `splits` fp32 split-K
// partials [splits][B][qkv width] (the same order and bf16 rounding as the
// split-K reduce), so a qkv projection can hand its partials straight over.
// ring > 0: page_table is a [B][ring] window-only page ring (logical page lp in
// column lp % ring, contexts not clamped); max_pages is then ring.
hipError_t launch_rope_append(uint16_t *qkv, int B, int n_q, int n_kv, int D, float theta,
                              const int32_t *ctx_lens, const int32_t *page_table, int max_pages, int ring,
                              uint16_t *pool, int64_t pool_pages, bool do_rope, bool do_append,
                              hipStream_t s, const float *partial = nullptr, int splits = 1);

// Paged GQA decode attention (the batch's pages split evenly over the waves)
// + exact log-sum-exp merge of sequences that span several waves.
hipError_t launch_attention(const uint16_t *qkv, int B, int n_q, int n_kv, int D, int window,
                            const int32_t *ctx_lens, const int32_t *page_table, int max_pages, int ring,
                            const uint16_t *pool, int64_t pool_pages, const AttnPlan &plan,
                            float *ws, uint16_t *o, hipStream_t s);

hipError_t launch_silu_mul(const uint16_t *gu, uint16_t *act, int rows, int F, hipStream_t s);

// Top-k routing of fp32 logits. With splits > 1 the logits are first summed
// from the router's split-K partials [splits][B][E] (the split-K reduce's
// order) and written to logits_out.
hipError_t launch_topk(const float *logits, int B, int E, int k, int32_t *ids, float *w, hipStream_t s,
                       const float *partial = nullptr, int splits = 1, float *logits_out = nullptr);
hipError_t launch_permute(const int32_t *ids, int B, int k, int E, int32_t *perm, int32_t *slot_pos,
                          int32_t *expert_off, hipStream_t s);
hipError_t launch_gather_rows(const uint16_t *src, const int32_t *perm, const int32_t *valid_rows,
                              int rows, int k, int H, uint16_t *dst, hipStream_t s);
hipError_t launch_moe_combine(const uint16_t *yp, const float *w, const int32_t *slot_pos, int B,
                              int k, int H, uint16_t *resid, hipStream_t s);

}  // namespace ods
