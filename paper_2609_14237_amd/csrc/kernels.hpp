// Internal launch interface between the host dispatcher and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ods {

enum Epilogue : int {
  EPI_BF16 = 0,   // C = bf16(acc)
  EPI_F32 = 1,    // C = acc (fp32 output)
  EPI_RESID = 2,  // C = bf16(C + acc), C is the residual stream (in place)
  EPI_SILU = 3,   // C[:, n] = bf16(silu(acc_gate) * acc_up), B rows n (gate) and n_up + n (up)
};

// C[m, n] = sum_k A[m, k] * B[n, k] with an epilogue. A, B, C row-major.
struct GemmArgs {
  const uint16_t *A; int64_t lda;
  const uint16_t *B; int64_t ldb; int64_t b_group_stride;
  void *C; int64_t ldc;
  int M, N, K;
  int n_up;                   // EPI_SILU: row offset of the "up" half inside B
  int epi;
  const int32_t *group_off;   // grouped GEMM: rows [off[g], off[g+1]) use B + g * b_group_stride
  int groups;
  int splits;                 // split-K count (>1: fp32 partials in `partial`, then a reduce)
  float *partial;
  int defer_reduce;           // splits > 1: leave the partials for a consumer that sums them itself
  int b_tiled;                // B in the streaming kernel's tile order (tile_weight); with n_up > 0
                              // the tiles pair gate and up rows, whatever the epilogue
};

// Tile order of a weight for the streaming GEMM: for each group, N tile and
// 64-wide K step, the 16 KB image of that step's 128 B rows in LDS (row r at
// r * 128 bytes, 16-byte chunk c of the row at position c ^ (r % 8)). Plain
// weights put rows 128 nt .. +127 in N tile nt; gated (gate rows, then up
// rows, `out` of each) put gate rows 64 nt .. +63 then the matching up rows.
// Rows past `out` are zero. `in` must be a multiple of 64.
int64_t tiled_weight_elems(int out, int in, bool gated, int groups);
hipError_t launch_tile_weight(const uint16_t *src, uint16_t *dst, int out, int in, bool gated, int groups,
                              hipStream_t s);

// Compute units of the current device (queried once per process and device).
int num_cus();

// Split-K plan for a dense GEMM (shared by sizing and launching).
int gemm_splits(int M, int N, int K, int epi, bool b_tiled = false);
size_t gemm_partial_bytes(int M, int N, int K, int epi, bool b_tiled = false);
hipError_t launch_gemm(const GemmArgs &a, hipStream_t s);
// Sum of split-K partials plus the epilogue (after a partial-writing launch).
hipError_t launch_splitk_reduce(const GemmArgs &a, hipStream_t s);
// Weight-streaming kernel (K % 64 == 0): dense GEMMs past 128 rows, of 33 to
// 64 rows but the SiLU-gated one, grouped GEMMs, and every GEMM on tiled weights.
bool gemm_use_stream(int M, int N, int K, int epi);
int gemm_stream_splits(int M, int N, int K, int epi);
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
constexpr int kMaxAttnBatch = 4096;  // the kernel keeps per-sequence contexts and a prefix in LDS
struct AttnPlan {
  int seg_pages;    // pages per wave range; 0: total / waves (at least 8)
  int grid;         // workgroups of the attention kernel
  int64_t records;  // partial-record slots per query-head group
  bool units_ok;    // batch * n_kv * span fits the kernel's 32-bit unit index
};
AttnPlan attn_plan(int B, int n_kv, int D, int max_pages, int window, int split_pages_req);
size_t attn_ws_bytes(int B, int n_q, int n_kv, int D, const AttnPlan &plan);
hipError_t launch_attention(const uint16_t *qkv, int B, int n_q, int n_kv, int D, int window,
                            const int32_t *ctx_lens, const int32_t *page_table, int max_pages, int ring,
                            const uint16_t *pool, int64_t pool_pages, const AttnPlan &plan,
                            float *ws, uint16_t *o, hipStream_t s);

hipError_t launch_silu_mul(const uint16_t *gu, uint16_t *act, int rows, int F, hipStream_t s);

hipError_t launch_topk(const float *logits, int B, int E, int k, int32_t *ids, float *w, hipStream_t s);
hipError_t launch_permute(const int32_t *ids, int B, int k, int E, int32_t *perm, int32_t *slot_pos,
                          int32_t *expert_off, hipStream_t s);
hipError_t launch_gather_rows(const uint16_t *src, const int32_t *perm, const int32_t *valid_rows,
                              int rows, int k, int H, uint16_t *dst, hipStream_t s);
hipError_t launch_moe_combine(const uint16_t *yp, const float *w, const int32_t *slot_pos, int B,
                              int k, int H, uint16_t *resid, hipStream_t s);

}  // namespace ods
