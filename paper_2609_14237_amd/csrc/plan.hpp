// Host-side planning of the ODS decode library, free of HIP: operator tables,
// argument validation, the KV page allocator, buffer and workspace sizing,
// the kernels' launch-shape choices (split-K counts, tile shapes, the
// attention work split), and the planner that turns one position of an
// operator range into one launch description. ods_host.cpp implements it as
// plain C++ (it builds with a host compiler alone, so it can run under the
// CPU sanitizers); ods_api.cpp executes the launches on a HIP stream.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include "../../include/ods.h"

namespace ods {

// ---------------------------------------------------------------- error state
// Thread-local message behind ods_last_error(). set_error returns `st`.
ods_status set_error(ods_status st, const char *fmt, ...);
void clear_error();
const char *error_text();

// ---------------------------------------------------------------- kernel launch shapes
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
  const int32_t *a_gather;    // streaming kernel only: row r of A is row a_gather[r] / a_gather_div
  int a_gather_div;           //   of the A pointer (clamped to [0, a_gather_rows)), e.g. the token
  int a_gather_rows;          //   of an expert slot, read straight from hn
};

constexpr int kDecodeBM = 64, kDecodeBK = 128;  // decode-tile GEMM block rows and K step

// Decode-tile GEMM shape choices (row-major weights).
bool use_big(int M, int N);            // 64 < M: the large-M tile
bool long_k(int N, int K, int epi);    // narrow output with K >= 2N (the down projection)
int tile_n(int N, int K, int epi);     // decode tile width
// Weight-streaming kernel: dense GEMMs past 128 rows, of 33 to 64 rows but
// the SiLU-gated one, grouped GEMMs, and every GEMM on tiled weights.
bool gemm_use_stream(int M, int N, int K, int epi);
int gemm_stream_rows(int M, int N, int K, int epi);  // dense block rows: 64 or 256
int gemm_stream_splits(int M, int N, int K, int epi);
// Split-K plan of a dense GEMM, and the fp32 partial bytes it needs.
int gemm_splits(int M, int N, int K, int epi, bool b_tiled = false);
size_t gemm_partial_bytes(int M, int N, int K, int epi, bool b_tiled = false);

// Tile order of a weight for the streaming GEMM: for each group, N tile and
// 64-wide K step, the 16 KB image of that step's 128 B rows in LDS (row r at
// r * 128 bytes, 16-byte chunk c of the row at position c ^ (r % 8)). Plain
// weights put rows 128 nt .. +127 in N tile nt; gated (gate rows, then up
// rows, `out` of each) put gate rows 64 nt .. +63 then the matching up rows.
// Rows past `out` are zero. `in` must be a multiple of 64.
int64_t tiled_weight_elems(int out, int in, bool gated, int groups);

// Paged decode attention: the batch's (sequence, KV head, window page) units
// split evenly over the waves of a grid of at most one 4-wave workgroup per
// compute unit, and a log-sum-exp merge of sequences that span several waves.
constexpr int kMaxAttnBatch = 4096;  // the kernel keeps per-sequence contexts and a prefix in LDS
struct AttnPlan {
  int seg_pages;    // pages per wave range; 0: total / waves (at least 8)
  int grid;         // workgroups of the attention kernel
  int64_t records;  // partial-record slots per query-head group
  bool units_ok;    // batch * n_kv * span fits the kernel's 32-bit unit index
};
int attn_span(int max_pages, int window);
int attn_grid(int B, int n_kv, int span, int cus);
AttnPlan attn_plan(int B, int n_kv, int D, int max_pages, int window, int split_pages_req, int cus);
size_t attn_ws_bytes(int B, int n_q, int n_kv, int D, const AttnPlan &plan);

// ---------------------------------------------------------------- blocks and ranges
enum OpKind {
  K_ATTN_NORM, K_QKV, K_ROPE, K_KV_APPEND, K_ATTN_CORE, K_O_PROJ, K_FFN_NORM,
  K_GATE_UP, K_SILU, K_DOWN,
  K_ROUTER, K_TOPK, K_PERMUTE, K_EXP_GATE_UP, K_EXP_SILU, K_EXP_DOWN, K_COMBINE
};
struct OpRef {
  int layer;  // -1: out of range
  OpKind kind;
};
const char *op_kind_name(OpKind k);
ods_status check_block(const ods_block *blk);
int num_ops(const ods_block *blk);              // block already checked
OpRef op_at(const ods_block *blk, int g);       // global operator g
int layer_offset(const ods_block *blk, int layer);
int layer_num_ops(const ods_layer_cfg &c);

// Workspace a range needs (the maximum over the layers it touches), for a
// device with `cus` compute units.
size_t range_ws_bytes(const ods_block *blk, int op_begin, int op_end, const ods_batch *batch, int cus);
size_t block_ws_bytes(const ods_block *blk, const ods_batch *batch, int cus);

// Every check ods_run_partition makes before it enqueues anything: block,
// range, batch fields, every pointer each operator of the range touches
// (non-null, 16-byte aligned), shape limits, and the workspace size. ODS_OK
// means the range can be planned and launched.
ods_status validate_range(const ods_block *blk, int op_begin, int op_end, const ods_batch *batch,
                          const ods_state *st, int cus);

// One launch of a validated range.
enum LaunchKind {
  LK_RMSNORM, LK_GEMM, LK_QKV_ROPE, LK_ROPE_APPEND, LK_ATTENTION, LK_SILU, LK_TOPK, LK_ROUTER_TOPK, LK_PERMUTE,
  LK_COMBINE
};
struct RopeArgs {
  uint16_t *qkv; int B, n_q, n_kv, D; float theta;
  const int32_t *ctx_lens, *table; int cols, ring;
  uint16_t *pool; int64_t pool_pages;
  bool do_rope, do_append;
  const float *partial; int splits;  // qkv split-K partials summed in place of a reduce (LK_QKV_ROPE)
};
struct AttnArgs {
  const uint16_t *qkv; int B, n_q, n_kv, D, window;
  const int32_t *ctx_lens, *table; int cols, ring;
  const uint16_t *pool; int64_t pool_pages;
  AttnPlan plan; float *ws; uint16_t *o;
};
struct Launch {
  LaunchKind kind;
  int layer;
  int n_ops;         // operators this launch covers (more than one when fused)
  const char *what;  // static name for traces and errors
  GemmArgs gemm;     // LK_GEMM, LK_QKV_ROPE, LK_ROUTER_TOPK
  RopeArgs rope;     // LK_QKV_ROPE, LK_ROPE_APPEND
  AttnArgs attn;     // LK_ATTENTION
  // LK_RMSNORM: x -> out with gain; LK_SILU: x (gate | up) -> out; LK_COMBINE: x (yp) into out (resid)
  const uint16_t *x, *gain; uint16_t *out; int rows, width; float eps;
  // LK_TOPK, LK_ROUTER_TOPK, LK_PERMUTE, LK_COMBINE
  const float *logits; float *weights; int32_t *ids, *perm, *slot_pos, *expert_off; int E, k;
  float *logits_out; const float *topk_partial; int topk_splits;  // LK_ROUTER_TOPK: router split-K partials
  uint16_t *xp;
};

// The launch that starts at position i of a validated range [op_begin,
// op_end) (operator op_begin + i). Adjacent operators of the same layer may
// be fused into it: out->n_ops says how many it covers.
void plan_launch(const ods_block *blk, int op_begin, int op_end, int i, const ods_batch *batch, const ods_state *st,
                 int cus, Launch *out);

}  // namespace ods
