/*
 * ods.h -- C ABI of the operator-level-disaggregated (ODS) decode hot path on
 * AMD Instinct MI355X (gfx950).
 *
 * The paper models one decode step as a fixed, ordered sequence of kernels
 * o_1..o_N (Appendix A.1) and a serving stage as a contiguous slice of the
 * operator sequence of a repeating partition block: stage j holds operators
 * q_{j-1}+1 .. q_j (Section 4, "Partition-block abstraction"; Appendix B.1).
 * Stages exchange an activation interface A_j at each boundary (Appendix B.3,
 * the stage-latency and transfer-latency equations), a worker loads only its
 * assigned components and state, buffers are bound once with only token,
 * position and KV metadata changing between steps, and one native call
 * enqueues a whole per-step action sequence (Section 6 and its "Single native
 * submission" optimisation). This library is that native call for one GPU.
 *
 * Operator index space. A block of layers is numbered globally, layer after
 * layer; indices are 0-based and ranges half-open, so the paper's stage j is
 * [q_{j-1}, q_j). Per layer (local index):
 *
 *   dense layer (10 ops)                  MoE layer (14 ops)
 *   0 attn_norm        resid -> xn        0..6 as in the dense layer
 *   1 qkv_proj         xn -> qkv          7  router          hn -> logits
 *   2 rope             qkv -> qkv         8  topk_softmax    logits -> topk_ids, topk_w
 *   3 kv_append        qkv -> KV pool     9  moe_permute     hn, topk_ids -> xp, perm,
 *   4 attn_core        qkv, pool -> o                            slot_pos, expert_off
 *   5 o_proj_residual  o, resid -> resid  10 expert_gate_up  xp -> gu_p
 *   6 ffn_norm         resid -> hn        11 silu_mul        gu_p -> act_p
 *   7 gate_up          hn -> gu           12 expert_down     act_p -> yp
 *   8 silu_mul         gu -> act          13 moe_combine_residual
 *   9 down_residual    act, resid -> resid                   yp, topk_w, slot_pos, resid -> resid
 *
 * Attention-FFN disaggregation cuts every layer at local 6; core-attention
 * disaggregation isolates [3, 5); the colocated template is [0, N_block)
 * (Section 4, "Design-space expressiveness").
 *
 * Numerics (the paper leaves the layer's arithmetic unspecified; these are the
 * library's conventions): bf16 storage, fp32 accumulation. RMSNorm
 * x * (mean(x^2) + eps)^-1/2 * gain. RoPE rotate-half pairs (i, i + d/2) at
 * position ctx - 1, angle (ctx - 1) * theta^(-2i/d) evaluated in double.
 * Attention softmax(q K^T / sqrt(d)) V over keys [ctx - window, ctx - 1]
 * (window 0: all keys); query head h reads KV head h / (n_q / n_kv).
 * SwiGLU silu(gate) * up. Routing: top-k of the fp32 router logits (ties go to
 * the lower expert index), weights = softmax over the chosen k. Every live
 * buffer is rounded to bf16 (round-to-nearest-even) except logits and routing
 * weights (fp32) and indices (int32).
 *
 * Ownership and errors. The caller owns all memory and the stream. The library
 * never allocates, frees, synchronises, or changes the current device, and
 * keeps no state between calls (apart from the static workspace array of
 * ods_run_partition_scratch). Every argument is checked on the host before
 * anything is enqueued: a non-OK status means nothing was enqueued, except
 * ODS_EHIP, which reports a launch failure after earlier kernels of the same
 * call were enqueued. Device faults surface at the caller's synchronisation.
 * All device pointers must be 16-byte aligned. Calls are thread-safe;
 * ods_last_error() is per thread.
 */
#ifndef ODS_H
#define ODS_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ODS_OK = 0,
  ODS_EINVAL = -1,        /* null / misaligned pointer, negative size, bad enum */
  ODS_ERANGE = -2,        /* operator range or context outside its bounds */
  ODS_ENOMEM = -3,        /* KV pool or workspace too small */
  ODS_EUNSUPPORTED = -4,  /* shape the kernels do not implement */
  ODS_EHIP = -5           /* HIP runtime reported an error while enqueuing */
} ods_status;

#define ODS_PAGE_TOKENS 16

/* Shape of one decoder layer. n_experts == 0 selects a dense SwiGLU FFN of
 * width ffn; otherwise a top_k-of-n_experts MoE with per-expert width moe_ffn.
 * window == 0 selects full attention, window > 0 a sliding window of that many
 * most recent tokens (the decoded token included).
 * Supported: head_dim in {64, 128}; n_q a multiple of n_kv with n_q / n_kv <= 16;
 * hidden, ffn, moe_ffn multiples of 8; n_experts <= 256; 1 <= top_k <= n_experts. */
typedef struct {
  int32_t hidden, n_q, n_kv, head_dim;
  int32_t ffn;
  int32_t n_experts, top_k, moe_ffn;
  int32_t window;
  float rope_theta, rms_eps;
} ods_layer_cfg;

/* Layout of a layer's projection weights (w_qkv, w_o, w_gate_up, w_down).
 *   ODS_WEIGHTS_ROWS:  row-major "out x in", as listed under ods_layer.
 *   ODS_WEIGHTS_TILED: the tile order ods_tile_weight() writes, which the
 *     weight-streaming GEMM reads as one contiguous run per block (faster at
 *     decode batches). Needs hidden, n_q * head_dim and ffn (dense) or moe_ffn
 *     (MoE) to be multiples of 64 (ODS_EUNSUPPORTED otherwise). w_router stays
 *     row-major. */
typedef enum { ODS_WEIGHTS_ROWS = 0, ODS_WEIGHTS_TILED = 1 } ods_weight_layout;

/* One layer's device-resident weights (bf16, row-major "out x in" unless
 * weight_layout says otherwise) and KV pool.
 *   g_attn, g_ffn  [hidden]
 *   w_qkv          [(n_q + 2 n_kv) head_dim, hidden]   q heads, then k heads, then v heads
 *   w_o            [hidden, n_q head_dim]
 *   dense: w_gate_up [2 ffn, hidden] (gate rows, then up rows); w_down [hidden, ffn]
 *   MoE:   w_router [n_experts, hidden]; w_gate_up [n_experts, 2 moe_ffn, hidden];
 *          w_down [n_experts, hidden, moe_ffn]
 *   kv_pool  [pool_pages][2][n_kv][16 * head_dim] bf16. Block (page, 0, g) holds the
 *            keys of 16 token slots row-major (slot t, dim i at t * head_dim + i);
 *            block (page, 1, g) holds the values dim-major (dim i, slot t at i * 16 + t).
 *            Token position t of a sequence lives in page page_table[b][t / 16],
 *            slot t % 16. Every block is 16 * head_dim * 2 bytes, contiguous. */
typedef struct {
  ods_layer_cfg cfg;
  const void *g_attn, *w_qkv, *w_o, *g_ffn, *w_gate_up, *w_down, *w_router;
  void *kv_pool;
  int64_t pool_pages;
  int32_t weight_layout;  /* ods_weight_layout */
} ods_layer;

/* A partition block: n_layers layers whose operators are numbered consecutively.
 * All layers share one batch, page table and live set. */
typedef struct {
  int32_t n_layers;
  const ods_layer *layers;
} ods_block;

/* Per-step metadata (device pointers). ctx_lens[b] counts the keys sequence b
 * attends to, the token being decoded included, so that token's position is
 * ctx_lens[b] - 1; valid values are 1 .. max_pages * 16 (larger values are
 * clamped; a row with a value < 1 is left alone by RoPE and KV append, and
 * its attention output is a row of zeros).
 * page_table [batch][max_pages] int32, -1 for unused entries; page ids outside
 * [0, pool_pages) are skipped by the kernels. attn_core numbers the (sequence,
 * KV head, window page) units of the batch and gives every wave of its grid an
 * equal contiguous range of them; split_pages fixes the range length in pages
 * (0: library choice, the batch's pages over all waves, at least 8 each).
 * attn_core takes batch <= 4096 and batch * n_kv * window pages < 2^30
 * (ODS_EUNSUPPORTED otherwise).
 *
 * Window-only page ring (ring_pages > 0). A sliding-window layer only ever
 * reads the most recent `window` tokens, so its KV pages can live in a ring
 * (a sliding-window layer reads at most its window of KV; Section 3, hybrid
 * architectures): with ring_pages = R > 0, every layer of
 * the call with window > 0 maps token position t of sequence b to page
 * ring_table[b][(t / 16) % R], slot t % 16, of its own kv_pool, and its
 * contexts are not clamped to max_pages * 16. Full-attention layers keep
 * page_table. R must be at least ceil(window / 16) + 1 for every such layer
 * the call touches (the window's pages plus the one the next token opens), so
 * a page is only reused once it has left the window (ODS_EINVAL otherwise).
 * ring_table is [batch][R] int32; ods_kv_alloc with max_pages = R and contexts
 * min(ctx, 16 R) fills one. A ring layer's pool needs at most batch * R pages
 * however long the contexts grow. ring_pages = 0: no ring (ring_table unused). */
typedef struct {
  int32_t batch, max_pages;
  const int32_t *ctx_lens;
  const int32_t *page_table;
  int32_t split_pages;
  int32_t ring_pages;
  const int32_t *ring_table;
} ods_batch;

/* Live buffers (the activation interface at any cut), device, caller-allocated.
 * Sizes per ods_live_bytes(). Only buffers read or written by the operators of
 * a call's range need to be non-null.
 *   resid [B, H] bf16 (updated in place by o_proj_residual, down_residual,
 *   moe_combine_residual); xn, hn [B, H]; qkv [B, (n_q + 2 n_kv) d]; o [B, n_q d];
 *   gu [B, 2F]; act [B, F]; logits [B, E] fp32; topk_ids [B, k] int32;
 *   topk_w [B, k] fp32; perm [B k] (sorted position -> token * k + slot);
 *   slot_pos [B k] (token * k + slot -> sorted position); expert_off [E + 1];
 *   xp [B k, H]; gu_p [B k, 2 I]; act_p [B k, I]; yp [B k, H] (all bf16);
 *   ws: scratch of at least ods_workspace_bytes() bytes. */
typedef struct {
  void *resid, *xn, *qkv, *o, *hn, *gu, *act;
  float *logits, *topk_w;
  int32_t *topk_ids, *perm, *slot_pos, *expert_off;
  void *xp, *gu_p, *act_p, *yp;
  void *ws;
  size_t ws_bytes;
} ods_state;

typedef enum {
  ODS_BUF_RESID = 0, ODS_BUF_XN, ODS_BUF_QKV, ODS_BUF_O, ODS_BUF_HN, ODS_BUF_GU, ODS_BUF_ACT,
  ODS_BUF_LOGITS, ODS_BUF_TOPK_W, ODS_BUF_TOPK_IDS, ODS_BUF_PERM, ODS_BUF_SLOT_POS,
  ODS_BUF_EXPERT_OFF, ODS_BUF_XP, ODS_BUF_GU_P, ODS_BUF_ACT_P, ODS_BUF_YP, ODS_BUF_COUNT
} ods_buffer;

/* Host-only page allocation for one step's batch (no device work). The pool's
 * page ids [0, pool_pages) are shuffled by a Fisher-Yates pass driven by
 * splitmix64(seed) (for i = P-1 down to 1, swap entries i and next() mod (i+1));
 * sequence b then takes the next ceil(ctx_lens_host[b] / 16) shuffled ids, in
 * batch order. Writes page_table_host [batch][max_pages] (caller memory), -1 in
 * unused entries. ODS_ENOMEM if the batch needs more than pool_pages pages,
 * ODS_ERANGE if a sequence needs more than max_pages, ODS_EINVAL for null
 * pointers or non-positive ctx. The paged cache itself follows the paper's use
 * of paged KV memory in its serving engine (Section 6). */
ods_status ods_kv_alloc(int64_t pool_pages, const int32_t *ctx_lens_host, int32_t batch,
                        uint64_t seed, int32_t max_pages, int32_t *page_table_host);

/* Bytes of one layer's KV pool of pool_pages pages (0 for an invalid cfg). */
size_t ods_kv_pool_bytes(const ods_layer_cfg *cfg, int64_t pool_pages);

/* Bytes of live buffer `which` for this block at this batch size (the maximum
 * over the block's layers; 0 when no layer uses the buffer). */
size_t ods_live_bytes(const ods_block *blk, int32_t batch, ods_buffer which);

/* Minimum ods_state.ws_bytes for any operator range of this block and batch. */
size_t ods_workspace_bytes(const ods_block *blk, const ods_batch *batch);

/* Number of operators of the block (sum over layers of 10 or 14); < 0 on error. */
int32_t ods_block_num_ops(const ods_block *blk);

/* Tiled weight layout (ODS_WEIGHTS_TILED). A weight of `groups` slabs (1, or
 * n_experts for the expert weights), each `out` x `in` row-major bf16 (gated:
 * 2 out rows, the gate rows then the up rows, as w_gate_up), is stored as
 * consecutive 16 KB tiles, slab by slab: for each N tile nt and each 64-wide
 * K step s, 128 rows of 64 columns, row r at byte r * 128 of the tile and the
 * row's 16-byte chunk c (columns 64 s + 8 c .. + 7) at position c ^ (r % 8)
 * of that row. Plain weights: tile row r is weight row 128 nt + r. Gated: tile
 * rows r < 64 are gate rows 64 nt + r, rows 64 + j the matching up rows
 * out + 64 nt + j, so both halves of an output column stream together (the
 * SwiGLU epilogue of the fused gate_up GEMM, Section 2's FFN operator). Rows
 * past `out` are zero. The XOR position of the chunks keeps the GEMM's LDS
 * fragment reads free of bank conflicts.
 *
 * ods_tiled_weight_bytes: bytes of that layout; 0 unless out >= 1, in >= 64,
 *   in % 64 == 0, groups >= 1 and gated in {0, 1}.
 * ods_tile_weight: enqueues on `stream` the conversion of the row-major weight
 *   at src (device, groups * (gated ? 2 : 1) * out * in bf16) into dst (device,
 *   ods_tiled_weight_bytes() bytes, not overlapping src). Both 16-byte aligned.
 *   ODS_EINVAL for null or misaligned pointers or sizes the layout rejects;
 *   ODS_EHIP if the launch fails. Nothing is enqueued on error. */
size_t ods_tiled_weight_bytes(int32_t out, int32_t in, int32_t gated, int32_t groups);
ods_status ods_tile_weight(const void *src, void *dst, int32_t out, int32_t in, int32_t gated, int32_t groups,
                           hipStream_t stream);

/* Static name of global operator `op` ("attn_core", ...), NULL if out of range. */
const char *ods_op_name(const ods_block *blk, int32_t op);

/* Enqueue operators [op_begin, op_end) of the block on `stream` (one native
 * submission for one stage; Section 6). Adjacent operators inside the range
 * may be fused; every buffer of the live set at op_end is materialised, so a
 * block run as any sequence of contiguous ranges computes the same step. A
 * buffer consumed inside the range may be left unwritten (with moe_permute
 * and expert_gate_up in one range the expert GEMM reads hn through perm and
 * xp is not written).
 * ODS_ERANGE unless 0 <= op_begin < op_end <= ods_block_num_ops(). An empty
 * batch (batch->batch == 0) returns ODS_OK once the block and the range are
 * valid, enqueueing nothing and reading no pointer of batch or state. */
ods_status ods_run_partition(const ods_block *blk, int32_t op_begin, int32_t op_end,
                             const ods_batch *batch, ods_state *state, hipStream_t stream);

/* Size of the workspace the library itself holds on each device for
 * ods_run_partition_scratch (64 MiB; every evaluated block needs at most
 * 32 MiB, as ods_workspace_bytes reports). */
#define ODS_SCRATCH_BYTES ((size_t)64 << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that forbid hipMalloc): the same as
 * ods_run_partition, except that the workspace is a static device array of
 * ODS_SCRATCH_BYTES bytes inside the library instead of state->ws (state->ws
 * and state->ws_bytes are ignored and may be NULL / 0). The caller still
 * passes every input and output buffer. Nothing is allocated or freed: each
 * device the library runs on holds its own copy of the array from module load
 * until the process ends; its address is resolved on the first call on a
 * device (with that device current). Nothing in the array needs to start at
 * zero; it keeps the contents the last call left. Calls that overlap on one
 * GPU (several streams or threads at once) share the array and race: the
 * caller must order them, e.g. on one stream per device.
 * Errors: those of ods_run_partition, plus ODS_ENOMEM when the range needs
 * more than ODS_SCRATCH_BYTES of workspace (nothing is enqueued) and ODS_EHIP
 * when the array's device address cannot be resolved. */
ods_status ods_run_partition_scratch(const ods_block *blk, int32_t op_begin, int32_t op_end,
                                     const ods_batch *batch, ods_state *state, hipStream_t stream);

/* The attention stage of layer `layer`: its operators 0..5 (attention-FFN
 * disaggregation's attention side; Section 2, "Attention-FFN Disaggregation"). */
ods_status ods_attn_stage(const ods_block *blk, int32_t layer, const ods_batch *batch,
                          ods_state *state, hipStream_t stream);

/* The FFN / MoE stage of layer `layer`: its operators 6 .. end of layer. */
ods_status ods_ffn_stage(const ods_block *blk, int32_t layer, const ods_batch *batch,
                         ods_state *state, hipStream_t stream);

/* Capture operators [op_begin, op_end) as an instantiated HIP graph, so a
 * stage replays as one submission with its buffers bound once (Section 6:
 * static plan capacity; graphs and buffers bound once, only token, position
 * and KV metadata change between iterations).
 * The graph holds the pointers of blk, batch and state and the host values
 * they carry (batch size, max_pages, split_pages, shapes) as of this call; the
 * device contents they point to (resid, ctx_lens, page_table, weights, pools)
 * are read at each launch, so a new decode step only rewrites those buffers.
 * Validation is that of ods_run_partition; on a non-OK status *exec is NULL.
 * The caller owns *exec: launch it with ods_graph_launch, free it with
 * ods_graph_destroy. Capture runs on a private stream and enqueues nothing. */
ods_status ods_partition_graph(const ods_block *blk, int32_t op_begin, int32_t op_end,
                               const ods_batch *batch, ods_state *state, hipGraphExec_t *exec);

/* Launch a graph from ods_partition_graph on `stream` (hipGraphLaunch). */
ods_status ods_graph_launch(hipGraphExec_t exec, hipStream_t stream);

/* Free a graph from ods_partition_graph (NULL is a no-op). */
ods_status ods_graph_destroy(hipGraphExec_t exec);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char *ods_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ODS_H */
