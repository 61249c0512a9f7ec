// Paged GQA decode attention for gfx950.
//
// Decode attention is the memory-bound operator class of the paper's cost
// model (Appendix A.2): each decoded token reads its whole KV context once.
// Work item = one wave = (sequence b, KV head g, a run of `split_pages` pages).
// All n_q / n_kv query heads of the group share the item, so every K/V byte is
// read from HBM exactly once. Per page (16 tokens):
//   S^T = K_page * Q_g^T    4 x MFMA 16x16x32 (d = 128): rows = tokens, cols = heads;
//                           lane l gets tokens (l/16)*4 .. +3 of head l%16.
//   online softmax          per lane (head l%16); page max over the 4 lane rows
//                           by two xor-shuffles; masked tokens get -inf.
//   O^T += V_page^T * P     8 x MFMA 16x16x16 (d = 128): V is stored dim-major in
//                           the page, so lane l reads 8 contiguous bytes, and P
//                           is already in the B-operand layout of S^T.
// The accumulator O^T keeps head l%16 in lane l, so the softmax rescale never
// leaves the lane. Partials (m, l, acc[d]) go to a workspace and a second
// kernel merges the splits exactly with their log-sum-exp weights.
#include <math.h>

#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace ods {

namespace {

template <int D>
__global__ __launch_bounds__(256) void attn_split_kernel(
    const uint16_t *__restrict__ qkv, int n_q, int n_kv, int window, const int32_t *__restrict__ ctx_lens,
    const int32_t *__restrict__ page_table, int max_pages, const uint16_t *__restrict__ pool,
    int64_t pool_pages, int split_pages, int n_splits, float scale_log2, float *__restrict__ ws_acc,
    float *__restrict__ ws_ml, int B) {
  constexpr int KK = D / 32;  // QK MFMAs per page
  constexpr int NB = D / 16;  // PV MFMAs per page
  constexpr int64_t BLK = (int64_t)kPage * D;

  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int split = gw % n_splits;
  const int g = (gw / n_splits) % n_kv;
  const int b = gw / (n_splits * n_kv);
  if (b >= B) return;
  const int group = n_q / n_kv;
  const int ctx = min(ctx_lens[b], max_pages * kPage);
  if (ctx < 1) return;
  const int p = ctx - 1;
  const int lo = window > 0 ? max(0, p - window + 1) : 0;
  const int first_page = lo / kPage, last_page = p / kPage;
  const int pg_begin = first_page + split * split_pages;
  if (pg_begin > last_page) return;
  const int pg_end = min(pg_begin + split_pages, last_page + 1);

  const int hl = lane & 15;   // head within the group (MFMA column)
  const int rq = lane >> 4;   // lane row-quad
  const bool head_ok = hl < group;

  bf16x8 qf[KK];
  {
    const uint16_t *q = qkv + (int64_t)b * (n_q + 2 * n_kv) * D + (int64_t)(g * group + hl) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      u32x4 w = head_ok ? *(const u32x4 *)(q + kk * 32 + rq * 8) : u32x4{0u, 0u, 0u, 0u};
      qf[kk] = __builtin_bit_cast(bf16x8, w);
    }
  }

  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const int32_t *pt = page_table + (int64_t)b * max_pages;
  const uint16_t *pool_g = pool + (int64_t)g * BLK;
  const int64_t page_stride = 2 * (int64_t)n_kv * BLK;
  const int64_t v_off = (int64_t)n_kv * BLK;

  // Page ids of this work item, one per lane (split_pages <= 64), broadcast
  // with readlane so the K/V loads never wait on a dependent scalar load.
  const int my_page = (lane < pg_end - pg_begin) ? pt[pg_begin + lane] : -1;

  u32x4 kf[KK];
  u32x2 vf[NB];
  auto fetch = [&](int pg, bool &ok) {
    int page = __builtin_amdgcn_readlane(my_page, pg - pg_begin);
    ok = (unsigned)page < (unsigned long long)pool_pages;
    if (!ok) page = 0;
    const uint16_t *kb = pool_g + (int64_t)page * page_stride;
    const uint16_t *vb = kb + v_off;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) kf[kk] = *(const u32x4 *)(kb + hl * D + kk * 32 + rq * 8);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) vf[nb] = *(const u32x2 *)(vb + (nb * 16 + hl) * kPage + rq * 4);
  };

  bool ok_next;
  fetch(pg_begin, ok_next);
  for (int pg = pg_begin; pg < pg_end; ++pg) {
    u32x4 kc[KK];
    u32x2 vc[NB];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) kc[kk] = kf[kk];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) vc[nb] = vf[nb];
    const bool ok = ok_next;
    if (pg + 1 < pg_end) fetch(pg + 1, ok_next);
    if (!ok) continue;

    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) s = mfma_16x16x32(__builtin_bit_cast(bf16x8, kc[kk]), qf[kk], s);

    const int tok0 = pg * kPage + rq * 4;
    const bool edge = (pg * kPage < lo) || (pg * kPage + kPage - 1 > p);
    float sv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = tok0 + i;
      sv[i] = (!edge || (t >= lo && t <= p)) ? s[i] * scale_log2 : -INFINITY;
    }
    float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);  // m_run = -inf -> 0
    float pv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) pv[i] = exp2f(sv[i] - m_new);
    l_run = l_run * alpha + ((pv[0] + pv[1]) + (pv[2] + pv[3]));
    m_run = m_new;
    bf16x4 pb;
#pragma unroll
    for (int i = 0; i < 4; ++i) pb[i] = (__bf16)pv[i];
    if (edge) {
      // Zero the values of masked slots: their P is 0, but stale slots may hold
      // non-finite bits and 0 * NaN would poison the accumulator.
      uint32_t m01 = (tok0 >= lo && tok0 <= p ? 0xffffu : 0u) |
                     (tok0 + 1 >= lo && tok0 + 1 <= p ? 0xffff0000u : 0u);
      uint32_t m23 = (tok0 + 2 >= lo && tok0 + 2 <= p ? 0xffffu : 0u) |
                     (tok0 + 3 >= lo && tok0 + 3 <= p ? 0xffff0000u : 0u);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        vc[nb][0] &= m01;
        vc[nb][1] &= m23;
      }
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      acc[nb] *= alpha;
      acc[nb] = mfma_16x16x16(__builtin_bit_cast(bf16x4, vc[nb]), pb, acc[nb]);
    }
  }

  l_run += __shfl_xor(l_run, 16, kWave);
  l_run += __shfl_xor(l_run, 32, kWave);
  if (head_ok) {
    const int h = g * group + hl;
    const int64_t rec = ((int64_t)b * n_q + h) * n_splits + split;
    float *dst = ws_acc + rec * D;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) *(f32x4 *)(dst + nb * 16 + rq * 4) = acc[nb];
    if (rq == 0) {
      ws_ml[rec * 2] = m_run;
      ws_ml[rec * 2 + 1] = l_run;
    }
  }
}

// o[b, h, d] = sum_s 2^(m_s - M) acc_s[d] / sum_s 2^(m_s - M) l_s over the splits
// that hold work for sequence b.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float *__restrict__ ws_acc,
                                                         const float *__restrict__ ws_ml, int n_q,
                                                         int window, const int32_t *__restrict__ ctx_lens,
                                                         int max_pages, int split_pages, int n_splits,
                                                         uint16_t *__restrict__ o, int B) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)B * n_q * D) return;
  const int d = (int)(idx % D);
  const int h = (int)((idx / D) % n_q);
  const int b = (int)(idx / ((int64_t)D * n_q));
  const int ctx = min(ctx_lens[b], max_pages * kPage);
  if (ctx < 1) {
    o[idx] = 0;
    return;
  }
  const int p = ctx - 1;
  const int lo = window > 0 ? max(0, p - window + 1) : 0;
  const int pages = p / kPage - lo / kPage + 1;
  const int ns = min(n_splits, (pages + split_pages - 1) / split_pages);
  const int64_t rec0 = ((int64_t)b * n_q + h) * n_splits;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, ws_ml[(rec0 + s) * 2]);
  float L = 0.f, acc = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < ns; ++s) {
      const float ms = ws_ml[(rec0 + s) * 2];
      if (ms == -INFINITY) continue;
      const float w = exp2f(ms - M);
      L += w * ws_ml[(rec0 + s) * 2 + 1];
      acc += w * ws_acc[(rec0 + s) * D + d];
    }
  }
  o[idx] = f2bf(L > 0.f ? acc / L : 0.f);
}

}  // namespace

AttnPlan attn_plan(int B, int n_kv, int D, int max_pages, int window, int split_pages_req) {
  (void)D;
  int span = max_pages;
  if (window > 0) span = std::min(max_pages, (window + kPage - 1) / kPage + 1);
  span = std::max(span, 1);
  int sp = split_pages_req;
  if (sp <= 0) {
    sp = 64;
    // Enough work items to give every compute unit many waves to switch between.
    while (sp > 4 && (int64_t)B * n_kv * ((span + sp - 1) / sp) < 8192) sp /= 2;
  }
  sp = std::min(sp, 64);  // one page id per lane of the work item's wave
  AttnPlan plan;
  plan.split_pages = sp;
  plan.n_splits = (span + sp - 1) / sp;
  return plan;
}

size_t attn_ws_bytes(int B, int n_q, int D, const AttnPlan &plan) {
  return (size_t)B * n_q * plan.n_splits * (D + 2) * sizeof(float);
}

hipError_t launch_attention(const uint16_t *qkv, int B, int n_q, int n_kv, int D, int window,
                            const int32_t *ctx_lens, const int32_t *page_table, int max_pages,
                            const uint16_t *pool, int64_t pool_pages, const AttnPlan &plan, float *ws,
                            uint16_t *o, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  float *ws_acc = ws;
  float *ws_ml = ws + (size_t)B * n_q * plan.n_splits * D;
  const int64_t waves = (int64_t)B * n_kv * plan.n_splits;
  const dim3 grid((unsigned)((waves + 3) / 4));
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
  const int64_t outs = (int64_t)B * n_q * D;
  const dim3 mgrid((unsigned)((outs + 255) / 256));
  if (D == 128) {
    hipLaunchKernelGGL(attn_split_kernel<128>, grid, dim3(256), 0, s, qkv, n_q, n_kv, window, ctx_lens,
                       page_table, max_pages, pool, pool_pages, plan.split_pages, plan.n_splits, scale_log2,
                       ws_acc, ws_ml, B);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_merge_kernel<128>, mgrid, dim3(256), 0, s, ws_acc, ws_ml, n_q, window, ctx_lens,
                       max_pages, plan.split_pages, plan.n_splits, o, B);
  } else {
    hipLaunchKernelGGL(attn_split_kernel<64>, grid, dim3(256), 0, s, qkv, n_q, n_kv, window, ctx_lens,
                       page_table, max_pages, pool, pool_pages, plan.split_pages, plan.n_splits, scale_log2,
                       ws_acc, ws_ml, B);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_merge_kernel<64>, mgrid, dim3(256), 0, s, ws_acc, ws_ml, n_q, window, ctx_lens,
                       max_pages, plan.split_pages, plan.n_splits, o, B);
  }
  return hipGetLastError();
}

}  // namespace ods
