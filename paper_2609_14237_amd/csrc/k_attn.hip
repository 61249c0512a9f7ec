// Paged GQA decode attention for gfx950.
//
// Decode attention is the memory-bound operator class of the paper's cost
// model (Appendix A.2): each decoded token reads its whole KV context once.
//
// Work item = one workgroup of 4 waves = (sequence b, KV head g, a chunk of
// `chunk_pages` consecutive pages of the attended window); the waves take the
// chunk's pages round-robin. All n_q / n_kv query heads of the group share the
// item, so every K/V byte is read from HBM exactly once. Per page (16 tokens):
//   S^T = K_page * Q_g^T    MFMA 16x16x32 (D/32 of them): rows = tokens, cols = heads;
//                           lane l gets tokens (l/16)*4 .. +3 of head l%16.
//   online softmax          per lane (head l%16); page max over the 4 lane rows
//                           by two xor-shuffles; masked tokens get -inf.
//   O^T += V_page^T * P     MFMA 16x16x16 (D/16 of them): V is stored dim-major in
//                           the page, so lane l reads 8 contiguous bytes, and P
//                           is already in the B-operand layout of S^T.
// The accumulator O^T keeps head l%16 in lane l, so the softmax rescale never
// leaves the lane. The 4 waves merge their (m, l, acc) through LDS; a sequence
// whose window fits in one chunk writes o directly, longer ones write one
// partial per chunk and a second kernel merges the chunks with their
// log-sum-exp weights. K/V registers are reloaded as soon as the MFMA that
// reads them has issued, so a wave keeps one page in flight with ~100 VGPRs
// and four waves fit per SIMD.
#include <math.h>

#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace ods {

namespace {

template <int D>
struct PageRegs {
  u32x4 k[D / 32];  // K rows: lane l holds K[t = l%16][kk*32 + (l/16)*8 .. +8]
  u32x2 v[D / 16];  // V dim-major: lane l holds V[d = nb*16 + l%16][t = (l/16)*4 .. +4]
  int pg;           // page index within the sequence (uniform)
  bool ok;          // page id inside the pool (uniform)
};

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3))) void attn_chunk_kernel(
    const uint16_t *__restrict__ qkv, int n_q, int n_kv, int window, const int32_t *__restrict__ ctx_lens,
    const int32_t *__restrict__ page_table, int max_pages, const uint16_t *__restrict__ pool,
    int64_t pool_pages, int chunk_pages, int n_chunks, float scale_log2, float *__restrict__ ws_acc,
    float *__restrict__ ws_ml, uint16_t *__restrict__ o, int B) {
  constexpr int KK = D / 32;  // QK MFMAs per page
  constexpr int NB = D / 16;  // PV MFMAs per page
  constexpr int64_t BLK = (int64_t)kPage * D;
  __shared__ float s_acc[3][NB * 4][64];  // waves 1..3, [register][lane]: conflict-free
  __shared__ float s_m[4][16], s_l[4][16];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: keeps control flow scalar
  const int group = n_q / n_kv;
  const int hl = lane & 15;  // head within the group (MFMA column)
  const int rq = lane >> 4;  // lane row-quad
  const bool head_ok = hl < group;
  const int64_t n_items = (int64_t)n_chunks * B * n_kv;
  // Persistent blocks stride over the virtual items, chunk index slowest, so
  // every block sees a similar mix of sequences and an empty item (a chunk
  // past the end of a short window) costs one lookup instead of a launch.
  for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
  const int chunk = (int)(item / ((int64_t)B * n_kv));
  const int bg = (int)(item % ((int64_t)B * n_kv));
  const int g = bg % n_kv;
  const int b = bg / n_kv;
  const int ctx = min(ctx_lens[b], max_pages * kPage);
  if (ctx < 1) continue;
  const int p = ctx - 1;
  const int lo = window > 0 ? max(0, p - window + 1) : 0;
  const int first_page = lo / kPage, last_page = p / kPage;
  const int pg_begin = first_page + chunk * chunk_pages;
  if (pg_begin > last_page) continue;  // uniform over the block
  const int pg_end = min(pg_begin + chunk_pages, last_page + 1);
  const int chunks_b = (last_page - first_page + chunk_pages) / chunk_pages;
  // this wave's contiguous share of the chunk
  const int per_wave = (pg_end - pg_begin + 3) / 4;
  const int w_begin = min(pg_end, pg_begin + wave * per_wave);
  const int n_my = min(pg_end, w_begin + per_wave) - w_begin;

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
  // Page ids of this wave's pages, one per lane (at most 16), broadcast with readlane.
  const int my_page = (lane < n_my) ? pt[w_begin + lane] : -1;

  // Issue the loads of this wave's page j (clamped to its last page so the
  // loads are unconditional and the compiler can count them in flight).
  auto issue = [&](PageRegs<D> &R, int j) {
    const int jj = min(j, n_my - 1);
    int page = __builtin_amdgcn_readlane(my_page, jj);
    R.pg = w_begin + j;
    R.ok = (unsigned)page < (unsigned long long)pool_pages;
    const uint16_t *kb = pool_g + (int64_t)(R.ok ? page : 0) * page_stride;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) R.k[kk] = *(const u32x4 *)(kb + hl * D + kk * 32 + rq * 8);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) R.v[nb] = *(const u32x2 *)(kb + v_off + (nb * 16 + hl) * kPage + rq * 4);
  };
  auto consume = [&](PageRegs<D> &R) {
    const int pg = R.pg;
    const bool ok = R.ok;
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) s = mfma_16x16x32(__builtin_bit_cast(bf16x8, R.k[kk]), qf[kk], s);
    const int tok0 = pg * kPage + rq * 4;
    const bool edge = !ok || (pg * kPage < lo) || (pg * kPage + kPage - 1 > p);
    float sv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = tok0 + i;
      sv[i] = (!edge || (ok && t >= lo && t <= p)) ? s[i] * scale_log2 : -INFINITY;
    }
    float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(m_run, mx);
    if (m_new == -INFINITY) return;  // only while every page so far had an invalid id
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
      // Zero the values of masked slots: their P is 0, but stale slots may
      // hold non-finite bits and 0 * NaN would poison the accumulator.
      const bool v0 = ok && tok0 >= lo && tok0 <= p, v1 = ok && tok0 + 1 >= lo && tok0 + 1 <= p;
      const bool v2 = ok && tok0 + 2 >= lo && tok0 + 2 <= p, v3 = ok && tok0 + 3 >= lo && tok0 + 3 <= p;
      const uint32_t m01 = (v0 ? 0xffffu : 0u) | (v1 ? 0xffff0000u : 0u);
      const uint32_t m23 = (v2 ? 0xffffu : 0u) | (v3 ? 0xffff0000u : 0u);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        R.v[nb][0] &= m01;
        R.v[nb][1] &= m23;
      }
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      acc[nb] *= alpha;
      acc[nb] = mfma_16x16x16(__builtin_bit_cast(bf16x4, R.v[nb]), pb, acc[nb]);
    }
  };

  if (n_my > 0) {
    // Two pages in flight per wave: while page j is consumed, j+1 is loading.
    PageRegs<D> R0, R1;
    issue(R0, 0);
    issue(R1, 1);
    for (int j = 0; j < n_my; j += 2) {
      consume(R0);
      issue(R0, j + 2);
      if (j + 1 < n_my) consume(R1);
      issue(R1, j + 3);
    }
  }

  l_run += __shfl_xor(l_run, 16, kWave);
  l_run += __shfl_xor(l_run, 32, kWave);

  // merge the four waves of the chunk
  if (wave > 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int e = 0; e < 4; ++e) s_acc[wave - 1][nb * 4 + e][lane] = acc[nb][e];
  }
  if (rq == 0) {
    s_m[wave][hl] = m_run;
    s_l[wave][hl] = l_run;
  }
  __syncthreads();
  if (wave == 0 && head_ok) {
  float M = s_m[0][hl];
#pragma unroll
  for (int w = 1; w < 4; ++w) M = fmaxf(M, s_m[w][hl]);
  float sc[4], L = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    sc[w] = (s_m[w][hl] == -INFINITY) ? 0.f : exp2f(s_m[w][hl] - M);
    L += sc[w] * s_l[w][hl];
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v = acc[nb][e] * sc[0];
#pragma unroll
      for (int w = 1; w < 4; ++w) v += sc[w] * s_acc[w - 1][nb * 4 + e][lane];
      acc[nb][e] = v;
    }
  const int h = g * group + hl;
  if (chunks_b == 1) {
    const float inv = L > 0.f ? 1.f / L : 0.f;
    uint16_t *dst = o + ((int64_t)b * n_q + h) * D;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      u32x2 w2;
      w2[0] = pack2(acc[nb][0] * inv, acc[nb][1] * inv);
      w2[1] = pack2(acc[nb][2] * inv, acc[nb][3] * inv);
      *(u32x2 *)(dst + nb * 16 + rq * 4) = w2;
    }
  } else {
    const int64_t rec = ((int64_t)b * n_q + h) * n_chunks + chunk;
    float *dst = ws_acc + rec * D;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) *(f32x4 *)(dst + nb * 16 + rq * 4) = acc[nb];
    if (rq == 0) {
      ws_ml[rec * 2] = M;
      ws_ml[rec * 2 + 1] = L;
    }
  }
  }
  __syncthreads();  // the next item reuses the merge buffers
  }
}

// One wave per (sequence, query head) with more than one chunk:
// o[d] = sum_c 2^(m_c - M) acc_c[d] / sum_c 2^(m_c - M) l_c.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float *__restrict__ ws_acc,
                                                         const float *__restrict__ ws_ml, int n_q, int window,
                                                         const int32_t *__restrict__ ctx_lens, int max_pages,
                                                         int chunk_pages, int n_chunks, uint16_t *__restrict__ o,
                                                         int B) {
  constexpr int DPL = D / 64;  // d values per lane
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wid >= (int64_t)B * n_q) return;
  const int b = (int)(wid / n_q);
  const int ctx = min(ctx_lens[b], max_pages * kPage);
  uint16_t *dst = o + wid * D + lane * DPL;
  if (ctx < 1) {
#pragma unroll
    for (int i = 0; i < DPL; ++i) dst[i] = 0;
    return;
  }
  const int p = ctx - 1;
  const int lo = window > 0 ? max(0, p - window + 1) : 0;
  const int chunks_b = (p / kPage - lo / kPage + chunk_pages) / chunk_pages;
  if (chunks_b <= 1) return;  // written by the chunk kernel
  const int64_t rec0 = wid * n_chunks;
  float mloc = -INFINITY;
  for (int c = lane; c < chunks_b; c += 64) mloc = fmaxf(mloc, ws_ml[(rec0 + c) * 2]);
  const float M = wave_max(mloc);
  auto weight = [&](int c) {
    const float mc = ws_ml[(rec0 + c) * 2];
    return mc == -INFINITY ? 0.f : exp2f(mc - M);
  };
  float lsum = 0.f;
  for (int c = lane; c < chunks_b; c += 64) lsum += weight(c) * ws_ml[(rec0 + c) * 2 + 1];
  const float L = wave_sum(lsum);
  float acc[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) acc[i] = 0.f;
  const float *src = ws_acc + rec0 * D + lane * DPL;
  for (int c0 = 0; c0 < chunks_b; c0 += 64) {
    const float wl = (c0 + lane < chunks_b) ? weight(c0 + lane) : 0.f;
    const int n = min(64, chunks_b - c0);
#pragma unroll 4
    for (int j = 0; j < n; ++j) {
      const float w = __shfl(wl, j, kWave);
#pragma unroll
      for (int i = 0; i < DPL; ++i) acc[i] += w * src[(int64_t)(c0 + j) * D + i];
    }
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
#pragma unroll
  for (int i = 0; i < DPL; ++i) dst[i] = f2bf(acc[i] * inv);
}

}  // namespace

// Compute units of the current device (queried once per process and device).
int num_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

AttnPlan attn_plan(int B, int n_kv, int D, int max_pages, int window, int split_pages_req) {
  (void)D;
  int span = max_pages;
  if (window > 0) span = std::min(max_pages, (window + kPage - 1) / kPage + 1);
  span = std::max(span, 1);
  int cp = split_pages_req;
  if (cp <= 0) {
    // A sliding window that fits in 128 pages is one chunk (no merge pass);
    // otherwise 128-page chunks, halved while the batch offers fewer items
    // than the persistent grid has blocks.
    if (window > 0 && span <= 128) {
      cp = span;
    } else {
      cp = 128;
      while (cp > 8 && (int64_t)B * n_kv * ((span + cp - 1) / cp) < 3 * num_cus()) cp /= 2;
    }
  }
  cp = std::min(cp, 128);  // a wave's share of a chunk must fit one page id per lane
  AttnPlan plan;
  plan.split_pages = cp;
  plan.n_splits = (span + cp - 1) / cp;
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
  // Persistent grid: three 4-wave blocks per compute unit (the occupancy the
  // kernel's registers allow), never more blocks than items.
  const int64_t n_items = (int64_t)B * n_kv * plan.n_splits;
  const dim3 grid((unsigned)std::min<int64_t>(n_items, 3 * num_cus()));
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
  const dim3 mgrid((unsigned)(((int64_t)B * n_q + 3) / 4));
  auto go = [&](auto kchunk, auto kmerge) {
    hipLaunchKernelGGL(kchunk, grid, dim3(256), 0, s, qkv, n_q, n_kv, window, ctx_lens, page_table, max_pages,
                       pool, pool_pages, plan.split_pages, plan.n_splits, scale_log2, ws_acc, ws_ml, o, B);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || plan.n_splits <= 1) return e;
    hipLaunchKernelGGL(kmerge, mgrid, dim3(256), 0, s, ws_acc, ws_ml, n_q, window, ctx_lens, max_pages,
                       plan.split_pages, plan.n_splits, o, B);
    return hipGetLastError();
  };
  if (D == 128) return go(attn_chunk_kernel<128>, attn_merge_kernel<128>);
  return go(attn_chunk_kernel<64>, attn_merge_kernel<64>);
}

}  // namespace ods
