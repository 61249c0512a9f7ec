// Row-wise and elementwise operators of the decode layer: RMSNorm, RoPE with
// KV-cache append, SiLU(gate) * up. All are a few MB per step at the largest
// batch; they stream rows with 16-byte vector accesses, one block per row.
#include "common.hpp"
#include "kernels.hpp"

namespace ods {

namespace {

// out[r] = x[r] * (mean(x[r]^2) + eps)^(-1/2) * gain, fp32 math, bf16 out.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const uint16_t *x, const uint16_t *gain,
                                                      uint16_t *out, int H, float eps) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const u32x4 *xr = (const u32x4 *)(x + row * H);
  const int nvec = H / 8;
  float ss = 0.f;
  for (int v = threadIdx.x; v < nvec; v += 256) {
    const u32x4 w = xr[v];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float a = bf_lo(w[j]), b = bf_hi(w[j]);
      ss += a * a + b * b;
    }
  }
  ss = block_sum_256(ss, red);
  const float inv = rsqrtf(ss / (float)H + eps);
  u32x4 *orow = (u32x4 *)(out + row * H);
  const u32x4 *g = (const u32x4 *)gain;
  for (int v = threadIdx.x; v < nvec; v += 256) {
    const u32x4 w = xr[v], gw = g[v];
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = pack2(bf_lo(w[j]) * inv * bf_lo(gw[j]), bf_hi(w[j]) * inv * bf_hi(gw[j]));
    orow[v] = o;
  }
}

// One block per sequence. RoPE (rotate-half) of the n_q + n_kv heads of
// qkv[b] at position ctx[b] - 1, in place, and/or store of k, v into the page
// slot of that position. With ring > 0 the table is a window-only page ring:
// position p lives in page_table[b][(p / 16) % ring] and is not clamped. The angle p * theta^(-2i/d) is formed in double and
// reduced modulo 2 pi there, so the fp32 sin / cos see |r| <= pi (positions
// reach 10^5 radians, where an fp32 angle would keep only ~2 decimals).
__global__ __launch_bounds__(256) void rope_append_kernel(uint16_t *qkv, int n_q, int n_kv, int D,
                                                          float theta, const int32_t *ctx_lens,
                                                          const int32_t *page_table, int max_pages, int ring,
                                                          uint16_t *pool, int64_t pool_pages,
                                                          int do_rope, int do_append) {
  __shared__ float cs[64], sn[64];
  const int b = blockIdx.x;
  const int ctx = ctx_lens[b];
  if (ctx < 1) return;
  const int p = (ring > 0 ? ctx : min(ctx, max_pages * kPage)) - 1;
  const int half = D / 2, nvh = half / 8;
  uint16_t *row = qkv + (int64_t)b * (n_q + 2 * n_kv) * D;

  uint16_t *kbase = nullptr, *vbase = nullptr;
  const int64_t blk = (int64_t)kPage * D;
  const int slot = p % kPage;
  if (do_append) {
    const int page = page_table[(int64_t)b * max_pages + (ring > 0 ? (p / kPage) % ring : p / kPage)];
    if (page >= 0 && page < pool_pages) {
      kbase = pool + (int64_t)page * 2 * n_kv * blk;
      vbase = kbase + n_kv * blk;
    }
  }
  if (do_rope) {
    if (threadIdx.x < half) {
      const double two_pi_hi = 6.283185307179586, two_pi_lo = 2.4492935982947064e-16;
      const double inv = exp2(-(2.0 * threadIdx.x / D) * log2((double)theta));
      const double a = (double)p * inv;
      const double k = rint(a * (1.0 / two_pi_hi));
      const double r = fma(-k, two_pi_lo, fma(-k, two_pi_hi, a));
      float sv, cv;
      sincosf((float)r, &sv, &cv);
      cs[threadIdx.x] = cv;
      sn[threadIdx.x] = sv;
    }
    __syncthreads();
  }
  // q and k heads: rotate (if asked) 8 pairs per item; k heads also go to the cache
  const int first = do_rope ? 0 : n_q;
  const int items = (n_q + n_kv - first) * nvh;
  for (int t = threadIdx.x; t < items; t += 256) {
    const int h = first + t / nvh, i0 = (t % nvh) * 8;
    uint16_t *u = row + h * D;
    u32x4 x0 = *(const u32x4 *)(u + i0), x1 = *(const u32x4 *)(u + half + i0);
    if (do_rope) {
      u32x4 y0, y1;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = i0 + 2 * j;
        const float a0 = bf_lo(x0[j]), a1 = bf_hi(x0[j]), b0 = bf_lo(x1[j]), b1 = bf_hi(x1[j]);
        y0[j] = pack2(a0 * cs[i] - b0 * sn[i], a1 * cs[i + 1] - b1 * sn[i + 1]);
        y1[j] = pack2(b0 * cs[i] + a0 * sn[i], b1 * cs[i + 1] + a1 * sn[i + 1]);
      }
      x0 = y0;
      x1 = y1;
      *(u32x4 *)(u + i0) = x0;
      *(u32x4 *)(u + half + i0) = x1;
    }
    if (kbase && h >= n_q) {
      uint16_t *dst = kbase + (h - n_q) * blk + slot * D;
      *(u32x4 *)(dst + i0) = x0;
      *(u32x4 *)(dst + half + i0) = x1;
    }
  }
  // v heads: dim-major in the page, one element per store
  if (vbase) {
    const uint16_t *v = row + (n_q + n_kv) * D;
    for (int t = threadIdx.x; t < n_kv * D; t += 256) {
      const int g = t / D, i = t % D;
      vbase[g * blk + i * kPage + slot] = v[t];
    }
  }
}

__global__ __launch_bounds__(256) void silu_mul_kernel(const uint16_t *gu, uint16_t *act, int F, int vblocks) {
  const int64_t row = blockIdx.x / vblocks;
  const int v = (blockIdx.x % vblocks) * 256 + threadIdx.x;  // 8-element vector index
  if (v * 8 >= F) return;
  const u32x4 g = *(const u32x4 *)(gu + row * 2 * F + v * 8);
  const u32x4 u = *(const u32x4 *)(gu + row * 2 * F + F + v * 8);
  u32x4 o;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    o[j] = pack2(silu(bf_lo(g[j])) * bf_lo(u[j]), silu(bf_hi(g[j])) * bf_hi(u[j]));
  *(u32x4 *)(act + row * F + v * 8) = o;
}

}  // namespace

hipError_t launch_rmsnorm(const uint16_t *x, const uint16_t *gain, uint16_t *out, int rows, int H,
                          float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(rows), dim3(256), 0, s, x, gain, out, H, eps);
  return hipGetLastError();
}

hipError_t launch_rope_append(uint16_t *qkv, int B, int n_q, int n_kv, int D, float theta,
                              const int32_t *ctx_lens, const int32_t *page_table, int max_pages, int ring,
                              uint16_t *pool, int64_t pool_pages, bool do_rope, bool do_append,
                              hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_append_kernel, dim3(B), dim3(256), 0, s, qkv, n_q, n_kv, D, theta, ctx_lens,
                     page_table, max_pages, ring, pool, pool_pages, (int)do_rope, (int)do_append);
  return hipGetLastError();
}

hipError_t launch_silu_mul(const uint16_t *gu, uint16_t *act, int rows, int F, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int vblocks = (F / 8 + 255) / 256;
  hipLaunchKernelGGL(silu_mul_kernel, dim3((unsigned)((int64_t)rows * vblocks)), dim3(256), 0, s, gu, act, F,
                     vblocks);
  return hipGetLastError();
}

}  // namespace ods
