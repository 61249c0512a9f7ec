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
  // The row's first 4 * 256 16-byte vectors (H <= 8192) and their gains are
  // loaded together and kept in registers; longer rows re-read the rest.
  constexpr int VPT = 4;
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const u32x4 *xr = (const u32x4 *)(x + row * H);
  const u32x4 *g = (const u32x4 *)gain;
  const int nvec = H / 8;
  u32x4 xv[VPT], gv[VPT];
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int v = threadIdx.x + i * 256;
    if (v < nvec) {
      xv[i] = xr[v];
      gv[i] = g[v];
    }
  }
  auto sumsq = [](const u32x4 &w) {
    float t = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float a = bf_lo(w[j]), b = bf_hi(w[j]);
      t += a * a + b * b;
    }
    return t;
  };
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < VPT; ++i)
    if (threadIdx.x + i * 256 < nvec) ss += sumsq(xv[i]);
  for (int v = threadIdx.x + VPT * 256; v < nvec; v += 256) ss += sumsq(xr[v]);
  ss = block_sum_256(ss, red);
  const float inv = rsqrtf(ss / (float)H + eps);
  u32x4 *orow = (u32x4 *)(out + row * H);
  auto scale = [&](const u32x4 &w, const u32x4 &gw) {
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = pack2(bf_lo(w[j]) * inv * bf_lo(gw[j]), bf_hi(w[j]) * inv * bf_hi(gw[j]));
    return o;
  };
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int v = threadIdx.x + i * 256;
    if (v < nvec) orow[v] = scale(xv[i], gv[i]);
  }
  for (int v = threadIdx.x + VPT * 256; v < nvec; v += 256) orow[v] = scale(xr[v], g[v]);
}

// One block per (sequence, group of kRopeHeads heads of its qkv row). RoPE
// (rotate-half) of the group's q and k heads at position ctx[b] - 1, in place,
// and/or store of its k, v heads into the page slot of that position. With
// ring > 0 the table is a window-only page ring: position p lives in
// page_table[b][(p / 16) % ring] and is not clamped. With splits > 1 the
// group's columns of the row are first summed from the split-K partials.
constexpr int kRopeHeads = 8;

__global__ __launch_bounds__(256) void rope_append_kernel(uint16_t *qkv, int n_q, int n_kv, int D,
                                                          float theta, const int32_t *ctx_lens,
                                                          const int32_t *page_table, int max_pages, int ring,
                                                          uint16_t *pool, int64_t pool_pages,
                                                          int do_rope, int do_append, const float *partial,
                                                          int splits, int B) {
  __shared__ float cs[64], sn[64];
  const int b = blockIdx.x;
  const int nh = n_q + 2 * n_kv, W = nh * D;
  const int h0 = blockIdx.y * kRopeHeads, h1 = min(nh, h0 + kRopeHeads);
  uint16_t *row = qkv + (int64_t)b * W;
  if (splits > 1) {
    // columns of heads [h0, h1) = bf16(sum over s of partial[s][b]), 4 per
    // thread, splits in order: what the split-K reduce would have written.
    for (int c = h0 * D + threadIdx.x * 4; c < h1 * D; c += 256 * 4) {
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      for (int sp = 0; sp < splits; ++sp) v += *(const f32x4 *)(partial + ((int64_t)sp * B + b) * W + c);
      u32x2 o;
      o[0] = pack2(v[0], v[1]);
      o[1] = pack2(v[2], v[3]);
      *(u32x2 *)(row + c) = o;
    }
    __syncthreads();  // the columns are read back below by other threads of this block
  }
  const int ctx = ctx_lens[b];
  if (ctx < 1) return;
  const int p = (ring > 0 ? ctx : min(ctx, max_pages * kPage)) - 1;
  const int half = D / 2, nvh = half / 8;

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
  // q and k heads of the group: rotate (if asked) 8 pairs per item; k heads also go to the cache
  const int qk0 = max(h0, do_rope ? 0 : n_q), qk1 = min(h1, n_q + n_kv);
  if (do_rope && qk0 < qk1) {
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
  const int items = max(0, qk1 - qk0) * nvh;
  for (int t = threadIdx.x; t < items; t += 256) {
    const int h = qk0 + t / nvh, i0 = (t % nvh) * 8;
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
  // v heads of the group: dim-major in the page, one element per store
  const int v0 = max(h0, n_q + n_kv);
  if (vbase && v0 < h1) {
    for (int t = threadIdx.x; t < (h1 - v0) * D; t += 256) {
      const int g = v0 - (n_q + n_kv) + t / D, i = t % D;
      vbase[g * blk + i * kPage + slot] = row[(int64_t)(v0 - (n_q + n_kv)) * D + (n_q + n_kv) * D + t];
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
                              hipStream_t s, const float *partial, int splits) {
  if (B <= 0) return hipSuccess;
  const int groups = (n_q + 2 * n_kv + kRopeHeads - 1) / kRopeHeads;
  hipLaunchKernelGGL(rope_append_kernel, dim3(B, groups), dim3(256), 0, s, qkv, n_q, n_kv, D, theta, ctx_lens,
                     page_table, max_pages, ring, pool, pool_pages, (int)do_rope, (int)do_append, partial,
                     partial ? splits : 1, B);
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
