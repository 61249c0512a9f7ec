// MoE routing and token permutation for the expert stage. In the paper's cost
// model only the routed experts count toward the activated parameters while
// every expert stays resident (Appendix A.4); these kernels turn per-token
// routing into contiguous per-expert row groups for the grouped GEMMs and
// scatter the expert outputs back. All integer outputs are deterministic.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace ods {

namespace {

// One wave per token: top-k of the fp32 logits (ties -> lower expert id), and
// softmax over the chosen k. E <= 256 (four logits per lane), k <= 64. With
// splits > 1 the token's logits are the sum of the router's split-K partials,
// added in split order as the reduce would, and are written to logits_out.
__global__ __launch_bounds__(256) void topk_kernel(const float *__restrict__ logits, int B, int E, int k,
                                                   int32_t *__restrict__ ids, float *__restrict__ w,
                                                   const float *__restrict__ partial, int splits,
                                                   float *__restrict__ logits_out) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  float v[4];
  bool taken[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + 64 * j;
    taken[j] = e >= E;
    if (e >= E) {
      v[j] = -INFINITY;
    } else if (splits > 1) {
      float t = 0.f;
      for (int sp = 0; sp < splits; ++sp) t += partial[((int64_t)sp * B + b) * E + e];
      v[j] = t;
      logits_out[(int64_t)b * E + e] = t;
    } else {
      v[j] = logits[(int64_t)b * E + e];
    }
  }
  float z0 = 0.f, sum = 0.f, my_z = 0.f;
  int my_i = 0;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane + 64 * j;
      if (!taken[j] && (v[j] > bv || (v[j] == bv && e < bi))) {
        bv = v[j];
        bi = e;
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float ov = __shfl_xor(bv, o, kWave);
      const int oi = __shfl_xor(bi, o, kWave);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (lane + 64 * j == bi) taken[j] = true;
    if (r == 0) z0 = bv;
    sum += __expf(bv - z0);
    if (lane == r) {
      my_z = bv;
      my_i = bi;
    }
  }
  if (lane < k) {
    ids[(int64_t)b * k + lane] = my_i;
    w[(int64_t)b * k + lane] = __expf(my_z - z0) / sum;
  }
}

// Stable counting sort of the n = B*k (token, slot) pairs by expert in one
// block of 16 waves. Pairs are taken in chunks of 64 (one per lane); wave w
// owns a contiguous run of chunks. Within a chunk, the lanes holding the same
// expert are found with one ballot per bit of the id, so a pair's rank among
// equal ids before it is a popcount and the group's lowest lane alone updates
// the shared counter. Pass 1 counts pairs per (expert, wave); an exclusive
// scan of those counts in expert-major order gives each wave's first slot in
// every expert's range; pass 2 places the pairs. Ids outside [0, E) are not
// placed and get slot_pos -1.
constexpr int kPermWaves = 16;

__device__ __forceinline__ uint64_t same_id_lanes(int e, int bits) {
  uint64_t m = ~0ull;
  for (int b = 0; b < bits; ++b) {
    const bool set = (e >> b) & 1;
    const uint64_t v = __ballot(set);
    m &= set ? v : ~v;
  }
  return m;
}

__global__ __launch_bounds__(64 * kPermWaves) void permute_kernel(const int32_t *__restrict__ ids, int n, int E,
                                                                 int32_t *__restrict__ perm,
                                                                 int32_t *__restrict__ slot_pos,
                                                                 int32_t *__restrict__ expert_off) {
  extern __shared__ uint32_t cnt[];  // [E][kPermWaves]: counts, then running slots
  __shared__ uint32_t wave_tot[kPermWaves];
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int chunks = (n + 63) / 64, per_wave = (chunks + kPermWaves - 1) / kPermWaves;
  const int c0 = min(chunks, w * per_wave), c1 = min(chunks, c0 + per_wave);
  int bits = 1;  // enough bits for the values 0..E (E marks an invalid id)
  while ((1 << bits) <= E) ++bits;
  const uint64_t below = (1ull << lane) - 1;
  for (int j = t; j < E * kPermWaves; j += blockDim.x) cnt[j] = 0;
  __syncthreads();
  for (int c = c0; c < c1; ++c) {
    const int i = c * 64 + lane;
    int e = i < n ? ids[i] : E;
    if ((unsigned)e >= (unsigned)E) e = E;
    const uint64_t same = same_id_lanes(e, bits);
    if (e < E && (same & below) == 0) cnt[e * kPermWaves + w] += (uint32_t)__popcll(same);
  }
  __syncthreads();
  // Exclusive scan over the E*16 counts; thread t scans a contiguous run.
  const int N = E * kPermWaves, per_t = (N + (int)blockDim.x - 1) / (int)blockDim.x;
  const int j0 = min(N, t * per_t), j1 = min(N, j0 + per_t);
  uint32_t local = 0;
  for (int j = j0; j < j1; ++j) local += cnt[j];
  uint32_t inc = local;
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(inc, d);
    if (lane >= d) inc += y;
  }
  if (lane == 63) wave_tot[w] = inc;
  __syncthreads();
  uint32_t run = inc - local, total = 0;
  for (int v = 0; v < kPermWaves; ++v) {
    const uint32_t x = wave_tot[v];
    if (v < w) run += x;
    total += x;
  }
  for (int j = j0; j < j1; ++j) {
    const uint32_t x = cnt[j];
    cnt[j] = run;
    run += x;
  }
  __syncthreads();
  for (int e = t; e < E; e += blockDim.x) expert_off[e] = (int32_t)cnt[e * kPermWaves];
  if (t == 0) expert_off[E] = (int32_t)total;
  __syncthreads();  // the placement below advances the slots read above
  for (int c = c0; c < c1; ++c) {
    const int i = c * 64 + lane;
    int e = i < n ? ids[i] : E;
    if ((unsigned)e >= (unsigned)E) e = E;
    const uint64_t same = same_id_lanes(e, bits);
    if (i >= n) continue;
    if (e == E) {
      slot_pos[i] = -1;
      continue;
    }
    const uint32_t first = cnt[e * kPermWaves + w];
    const uint32_t pos = first + (uint32_t)__popcll(same & below);
    perm[pos] = i;
    slot_pos[i] = (int32_t)pos;
    if ((same & below) == 0) cnt[e * kPermWaves + w] = first + (uint32_t)__popcll(same);
  }
}

// dst[r] = src[perm[r] / k] for sorted rows r < expert_off[E]; rows past the end are zeroed.
__global__ __launch_bounds__(256) void gather_rows_kernel(const uint16_t *__restrict__ src,
                                                          const int32_t *__restrict__ perm, int k, int H,
                                                          const int32_t *__restrict__ valid_rows,
                                                          uint16_t *__restrict__ dst) {
  const int r = blockIdx.x;
  const int nvec = H / 8;
  u32x4 *d = (u32x4 *)(dst + (int64_t)r * H);
  if (r >= min((int)gridDim.x, *valid_rows)) {
    for (int v = threadIdx.x; v < nvec; v += 256) d[v] = u32x4{0u, 0u, 0u, 0u};
    return;
  }
  const int pr = perm[r];
  if (pr < 0 || pr >= gridDim.x) {  // perm comes from device memory
    for (int v = threadIdx.x; v < nvec; v += 256) d[v] = u32x4{0u, 0u, 0u, 0u};
    return;
  }
  const u32x4 *s = (const u32x4 *)(src + (int64_t)(pr / k) * H);
  for (int v = threadIdx.x; v < nvec; v += 256) d[v] = s[v];
}

// resid[b] = bf16(resid[b] + sum_j w[b, j] * yp[slot_pos[b*k + j]]), fp32 accumulation.
__global__ __launch_bounds__(256) void moe_combine_kernel(const uint16_t *__restrict__ yp,
                                                          const float *__restrict__ w,
                                                          const int32_t *__restrict__ slot_pos, int k, int H,
                                                          int n_rows, uint16_t *__restrict__ resid) {
  const int b = blockIdx.x;
  const int nvec = H / 8;
  u32x4 *r = (u32x4 *)(resid + (int64_t)b * H);
  for (int v = threadIdx.x; v < nvec; v += 256) {
    float acc[8];
    const u32x4 x = r[v];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc[2 * j] = 0.f;
      acc[2 * j + 1] = 0.f;
    }
    for (int j = 0; j < k; ++j) {
      const int pos = slot_pos[(int64_t)b * k + j];
      if (pos < 0 || pos >= n_rows) continue;
      const float wj = w[(int64_t)b * k + j];
      const u32x4 y = *((const u32x4 *)(yp + (int64_t)pos * H) + v);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += wj * bf_lo(y[q]);
        acc[2 * q + 1] += wj * bf_hi(y[q]);
      }
    }
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = pack2(bf_lo(x[q]) + acc[2 * q], bf_hi(x[q]) + acc[2 * q + 1]);
    r[v] = o;
  }
}

}  // namespace

hipError_t launch_topk(const float *logits, int B, int E, int k, int32_t *ids, float *w, hipStream_t s,
                       const float *partial, int splits, float *logits_out) {
  if (B <= 0) return hipSuccess;
  if (splits > 1 && (!partial || !logits_out)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(topk_kernel, dim3((B + 3) / 4), dim3(256), 0, s, logits, B, E, k, ids, w, partial,
                     splits > 1 ? splits : 1, logits_out);
  return hipGetLastError();
}

hipError_t launch_permute(const int32_t *ids, int B, int k, int E, int32_t *perm, int32_t *slot_pos,
                          int32_t *expert_off, hipStream_t s) {
  const int n = B * k;
  const size_t lds = (size_t)E * kPermWaves * sizeof(uint32_t);  // 16 KiB at E = 256
  hipLaunchKernelGGL(permute_kernel, dim3(1), dim3(64 * kPermWaves), lds, s, ids, n, E, perm, slot_pos,
                     expert_off);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const uint16_t *src, const int32_t *perm, const int32_t *valid_rows,
                                  int rows, int k, int H, uint16_t *dst, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(rows), dim3(256), 0, s, src, perm, k, H, valid_rows, dst);
  return hipGetLastError();
}

hipError_t launch_moe_combine(const uint16_t *yp, const float *w, const int32_t *slot_pos, int B, int k,
                              int H, uint16_t *resid, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(moe_combine_kernel, dim3(B), dim3(256), 0, s, yp, w, slot_pos, k, H, B * k, resid);
  return hipGetLastError();
}

}  // namespace ods
