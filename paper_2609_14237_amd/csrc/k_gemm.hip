// bf16 MFMA GEMM for the decode projections, the SwiGLU FFN and the grouped
// expert GEMMs: C[m, n] = sum_k A[m, k] * B[n, k] (both operands K-contiguous,
// "out x in" weights), fp32 accumulation, fused epilogues.
//
// Tiling: 256 threads = 4 waves; block tile BM x BN outputs, K step BK; LDS
// double buffering (global loads of step k+1 are in flight while step k runs
// on the matrix cores). Decode GEMMs are weight-streaming (M <= 64 rows against
// megabytes of weights), so the tile covers all rows it can and narrow outputs
// are split along K to keep every compute unit streaming. Dense GEMMs past 128
// rows, those of 33 to 64 rows but the SiLU-gated one, and the grouped expert
// GEMMs with K % 64 = 0 go to the direct-to-LDS streaming kernel
// (k_gemm_stream.hip); the large-M kernel here takes 64 < M <= 128 and the
// grouped GEMMs with other K. MFMA 16x16x32 bf16: lane l holds A[m = l%16][8 k's
// starting at (l/16)*8] and B[same k's][n = l%16]; the 16x16 fp32 result puts
// rows (l/16)*4 .. +3 of column l%16 in lane l.
#include "common.hpp"
#include "kernels.hpp"

namespace ods {

namespace {

template <int BM, int BN, int BK, int WM, int WN, int EPI, bool PARTIAL>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs p) {
  constexpr int LDS_STRIDE = BK + 8;  // elements; 16-byte row pad against bank conflicts
  constexpr bool SILU = EPI == EPI_SILU;
  constexpr int BNL = SILU ? 2 * BN : BN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int NB = SILU ? 2 * TN : TN;  // B fragments (gate then up) per wave
  constexpr int CPR = BK / 8;  // 16-byte chunks per tile row
  constexpr int A_CHUNKS = BM * CPR / 256;
  constexpr int B_CHUNKS = BNL * CPR / 256;
  static_assert(WM * WN == 4, "4 waves");
  static_assert(A_CHUNKS * 256 == BM * CPR && B_CHUNKS * 256 == BNL * CPR, "tile");

  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  uint16_t(*As)[BM * LDS_STRIDE] = (uint16_t(*)[BM * LDS_STRIDE])smem;
  uint16_t(*Bs)[BNL * LDS_STRIDE] = (uint16_t(*)[BNL * LDS_STRIDE])(smem + 2 * BM * LDS_STRIDE);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform
  const int wm = wave / WN, wn = wave % WN;
  const int n0 = blockIdx.x * BN;

  const int m_begin = 0, m_end = p.M;
  const uint16_t *Bg = p.B;
  int k_begin = 0, k_end = p.K;
  int split = 0;
  if (PARTIAL) {
    split = blockIdx.z;
    const int steps = (p.K + BK - 1) / BK;
    const int per = (steps + p.splits - 1) / p.splits;
    k_begin = split * per * BK;
    k_end = min(p.K, k_begin + per * BK);
  }
  if (k_begin >= k_end && !PARTIAL) return;

  // Global row of each B-tile row this thread loads (-1: outside N).
  int64_t b_row_off[B_CHUNKS];
#pragma unroll
  for (int i = 0; i < B_CHUNKS; ++i) {
    const int r = (tid + i * 256) / CPR;
    int n, row;
    if (SILU) {
      n = n0 + (r % BN);
      row = (r < BN) ? n : p.n_up + n;
    } else {
      n = n0 + r;
      row = n;
    }
    b_row_off[i] = (n < p.N) ? (int64_t)row * p.ldb : -1;
  }

  for (int m0 = m_begin + blockIdx.y * BM; m0 < m_end; m0 += gridDim.y * BM) {
    f32x4 acc[TM][NB];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    u32x4 ra[A_CHUNKS], rb[B_CHUNKS];
    auto load = [&](int k0) {
#pragma unroll
      for (int i = 0; i < A_CHUNKS; ++i) {
        const int c = tid + i * 256, r = c / CPR, kc = (c % CPR) * 8;
        const int m = m0 + r, k = k0 + kc;
        ra[i] = (m < m_end && k < k_end) ? *(const u32x4 *)(p.A + (int64_t)m * p.lda + k)
                                         : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int i = 0; i < B_CHUNKS; ++i) {
        const int c = tid + i * 256, kc = (c % CPR) * 8;
        const int k = k0 + kc;
        rb[i] = (b_row_off[i] >= 0 && k < k_end)
                    ? __builtin_nontemporal_load((const u32x4 *)(Bg + b_row_off[i] + k))
                    : u32x4{0u, 0u, 0u, 0u};
      }
    };
    auto store = [&](int buf) {
#pragma unroll
      for (int i = 0; i < A_CHUNKS; ++i) {
        const int c = tid + i * 256, r = c / CPR, kc = (c % CPR) * 8;
        *(u32x4 *)&As[buf][r * LDS_STRIDE + kc] = ra[i];
      }
#pragma unroll
      for (int i = 0; i < B_CHUNKS; ++i) {
        const int c = tid + i * 256, r = c / CPR, kc = (c % CPR) * 8;
        *(u32x4 *)&Bs[buf][r * LDS_STRIDE + kc] = rb[i];
      }
    };

    const int nk = (k_end - k_begin + BK - 1) / BK;
    if (nk > 0) {
      load(k_begin);
      store(0);
    }
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      if (kt + 1 < nk) load(k_begin + (kt + 1) * BK);
#pragma unroll
      for (int ks = 0; ks < BK / 32; ++ks) {
        bf16x8 af[TM], bfr[NB];
        const int col = ks * 32 + (lane >> 4) * 8;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int r = wm * WTM + i * 16 + (lane & 15);
          af[i] = __builtin_bit_cast(bf16x8, *(const u32x4 *)&As[cur][r * LDS_STRIDE + col]);
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int jj = SILU ? (j % TN) : j;
          const int r = (SILU && j >= TN ? BN : 0) + wn * WTN + jj * 16 + (lane & 15);
          bfr[j] = __builtin_bit_cast(bf16x8, *(const u32x4 *)&Bs[cur][r * LDS_STRIDE + col]);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j) acc[i][j] = mfma_16x16x32(af[i], bfr[j], acc[i][j]);
      }
      if (kt + 1 < nk) store(cur ^ 1);
      __syncthreads();
    }

    // Epilogue: lane holds rows (lane>>4)*4 + e of column lane&15 of each 16x16 tile.
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = n0 + wn * WTN + j * 16 + (lane & 15);
        if (n >= p.N) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = m0 + wm * WTM + i * 16 + (lane >> 4) * 4 + e;
          if (m >= m_end) continue;
          const float v = acc[i][j][e];
          if (PARTIAL) {
            const int64_t ncols = SILU ? 2 * (int64_t)p.N : p.N;
            float *dst = p.partial + ((int64_t)split * p.M + m) * ncols;
            dst[n] = v;
            if (SILU) dst[p.N + n] = acc[i][TN + j][e];
          } else if (EPI == EPI_BF16) {
            ((uint16_t *)p.C)[(int64_t)m * p.ldc + n] = f2bf(v);
          } else if (EPI == EPI_F32) {
            ((float *)p.C)[(int64_t)m * p.ldc + n] = v;
          } else if (EPI == EPI_RESID) {
            uint16_t *c = (uint16_t *)p.C + (int64_t)m * p.ldc + n;
            *c = f2bf(bf2f(*c) + v);
          } else {  // SILU
            const float up = acc[i][TN + j][e];
            ((uint16_t *)p.C)[(int64_t)m * p.ldc + n] = f2bf(silu(v) * up);
          }
        }
      }
    }
  }
}

// Large-M variant (grouped expert GEMMs; dense GEMMs with 64 < M <= 128 or K
// not a multiple of 64): 512 threads = 8 waves as 4 (M) x 2 (N), block tile
// BM x BN with BN = 128 columns of B rows (SiLU: 64 gate + 64 up rows), wave
// tile (BM/4) x 64. The whole batch fits one or two M tiles, so the weights
// stream from HBM once. Pipeline: step k+1 arrives in registers while step k
// is on the matrix cores; its LDS stores are issued between the two MFMA
// halves of step k (into the buffer the previous barrier freed) so the LDS,
// matrix and load units overlap; one barrier per K step. A 128-row tile's
// LDS (74 KB) leaves room for two blocks per CU, so without split-K partials
// (whose extra addressing would spill) its registers are capped at 128 to let
// the second block in; a 256-row tile (110 KB) runs alone.
template <int BM, int EPI, bool PARTIAL>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(BM == 128 && !PARTIAL ? 4 : 2)))
void gemm_big_kernel(GemmArgs p) {
  constexpr int BK = 64, LS = BK + 8, CPR = BK / 8;
  constexpr bool SILU = EPI == EPI_SILU;
  constexpr int BNL = 128;                 // B-tile rows
  constexpr int BN = SILU ? 64 : 128;      // output columns per block
  constexpr int WTM = BM / 4, TM = WTM / 16;
  constexpr int TN = SILU ? 2 : 4;         // output n-tiles per wave
  constexpr int NB = SILU ? 4 : 4;         // B fragments per wave (gate+up for SiLU)
  constexpr int AC = BM * CPR / 512, BC = BNL * CPR / 512;
  static_assert(AC * 512 == BM * CPR && BC * 512 == BNL * CPR, "tile");
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  uint16_t *As = smem;
  uint16_t *Bs = smem + 2 * BM * LS;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int n0 = blockIdx.x * BN;
  int m_begin = 0, m_end = p.M;
  const uint16_t *Bg = p.B;
  if (p.group_off) {  // grouped (expert) GEMM: rows [off[g], off[g+1]) against weight slab g
    const int g = blockIdx.z;
    m_begin = max(0, p.group_off[g]);      // offsets come from device memory:
    m_end = min(p.M, p.group_off[g + 1]);  // never step outside the M rows
    Bg += (int64_t)g * p.b_group_stride;
  }
  int k_begin = 0, k_end = p.K, split = 0;
  if (PARTIAL) {
    split = blockIdx.z;
    const int steps = (p.K + BK - 1) / BK;
    const int per = (steps + p.splits - 1) / p.splits;
    k_begin = split * per * BK;
    k_end = min(p.K, k_begin + per * BK);
  }
  const int nk = max(0, (k_end - k_begin + BK - 1) / BK);

  // Sources of this thread's chunks; rows outside M / N read a valid row and are zeroed at the LDS store.
  const uint16_t *bsrc[BC];
  bool bok[BC];
#pragma unroll
  for (int i = 0; i < BC; ++i) {
    const int c = tid + i * 512, r = c / CPR;
    int n, row;
    if (SILU) {
      n = n0 + (r % BN);
      row = (r < BN) ? n : p.n_up + n;
    } else {
      n = n0 + r;
      row = n;
    }
    bok[i] = n < p.N;
    bsrc[i] = Bg + (int64_t)(bok[i] ? row : 0) * p.ldb + (c % CPR) * 8;
  }
  for (int m0 = m_begin + blockIdx.y * BM; m0 < m_end; m0 += gridDim.y * BM) {
  const uint16_t *asrc[AC];
  bool aok[AC];
#pragma unroll
  for (int i = 0; i < AC; ++i) {
    const int c = tid + i * 512, m = m0 + c / CPR;
    aok[i] = m < m_end;
    asrc[i] = p.A + (int64_t)(aok[i] ? m : m_begin) * p.lda + (c % CPR) * 8;
  }
  struct St {
    u32x4 a[AC];
    u32x4 b[BC];
  };
  auto issue = [&](St &S, int kt) {
    const int k0 = k_begin + min(kt, max(nk - 1, 0)) * BK;
#pragma unroll
    for (int i = 0; i < AC; ++i) {
      const int kc = ((tid + i * 512) % CPR) * 8;
      S.a[i] = *(const u32x4 *)(asrc[i] + (min(k0 + kc, p.K - 8) - kc));
    }
#pragma unroll
    for (int i = 0; i < BC; ++i) {
      const int kc = ((tid + i * 512) % CPR) * 8;
      S.b[i] = __builtin_nontemporal_load((const u32x4 *)(bsrc[i] + (min(k0 + kc, p.K - 8) - kc)));
    }
  };
  auto store = [&](const St &S, int kt, int buf) {
    const int k0 = k_begin + kt * BK;
#pragma unroll
    for (int i = 0; i < AC; ++i) {
      const int c = tid + i * 512, kc = (c % CPR) * 8;
      *(u32x4 *)&As[buf * BM * LS + (c / CPR) * LS + kc] =
          (aok[i] && k0 + kc < k_end) ? S.a[i] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < BC; ++i) {
      const int c = tid + i * 512, kc = (c % CPR) * 8;
      *(u32x4 *)&Bs[buf * BNL * LS + (c / CPR) * LS + kc] =
          (bok[i] && k0 + kc < k_end) ? S.b[i] : u32x4{0u, 0u, 0u, 0u};
    }
  };
  f32x4 acc[TM][NB];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // B-tile row of wave fragment j: SiLU pairs gate tile j with up tile j (rows + BN).
  auto brow = [&](int j) {
    if (SILU) return (j >= TN ? BN : 0) + wn * (BN / 2) + (j % TN) * 16;
    return wn * 64 + j * 16;
  };
  // Waves whose rows all lie past the end of the tile's rows (a short expert
  // group) skip the LDS reads and matrix work; the test is wave-uniform.
  const bool rows_live = m0 + wm * WTM < m_end;
  auto compute_ks = [&](int buf, int ks) {
    if (!rows_live) return;
    bf16x8 af[TM], bfr[NB];
    const int col = ks * 32 + (lane >> 4) * 8;
#pragma unroll
    for (int i = 0; i < TM; ++i)
      af[i] = __builtin_bit_cast(bf16x8, *(const u32x4 *)&As[buf * BM * LS + (wm * WTM + i * 16 + (lane & 15)) * LS + col]);
#pragma unroll
    for (int j = 0; j < NB; ++j)
      bfr[j] = __builtin_bit_cast(bf16x8, *(const u32x4 *)&Bs[buf * BNL * LS + (brow(j) + (lane & 15)) * LS + col]);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] = mfma_16x16x32(af[i], bfr[j], acc[i][j]);
  };
  auto step = [&](int buf, St &Rnext, int kt) {
    // buf holds step kt; Rnext holds step kt+1 (arriving); the other slot holds step kt+2
    compute_ks(buf, 0);
    store(Rnext, kt + 1, buf ^ 1);
    compute_ks(buf, 1);
    __syncthreads();
    issue(Rnext, kt + 3);
  };
  if (nk > 0) {
    St R0, R1;
    issue(R0, 0);
    issue(R1, 1);
    store(R0, 0, 0);
    __syncthreads();
    issue(R0, 2);
    for (int kt = 0; kt < nk; kt += 2) {
      step(0, R1, kt);
      if (kt + 1 < nk) step(1, R0, kt + 1);
    }
  }

  // Epilogue: lane holds rows (lane>>4)*4 + e of column lane&15 of each 16x16 tile.
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + (SILU ? wn * (BN / 2) + j * 16 : wn * 64 + j * 16) + (lane & 15);
      if (n >= p.N) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm * WTM + i * 16 + (lane >> 4) * 4 + e;
        if (m >= m_end) continue;
        const float v = acc[i][j][e];
        if (PARTIAL) {
          const int64_t ncols = SILU ? 2 * (int64_t)p.N : p.N;
          float *dst = p.partial + ((int64_t)split * p.M + m) * ncols;
          dst[n] = v;
          if (SILU) dst[p.N + n] = acc[i][TN + j][e];
        } else if (EPI == EPI_BF16) {
          ((uint16_t *)p.C)[(int64_t)m * p.ldc + n] = f2bf(v);
        } else if (EPI == EPI_F32) {
          ((float *)p.C)[(int64_t)m * p.ldc + n] = v;
        } else if (EPI == EPI_RESID) {
          uint16_t *c = (uint16_t *)p.C + (int64_t)m * p.ldc + n;
          *c = f2bf(bf2f(*c) + v);
        } else {
          ((uint16_t *)p.C)[(int64_t)m * p.ldc + n] = f2bf(silu(v) * acc[i][TN + j][e]);
        }
      }
    }
  }
  __syncthreads();  // the next M tile reuses the LDS buffers
  }
}

// Sum split-K partials and apply the epilogue, 4 outputs per thread (N % 4 == 0).
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs p) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)p.M * p.N;
  if (q * 4 >= total) return;
  const int m = (int)(q * 4 / p.N), n = (int)(q * 4 % p.N);
  const int64_t ncols = EPI == EPI_SILU ? 2 * (int64_t)p.N : p.N;
  f32x4 v = {0.f, 0.f, 0.f, 0.f}, up = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < p.splits; ++s) {
    const float *row = p.partial + ((int64_t)s * p.M + m) * ncols;
    v += *(const f32x4 *)(row + n);
    if (EPI == EPI_SILU) up += *(const f32x4 *)(row + p.N + n);
  }
  if (EPI == EPI_F32) {
    *(f32x4 *)((float *)p.C + (int64_t)m * p.ldc + n) = v;
    return;
  }
  uint16_t *c = (uint16_t *)p.C + (int64_t)m * p.ldc + n;
  if (EPI == EPI_RESID) {
    const u32x2 old = *(const u32x2 *)c;
    v[0] += bf_lo(old[0]);
    v[1] += bf_hi(old[0]);
    v[2] += bf_lo(old[1]);
    v[3] += bf_hi(old[1]);
  } else if (EPI == EPI_SILU) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = silu(v[e]) * up[e];
  }
  u32x2 o;
  o[0] = pack2(v[0], v[1]);
  o[1] = pack2(v[2], v[3]);
  *(u32x2 *)c = o;
}

constexpr int kBM = kDecodeBM, kBK = kDecodeBK;

size_t lds_bytes(int BM, int BN, int BK, bool silu) { return (size_t)2 * (BM + (silu ? 2 : 1) * BN) * (BK + 8) * 2; }

template <int BM, int BN, int BK, int EPI, bool PARTIAL>
hipError_t launch_tile(const GemmArgs &a, dim3 grid, hipStream_t s) {
  auto kern = gemm_kernel<BM, BN, BK, 2, 2, EPI, PARTIAL>;
  const size_t lds = lds_bytes(BM, BN, BK, EPI == EPI_SILU);
  static std::atomic<uint64_t> lds_set{0};  // devices whose limit this kernel already raised
  if (hipError_t e = ensure_lds_limit((const void *)kern, lds, lds_set); e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, grid, dim3(256), lds, s, a);
  return hipGetLastError();
}

template <int BM, int EPI, bool PARTIAL>
hipError_t launch_big(const GemmArgs &a, dim3 grid, hipStream_t s) {
  auto kern = gemm_big_kernel<BM, EPI, PARTIAL>;
  const size_t lds = (size_t)2 * (BM + 128) * (64 + 8) * 2;
  static std::atomic<uint64_t> lds_set{0};  // devices whose limit this kernel already raised
  if (hipError_t e = ensure_lds_limit((const void *)kern, lds, lds_set); e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, grid, dim3(512), lds, s, a);
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_epi(const GemmArgs &a, hipStream_t s) {
  const int bn = tile_n(a.N, a.K, EPI);
  const int n_tiles = (a.N + bn - 1) / bn;
  if (a.b_tiled) return launch_gemm_stream(a, s);  // tiled weights: K % 64 == 0 by contract
  if (a.a_gather && !(a.group_off && a.K % 64 == 0)) return hipErrorInvalidValue;  // only the streaming kernel gathers
  if (a.group_off) {
    // Expert row groups average B*k/E rows (64 at the MoE workload). The
    // streaming kernel takes them when K is a whole number of 64-wide steps
    // (one block per N tile and expert, the expert's rows in 64- or 256-row
    // tiles).
    if (a.K % 64 == 0) {
      GemmArgs g = a;
      g.splits = 1;
      return launch_gemm_stream(g, s);
    }
    // Otherwise a 128-row large-M tile covers a whole group, so each expert's
    // weights stream once, and 128 weight rows per block keep the re-reads of
    // the group's activations to one per 128 output columns.
    const int bnb = EPI == EPI_SILU ? 64 : 128;
    dim3 grid((a.N + bnb - 1) / bnb, 1, a.groups);
    return launch_big<128, EPI, false>(a, grid, s);
  }
  const bool part = a.splits > 1;
  hipError_t e;
  if (gemm_use_stream(a.M, a.N, a.K, EPI)) return launch_gemm_stream(a, s);  // launches its own reduce
  if (use_big(a.M, a.N)) {
    const int bm = a.M > 128 ? 256 : 128;
    const int bnb = EPI == EPI_SILU ? 64 : 128;
    dim3 grid((a.N + bnb - 1) / bnb, (a.M + bm - 1) / bm, part ? a.splits : 1);
    if (bm == 256)
      e = part ? launch_big<256, EPI, true>(a, grid, s) : launch_big<256, EPI, false>(a, grid, s);
    else
      e = part ? launch_big<128, EPI, true>(a, grid, s) : launch_big<128, EPI, false>(a, grid, s);
  } else {
  const int m_tiles = (a.M + kBM - 1) / kBM;
  dim3 grid(n_tiles, m_tiles, part ? a.splits : 1);
  if (bn == 32)
    e = part ? launch_tile<kBM, 32, kBK, EPI, true>(a, grid, s) : launch_tile<kBM, 32, kBK, EPI, false>(a, grid, s);
  else
    e = part ? launch_tile<kBM, 64, kBK, EPI, true>(a, grid, s) : launch_tile<kBM, 64, kBK, EPI, false>(a, grid, s);
  }
  if (e != hipSuccess || !part || a.defer_reduce) return e;
  return launch_splitk_reduce(a, s);
}

}  // namespace

hipError_t launch_splitk_reduce(const GemmArgs &a, hipStream_t s) {
  const int64_t quads = (int64_t)a.M * a.N / 4;
  const dim3 grid((unsigned)((quads + 255) / 256));
  switch (a.epi) {
    case EPI_BF16: hipLaunchKernelGGL((splitk_reduce_kernel<EPI_BF16>), grid, dim3(256), 0, s, a); break;
    case EPI_F32: hipLaunchKernelGGL((splitk_reduce_kernel<EPI_F32>), grid, dim3(256), 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((splitk_reduce_kernel<EPI_RESID>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((splitk_reduce_kernel<EPI_SILU>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  switch (a.epi) {
    case EPI_BF16: return launch_epi<EPI_BF16>(a, s);
    case EPI_F32: return launch_epi<EPI_F32>(a, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, s);
    default: return launch_epi<EPI_SILU>(a, s);
  }
}

}  // namespace ods
