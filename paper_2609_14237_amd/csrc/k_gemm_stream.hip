// Weight-streaming bf16 MFMA GEMM for M > 128 rows (the 256-row decode batch,
// the 512-row MoE attention projections, larger prefill-sized batches), for
// 33 to 64 rows outside the SiLU-gated FFN GEMM, and for the grouped expert
// GEMMs (any rows per group), and for every GEMM on tiled weights (B stored
// as the LDS image of each K step's tile, read as one contiguous run per
// block): C[m, n] = sum_k A[m, k] * B[n, k] with the same epilogues as the
// other GEMM kernels. Built on its own with MFMA results in
// VGPRs (build.py passes -amdgpu-mfma-vgpr-form for this file only), which
// keeps the accumulators in place across the K loop.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace ods {

namespace {

constexpr int kNonTemporal = 2;  // cache-policy operand of the direct-to-LDS load: nt
// Row pitch (floats) of the epilogue's LDS tile: 128 columns plus 4, so the
// four rows one fragment write touches fall in different banks.
constexpr int kStageRow = 132;

// Three tile shapes (K % 64 == 0), all with two waves per SIMD and 128 rows
// of B per block (SiLU: 64 gate + 64 up rows, each wave taking the gate and
// up rows of the same output columns, so both halves of a column meet in one
// lane). MG = 4: 512 threads = 8 waves as 4 (M) x 2 (N) over a 256-row tile of
// A, three K steps of LDS (144 KB), one block per CU. MG = 2: 256 threads =
// 4 waves as 2 x 2 over a 128-row tile, two K steps (64 KB), two blocks per
// CU. MG = 1: 256 threads = 4 waves as 1 x 4 over a 64-row tile, three K
// steps (72 KB), two blocks per CU. Wave (wm, wn) computes rows
// [64 wm, 64 wm + 64) against its 128 / WN rows of B.
//
// Both operands go from global memory straight into LDS (direct-to-LDS loads:
// no registers and no LDS store instructions), eight lanes per 128-byte row
// segment so every load reads whole cache lines. A load writes its 64 lanes'
// 16 bytes in lane order; choosing which chunk each lane fetches XOR-swizzles
// the chunks of each row by row index, so the MFMA fragment reads are
// conflict-free. A rows land in an area per M group (shared by that group's
// waves), B rows in an area all waves share; both are rings of NSLOT K steps,
// filled NSLOT - 1 steps ahead. Two waves per SIMD matter: one wave per SIMD
// draws about 25 B/clk from LDS, two about 50, and each wave reads 16 KB
// (MG = 4, 2) or 12 KB (MG = 1) of fragments per K step.
//
// Synchronisation is explicit: the only vector-memory instructions in the
// loop are these loads (one event type, completed in order), so at the top of
// step t "vmcnt <= loads of NSLOT - 2 steps" means this wave's loads of step
// t + 1 have landed, and the barrier that follows publishes every wave's
// share. The loads of step t + NSLOT are issued after that barrier, into the
// slot of step t, whose fragments are in registers by then. The barrier is a
// bare s_barrier (the workgroup fence of __syncthreads would wait for every
// load in flight).
//
// Blocks are placed so that the compute units of one XCD share a K range
// (split-K) and the M tiles of one weight slab run on one XCD at the same
// time, so A slices and weight slabs are served by that XCD's L2. This file
// is built with MFMA results in VGPRs, which keeps the accumulators in place.
// MG = 64-row M groups per block (4, 2 or 1, above); NSLOT = K steps of LDS.
template <int MG, int NSLOT, int EPI, bool PARTIAL>
__global__ __launch_bounds__(MG == 4 ? 512 : 256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_stream_kernel(GemmArgs p, int n_tiles, int m_tiles) {
  constexpr int BK = 64, BNR = 128;
  constexpr int WN = MG == 1 ? 4 : 2, WAVES = MG * WN, BM = 64 * MG;
  constexpr bool SILU = EPI == EPI_SILU;
  constexpr int BN = SILU ? BNR / 2 : BNR;  // output columns per block
  constexpr int TN = 8 / WN;                // B fragments per wave and K half
  constexpr int AL = 8 / WN, BL = 16 / WAVES;
  constexpr int LOADS = AL + BL;            // loads per wave per step: its part of an M group's A and of B
  constexpr int BSTAGE = BNR * BK * 2;      // bytes of one B tile (16 KB)
  constexpr int ASTAGE = 64 * BK * 2;       // bytes of one M group's A tile (8 KB)
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];  // B slots, then A slots per M group

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  uint8_t *const lds_b = (uint8_t *)smem;
  uint8_t *const lds_a = lds_b + NSLOT * BSTAGE + wm * NSLOT * ASTAGE;

  // The block's task: an N tile, a K range and the rows [m_first, m_last).
  int nt, split = 0, m_first, m_last;
  const uint16_t *Bg = p.B;
  if (p.group_off) {
    // Grouped (expert) GEMM: block (N tile, group g) over the group's rows,
    // whatever their count, against weight slab g (no split-K).
    nt = blockIdx.x;
    const int gi = blockIdx.y;
    m_first = max(0, p.group_off[gi]);      // offsets come from device memory:
    m_last = min(p.M, p.group_off[gi + 1]);  // never step outside the M rows
    Bg += (int64_t)gi * p.b_group_stride;
    if (m_first >= m_last) return;
  } else {
    // Blocks are dispatched to the 8 XCDs round-robin by index.
    const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
    const int g = 8 / p.splits;  // XCDs per K range
    split = xcd / g;
    const int mt = j % m_tiles;
    nt = (j / m_tiles) * g + xcd % g;
    if (nt >= n_tiles) return;
    m_first = mt * BM;
    m_last = min(p.M, m_first + BM);
  }
  const int n0 = nt * BN;
  // When a weight tile is read by exactly one block, once (a dense GEMM with
  // one M tile, an expert whose rows fit one tile), its loads carry the
  // non-temporal policy, so the weight stream does not evict the activation
  // rows every block re-reads (B = 64: gate_up 43 -> 40 us, down 27.5 -> 26
  // us). Weight tiles shared by the M tiles of one XCD keep the default
  // policy (the L2 serves their re-reads), and so do the split-K blocks of
  // the 256-row tile, which measured slower with it (down at B = 256: 34 ->
  // 46 us).
  const bool b_once = (MG == 1 || p.splits == 1) && (p.group_off ? m_last - m_first <= BM : m_tiles == 1);
  // The staged epilogue stores whole 16-byte chunks: every chunk must lie
  // inside or outside the output columns, and start 16-byte aligned.
  constexpr int VEC_W = PARTIAL || EPI == EPI_F32 ? 4 : 8;  // outputs per chunk
  const int n_lim = !SILU && p.b_tiled && p.n_up > 0 ? p.n_up : p.N;
  const bool vec = p.N % VEC_W == 0 && n_lim % VEC_W == 0 &&
                   (PARTIAL ? ((uintptr_t)p.partial & 15) == 0 : p.ldc % VEC_W == 0 && ((uintptr_t)p.C & 15) == 0);

  const int steps = p.K / BK;
  const int per = (steps + p.splits - 1) / p.splits;
  const int s_begin = split * per;
  const int nk = min(per, steps - s_begin);  // may be <= 0 for a trailing split: it writes zeros
  const int last = max(nk - 1, 0);

  // Load q fills LDS row 8q + lane / 8 of its tile, position lane % 8, with
  // chunk c = (lane % 8) ^ (row % 8) of that row, so chunk c of row r sits at
  // position c ^ (r % 8).
  const int chunk = ((lane & 7) ^ (lane >> 3)) * 8;
  // Tiled weights hold each step's tile as its LDS image, so load q of a wave
  // copies 1 KB of it verbatim: the block streams one contiguous run of its
  // N tile's K range instead of 128 separate rows.
  const uint16_t *bptr[BL];
  const int64_t bstep = p.b_tiled ? BNR * BK : BK;  // elements between consecutive K steps of a load
#pragma unroll
  for (int q = 0; q < BL; ++q) {
    if (p.b_tiled) {
      bptr[q] = Bg + ((int64_t)nt * steps + s_begin) * (BNR * BK) + (wave * BL + q) * 512 + lane * 8;
    } else {
      const int r = (wave * BL + q) * 8 + (lane >> 3);
      const int n = min(n0 + (SILU ? r % BN : r), p.N - 1);
      const int row = SILU && r >= BN ? p.n_up + n : n;
      bptr[q] = Bg + (int64_t)row * p.ldb + (int64_t)s_begin * BK + chunk;
    }
  }
  // Fragment read: row 16i + lane % 16, chunk 4 ks + lane / 16. B tile row of
  // fragment jt: SiLU takes gate rows (64 / WN) wn + 16 jt (jt < TN / 2) and the
  // matching up rows 64 + (64 / WN) wn + 16 (jt - TN / 2), so gate fragment jt
  // pairs with up fragment jt + TN / 2.
  const int rd_off0 = (lane & 15) * 128 + (((lane >> 4) ^ (lane & 7)) << 4);
  const int rd_off1 = (lane & 15) * 128 + (((4 + (lane >> 4)) ^ (lane & 7)) << 4);
  auto brow = [&](int jt) {
    return SILU ? (jt / (TN / 2)) * 64 + wn * (64 / WN) + (jt % (TN / 2)) * 16 : wn * (128 / WN) + jt * 16;
  };

  // Fragments of one K step: A row groups i and B fragments jt, both K halves.
  struct Frags {
    bf16x8 a[2][4], b[2][TN];
  };
  f32x4 acc[4][TN];

  for (int m0 = m_first; m0 < m_last; m0 += BM) {
    // A rows past the tile's last row re-read that row and are never stored.
    const uint16_t *aptr[AL];
#pragma unroll
    for (int q = 0; q < AL; ++q) {
      const int m = min(m0 + wm * 64 + (wn * AL + q) * 8 + (lane >> 3), m_last - 1);
      int64_t row = m;
      if (p.a_gather) row = min(max(p.a_gather[m] / p.a_gather_div, 0), p.a_gather_rows - 1);  // device data: clamp
      aptr[q] = p.A + row * p.lda + (int64_t)s_begin * BK + chunk;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jt = 0; jt < TN; ++jt) acc[i][jt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Waves whose 64 rows all lie past the tile's end (a short expert group)
    // only load their share of B; they issue fewer loads per step, so they
    // wait for their own count. Every wave passes the same barriers.
    const bool live = m0 + wm * 64 < m_last;
    auto pipeline = [&](auto live_c, auto nt_c) {
      constexpr bool LIVE = decltype(live_c)::value;
      constexpr bool NT = decltype(nt_c)::value;  // weight loads with the non-temporal policy
      constexpr int LW = LIVE ? LOADS : BL;  // loads per step of this wave
      auto issue = [&](int t, int slot) {
        const int64_t k = (int64_t)t * BK;  // t <= last
        if (LIVE) {
#pragma unroll
          for (int q = 0; q < AL; ++q)
            __builtin_amdgcn_global_load_lds(
                (const void *)(aptr[q] + k),
                (__attribute__((address_space(3))) void *)(lds_a + slot * ASTAGE + (wn * AL + q) * 1024), 16, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < BL; ++q)
          __builtin_amdgcn_global_load_lds(
              (const void *)(bptr[q] + t * bstep),
              (__attribute__((address_space(3))) void *)(lds_b + slot * BSTAGE + (wave * BL + q) * 1024), 16, 0,
              NT ? kNonTemporal : 0);
      };
      auto read_frags = [&](Frags &f, int slot) {
        const uint8_t *as = lds_a + slot * ASTAGE, *bs = lds_b + slot * BSTAGE;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int off = ks ? rd_off1 : rd_off0;
#pragma unroll
          for (int i = 0; i < 4; ++i) f.a[ks][i] = __builtin_bit_cast(bf16x8, *(const u32x4 *)(as + i * 2048 + off));
#pragma unroll
          for (int jt = 0; jt < TN; ++jt)
            f.b[ks][jt] = __builtin_bit_cast(bf16x8, *(const u32x4 *)(bs + brow(jt) * 128 + off));
        }
      };
      auto mma = [&](const Frags &f) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int jt = 0; jt < TN; ++jt) acc[i][jt] = mfma_16x16x32(f.a[ks][i], f.b[ks][jt], acc[i][jt]);
      };
      // Step t runs its MFMAs on fragments read during step t - 1, reads the
      // fragments of step t + 1, and refills the slot of step t (free once its
      // fragments are in registers) with the loads of step t + NSLOT.
      issue(0, 0);
#pragma unroll
      for (int s = 1; s < NSLOT; ++s) issue(min(s, last), s);
      Frags f0, f1;
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"((NSLOT - 1) * LW) : "memory");
      __builtin_amdgcn_sched_barrier(0);
      if (LIVE) read_frags(f0, 0);
      int slot = 0;  // slot of step t
      auto step = [&](int t, const Frags &cur, Frags &nxt) {
        // Loads of step t + 1 have landed once only those of the NSLOT - 2
        // steps after it are outstanding; lgkmcnt(0) retires this wave's
        // reads of slot t (issued a step ago) before the barrier lets step
        // t + NSLOT overwrite it.
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"((NSLOT - 2) * LW) : "memory");
        __builtin_amdgcn_sched_barrier(0);
        const int s1 = slot == NSLOT - 1 ? 0 : slot + 1;
        issue(min(t + NSLOT, last), slot);
        if (LIVE) {
          read_frags(nxt, s1);
          mma(cur);
          // Interleave one global load per MFMA, then one fragment read per
          // MFMA, then the rest of the MFMAs. Loads issued in one burst by all
          // eight waves back up the address unit and stall the issuing waves;
          // reads issued in one burst ahead of the MFMAs make the compiler
          // drain them all (lgkmcnt counts only to 15) before the first MFMA.
          constexpr int NM = 8 * TN, NR = 8 + 2 * TN;  // MFMAs and fragment reads per step
          constexpr int NMR = NR < NM - LOADS ? NR : NM - LOADS;
#pragma unroll
          for (int k = 0; k < LOADS; ++k) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
          }
#pragma unroll
          for (int k = 0; k < NMR; ++k) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          if (NM - LOADS - NMR > 0) __builtin_amdgcn_sched_group_barrier(0x008, NM - LOADS - NMR, 0);
        }
        slot = s1;
      };
      int t = 0;
      for (; t + 2 <= nk; t += 2) {
        step(t, f0, f1);
        step(t + 1, f1, f0);
      }
      if (t < nk) step(t, f0, f1);
      // Nothing may still be reading the LDS slots when they are reused or the block retires.
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    };
    if (nk > 0) {
      if (live) {
        if (b_once) pipeline(std::true_type{}, std::true_type{});
        else pipeline(std::true_type{}, std::false_type{});
      } else {
        if (b_once) pipeline(std::false_type{}, std::true_type{});
        else pipeline(std::false_type{}, std::false_type{});
      }
    }
    // Epilogue: lane holds rows (lane >> 4) * 4 + e of column lane & 15 of each 16x16 tile.
    // A plain epilogue over gated tiles maps tile row rr to gate column
    // 64 nt + rr (rr < 64) or up column n_up + 64 nt + rr - 64.
    constexpr int TO = SILU ? TN / 2 : TN;  // output fragments (SiLU pairs gate jt with up jt + TO)
    if (vec) {
      // Staged through LDS (the drained slots): every live wave writes its
      // fp32 results (SiLU: silu(gate) * up; SiLU partials: gate columns, then
      // up columns) into a row-major tile, and the whole block stores it as
      // 16-byte chunks, whole cache lines per row, instead of one 2- or 4-byte
      // store per lane and value. The arithmetic is the scalar path's.
      float *stage = (float *)smem;
      if (live) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int jt = 0; jt < TO; ++jt) {
            const int col = (SILU ? wn * (64 / WN) : wn * (128 / WN)) + jt * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float *row = stage + (wm * 64 + i * 16 + (lane >> 4) * 4 + e) * kStageRow;
              if (SILU && !PARTIAL) {
                row[col] = silu(acc[i][jt][e]) * acc[i][jt + TO][e];
              } else {
                row[col] = acc[i][jt][e];
                if (SILU) row[64 + col] = acc[i][jt + TO][e];
              }
            }
          }
      }
      __syncthreads();
      constexpr bool F32OUT = PARTIAL || EPI == EPI_F32;
      constexpr int CW = F32OUT ? 4 : 8;                      // outputs per 16-byte chunk
      constexpr int CH = (SILU && !PARTIAL ? 64 : 128) / CW;  // chunks per tile row
      const bool gated_cols = !SILU && p.b_tiled && p.n_up > 0;
      const int rows = min(BM, m_last - m0);
      for (int idx = tid; idx < rows * CH; idx += WAVES * 64) {
        const int r = idx / CH, sc = (idx % CH) * CW, m = m0 + r;
        const float *src = stage + r * kStageRow + sc;
        int64_t dst;  // element offset of the chunk in C or in the partials
        if (PARTIAL) {
          const int64_t ncols = SILU ? 2 * (int64_t)p.N : p.N;
          int n;
          if (SILU) {
            n = n0 + (sc & 63);
            if (n >= p.N) continue;
            if (sc >= 64) n += p.N;
          } else if (gated_cols) {
            const int c = nt * 64 + (sc & 63);
            if (c >= p.n_up) continue;
            n = sc < 64 ? c : p.n_up + c;
          } else {
            n = n0 + sc;
            if (n >= p.N) continue;
          }
          dst = ((int64_t)split * p.M + m) * ncols + n;
          *(f32x4 *)(p.partial + dst) = *(const f32x4 *)src;
          continue;
        }
        int n;
        if (gated_cols) {
          const int c = nt * 64 + (sc & 63);
          if (c >= p.n_up) continue;
          n = sc < 64 ? c : p.n_up + c;
        } else {
          n = n0 + sc;
          if (n >= p.N) continue;
        }
        dst = (int64_t)m * p.ldc + n;
        if (EPI == EPI_F32) {
          *(f32x4 *)((float *)p.C + dst) = *(const f32x4 *)src;
          continue;
        }
        const f32x4 lo = *(const f32x4 *)src, hi = *(const f32x4 *)(src + 4);
        float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        uint16_t *c = (uint16_t *)p.C + dst;
        if (EPI == EPI_RESID) {
          const u32x4 old = *(const u32x4 *)c;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            v[2 * q] += bf_lo(old[q]);
            v[2 * q + 1] += bf_hi(old[q]);
          }
        }
        u32x4 out;
#pragma unroll
        for (int q = 0; q < 4; ++q) out[q] = pack2(v[2 * q], v[2 * q + 1]);
        *(u32x4 *)c = out;
      }
      __syncthreads();  // the stage is read before the next tile's loads refill the slots
      continue;
    }
    if (!live) continue;
    const bool gated_cols = !SILU && p.b_tiled && p.n_up > 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int jt = 0; jt < TO; ++jt) {
        const int rr = (SILU ? wn * (64 / WN) : wn * (128 / WN)) + jt * 16 + (lane & 15);
        int n = n0 + rr;
        if (gated_cols) {
          const int c = nt * 64 + (rr & 63);
          if (c >= p.n_up) continue;
          n = rr < 64 ? c : p.n_up + c;
        } else if (n >= p.N) {
          continue;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + e;
          if (m >= m_last) continue;
          const float v = acc[i][jt][e];
          if (PARTIAL) {
            const int64_t ncols = SILU ? 2 * (int64_t)p.N : p.N;
            float *dst = p.partial + ((int64_t)split * p.M + m) * ncols;
            dst[n] = v;
            if (SILU) dst[p.N + n] = acc[i][jt + TO][e];
          } else if (EPI == EPI_BF16) {
            ((uint16_t *)p.C)[(int64_t)m * p.ldc + n] = f2bf(v);
          } else if (EPI == EPI_F32) {
            ((float *)p.C)[(int64_t)m * p.ldc + n] = v;
          } else if (EPI == EPI_RESID) {
            uint16_t *c = (uint16_t *)p.C + (int64_t)m * p.ldc + n;
            *c = f2bf(bf2f(*c) + v);
          } else {
            ((uint16_t *)p.C)[(int64_t)m * p.ldc + n] = f2bf(silu(v) * acc[i][jt + TO][e]);
          }
        }
      }
    }
  }
}

template <int MG, int NSLOT, int EPI, bool PARTIAL>
hipError_t launch_stream(const GemmArgs &a, hipStream_t s) {
  constexpr int BN = EPI == EPI_SILU ? 64 : 128;
  const int n_tiles = (a.N + BN - 1) / BN, m_tiles = (a.M + 64 * MG - 1) / (64 * MG);
  const int g = 8 / a.splits;  // splits is 1, 2, 4 or 8 (gemm_stream_splits)
  // dense: a 1-D grid placed on the XCDs; grouped: (N tile, group)
  const dim3 grid = a.group_off ? dim3(n_tiles, a.groups) : dim3(8 * m_tiles * ((n_tiles + g - 1) / g));
  auto kern = gemm_stream_kernel<MG, NSLOT, EPI, PARTIAL>;
  // per slot: B tile + A tile per M group; at least the epilogue's fp32 tile
  const size_t lds = std::max<size_t>((size_t)NSLOT * (128 * 64 * 2 + MG * 64 * 64 * 2), (size_t)64 * MG * kStageRow * 4);
  static std::atomic<uint64_t> lds_set{0};  // devices whose limit this kernel already raised
  if (hipError_t e = ensure_lds_limit((const void *)kern, lds, lds_set); e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, grid, dim3(MG == 4 ? 512 : 256), lds, s, a, n_tiles, m_tiles);
  return hipGetLastError();
}

// Tile shapes. Dense GEMMs: 64-row tiles (two blocks per CU) up to 64 rows,
// 256-row tiles past that (at 96 and 128 rows the 256-row tile with idle
// waves beats the 128-row one on every 8B-shaped GEMM, by 3-14 us), except
// where the 256-row grid would leave most compute units idle
// (gemm_stream_rows: 64-row tiles again). Grouped
// (expert) GEMMs, by the average rows per group:
//  - up to 32: 64-row tiles;
//  - up to 96: 128-row tiles (two blocks per CU on a two-slot ring), which
//    cover nearly every group in one pass while one block's start and end
//    overlap the other's stream (top-8 of 64 experts, expert width 1536:
//    down 182-185 -> 166 us and gate_up 287-295 -> 283 us at 64 rows per
//    expert, 199 -> 175 and 312 -> 295 us at 96);
//  - more: 256-row tiles (a 128-row tile would stream the weights of every
//    group past 128 rows twice: at 128 rows per expert 237 against 209 us for
//    down).
enum StreamTile { TILE_64 = 0, TILE_128 = 1, TILE_256 = 2 };
StreamTile gemm_stream_tile(const GemmArgs &a) {
  if (a.group_off) {
    if (a.groups <= 0 || a.M <= 32 * a.groups) return TILE_64;
    return a.M <= 96 * a.groups ? TILE_128 : TILE_256;
  }
  return gemm_stream_rows(a.M, a.N, a.K, a.epi) == 64 ? TILE_64 : TILE_256;
}

template <int MG, int NSLOT, int EPI>
hipError_t launch_part(const GemmArgs &a, hipStream_t s) {
  return a.splits > 1 ? launch_stream<MG, NSLOT, EPI, true>(a, s) : launch_stream<MG, NSLOT, EPI, false>(a, s);
}

template <int EPI>
hipError_t launch_epi(const GemmArgs &a, hipStream_t s) {
  hipError_t e;
  switch (gemm_stream_tile(a)) {
    case TILE_64: e = launch_part<1, 3, EPI>(a, s); break;
    case TILE_128: e = launch_part<2, 2, EPI>(a, s); break;
    default: e = launch_part<4, 3, EPI>(a, s); break;
  }
  if (e != hipSuccess || a.splits <= 1 || a.defer_reduce) return e;
  return launch_splitk_reduce(a, s);
}

// One thread per 16-byte chunk of the tiled weight (the order tile_weight
// documents); rows past `out` are written as zeros.
__global__ __launch_bounds__(256) void tile_weight_kernel(const uint16_t *__restrict__ src,
                                                          uint16_t *__restrict__ dst, int out, int in, int gated,
                                                          int n_tiles, int64_t n_chunks) {
  const int ks = in / 64;
  const int64_t src_rows = gated ? 2 * (int64_t)out : out;
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < n_chunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int pos = (int)(c & 7);
    const int r = (int)((c >> 3) & 127);
    const int64_t tile = c >> 10;  // (slab * n_tiles + nt) * ks + s
    const int s = (int)(tile % ks);
    const int64_t st = tile / ks;
    const int nt = (int)(st % n_tiles);
    const int64_t slab = st / n_tiles;
    const int n = gated ? nt * 64 + (r & 63) : nt * 128 + r;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (n < out) {
      const int64_t row = slab * src_rows + (gated && r >= 64 ? out + n : n);
      v = *(const u32x4 *)(src + row * in + s * 64 + ((pos ^ (r & 7)) << 3));
    }
    *(u32x4 *)(dst + c * 8) = v;
  }
}

}  // namespace

hipError_t launch_tile_weight(const uint16_t *src, uint16_t *dst, int out, int in, bool gated, int groups,
                              hipStream_t s) {
  const int n_tiles = gated ? (out + 63) / 64 : (out + 127) / 128;
  const int64_t n_chunks = tiled_weight_elems(out, in, gated, groups) / 8;
  const int64_t blocks = std::min<int64_t>((n_chunks + 255) / 256, 65536);
  hipLaunchKernelGGL(tile_weight_kernel, dim3((unsigned)blocks), dim3(256), 0, s, src, dst, out, in, gated ? 1 : 0,
                     n_tiles, n_chunks);
  return hipGetLastError();
}

hipError_t launch_gemm_stream(const GemmArgs &a, hipStream_t s) {
  if (a.splits != 1 && a.splits != 2 && a.splits != 4 && a.splits != 8) return hipErrorInvalidValue;
  if (a.group_off && (a.splits != 1 || a.groups <= 0)) return hipErrorInvalidValue;
  switch (a.epi) {
    case EPI_BF16: return launch_epi<EPI_BF16>(a, s);
    case EPI_F32: return launch_epi<EPI_F32>(a, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, s);
    default: return launch_epi<EPI_SILU>(a, s);
  }
}

}  // namespace ods
