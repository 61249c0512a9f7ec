// Paged GQA decode attention for gfx950.
//
// Decode attention is the memory-bound operator class of the paper's cost
// model (Appendix A.2): each decoded token reads its whole KV context once.
//
// Work split: the (sequence b, KV head g, page of b's attended window) units
// of the whole batch are numbered b-major, and wave r of the grid takes the
// contiguous unit range [r*S, (r+1)*S) with S = ceil(total / waves) (at least
// 8 pages), so every wave streams the same number of KV bytes however ragged
// the contexts are. A range may end inside a sequence or cover several short
// ones; each (b, g) piece is a segment. A sequence that one segment covers is
// written to o directly; otherwise every segment leaves a partial record
// (acc, running max, running sum) and a second kernel merges the records with
// their log-sum-exp weights. Each workgroup first builds the unit prefix over
// the batch in LDS from ctx_lens, so the split needs no host knowledge of the
// contexts.
//
// All n_q / n_kv query heads of the group share a segment, so every K/V byte
// is read from HBM exactly once. Per page (16 tokens):
//   S^T = K_page * Q_g^T    MFMA 16x16x32 (D/32 of them): rows = tokens, cols = heads;
//                           lane l gets tokens (l/16)*4 .. +3 of head l%16.
//   online softmax          per lane (head l%16); page max over the 4 lane rows
//                           by two xor-shuffles; masked tokens get -inf.
//   O^T += V_page^T * P     MFMA 16x16x16 (D/16 of them): V is stored dim-major in
//                           the page, so lane l reads 8 contiguous bytes, and P
//                           is already in the B-operand layout of S^T.
// The accumulator O^T keeps head l%16 in lane l, so the softmax rescale never
// leaves the lane. K and V reach registers through LDS: each wave streams its
// pages with direct-to-LDS loads into a ring of two page slots of its own and
// reads a slot into registers once its loads have landed, so the page in
// flight costs no registers. The group's q rows are read once per segment,
// not once per page. The page ids of the next 64 pages load while the current
// 64 are streamed.
#include <math.h>

#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace ods {

namespace {

constexpr int kNonTemporal = 2;  // cache-policy operand of the direct-to-LDS load: nt
// Largest dynamic LDS a launch asks for: the per-sequence arrays at the batch
// limit plus two K+V page slots for each of the four waves at D = 128.
constexpr size_t kMaxAttnLds = ((2 * (size_t)kMaxAttnBatch + 1) * sizeof(int) + 15) / 16 * 16 + 4 * 2 * 2 * 16 * 128 * 2;

template <int D>
struct PageRegs {
  u32x4 k[D / 32];  // K rows: lane l holds K[t = l%16][kk*32 + (l/16)*8 .. +8]
  u32x2 v[D / 16];  // V dim-major: lane l holds V[d = nb*16 + l%16][t = (l/16)*4 .. +4]
  u32x4 q[D / 32];  // the page's query heads: lane l holds q[head l%16][kk*32 + (l/16)*8 .. +8]
  int pg;           // page index within the sequence (uniform)
  int seq;          // b * n_kv + g, -1 for a padding slot past the range (uniform)
  int lo, p;        // attended token positions [lo, p] of the sequence (uniform)
  bool ok;          // page id inside the pool (uniform)
};

// Uniform description of a page whose K / V loads are in flight in an LDS slot.
struct PageMeta {
  int pg, seq, lo, p;  // as in PageRegs
  bool ok;
};

// Attended window of a sequence from its (clamped) context: token positions
// [lo, p] and window pages [first_page, first_page + n_pages).
__device__ __forceinline__ void window_of(int ctx, int window, int &p, int &lo, int &first_page, int &n_pages) {
  if (ctx < 1) {
    p = lo = first_page = n_pages = 0;
    return;
  }
  p = ctx - 1;
  lo = window > 0 ? max(0, p - window + 1) : 0;
  first_page = lo / kPage;
  n_pages = p / kPage - first_page + 1;
}

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_flat_kernel(
    const uint16_t *__restrict__ qkv, int n_q, int n_kv, int window, const int32_t *__restrict__ ctx_lens,
    const int32_t *__restrict__ page_table, int max_pages, int ring, const uint16_t *__restrict__ pool,
    int64_t pool_pages, int seg_pages, float scale_log2, float *__restrict__ ws_acc, float *__restrict__ ws_ml,
    int2 *__restrict__ ws_meta, uint16_t *__restrict__ o, int B) {
  constexpr int KK = D / 32;  // QK MFMAs per page
  constexpr int NB = D / 16;  // PV MFMAs per page
  constexpr int64_t BLK = (int64_t)kPage * D;
  extern __shared__ int smem_i[];
  int *s_pre = smem_i;          // [B + 1]: first unit of sequence b (its KV head 0)
  int *s_ctx = smem_i + B + 1;  // [B]: context (clamped to the page table unless it is a ring)
  __shared__ int s_wtot[4];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keeps control flow scalar
  const int group = n_q / n_kv;
  const int hl = lane & 15;  // head within the group (MFMA column)
  const int rq = lane >> 4;  // lane row-quad
  const bool head_ok = hl < group;
  const int row_elems = (n_q + 2 * n_kv) * D;

  // ---- per-sequence contexts and the unit prefix s_pre[b] = n_kv * sum_{b' < b} pages(b')
  {
    const int per = (B + 255) / 256;
    const int b0 = min(B, tid * per), b1 = min(B, b0 + per);
    int loc = 0;
    for (int b = b0; b < b1; ++b) {
      const int c = ring > 0 ? ctx_lens[b] : min(ctx_lens[b], max_pages * kPage);
      int p, lo, fp, n;
      window_of(c, window, p, lo, fp, n);
      s_ctx[b] = c;
      loc += n;
    }
    int inc = loc;
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(inc, d, kWave);
      if (lane >= d) inc += y;
    }
    if (lane == 63) s_wtot[wave] = inc;
    __syncthreads();
    int run = inc - loc;
    for (int w = 0; w < wave; ++w) run += s_wtot[w];
    for (int b = b0; b < b1; ++b) {
      int p, lo, fp, n;
      window_of(s_ctx[b], window, p, lo, fp, n);
      s_pre[b] = run * n_kv;
      run += n;
    }
    if (tid == 255) s_pre[B] = run * n_kv;
    __syncthreads();
  }
  // This wave's LDS page slots, after the per-sequence arrays: K block, then V block.
  constexpr int kSlots = 2;
  constexpr int SLOT = 2 * kPage * D * 2;
  constexpr int LPP = 2 * (kPage * D * 2 / 1024);  // 16-byte direct-to-LDS loads per page and lane
  uint8_t *const slots = (uint8_t *)smem_i + (((2 * B + 1) * 4 + 15) & ~15) + wave * kSlots * SLOT;
  const int total = __builtin_amdgcn_readfirstlane(s_pre[B]);
  const int n_waves = gridDim.x * 4;
  const int S = seg_pages > 0 ? seg_pages : max(8, (total + n_waves - 1) / n_waves);
  const int64_t page_stride = 2 * (int64_t)n_kv * BLK;
  const int64_t v_off = (int64_t)n_kv * BLK;

  // last b with s_pre[b] <= u (a non-empty sequence when u < total)
  auto find_seq = [&](int u) {
    int b = 0, hi = B;
    while (hi - b > 1) {
      const int mid = (b + hi) >> 1;
      if (s_pre[mid] <= u) b = mid; else hi = mid;
    }
    return b;
  };

  for (int r = blockIdx.x * 4 + wave; (int64_t)r * S < total; r += n_waves) {
    const int u0 = r * S, n_w = min(total, u0 + S) - u0;  // this range: units [u0, u0 + n_w)

    // Page ids of range pages [t0, t0 + 64), one per lane (-1 past the range):
    // each lane locates its own unit.
    auto gather_ids = [&](int t0) {
      const int t = t0 + lane;
      if (t >= n_w) return -1;
      const int u = u0 + t;
      const int b = find_seq(u);
      int p, lo, fp, n;
      window_of(s_ctx[b], window, p, lo, fp, n);
      const int lp = fp + (u - s_pre[b]) % n;  // logical page of the sequence
      return page_table[(int64_t)b * max_pages + (ring > 0 ? lp % ring : lp)];
    };

    // ---- issue cursor: the next range page to load, as (sequence, head, window page)
    int ib = __builtin_amdgcn_readfirstlane(find_seq(u0));
    int ig, ipage, in_b, ifp, ilo, ip;
    auto cursor_seq = [&]() {
      int p, lo, fp, n;
      window_of(s_ctx[ib], window, p, lo, fp, n);
      ip = __builtin_amdgcn_readfirstlane(p);
      ilo = __builtin_amdgcn_readfirstlane(lo);
      ifp = __builtin_amdgcn_readfirstlane(fp);
      in_b = __builtin_amdgcn_readfirstlane(n);
    };
    cursor_seq();
    {
      const int off = u0 - __builtin_amdgcn_readfirstlane(s_pre[ib]);
      ig = off / in_b;
      ipage = off % in_b;
    }
    int it = 0;  // range page index of the next issue
    int ids_cur = gather_ids(0), ids_nxt = gather_ids(64);

    // Issue the loads of the cursor's page into LDS slot `slot`, describe it
    // in R and advance the cursor. Past the range the slot re-reads a valid
    // page and is marked as padding, so every issue makes the same loads and
    // the waits can count them.
    auto issue = [&](PageMeta &R, int slot) {
      if (it > 0 && (it & 63) == 0) {
        ids_cur = ids_nxt;
        ids_nxt = gather_ids(it + 64);
      }
      const bool live = it < n_w;
      const int page = __builtin_amdgcn_readlane(ids_cur, it & 63);
      R.seq = live ? ib * n_kv + ig : -1;
      R.pg = ifp + ipage;
      R.lo = ilo;
      R.p = ip;
      R.ok = live && (unsigned)page < (unsigned long long)pool_pages;
      const uint16_t *kb = pool + (int64_t)ig * BLK + (int64_t)(R.ok ? page : 0) * page_stride;
      uint8_t *const dst = slots + slot * SLOT;
      // A direct-to-LDS load writes lane l's 16 bytes at byte 16 l of its
      // destination. K: lane l fetches the 16 bytes it will read as its MFMA
      // fragment (K[t = l % 16][kk * 32 + (l / 16) * 8 ..]), so its read-back is
      // at 16 l, conflict-free. V: the dim-major block is copied verbatim and
      // lane l reads its 8 bytes (dim nb * 16 + l % 16, slots (l / 16) * 4 ..)
      // at (nb * 16 + l % 16) * 32 + (l / 16) * 8. K/V bytes are read once per
      // launch: the loads carry the non-temporal cache policy.
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        __builtin_amdgcn_global_load_lds((const void *)(kb + hl * D + kk * 32 + rq * 8),
                                         (__attribute__((address_space(3))) void *)(dst + kk * 1024), 16, 0,
                                         kNonTemporal);
#pragma unroll
      for (int j = 0; j < KK; ++j)
        __builtin_amdgcn_global_load_lds((const void *)((const uint8_t *)(kb + v_off) + j * 1024 + lane * 16),
                                         (__attribute__((address_space(3))) void *)(dst + kPage * D * 2 + j * 1024),
                                         16, 0, kNonTemporal);
      if (live) {
        ++it;
        if (++ipage == in_b) {
          ipage = 0;
          if (++ig == n_kv) {
            ig = 0;
            if (it < n_w) {
              ++ib;
              while (__builtin_amdgcn_readfirstlane(s_pre[ib + 1]) == __builtin_amdgcn_readfirstlane(s_pre[ib])) ++ib;
              cursor_seq();
            }
          }
        }
      }
    };

    // ---- consume side: the segment being accumulated
    int cur_seq = -1, cur_first_pg = 0;
    f32x4 acc[NB];
    float m_run = -INFINITY, l_run = 0.f;
    auto finish = [&]() {  // write the current segment's output or record
      float l = l_run;
      l += __shfl_xor(l, 16, kWave);
      l += __shfl_xor(l, 32, kWave);
      const int b = cur_seq / n_kv, g = cur_seq % n_kv;
      const int n_b = (__builtin_amdgcn_readfirstlane(s_pre[b + 1]) - __builtin_amdgcn_readfirstlane(s_pre[b])) / n_kv;
      const int s0 = __builtin_amdgcn_readfirstlane(s_pre[b]) + g * n_b;
      const int first_r = s0 / S, n_seg = (s0 + n_b - 1) / S - first_r + 1;
      int p, lo, fp, n;
      window_of(s_ctx[b], window, p, lo, fp, n);
      if (cur_first_pg == __builtin_amdgcn_readfirstlane(fp) && lane == 0)
        ws_meta[cur_seq] = make_int2(first_r + cur_seq, n_seg);
      if (!head_ok) return;
      if (n_seg == 1) {
        const float inv = l > 0.f ? 1.f / l : 0.f;
        uint16_t *dst = o + ((int64_t)b * n_q + g * group + hl) * D;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          u32x2 w2;
          w2[0] = pack2(acc[nb][0] * inv, acc[nb][1] * inv);
          w2[1] = pack2(acc[nb][2] * inv, acc[nb][3] * inv);
          *(u32x2 *)(dst + nb * 16 + rq * 4) = w2;
        }
      } else {
        // record r + seq is unique: the sequences one range meets are consecutive
        const int64_t rec = (int64_t)(r + cur_seq) * group + hl;
        float *dst = ws_acc + rec * D;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) *(f32x4 *)(dst + nb * 16 + rq * 4) = acc[nb];
        if (rq == 0) {
          ws_ml[rec * 2] = m_run;
          ws_ml[rec * 2 + 1] = l;
        }
      }
    };

    auto consume = [&](PageRegs<D> &R) {
      if (R.seq != cur_seq) {  // uniform: the page opens a new segment
        if (cur_seq >= 0) finish();
        cur_seq = R.seq;
        cur_first_pg = R.pg;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        m_run = -INFINITY;
        l_run = 0.f;
      }
      const int pg = R.pg, lo = R.lo, p = R.p;
      const bool ok = R.ok;
      f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        s = mfma_16x16x32(__builtin_bit_cast(bf16x8, R.k[kk]), __builtin_bit_cast(bf16x8, R.q[kk]), s);
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

    // Two pages in flight through the wave's LDS slots: while one is consumed
    // the next is loading; the stream runs across segment boundaries without
    // draining. A wave's loads complete in order, so slot s has landed once
    // only the other slot's LPP loads are outstanding. The q rows of a segment
    // are loaded when its first page is consumed, and that path alone waits
    // for every load.
    PageMeta ms[kSlots];
    u32x4 qreg[KK];
    int q_seq = -1;
#pragma unroll
    for (int sl = 0; sl < kSlots; ++sl) issue(ms[sl], sl);
    for (int t = 0; t < n_w; t += kSlots) {
#pragma unroll
      for (int sl = 0; sl < kSlots; ++sl) {
        if (t + sl < n_w) {
          asm volatile("s_waitcnt vmcnt(%0)" ::"n"((kSlots - 1) * LPP) : "memory");
          PageRegs<D> R;
          const uint8_t *src = slots + sl * SLOT;
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) R.k[kk] = *(const u32x4 *)(src + kk * 1024 + lane * 16);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            R.v[nb] = *(const u32x2 *)(src + kPage * D * 2 + (nb * 16 + hl) * 32 + rq * 8);
          if (ms[sl].seq >= 0 && ms[sl].seq != q_seq) {
            q_seq = ms[sl].seq;
            const int qb = q_seq / n_kv, qg = q_seq % n_kv;
            const uint16_t *qp = qkv + (int64_t)qb * row_elems + (int64_t)(qg * group + (head_ok ? hl : 0)) * D;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) qreg[kk] = *(const u32x4 *)(qp + kk * 32 + rq * 8);
            // vmcnt(0) on this path only (a builtin, so the compiler knows the q
            // registers have landed and adds no wait on the common path)
            __builtin_amdgcn_s_waitcnt(0x0F70);
          }
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) R.q[kk] = qreg[kk];
          R.pg = ms[sl].pg;
          R.seq = ms[sl].seq;
          R.lo = ms[sl].lo;
          R.p = ms[sl].p;
          R.ok = ms[sl].ok;
          consume(R);
        }
        issue(ms[sl], sl);
      }
    }
    // No load may still be writing the slots when the next range reuses them
    // or the wave retires.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    finish();
  }
}

// One wave per (sequence, query head): a sequence split into several segments
// gets o[d] = sum_c 2^(m_c - M) acc_c[d] / sum_c 2^(m_c - M) l_c over its
// records; a row with no context gets zeros; single-segment rows were written
// by the attention kernel.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float *__restrict__ ws_acc,
                                                         const float *__restrict__ ws_ml,
                                                         const int2 *__restrict__ ws_meta, int n_q, int n_kv,
                                                         const int32_t *__restrict__ ctx_lens,
                                                         uint16_t *__restrict__ o, int B) {
  constexpr int DPL = D / 64;  // d values per lane
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wid >= (int64_t)B * n_q) return;
  const int b = (int)(wid / n_q), h = (int)(wid % n_q);
  const int group = n_q / n_kv;
  uint16_t *dst = o + wid * D + lane * DPL;
  // The context and the merge metadata load together (the metadata of an
  // empty sequence is never used).
  const int ctx = ctx_lens[b];
  const int2 meta = ws_meta[(int64_t)b * n_kv + h / group];
  // Keeps the metadata load ahead of the context test (the compiler would
  // otherwise sink it past the branch and wait for the context first).
  asm volatile("" ::"v"(meta.x), "v"(meta.y));
  if (ctx < 1) {
#pragma unroll
    for (int i = 0; i < DPL; ++i) dst[i] = 0;
    return;
  }
  const int n_seg = meta.y;
  if (n_seg <= 1) return;  // written by the attention kernel
  const int64_t rec0 = (int64_t)meta.x * group + h % group;  // records rec0 + c * group
  // The accumulators of the first kPre records load together with the (m, l)
  // pairs (neither depends on the other), so a sequence split a few ways costs
  // one round trip after the metadata instead of two.
  constexpr int kPre = 4;
  float pre[kPre][DPL];
#pragma unroll
  for (int c = 0; c < kPre; ++c) {
    if (c < n_seg) {
      const float *src = ws_acc + (rec0 + (int64_t)c * group) * D + lane * DPL;
#pragma unroll
      for (int i = 0; i < DPL; ++i) pre[c][i] = src[i];
    }
  }
  // (m, l) of record c as one 8-byte load; lane c keeps record c (< 64).
  auto ml_of = [&](int c) { return *(const float2 *)(ws_ml + (rec0 + (int64_t)c * group) * 2); };
  const float2 own = lane < n_seg ? ml_of(lane) : make_float2(-INFINITY, 0.f);
  float mloc = own.x;
  for (int c = lane + 64; c < n_seg; c += 64) mloc = fmaxf(mloc, ml_of(c).x);
  const float M = wave_max(mloc);
  auto weight_of = [&](float mc) { return mc == -INFINITY ? 0.f : exp2f(mc - M); };
  float lsum = weight_of(own.x) * own.y;
  for (int c = lane + 64; c < n_seg; c += 64) {
    const float2 r = ml_of(c);
    lsum += weight_of(r.x) * r.y;
  }
  const float L = wave_sum(lsum);
  float acc[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) acc[i] = 0.f;
  if (n_seg <= kPre) {
    const float wl = lane < n_seg ? weight_of(own.x) : 0.f;
#pragma unroll
    for (int c = 0; c < kPre; ++c) {
      if (c < n_seg) {
        const float w = __shfl(wl, c, kWave);
#pragma unroll
        for (int i = 0; i < DPL; ++i) acc[i] += w * pre[c][i];
      }
    }
  }
  for (int c0 = 0; n_seg > kPre && c0 < n_seg; c0 += 64) {
    const float wl = (c0 + lane < n_seg) ? (c0 == 0 ? weight_of(own.x) : weight_of(ml_of(c0 + lane).x)) : 0.f;
    const int n = min(64, n_seg - c0);
#pragma unroll 4
    for (int j = 0; j < n; ++j) {
      const float w = __shfl(wl, j, kWave);
      const float *src = ws_acc + (rec0 + (int64_t)(c0 + j) * group) * D + lane * DPL;
#pragma unroll
      for (int i = 0; i < DPL; ++i) acc[i] += w * src[i];
    }
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
#pragma unroll
  for (int i = 0; i < DPL; ++i) dst[i] = f2bf(acc[i] * inv);
}

}  // namespace

// Compute units of the current device (queried once per process and device).
int num_cus() {
  static std::atomic<int> cached[64] = {};  // 0: not queried yet (threads may race to fill a slot, same value)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

hipError_t launch_attention(const uint16_t *qkv, int B, int n_q, int n_kv, int D, int window,
                            const int32_t *ctx_lens, const int32_t *page_table, int max_pages, int ring,
                            const uint16_t *pool, int64_t pool_pages, const AttnPlan &plan, float *ws,
                            uint16_t *o, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  const size_t group = n_q / n_kv;
  float *ws_acc = ws;  // [records][group][D], 16-byte aligned rows
  float *ws_ml = ws_acc + (size_t)plan.records * group * D;
  int2 *ws_meta = (int2 *)(ws_ml + (size_t)plan.records * group * 2);
  // per-sequence arrays, then two K+V page slots per wave (64 KB at D = 128)
  const size_t lds = (((2 * (size_t)B + 1) * sizeof(int) + 15) & ~(size_t)15) + (size_t)4 * 2 * 2 * kPage * D * 2;
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
  const dim3 mgrid((unsigned)(((int64_t)B * n_q + 3) / 4));
  auto go = [&](auto kflat, auto kmerge, std::atomic<uint64_t> &lds_set) {
    if (hipError_t e = ensure_lds_limit((const void *)kflat, kMaxAttnLds, lds_set); e != hipSuccess) return e;
    hipLaunchKernelGGL(kflat, dim3(plan.grid), dim3(256), lds, s, qkv, n_q, n_kv, window, ctx_lens, page_table,
                       max_pages, ring, pool, pool_pages, plan.seg_pages, scale_log2, ws_acc, ws_ml, ws_meta, o, B);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kmerge, mgrid, dim3(256), 0, s, ws_acc, ws_ml, ws_meta, n_q, n_kv, ctx_lens, o, B);
    return hipGetLastError();
  };
  static std::atomic<uint64_t> lds_set_128{0}, lds_set_64{0};  // devices whose limit each kernel already raised
  if (D == 128) return go(attn_flat_kernel<128>, attn_merge_kernel<128>, lds_set_128);
  return go(attn_flat_kernel<64>, attn_merge_kernel<64>, lds_set_64);
}

}  // namespace ods
