// Gradients of the channel attention (Section 3.1 Step 3 with the dummy slot of Section
// 3.2), the attention half of the backward pass that training runs through its
// gradient-carrying passes (Section 3.3, truncated backpropagation).
//
// For a query row with scores s_j = q.k_j / sqrt(d) over its visible slots and the dummy,
// P_j = exp(s_j - LSE) and O = sum_j P_j v_j. Given dO:
//   dP_j = dO.v_j,  D = dO.O = sum_j P_j dP_j,  dS_j = P_j (dP_j - D),
//   dq = sum_j dS_j k_j / sqrt(d),  dk_j += dS_j q / sqrt(d),  dv_j += P_j dO.
// Three kernels:
//   attend_bwd_dq_kernel   query-major, like the forward: LSE (one pass over the slots),
//                          then dq (a second pass); writes per-row LSE, D and the dummy's
//                          P and dS.
//   attend_bwd_dkv_kernel  slot-major: a workgroup owns 256 slots of one channel, sequence
//                          and KV head and walks every query that reads them (all
//                          consumers of the channel, all grouped query heads), so each
//                          slot's dk and dv are summed in registers and written once.
//   attend_bwd_dummy_*     the dummy's dk, dv: a sum over every row of its readers.
// Products run on the matrix cores in bf16 (P and dS rounded to bf16 as operands), sums
// in fp32; gradients leave in fp32.
#include <algorithm>

#include "wm_device.hpp"
#include "wm_frag.hpp"
#include "wm_internal.hpp"

namespace wm {

struct BwdArgs {
  const bf16 *Q, *Kc, *Vc, *Kd, *Vd, *O, *dO;
  const int32_t* ctx_len;
  float *dQ, *dKc, *dVc, *dKd, *dVd;
  float *lse, *dlt, *pd, *dsd;  // per query row [L][B][Hq][T] (workspace)
  int B, T, L, Hq, Hkv, S_cap, mask_paper, ctx_hi, n_qtiles, n_stiles;
  float scale_log2, scale;  // log2(e) / sqrt(d), 1 / sqrt(d)
  LayerTable chan;
  ChannelGroups grp;
  int accumulate;  // add the slot and dummy gradients into dKc, dVc, dKd, dVd
  int dchunks;     // partial sums per (channel, KV head) of the dummy's gradients
  int gs, gq;      // query i of sequence b sits at position ctx_len[b] + gq + gs i
  int kv_heavy_first;  // slot-major grid: each XCD takes its (channel, sequence, KV head)
                       // slices' slot tiles lowest slots (most readers) first
};

// waves per workgroup of the query-major and the slot-major kernel (32 rows each)
#ifndef WM_BWD_QWAVES
#define WM_BWD_QWAVES 8
#endif
#ifndef WM_BWD_KWAVES
#define WM_BWD_KWAVES 8
#endif
constexpr int kBwdQWaves = WM_BWD_QWAVES, kBwdKWaves = WM_BWD_KWAVES;

__device__ __forceinline__ float bwd_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Copies rows row0 .. row0 + ROWS - 1 (DH bf16 each, row_bytes apart in the view) into the
// LDS block at lds_base with LDS DMA, in the fragment readers' chunk swizzle: wave w's
// n-th instruction fills LDS chunks 64 (NI w + n) + lane, and each lane fetches the chunk
// the swizzle puts there. Rows at or past nvalid arrive as zeros. Every wave of the NW
// issues up to NI copies (the block's 16-byte chunks in whole 64-lane instructions); the
// caller waits for them (vmcnt) before the barrier that publishes the block.
template <int DH, int ROWS, int NW>
__device__ __forceinline__ void bwd_dma(uint32_t lds_base, __amdgpu_buffer_rsrc_t view,
                                        uint32_t row_bytes, int row0, int nvalid, int w,
                                        int lane) {
  constexpr int CPR = DH * 2 / 16, TOT = ROWS * CPR, NI = (TOT + 64 * NW - 1) / (64 * NW);
  static_assert(TOT % 64 == 0, "whole 64-lane instructions");
#pragma unroll
  for (int n = 0; n < NI; ++n) {
    if ((NI * w + n) * 64 >= TOT) break;  // wave-uniform: the block is complete
    const int pos = (NI * w + n) * 64 + lane, row = pos / CPR, cc = pos - row * CPR;
    const int gr = row0 + row;
    const uint32_t off = gr < nvalid ? (uint32_t)gr * row_bytes + 16u * (uint32_t)(cc ^ pf_swz<DH>(row))
                                     : kOffOob;
    lds_dma16(__builtin_amdgcn_readfirstlane(lds_base + (NI * w + n) * 1024), off, view);
  }
}

__device__ __forceinline__ bf16x4 bwd_ld8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

// --------------------------------------------------------------- dq, LSE, D
// Tile: 32 NW query rows of one (consumer, sequence, query head), 32 per wave; S^T = K q^T
// puts one query in a lane (as in the forward), dP^T = V dO^T likewise, and
// dq^T += K^T dS^T takes dS^T straight from those registers through the transposing
// read of the K block.
template <int DH, int NW>
__global__ __launch_bounds__(64 * NW) void attend_bwd_dq_kernel(BwdArgs a) {
  constexpr int NKS = DH / 16, NDT = DH / 32, ROW = 2 * DH, BLK = 64, NH = DH == 64 ? 2 : 1;
  // two buffers, each a K block then a V block
  __shared__ __align__(16) char smem[4 * BLK * ROW];
  const uint32_t lbase = (uint32_t)(uintptr_t)smem;
  // XCD-aware order: each XCD walks a contiguous run of tiles, so the query tiles of one
  // head (which read the same K/V slice) share its L2
  const int tile = xcd_tile(blockIdx.x, (int)gridDim.x);
  const int qtile = a.n_qtiles - 1 - tile % a.n_qtiles;
  int y = tile / a.n_qtiles;
  const int hq = y % a.Hq;
  y /= a.Hq;
  const int b = y % a.B, l = y / a.B;
  const int c = a.chan.v[l], kvh = hq / (a.Hq / a.Hkv);
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pos0 = __builtin_amdgcn_readfirstlane(ctx_at(a.ctx_len, b, a.ctx_hi));
  const int incl = a.mask_paper ? 0 : 1;
  const int q0 = qtile * 32 * NW, qw0 = q0 + 32 * w, qi = qw0 + r;
  const bool valid = qi < a.T;
  const float cl2 = a.scale_log2;

  // the row's query, dO and O at this lane's columns (buffer loads: rows past T are zeros)
  bf16x8 qf[NKS], df[NKS], of[NKS];
  {
    const long rowl = ((long)l * a.B + b) * a.T;  // (l, b, 0) in [L][B][T][Hq d]
    const uint32_t ostride = (uint32_t)a.Hq * DH * 2u;
    const auto qv = make_view(a.Q + (((long)l * a.B + b) * a.Hq + hq) * (long)a.T * DH,
                              (uint32_t)a.T * DH * 2u);
    const auto dv = make_view(a.dO + rowl * a.Hq * DH + (long)hq * DH, (uint32_t)a.T * ostride);
    const auto ov = make_view(a.O + rowl * a.Hq * DH + (long)hq * DH, (uint32_t)a.T * ostride);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const uint32_t col = (uint32_t)(16 * ks + 8 * h) * 2u;
      qf[ks] = buf_frag<bf16>(qv, valid ? (uint32_t)qi * DH * 2u + col : kOffOob);
      df[ks] = buf_frag<bf16>(dv, valid ? (uint32_t)qi * ostride + col : kOffOob);
      of[ks] = buf_frag<bf16>(ov, valid ? (uint32_t)qi * ostride + col : kOffOob);
    }
  }
  // dummy key and value (zeros without the paper mask)
  const long dofs = ((long)c * a.Hkv + kvh) * DH;
  const uint32_t dbytes = a.mask_paper ? DH * 2u : 0u;
  const auto kdv = make_view(a.mask_paper ? a.Kd + dofs : nullptr, dbytes);
  const auto vdv = make_view(a.mask_paper ? a.Vd + dofs : nullptr, dbytes);
  float dl = 0.f, sdp = 0.f, dpd = 0.f;
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const bf16x8 kd = buf_frag<bf16>(kdv, (16 * ks + 8 * h) * 2u);
    const bf16x8 vd = buf_frag<bf16>(vdv, (16 * ks + 8 * h) * 2u);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      dl += (float)df[ks][e] * (float)of[ks][e];
      sdp += (float)qf[ks][e] * (float)kd[e];
      dpd += (float)df[ks][e] * (float)vd[e];
    }
  }
  const float delta = halves_sum(dl);
  const float sd = halves_sum(sdp) * cl2;  // the dummy's score, log2 units
  dpd = halves_sum(dpd);

  const int pq = pos0 + a.gq + incl;  // position (+ incl) of query 0; query i adds gs i
  const int qlast = min(q0 + 32 * NW - 1, a.T - 1);
  const int kend = min(pq + a.gs * qlast, a.S_cap);              // slots the tile may see
  const int wq_last = min(qw0 + 31, a.T - 1);
  const int wkend = wq_last >= qw0 ? pq + a.gs * wq_last : 0;    // ... this wave
  const int lim = pq + a.gs * qi;                                // ... this lane's row
  const int wlim0 = pq + a.gs * qw0;                             // ... the wave's first row
  const int nblk = (kend + BLK - 1) / BLK;
  const long cbase = (((long)c * a.B + b) * a.Hkv + kvh) * (long)a.S_cap * DH;
  const auto kv = make_view(a.Kc + cbase, (uint32_t)max(kend, 0) * ROW);
  const auto vv = make_view(a.Vc + cbase, (uint32_t)max(kend, 0) * ROW);
  const PfLane<DH> lo = pf_lane<DH>(lane);

  // One walk over the blocks with an online normaliser: the row keeps a running maximum m
  // (log2 units, shared by the two lanes of the row) and sums l = sum 2^(s - m) and
  // dq~ = sum 2^(s - m) (dP - D) k, both rescaled when m grows; at the end
  // lse = m + log2 l and dq = dq~ / l, since dS = P (dP - D) with P = 2^(s - lse).
  float m = a.mask_paper ? sd : kNegBig;
  float sum = a.mask_paper && h == 0 ? 1.f : 0.f;
  f32x16 dq[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) dq[dt] = zero16();
  // blocks are double-buffered: block j + 1 is copied while block j is multiplied
  if (nblk > 0) {
    bwd_dma<DH, BLK, NW>(lbase, kv, ROW, 0, kend, w, lane);
    bwd_dma<DH, BLK, NW>(lbase + BLK * ROW, vv, ROW, 0, kend, w, lane);
  }
  for (int j = 0; j < nblk; ++j) {
    const uint32_t kb = (uint32_t)(j & 1) * 2 * BLK * ROW;
    wait_vmcnt<0>();
    __syncthreads();  // block j is in LDS; every wave is done with block j - 1
    if (j + 1 < nblk) {
      const uint32_t nb = lbase + (kb ^ (2 * BLK * ROW));
      bwd_dma<DH, BLK, NW>(nb, kv, ROW, (j + 1) * BLK, kend, w, lane);
      bwd_dma<DH, BLK, NW>(nb + BLK * ROW, vv, ROW, (j + 1) * BLK, kend, w, lane);
    }
#pragma unroll
    for (int hg = 0; hg < 2 / NH; ++hg) {
      const int sb = j * BLK + 32 * NH * hg;  // the group's first slot
      if (sb < wkend) {
        f32x16 sc[NH], dp[NH];
#pragma unroll
        for (int x = 0; x < NH; ++x) sc[x] = dp[x] = zero16();
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
          for (int x = 0; x < NH; ++x) {
            const uint32_t ho = kb + (NH * hg + x) * 32 * ROW;
            sc[x] = mma32(sc[x], pf_ldk<DH>(smem, lo, ho, ks), qf[ks]);
            dp[x] = mma32(dp[x], pf_ldk<DH>(smem, lo, ho + BLK * ROW, ks), df[ks]);
          }
        // the group's largest raw score (hidden slots at -inf, whose weight is 0 against any
        // reference, and which leave the maximum alone); cl2 > 0 scales it to log2 units,
        // and each weight is 2^(s cl2 - m) from one fma
        constexpr float kHidden = -__builtin_inff();
        float mx = kHidden;
        if (sb + 32 * NH - 1 < wlim0) {  // every row of the wave sees the group
#pragma unroll
          for (int x = 0; x < NH; ++x)
#pragma unroll
            for (int q = 0; q < 16; ++q) mx = fmaxf(mx, sc[x][q]);
        } else {
          const int thr = lim - sb - 4 * h;  // slot sb + 32 x + 8 (q / 4) + 4 h + q % 4 < lim
#pragma unroll
          for (int x = 0; x < NH; ++x)
#pragma unroll
            for (int q = 0; q < 16; ++q) {
              sc[x][q] = 32 * x + 8 * (q >> 2) + (q & 3) < thr ? sc[x][q] : kHidden;
              mx = fmaxf(mx, sc[x][q]);
            }
        }
        const float mn = fmaxf(m, halves_max(mx) * cl2);
        if (__builtin_expect(__any(mn > m), 0)) {  // the maximum grew: rescale the sums
          const float f = bwd_exp2(m - mn);
          sum *= f;
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) dq[dt] *= f;
          m = mn;
        }
        bf16x8 ds[NH][2];
        float part = 0.f;
#pragma unroll
        for (int x = 0; x < NH; ++x)
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const float p = bwd_exp2(__builtin_fmaf(sc[x][q], cl2, -m));  // 0 when hidden
            part += p;
            ds[x][q >> 3][q & 7] = (bf16)(p * (dp[x][q] - delta));
          }
        sum += part;
#pragma unroll
        for (int x = 0; x < NH; ++x)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int kh = 0; kh < 2; ++kh)
              dq[dt] = mma32(dq[dt], pf_ldv<DH>(smem, lo, kb + (NH * hg + x) * 32 * ROW, kh, dt),
                             ds[x][kh]);
      }
    }
  }
  const float ltot = halves_sum(sum);
  const float lse = m + __log2f(ltot), inv = 1.0f / ltot;
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) dq[dt] *= inv;

  // the dummy's term, then dq / sqrt(d) out
  const float p_d = a.mask_paper ? bwd_exp2(sd - lse) : 0.f;
  const float ds_d = p_d * (dpd - delta);
  if (valid) {
    float* dst = a.dQ + ((((long)l * a.B + b) * a.Hq + hq) * a.T + qi) * DH;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const bf16x4 kd = bwd_ld8(kdv, (32 * dt + 8 * g + 4 * h) * 2u);
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = (dq[dt][4 * g + i] + ds_d * (float)kd[i]) * a.scale;
        *(f32x4*)(dst + 32 * dt + 8 * g + 4 * h) = v;
      }
    if (h == 0) {
      const long idx = (((long)l * a.B + b) * a.Hq + hq) * a.T + qi;
      a.lse[idx] = lse;
      a.dlt[idx] = delta;
      a.pd[idx] = p_d;
      a.dsd[idx] = ds_d;
    }
  }
}

// ------------------------------------------------------------------- dk, dv
// Tile: 32 NW slots of one (channel, sequence, KV head), 32 per wave; the wave's K and V
// rows stay in registers as the column operand. The tile walks every query block of 64
// rows that may read its slots, for every consumer of the channel and every query head of
// the KV head, as one flat sequence, so the next block (queries and dO by LDS DMA, the
// rows' LSE and D through registers) is fetched while the current one is multiplied. For
// each 32-row half: S = Q K^T and dP = dO V^T put one slot in a lane, and dv^T += dO^T P
// and dk^T += Q^T dS take P and dS from those registers through the transposing reads
// of the dO and Q blocks.
template <int DH, int NW>
__global__ __launch_bounds__(64 * NW) void attend_bwd_dkv_kernel(BwdArgs a) {
  constexpr int NKS = DH / 16, NDT = DH / 32, ROW = 2 * DH, QB = 64, NH = DH == 64 ? 2 : 1;
  constexpr uint32_t BUF = 2 * QB * ROW;  // one buffer: a Q block, then a dO block
  __shared__ __align__(16) char smem[2 * BUF];
  __shared__ __align__(16) float s_lse[2][QB], s_dlt[2][QB];
  const uint32_t lbase = (uint32_t)(uintptr_t)smem;
  // XCD-aware order: the slot tiles of one (channel, sequence, KV head), which read the
  // same queries and output gradients, run on one XCD
  int stile, y;
  if (a.kv_heavy_first) {
    // a grid of at most two rounds: XCD x owns a contiguous band of the slices and starts
    // every slice's first slot tile, then every second, ..., so the long tiles start first
    const int px = (int)gridDim.x / (a.n_stiles * kNumXcd), sidx = blockIdx.x / kNumXcd;
    stile = sidx / px;
    y = (blockIdx.x % kNumXcd) * px + sidx % px;
  } else {
    const int tile = xcd_tile(blockIdx.x, (int)gridDim.x);
    stile = tile % a.n_stiles;
    y = tile / a.n_stiles;
  }
  const int kvh = y % a.Hkv;
  y /= a.Hkv;
  const int b = y % a.B, c = y / a.B;
  const int G = a.Hq / a.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pos0 = __builtin_amdgcn_readfirstlane(ctx_at(a.ctx_len, b, a.ctx_hi));
  const int incl = a.mask_paper ? 0 : 1;
  const int pq = pos0 + a.gq + incl;  // query qr sees slots below pq + gs qr
  const int send = pos0 + a.gq + a.gs * (a.T - 1) + 1;  // slots written: [0, send)
  const int sbase = stile * 32 * NW;
  if (sbase >= send) return;
  const int ws0 = sbase + 32 * w, slot = ws0 + r;
  const bool slot_ok = slot < send;
  const float cl2 = a.scale_log2;

  const long cbase = (((long)c * a.B + b) * a.Hkv + kvh) * (long)a.S_cap * DH;
  bf16x8 kf[NKS], vf[NKS];
  {
    const auto kv = make_view(a.Kc + cbase, (uint32_t)send * ROW);
    const auto vv = make_view(a.Vc + cbase, (uint32_t)send * ROW);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const uint32_t off = slot_ok ? (uint32_t)slot * ROW + (16 * ks + 8 * h) * 2u : kOffOob;
      kf[ks] = buf_frag<bf16>(kv, off);
      vf[ks] = buf_frag<bf16>(vv, off);
    }
  }
  f32x16 dk[NDT], dv[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) dk[dt] = dv[dt] = zero16();
  const PfLane<DH> lo = pf_lane<DH>(lane);
  // the first query that sees slot sbase: the least qr with pq + gs qr > sbase
  const int i_num = sbase - pq;
  const int i_first = i_num < 0 ? 0 : i_num / a.gs + 1;
  const int qb0 = i_first / QB, nqb = (a.T + QB - 1) / QB - qb0;
  const int nmem = a.grp.offsets[c + 1] - a.grp.offsets[c];
  const int nit = nqb > 0 ? nmem * G * nqb : 0;
  const uint32_t ostride = (uint32_t)a.Hq * DH * 2u;

  // iteration it -> (consumer, query head, query block)
  auto where = [&](int it, int& l, int& hq, int& qb) {
    qb = qb0 + it % nqb;
    const int x = it / nqb;
    hq = kvh * G + x % G;
    l = a.grp.members[a.grp.offsets[c] + x / G];
  };
  float lse_n = 0.f, dlt_n = 0.f;  // the next block's row statistics (threads < QB)
  auto fetch = [&](int it, uint32_t buf) {
    int l, hq, qb;
    where(it, l, hq, qb);
    const long rows0 = (((long)l * a.B + b) * a.Hq + hq) * a.T;
    const long rowl = ((long)l * a.B + b) * a.T;
    const auto qv = make_view(a.Q + rows0 * DH, (uint32_t)a.T * DH * 2u);
    const auto dov = make_view(a.dO + rowl * a.Hq * DH + (long)hq * DH, (uint32_t)a.T * ostride);
    bwd_dma<DH, QB, NW>(buf, qv, DH * 2u, qb * QB, a.T, w, lane);
    bwd_dma<DH, QB, NW>(buf + QB * ROW, dov, ostride, qb * QB, a.T, w, lane);
    if (tid < QB) {
      const int qr = qb * QB + tid;
      lse_n = qr < a.T ? a.lse[rows0 + qr] : 1.0e30f;  // a row past T weighs 0
      dlt_n = qr < a.T ? a.dlt[rows0 + qr] : 0.f;
    }
  };
  if (nit > 0) fetch(0, lbase);
  for (int it = 0; it < nit; ++it) {
    const int u = it & 1;
    const uint32_t kb = (uint32_t)u * BUF;
    if (tid < QB) {
      s_lse[u][tid] = lse_n;
      s_dlt[u][tid] = dlt_n;
    }
    wait_vmcnt<0>();
    __syncthreads();  // block it is in LDS; every wave is done with block it - 1
    int l, hq, qb;
    where(it, l, hq, qb);
    (void)l;
    (void)hq;
    if (it + 1 < nit) fetch(it + 1, lbase + (kb ^ BUF));
    // the block's 32-row halves NH at a time (NH = 2: their products interleave; NH = 1
    // where two halves' registers would not fit): S = Q K^T and dP = dO V^T put one slot in a
    // lane; a group is skipped when its last row cannot see the wave's first slot
#pragma unroll
    for (int hg = 0; hg < 2 / NH; ++hg) {
      const int qg = qb * QB + 32 * NH * hg;  // the group's first row
      if (qg < a.T && pq + a.gs * min(qg + 32 * NH - 1, a.T - 1) > ws0) {
        f32x16 sc[NH], dp[NH];
#pragma unroll
        for (int x = 0; x < NH; ++x) sc[x] = dp[x] = zero16();
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
          for (int x = 0; x < NH; ++x) {
            const uint32_t ho = kb + (NH * hg + x) * 32 * ROW;
            sc[x] = mma32(sc[x], pf_ldk<DH>(smem, lo, ho, ks), kf[ks]);
            dp[x] = mma32(dp[x], pf_ldk<DH>(smem, lo, ho + QB * ROW, ks), vf[ks]);
          }
        // lane (h, r): slot r of the wave, rows 32 x + 8 (i / 4) + 4 h + i % 4 of the group
        bf16x8 pp[NH][2], pds[NH][2];
        const int hb = 32 * NH * hg;  // the group's rows in the staged block
        if (ws0 + 31 < pq + a.gs * qg) {  // every row of the group sees every slot
#pragma unroll
          for (int x = 0; x < NH; ++x)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const f32x4 lz = *(const f32x4*)(&s_lse[u][hb + 32 * x + 8 * g + 4 * h]);
              const f32x4 dz = *(const f32x4*)(&s_dlt[u][hb + 32 * x + 8 * g + 4 * h]);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int i = 4 * g + e;
                const float p = bwd_exp2(sc[x][i] * cl2 - lz[e]);
                pp[x][i >> 3][i & 7] = (bf16)p;
                pds[x][i >> 3][i & 7] = (bf16)(p * (dp[x][i] - dz[e]));
              }
            }
        } else {
          // row qg + 32 x + 8 g + 4 h + e sees the slot iff thr + gs (32 x + 8 g + e) > 0
          const int thr = pq + a.gs * (qg + 4 * h) - slot;
#pragma unroll
          for (int x = 0; x < NH; ++x)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const f32x4 lz = *(const f32x4*)(&s_lse[u][hb + 32 * x + 8 * g + 4 * h]);
              const f32x4 dz = *(const f32x4*)(&s_dlt[u][hb + 32 * x + 8 * g + 4 * h]);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int i = 4 * g + e;
                const float p = thr + a.gs * (32 * x + 8 * g + e) > 0
                                    ? bwd_exp2(sc[x][i] * cl2 - lz[e]) : 0.f;
                pp[x][i >> 3][i & 7] = (bf16)p;
                pds[x][i >> 3][i & 7] = (bf16)(p * (dp[x][i] - dz[e]));
              }
            }
        }
        // dv^T += dO^T P and dk^T += Q^T dS, P and dS through the transposing reads
#pragma unroll
        for (int x = 0; x < NH; ++x)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int kh = 0; kh < 2; ++kh) {
              const uint32_t ho = kb + (NH * hg + x) * 32 * ROW;
              dv[dt] = mma32(dv[dt], pf_ldv<DH>(smem, lo, ho + QB * ROW, kh, dt), pp[x][kh]);
              dk[dt] = mma32(dk[dt], pf_ldv<DH>(smem, lo, ho, kh, dt), pds[x][kh]);
            }
      }
    }
  }
  if (slot_ok) {
    float* dkd = a.dKc + cbase + (long)slot * DH;
    float* dvd = a.dVc + cbase + (long)slot * DH;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 kq, vq;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          kq[i] = dk[dt][4 * g + i] * a.scale;
          vq[i] = dv[dt][4 * g + i];
        }
        if (a.accumulate) {
          kq += *(const f32x4*)(dkd + 32 * dt + 8 * g + 4 * h);
          vq += *(const f32x4*)(dvd + 32 * dt + 8 * g + 4 * h);
        }
        *(f32x4*)(dkd + 32 * dt + 8 * g + 4 * h) = kq;
        *(f32x4*)(dvd + 32 * dt + 8 * g + 4 * h) = vq;
      }
  }
}

// -------------------------------------------------------------------- dummy
// The dummy's gradients sum over every row that reads its channel and KV head: the rows
// (consumer, query head, sequence, position) are split into dummy_chunks(sh) contiguous
// chunks, one workgroup of 4 DH threads each, and a second kernel adds the chunks in order.
// In a chunk, thread (rl, cg) of 32 x DH / 8 sums columns 8 cg .. 8 cg + 7 over every 32nd
// row from rl (16-byte loads of the row's output gradient and query), and the 32 partial
// rows are added in order.
// chunks per (channel, KV head): at least 32, and enough for ~4096 workgroups in all, but
// no more than one per 128 rows of an even spread of the consumers over the channels (a
// fixed function of the shape, so the sums keep one order on any device)
static int dummy_chunks(const Shape& sh) {
  const int pairs = sh.k * sh.Hkv;
  const long rows = (long)((sh.L + sh.k - 1) / sh.k) * (sh.Hq / sh.Hkv) * sh.B * sh.T_new;
  const int by_rows = (int)std::min(1024L, std::max(1L, (rows + 127) / 128));
  return std::min(by_rows, std::max(32, std::min(1024, (2048 + pairs - 1) / pairs)));
}

template <int DH>
__global__ __launch_bounds__(4 * DH) void attend_bwd_dummy_part_kernel(BwdArgs a, float* part) {
  constexpr int CG = DH / 8, R = 4 * DH / CG;  // column groups, rows per pass (32)
  __shared__ float s_v[R][DH], s_k[R][DH];
  const int nch = a.dchunks;
  const int ck = blockIdx.x / nch, chunk = blockIdx.x % nch;
  const int c = ck / a.Hkv, kvh = ck % a.Hkv;
  const int tid = threadIdx.x, cg = tid % CG, rl = tid / CG;
  const int G = a.Hq / a.Hkv;
  const long per_b = a.T, per_h = (long)a.B * per_b, per_m = G * per_h;
  const long nrow = (long)(a.grp.offsets[c + 1] - a.grp.offsets[c]) * per_m;
  const long r0 = nrow * chunk / nch, r1 = nrow * (chunk + 1) / nch;
  float av[8], ak[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) av[u] = ak[u] = 0.f;
  if (a.mask_paper && r0 + rl < r1) {
    // row rr = ((mi G + hg) B + b) T + i, stepped by R without divisions in the loop
    long rr = r0 + rl;
    int mi = (int)(rr / per_m), hg = (int)(rr / per_h % G), b = (int)(rr / per_b % a.B);
    int i = (int)(rr % per_b);
    for (; rr < r1; rr += R) {
      const int l = a.grp.members[a.grp.offsets[c] + mi], hq = kvh * G + hg;
      const long row = (((long)l * a.B + b) * a.Hq + hq) * a.T + i;
      const float pd = a.pd[row], ds = a.dsd[row];
      const bf16x8 dov = *(const bf16x8*)(a.dO + (((long)l * a.B + b) * a.T + i) * a.Hq * DH +
                                          (long)hq * DH + 8 * cg);
      const bf16x8 qv = *(const bf16x8*)(a.Q + row * DH + 8 * cg);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        av[u] += pd * (float)dov[u];
        ak[u] += ds * (float)qv[u];
      }
      i += R;
      while (i >= a.T) {
        i -= a.T;
        if (++b == a.B) {
          b = 0;
          if (++hg == G) {
            hg = 0;
            ++mi;
          }
        }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    s_v[rl][8 * cg + u] = av[u];
    s_k[rl][8 * cg + u] = ak[u];
  }
  __syncthreads();
  if (tid < 2 * DH) {
    const int e = tid % DH;
    const float(*src)[DH] = tid < DH ? s_v : s_k;
    float v = 0.f;
    for (int q = 0; q < R; ++q) v += src[q][e];
    part[(long)blockIdx.x * 2 * DH + tid] = v;  // V's sums, then K's
  }
}

// The chunks' partial sums, added in a fixed order: thread (q, e) of 4 DH sums chunks
// q, q + 4, ... of column e, then the four in order.
template <int DH>
__global__ __launch_bounds__(4 * DH) void attend_bwd_dummy_sum_kernel(BwdArgs a,
                                                                       const float* part) {
  __shared__ float s_v[4 * DH], s_k[4 * DH];
  const int ck = blockIdx.x, tid = threadIdx.x, e = tid % DH, q = tid / DH;
  float v = 0.f, k = 0.f;
  for (int ch = q; ch < a.dchunks; ch += 4) {
    const float* p = part + ((long)ck * a.dchunks + ch) * 2 * DH;
    v += p[e];
    k += p[DH + e];
  }
  s_v[tid] = v;
  s_k[tid] = k;
  __syncthreads();
  if (q == 0) {
    v = (s_v[e] + s_v[DH + e]) + (s_v[2 * DH + e] + s_v[3 * DH + e]);
    k = (s_k[e] + s_k[DH + e]) + (s_k[2 * DH + e] + s_k[3 * DH + e]);
    float* pv = a.dVd + (long)ck * DH + e;
    float* pk = a.dKd + (long)ck * DH + e;
    *pv = a.accumulate ? *pv + v : v;
    *pk = a.accumulate ? *pk + k * a.scale : k * a.scale;
  }
}

size_t attend_backward_rows_bytes(const Shape& sh) {
  return (4ul * sh.L * sh.B * sh.Hq * sh.T_new + 2ul * sh.k * sh.Hkv * dummy_chunks(sh) * sh.d) *
         sizeof(float);
}

void launch_attend_backward(const Shape& sh, const LayerTable& chan_map,
                            const ChannelGroups& groups, const bf16* Q, const bf16* Kc,
                            const bf16* Vc, const bf16* Kd, const bf16* Vd, const bf16* O,
                            const bf16* dO, const int32_t* ctx_len, float* dQ, float* dKc,
                            float* dVc, float* dKd, float* dVd, float* rows, hipStream_t s,
                            bool accumulate) {
  if (sh.N() <= 0) return;
  const long nrow = (long)sh.L * sh.B * sh.Hq * sh.T_new;
  BwdArgs a{Q, Kc, Vc, Kd, Vd, O, dO, ctx_len, dQ, dKc, dVc, dKd, dVd, rows, rows + nrow,
            rows + 2 * nrow, rows + 3 * nrow, sh.B, sh.T_new, sh.L, sh.Hq, sh.Hkv, sh.S_cap,
            sh.mask_paper, sh.ctx_hi, (sh.T_new + 32 * kBwdQWaves - 1) / (32 * kBwdQWaves),
            (int)(((long)sh.ctx_max + sh.span() + 32 * kBwdKWaves - 1) / (32 * kBwdKWaves)),
            kLog2e / sqrtf((float)sh.d),
            1.0f / sqrtf((float)sh.d), chan_map, groups, accumulate ? 1 : 0,
            dummy_chunks(sh), sh.gs, sh.gq, 0};
  {
    // small slot-major grids (two rounds at most) take their heavy tiles first; larger ones
    // keep each slice's tiles together, so they share its queries in one L2
    const long slices = (long)sh.Hkv * sh.B * sh.k;
    a.kv_heavy_first = slices % kNumXcd == 0 && (long)a.n_stiles * slices <= 2L * device_cus();
  }
  const dim3 ga(a.n_qtiles * sh.Hq * sh.B * sh.L), gb(a.n_stiles * sh.Hkv * sh.B * sh.k),
      gp(sh.k * sh.Hkv * a.dchunks), gs(sh.k * sh.Hkv);
  float* part = rows + 4 * nrow;
  if (sh.d == 64) {
    hipLaunchKernelGGL((attend_bwd_dq_kernel<64, kBwdQWaves>), ga, dim3(64 * kBwdQWaves), 0, s, a);
    hipLaunchKernelGGL((attend_bwd_dkv_kernel<64, kBwdKWaves>), gb, dim3(64 * kBwdKWaves), 0, s,
                       a);
    hipLaunchKernelGGL(attend_bwd_dummy_part_kernel<64>, gp, dim3(4 * 64), 0, s, a, part);
    hipLaunchKernelGGL(attend_bwd_dummy_sum_kernel<64>, gs, dim3(4 * 64), 0, s, a,
                       (const float*)part);
  } else {
    hipLaunchKernelGGL((attend_bwd_dq_kernel<96, kBwdQWaves>), ga, dim3(64 * kBwdQWaves), 0, s, a);
    hipLaunchKernelGGL((attend_bwd_dkv_kernel<96, kBwdKWaves>), gb, dim3(64 * kBwdKWaves), 0, s,
                       a);
    hipLaunchKernelGGL(attend_bwd_dummy_part_kernel<96>, gp, dim3(4 * 96), 0, s, a, part);
    hipLaunchKernelGGL(attend_bwd_dummy_sum_kernel<96>, gs, dim3(4 * 96), 0, s, a,
                       (const float*)part);
  }
}

}  // namespace wm
