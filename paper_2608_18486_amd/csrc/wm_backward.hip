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
//   attend_bwd_dkv_kernel  slot-major: a workgroup owns 128 slots of one channel, sequence
//                          and KV head and walks every query that reads them (all
//                          consumers of the channel, all grouped query heads), so each
//                          slot's dk and dv are summed in registers and written once.
//   attend_bwd_dummy_kernel  the dummy's dk, dv: a sum over every row of its readers.
// Products run on the matrix cores in bf16 (P and dS rounded to bf16 as operands), sums
// in fp32; gradients leave in fp32.
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
};

constexpr int kBwdThreads = 256;

__device__ __forceinline__ float bwd_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Copies rows row0 .. row0 + ROWS - 1 (DH bf16 each, row_bytes apart in the view) into an
// LDS block with the fragment readers' chunk swizzle; rows at or past nvalid read zeros.
template <int DH, int ROWS>
__device__ __forceinline__ void bwd_stage(char* dst, __amdgpu_buffer_rsrc_t view,
                                          uint32_t row_bytes, int row0, int nvalid, int tid) {
  constexpr int CPR = DH * 2 / 16;
#pragma unroll
  for (int ch = tid; ch < ROWS * CPR; ch += kBwdThreads) {
    const int r = ch / CPR, c = ch - r * CPR, gr = row0 + r;
    const uint32_t off = gr < nvalid ? (uint32_t)gr * row_bytes + 16u * c : kOffOob;
    *(i32x4*)(dst + r * 2 * DH + 16 * (c ^ pf_swz<DH>(r))) = buf_ld16(view, off);
  }
}

__device__ __forceinline__ bf16x4 bwd_ld8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

// --------------------------------------------------------------- dq, LSE, D
// Tile: 128 query rows of one (consumer, sequence, query head), 32 per wave; S^T = K q^T
// puts one query in a lane (as in the forward), dP^T = V dO^T likewise, and
// dq^T += K^T dS^T takes dS^T straight from those registers through the transposing
// read of the K block.
template <int DH>
__global__ __launch_bounds__(kBwdThreads) void attend_bwd_dq_kernel(BwdArgs a) {
  constexpr int NKS = DH / 16, NDT = DH / 32, ROW = 2 * DH, BLK = 64;
  __shared__ __align__(16) char smem[2 * BLK * ROW];  // K block, then V block
  const int tile = blockIdx.x;
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
  const int q0 = qtile * 128, qw0 = q0 + 32 * w, qi = qw0 + r;
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

  const int qlast = min(q0 + 127, a.T - 1);
  const int kend = min(pos0 + qlast + incl, a.S_cap);            // slots the tile may see
  const int wq_last = min(qw0 + 31, a.T - 1);
  const int wkend = wq_last >= qw0 ? pos0 + wq_last + incl : 0;  // ... this wave
  const int lim = pos0 + qi + incl;                              // ... this lane's row
  const int nblk = (kend + BLK - 1) / BLK;
  const long cbase = (((long)c * a.B + b) * a.Hkv + kvh) * (long)a.S_cap * DH;
  const auto kv = make_view(a.Kc + cbase, (uint32_t)max(kend, 0) * ROW);
  const auto vv = make_view(a.Vc + cbase, (uint32_t)max(kend, 0) * ROW);
  const PfLane<DH> lo = pf_lane<DH>(lane);

  // pass 1: the row's log-sum-exp (log2 units) over the dummy and the visible slots; the
  // two lanes of a row share the running maximum and keep partial sums
  float m = a.mask_paper ? sd : kNegBig;
  float sum = a.mask_paper && h == 0 ? 1.f : 0.f;
  for (int j = 0; j < nblk; ++j) {
    bwd_stage<DH, BLK>(smem, kv, ROW, j * BLK, kend, tid);
    __syncthreads();
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int s0 = j * BLK + 32 * hf;
      if (s0 < wkend) {
        f32x16 sc = zero16();
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) sc = mma32(sc, pf_ldk<DH>(smem, lo, hf * 32 * ROW, ks), qf[ks]);
        float mx = kNegBig;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int s = s0 + 8 * (q >> 2) + 4 * h + (q & 3);
          sc[q] = s < lim ? sc[q] * cl2 : kNegBig;
          mx = fmaxf(mx, sc[q]);
        }
        const float mn = fmaxf(m, halves_max(mx));
        float part = 0.f;
#pragma unroll
        for (int q = 0; q < 16; ++q) part += bwd_exp2(sc[q] - mn);
        sum = sum * bwd_exp2(m - mn) + part;
        m = mn;
      }
    }
    __syncthreads();
  }
  const float lse = m + __log2f(halves_sum(sum));

  // pass 2: dS and dq^T += K^T dS^T
  f32x16 dq[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) dq[dt] = zero16();
  for (int j = 0; j < nblk; ++j) {
    bwd_stage<DH, BLK>(smem, kv, ROW, j * BLK, kend, tid);
    bwd_stage<DH, BLK>(smem + BLK * ROW, vv, ROW, j * BLK, kend, tid);
    __syncthreads();
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int s0 = j * BLK + 32 * hf;
      if (s0 < wkend) {
        f32x16 sc = zero16(), dp = zero16();
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          sc = mma32(sc, pf_ldk<DH>(smem, lo, hf * 32 * ROW, ks), qf[ks]);
          dp = mma32(dp, pf_ldk<DH>(smem, lo, BLK * ROW + hf * 32 * ROW, ks), df[ks]);
        }
        bf16x8 ds[2];
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int s = s0 + 8 * (q >> 2) + 4 * h + (q & 3);
          const float p = s < lim ? bwd_exp2(sc[q] * cl2 - lse) : 0.f;
          ds[q >> 3][q & 7] = (bf16)(p * (dp[q] - delta));
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int kh = 0; kh < 2; ++kh)
            dq[dt] = mma32(dq[dt], pf_ldv<DH>(smem, lo, hf * 32 * ROW, kh, dt), ds[kh]);
      }
    }
    __syncthreads();
  }

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
// Tile: 128 slots of one (channel, sequence, KV head), 32 per wave; the wave's K and V
// rows stay in registers as the column operand. For each 32-row query block (staged in
// LDS with its LSE and D): S = Q K^T and dP = dO V^T put one slot in a lane, and
// dv^T += dO^T P and dk^T += Q^T dS take P and dS from those registers through the
// transposing reads of the dO and Q blocks.
template <int DH>
__global__ __launch_bounds__(kBwdThreads) void attend_bwd_dkv_kernel(BwdArgs a) {
  constexpr int NKS = DH / 16, NDT = DH / 32, ROW = 2 * DH, QB = 32;
  __shared__ __align__(16) char smem[2 * QB * ROW];  // Q block, then dO block
  __shared__ __align__(16) float s_lse[QB], s_dlt[QB];
  const int tile = blockIdx.x;
  const int stile = tile % a.n_stiles;
  int y = tile / a.n_stiles;
  const int kvh = y % a.Hkv;
  y /= a.Hkv;
  const int b = y % a.B, c = y / a.B;
  const int G = a.Hq / a.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pos0 = __builtin_amdgcn_readfirstlane(ctx_at(a.ctx_len, b, a.ctx_hi));
  const int incl = a.mask_paper ? 0 : 1;
  const int send = pos0 + a.T;  // slots written: [0, send)
  const int sbase = stile * 128;
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
  // the first query that sees slot sbase sits at position sbase + 1 - incl
  const int i_first = max(0, sbase + 1 - incl - pos0);
  const uint32_t ostride = (uint32_t)a.Hq * DH * 2u;

  for (int mi = a.grp.offsets[c]; mi < a.grp.offsets[c + 1]; ++mi) {
    const int l = a.grp.members[mi];
    for (int hg = 0; hg < G; ++hg) {
      const int hq = kvh * G + hg;
      const long rows0 = (((long)l * a.B + b) * a.Hq + hq) * a.T;  // (l, b, hq, 0) in [L][B][Hq][T]
      const long rowl = ((long)l * a.B + b) * a.T;                 // (l, b, 0) in [L][B][T][Hq d]
      const auto qv = make_view(a.Q + rows0 * DH, (uint32_t)a.T * DH * 2u);
      const auto dov = make_view(a.dO + rowl * a.Hq * DH + (long)hq * DH, (uint32_t)a.T * ostride);
      for (int qb = i_first / QB; qb * QB < a.T; ++qb) {
        bwd_stage<DH, QB>(smem, qv, DH * 2u, qb * QB, a.T, tid);
        bwd_stage<DH, QB>(smem + QB * ROW, dov, ostride, qb * QB, a.T, tid);
        if (tid < QB) {
          const int qr = qb * QB + tid;
          s_lse[tid] = qr < a.T ? a.lse[rows0 + qr] : 1.0e30f;  // a row past T weighs 0
          s_dlt[tid] = qr < a.T ? a.dlt[rows0 + qr] : 0.f;
        }
        __syncthreads();
        // the block's last row, at position pos0 + qb QB + QB - 1, sees slots below
        // that + incl: skip when the wave's first slot is not among them
        if (pos0 + min(qb * QB + QB - 1, a.T - 1) + incl > ws0) {
          f32x16 sc = zero16(), dp = zero16();
#pragma unroll
          for (int ks = 0; ks < NKS; ++ks) {
            sc = mma32(sc, pf_ldk<DH>(smem, lo, 0, ks), kf[ks]);
            dp = mma32(dp, pf_ldk<DH>(smem, lo, QB * ROW, ks), vf[ks]);
          }
          // lane (h, r): slot r of the wave, query rows 8 (i / 4) + 4 h + i % 4 of the block
          bf16x8 pp[2], pds[2];
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x4 lz = *(const f32x4*)(s_lse + 8 * g + 4 * h);
            const f32x4 dz = *(const f32x4*)(s_dlt + 8 * g + 4 * h);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int i = 4 * g + e, qr = qb * QB + 8 * g + 4 * h + e;
              const float p = slot < pos0 + qr + incl ? bwd_exp2(sc[i] * cl2 - lz[e]) : 0.f;
              pp[i >> 3][i & 7] = (bf16)p;
              pds[i >> 3][i & 7] = (bf16)(p * (dp[i] - dz[e]));
            }
          }
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int kh = 0; kh < 2; ++kh) {
              dv[dt] = mma32(dv[dt], pf_ldv<DH>(smem, lo, QB * ROW, kh, dt), pp[kh]);
              dk[dt] = mma32(dk[dt], pf_ldv<DH>(smem, lo, 0, kh, dt), pds[kh]);
            }
        }
        __syncthreads();
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
        *(f32x4*)(dkd + 32 * dt + 8 * g + 4 * h) = kq;
        *(f32x4*)(dvd + 32 * dt + 8 * g + 4 * h) = vq;
      }
  }
}

// -------------------------------------------------------------------- dummy
// One workgroup per (channel, KV head), 4 DH threads: thread (rl, e) sums column e over
// every fourth row of the channel's readers, then the four partial sums are added.
template <int DH>
__global__ __launch_bounds__(4 * DH) void attend_bwd_dummy_kernel(BwdArgs a) {
  __shared__ float s_v[4 * DH], s_k[4 * DH];
  const int c = blockIdx.x / a.Hkv, kvh = blockIdx.x % a.Hkv;
  const int tid = threadIdx.x, e = tid % DH, rl = tid / DH;
  const int G = a.Hq / a.Hkv;
  float av = 0.f, ak = 0.f;
  if (a.mask_paper) {
    for (int mi = a.grp.offsets[c]; mi < a.grp.offsets[c + 1]; ++mi) {
      const int l = a.grp.members[mi];
      for (int hg = 0; hg < G; ++hg) {
        const int hq = kvh * G + hg;
        for (int b = 0; b < a.B; ++b) {
          const long rows0 = (((long)l * a.B + b) * a.Hq + hq) * a.T;
          const long rowl = ((long)l * a.B + b) * a.T;
          for (int i = rl; i < a.T; i += 4) {
            av += a.pd[rows0 + i] * (float)a.dO[(rowl + i) * a.Hq * DH + (long)hq * DH + e];
            ak += a.dsd[rows0 + i] * (float)a.Q[(rows0 + i) * DH + e];
          }
        }
      }
    }
  }
  s_v[tid] = av;
  s_k[tid] = ak;
  __syncthreads();
  if (rl == 0) {
    const long o = ((long)c * a.Hkv + kvh) * DH + e;
    a.dVd[o] = (s_v[e] + s_v[DH + e]) + (s_v[2 * DH + e] + s_v[3 * DH + e]);
    a.dKd[o] = ((s_k[e] + s_k[DH + e]) + (s_k[2 * DH + e] + s_k[3 * DH + e])) * a.scale;
  }
}

size_t attend_backward_rows_bytes(const Shape& sh) {
  return 4ul * sh.L * sh.B * sh.Hq * sh.T_new * sizeof(float);
}

void launch_attend_backward(const Shape& sh, const LayerTable& chan_map,
                            const ChannelGroups& groups, const bf16* Q, const bf16* Kc,
                            const bf16* Vc, const bf16* Kd, const bf16* Vd, const bf16* O,
                            const bf16* dO, const int32_t* ctx_len, float* dQ, float* dKc,
                            float* dVc, float* dKd, float* dVd, float* rows, hipStream_t s) {
  if (sh.N() <= 0) return;
  const long nrow = (long)sh.L * sh.B * sh.Hq * sh.T_new;
  BwdArgs a{Q, Kc, Vc, Kd, Vd, O, dO, ctx_len, dQ, dKc, dVc, dKd, dVd, rows, rows + nrow,
            rows + 2 * nrow, rows + 3 * nrow, sh.B, sh.T_new, sh.L, sh.Hq, sh.Hkv, sh.S_cap,
            sh.mask_paper, sh.ctx_hi, (sh.T_new + 127) / 128,
            (int)(((long)sh.ctx_max + sh.T_new + 127) / 128), kLog2e / sqrtf((float)sh.d),
            1.0f / sqrtf((float)sh.d), chan_map, groups};
  const dim3 ga(a.n_qtiles * sh.Hq * sh.B * sh.L), gb(a.n_stiles * sh.Hkv * sh.B * sh.k),
      gc(sh.k * sh.Hkv);
  if (sh.d == 64) {
    hipLaunchKernelGGL(attend_bwd_dq_kernel<64>, ga, dim3(kBwdThreads), 0, s, a);
    hipLaunchKernelGGL(attend_bwd_dkv_kernel<64>, gb, dim3(kBwdThreads), 0, s, a);
    hipLaunchKernelGGL(attend_bwd_dummy_kernel<64>, gc, dim3(4 * 64), 0, s, a);
  } else {
    hipLaunchKernelGGL(attend_bwd_dq_kernel<96>, ga, dim3(kBwdThreads), 0, s, a);
    hipLaunchKernelGGL(attend_bwd_dkv_kernel<96>, gb, dim3(kBwdThreads), 0, s, a);
    hipLaunchKernelGGL(attend_bwd_dummy_kernel<96>, gc, dim3(4 * 96), 0, s, a);
  }
}

}  // namespace wm
