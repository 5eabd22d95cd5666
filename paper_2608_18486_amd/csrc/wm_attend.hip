// Per-layer channel attention (paper Section 3.1 Step 3, Section 3.2).
//
// Consumer layer l reads channel c = map[l] of the channel-major cache
// Kc/Vc[k][B][Hkv][S_cap][d]. A query at position t sees, in the paper's mask,
// the learned dummy slot of its channel and the cached slots s < t (a token
// never reads its own channels); in the inclusive mask it sees slots s <= t and
// no dummy. The dummy enters the online softmax as its initial state
// (m = q.Kd, l = 1, acc = Vd), which is exactly a prepended KV slot.
//
// Full-sequence form (attend_prefill): flash attention on the matrix cores.
// Each wave owns 64 queries and computes S^T = K Q^T so that a lane holds one
// query's scores in registers (row max and sum need one cross-half exchange),
// then O^T = V^T P^T with P^T taken straight from those registers (the MFMA
// k-slot order is chosen to match; see wm_device.hpp). K blocks are staged
// row-major in LDS; bf16 V blocks too, read as V^T fragments with the transposing
// LDS read (fp32 V is stored transposed).
//
// Decode form (attend_decode + combine): split-S over the cache, one
// workgroup per (split, channel, sequence, KV head) serving every query row
// that reads that channel and head (all its consumer layers, grouped query
// heads and new tokens), so each channel slice is streamed from HBM once.
#include <atomic>
#include <type_traits>

#include "wm_device.hpp"
#include "wm_frag.hpp"
#include "wm_internal.hpp"

namespace wm {

template <typename T>
__device__ __forceinline__ frag_t<T> ld_frag_4_4(const T* p0, const T* p1);
template <>
__device__ __forceinline__ bf16x8 ld_frag_4_4<bf16>(const bf16* p0, const bf16* p1) {
  bf16x4 a = *(const bf16x4*)p0, b = *(const bf16x4*)p1;
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
template <>
__device__ __forceinline__ f32x8 ld_frag_4_4<float>(const float* p0, const float* p1) {
  f32x4 a = *(const f32x4*)p0, b = *(const f32x4*)p1;
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// A lane's sum of 16 softmax weights above this (some weight above 2^12) triggers the
// rescale of the running state; `!(ps <= kGrowSum)` also catches inf and NaN.
constexpr float kGrowSum = 65536.0f;
// Reference of a row that has seen no slot yet, in log2 units. Finite and small, so
// scores offset by it keep their digits; a row still at kNoRef always takes the
// exact-max rescale, which then sets the reference to the row's exact maximum (up or
// down: its state is still zero). Only a step that hides every slot from the row
// leaves it at kNoRef.
constexpr float kNoRef = -100.0f;

// Growth of a row's reference at a rescale, from the step's row maximum mx (in log2
// units relative to the current reference m): never down once a slot has been read;
// from kNoRef, exactly to the row maximum unless the step hid every slot from the row.
__device__ __forceinline__ float ref_growth(float mx, float m) {
  return m == kNoRef ? (mx > 0.5f * kNegBig ? mx : 0.f) : fmaxf(mx, 0.f);
}
// Factor of the running state at that rescale: a row still at kNoRef has a zero state,
// and exp2(-growth) could overflow when the reference moves down.
__device__ __forceinline__ float ref_rescale(float growth, float m) {
  return m == kNoRef ? 0.f : fast_exp2(-growth);
}

// Document mask (packed sequences, Section 4.1): query i of sequence b, at position
// ctx + i, reads cached slots from its document's first position on (clamped into
// [0, position]); the dummy slot stays visible. Without a document array every row
// starts at slot 0.
__device__ __forceinline__ int doc_first(const int32_t* doc, int b, int T_new, int i, int pos) {
  if (!doc) return 0;
  return min(max(doc[(long)b * T_new + i], 0), pos);
}
__device__ __forceinline__ int wave_min_i(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = min(v, __shfl_xor(v, m, 64));
  return v;
}
__device__ __forceinline__ int wave_max_i(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = max(v, __shfl_xor(v, m, 64));
  return v;
}

template <typename T> struct AttnArgs {
  const T *Q, *Kc, *Vc, *Kd, *Vd;
  const int32_t* ctx_len;
  const int32_t* doc;  // [B][T_new] first position of each token's document, or null
  T* O;
  int B, T_new, L, Hq, Hkv, S_cap, mask_paper, n_qtiles;
  int gs, gq, ctx_hi;  // query i of sequence b sits at position ctx_len[b] + gq + gs i
  float scale_log2;  // log2(e) / sqrt(d)
  LayerTable chan;
  LayerTable lord;  // the consumers in channel order (the bf16 kernels' tile order)
  // split slot ranges (bf16 full-sequence kernel, small grids): each query tile's walk is
  // cut into nsplit ranges of split_blk 64-slot blocks, one workgroup each, whose partial
  // softmax states go to part and are merged by attend_split_combine_kernel (nsplit = 1:
  // one workgroup walks the whole range and writes O)
  int nsplit, split_blk;
  float* part;
};

#ifndef WM_PREFILL_WAVES
#define WM_PREFILL_WAVES 8
#endif
constexpr int kPrefillWaves = WM_PREFILL_WAVES;  // waves per prefill workgroup

template <typename T, int DH> struct PrefillCfg {
  static constexpr int NW = kPrefillWaves;
  static constexpr int QT = 256 / (32 * NW);  // 32-query tiles per wave (256 queries per block)
  static constexpr int NT = 64 * NW;    // threads
  static constexpr int BQ = 32 * QT * NW;  // queries per workgroup
  static constexpr int BKV = 64;        // keys per block
  static constexpr int PAD = sizeof(T) == 2 ? 8 : 4;
  static constexpr int LDK = DH + PAD;   // Ks: [BKV][LDK]
  // bf16 V is staged row-major like K ([BKV][LDV], read transposed by ds_read_b64_tr_b16);
  // fp32 V is stored transposed ([DH][LDV])
  static constexpr bool VTR = sizeof(T) == 2;
  static constexpr int LDV = VTR ? DH + 16 : BKV + PAD;
  static constexpr int VS = VTR ? BKV * LDV : DH * LDV;  // V stage (elements)
  static constexpr int NKS = DH / 16;    // k16 steps of Q K^T
  static constexpr int NDT = DH / 32;    // 32-row tiles of O^T
  static constexpr int KIT = BKV * DH / 8;             // K fragments per block
  static constexpr int KFR = (KIT + NT - 1) / NT;      // ... per thread
  static constexpr int VIT = VTR ? KIT : (BKV / 2) * (DH / 8);  // V items per block (16-B
                                                                 // fragments, or key pairs)
  static constexpr int VPT = (VIT + NT - 1) / NT;      // ... per thread
};

// Paired-key transposed store of two V rows' 8 columns: Vt[c][key], Vt[c][key+1].
__device__ __forceinline__ void st_pair_t(bf16* vt, int ld, const bf16x8& a, const bf16x8& b) {
#pragma unroll
  for (int i = 0; i < 8; ++i) *(bf16x2*)(vt + i * ld) = bf16x2{a[i], b[i]};
}
__device__ __forceinline__ void st_pair_t(float* vt, int ld, const f32x8& a, const f32x8& b) {
  typedef __attribute__((ext_vector_type(2))) float f32x2;
#pragma unroll
  for (int i = 0; i < 8; ++i) *(f32x2*)(vt + i * ld) = f32x2{a[i], b[i]};
}

// V^T fragment for keys kb + 4h + {0..3, 8..11} and value column 32 dt + r from a
// row-major bf16 V tile, with two transposing LDS reads: within each 16-lane group,
// lane i's element t comes from element i % 4 of the 8-byte chunk addressed by lane
// 4t + i / 4, so lane j addresses key (kb + 4h + 8s + j / 4), columns
// 32 dt + 16 (group & 1) + 4 (j % 4) .. + 3, and receives 4 keys of its own column.
__device__ __forceinline__ bf16x8 ld_vt_tr(const bf16* vs, int ldv, int kb, int dt, int lane) {
  const int j = lane & 15, grp = lane >> 4, h = lane >> 5;
  const bf16* p = vs + (kb + 4 * h + (j >> 2)) * ldv + 32 * dt + 16 * (grp & 1) + 4 * (j & 3);
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 8 * ldv));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// One 64-key block for one wave (QT tiles of 32 queries): two 32-key halves, each
// S^T = K Q^T, online-softmax update (lazy rescale), O^T += V^T P^T. MASK selects the
// code for blocks that straddle the causal boundary of some of the wave's rows.
template <typename T, int DH, bool MASK>
__device__ __forceinline__ void attend_block(
    const T* __restrict__ ks_, const T* __restrict__ vt_,
    const frag_t<T> (&qf)[PrefillCfg<T, DH>::QT][DH / 16], float (&m)[PrefillCfg<T, DH>::QT],
    float (&lsum)[PrefillCfg<T, DH>::QT], f32x16 (&o)[DH / 32][PrefillCfg<T, DH>::QT], int k0,
    int wkend, int tq0, int gs, int incl, const int (&dlo)[PrefillCfg<T, DH>::QT], int h,
    int r) {
  using C = PrefillCfg<T, DH>;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    if (MASK && k0 + 32 * kt >= wkend) break;  // this half is past every row of the wave
    // Q is pre-scaled by log2(e)/sqrt(d): s' is the score in log2 units, m' the row's
    // reference. In bf16 the scores start from -m', so the MFMAs leave s' - m' and the
    // weight needs no subtraction; fp32 starts from 0 (summing on top of m' would cost
    // fp32 parity a few ulps of m') and subtracts m' itself.
    constexpr bool kOffsetInit = sizeof(T) == 2;
    f32x16 st[C::QT];
    float off[C::QT];
#pragma unroll
    for (int qt = 0; qt < C::QT; ++qt) {
      off[qt] = kOffsetInit ? 0.f : m[qt];
#pragma unroll
      for (int q = 0; q < 16; ++q) st[qt][q] = kOffsetInit ? -m[qt] : 0.f;
    }
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks) {
      frag_t<T> kf = ld_frag<T>(ks_ + (32 * kt + r) * C::LDK + 16 * ks + 8 * h);
#pragma unroll
      for (int qt = 0; qt < C::QT; ++qt) st[qt] = mma32(st[qt], kf, qf[qt][ks]);
    }
    frag_t<T> pf[C::QT][2];  // [qt][hf]
#pragma unroll
    for (int qt = 0; qt < C::QT; ++qt) {
      if (MASK) {
        // slot k0 + 32kt + 8(q/4) + 4h + q%4 is visible to the row at position t iff
        // it is < t + incl and at least the row's document start (row 32 qt + r of the
        // wave sits at position tq0 + gs (32 qt + r))
        const int base = k0 + 32 * kt + 4 * h;
        const int lim = tq0 + gs * (32 * qt + r) + incl - base, lo = dlo[qt] - base;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int off = 8 * (q >> 2) + (q & 3);
          if (off >= lim || off < lo) st[qt][q] = kNegBig;
        }
      }
      // Weights against the current reference m first: while every weight stays below
      // 2^12 (so a lane's sum of 16 stays below 2^16) no rescale is needed. Otherwise
      // (rare: a row's first block, or a score far above m) take the exact row max,
      // rescale the running state to it and recompute. Masked slots hold -1e30: weight 0.
      float pv[16], ps = 0.f;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        pv[q] = fast_exp2(st[qt][q] - off[qt]);
        ps += pv[q];
      }
      if (__any(!(ps <= kGrowSum) || m[qt] == kNoRef)) {
        float mx = st[qt][0];
#pragma unroll
        for (int q = 1; q < 16; ++q) mx = fmaxf(mx, st[qt][q]);
        mx = ref_growth(halves_max(mx) - off[qt], m[qt]);  // growth of the reference
        const float alpha = ref_rescale(mx, m[qt]);
        m[qt] += mx;
        lsum[qt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < C::NDT; ++dt) o[dt][qt] *= alpha;
        ps = 0.f;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          pv[q] = fast_exp2(st[qt][q] - off[qt] - mx);
          ps += pv[q];
        }
      }
#pragma unroll
      for (int q = 0; q < 16; ++q) pf[qt][q >> 3][q & 7] = from_f32<T>(pv[q]);
      lsum[qt] += ps;
    }
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int kc = 32 * kt + 16 * hf + 4 * h;
#pragma unroll
      for (int dt = 0; dt < C::NDT; ++dt) {
        frag_t<T> vf;
        if constexpr (C::VTR) {
          vf = ld_vt_tr(vt_, C::LDV, 32 * kt + 16 * hf, dt, 32 * h + r);
        } else {
          const T* vrow = vt_ + (32 * dt + r) * C::LDV;
          vf = ld_frag_4_4<T>(vrow + kc, vrow + kc + 8);
        }
#pragma unroll
        for (int qt = 0; qt < C::QT; ++qt) o[dt][qt] = mma32(o[dt][qt], vf, pf[qt][hf]);
      }
    }
  }
}

template <typename T, int DH>
__global__ __launch_bounds__(64 * kPrefillWaves) void attend_prefill_kernel(AttnArgs<T> a) {
  using C = PrefillCfg<T, DH>;
  constexpr int QT = C::QT;
  __shared__ __align__(16) T Ks[2][C::BKV * C::LDK];
  __shared__ __align__(16) T Vt[2][C::VS];

  // 1-D grid over (consumer, sequence, head, query tile); each XCD takes a contiguous
  // run of heads, and a head's tiles run longest causal rows first on one L2
  const int tile = xcd_tile(blockIdx.x, a.n_qtiles * a.Hq * a.B * a.L);
  const int qtile = a.n_qtiles - 1 - tile % a.n_qtiles;
  int y = tile / a.n_qtiles;
  const int hq = y % a.Hq;
  y /= a.Hq;
  const int b = y % a.B, l = y / a.B;
  const int c = a.chan.v[l];
  const int kvh = hq / (a.Hq / a.Hkv);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, r = lane & 31;
  const int ctx = __builtin_amdgcn_readfirstlane(ctx_at(a.ctx_len, b, a.ctx_hi));
  const int incl = a.mask_paper ? 0 : 1;
  const int q0 = qtile * C::BQ, qw0 = q0 + 32 * QT * w;
  const float cl2 = a.scale_log2;
  const int gs = a.gs, pos0 = ctx + a.gq;  // query i sits at position pos0 + gs i

  // document mask: each row's first readable slot; the walk starts at the block holding
  // the workgroup's least one (base0), and slot indices below are relative to base0
  __shared__ int s_lo[C::NW];
  int dlo[QT], base0 = 0, wlo_max = 0, wlo_min = 0;  // wlo_min: blocks below it are skipped
  if (a.doc) {
    int wmin = 0x7fffffff;
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const int qi = qw0 + 32 * qt + r;
      dlo[qt] = qi < a.T_new ? doc_first(a.doc, b, a.T_new, qi, pos0 + gs * qi) : 0;
      wmin = min(wmin, qi < a.T_new ? dlo[qt] : 0x7fffffff);
      wlo_max = max(wlo_max, dlo[qt]);
    }
    wmin = __builtin_amdgcn_readfirstlane(wave_min_i(wmin));
    wlo_max = __builtin_amdgcn_readfirstlane(wave_max_i(wlo_max));
    if (lane == 0) s_lo[w] = wmin;
    __syncthreads();
    int gmin = s_lo[0];
#pragma unroll
    for (int k = 1; k < C::NW; ++k) gmin = min(gmin, s_lo[k]);
    base0 = __builtin_amdgcn_readfirstlane(gmin / C::BKV * C::BKV);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) dlo[qt] -= base0;
    wlo_max -= base0;
    wlo_min = wmin == 0x7fffffff ? 0 : wmin - base0;
  } else {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) dlo[qt] = 0;
  }
  const int ctxr = pos0 - base0, scap = a.S_cap - base0;  // query 0's position from base0

  const long cbase = (((long)c * a.B + b) * a.Hkv + kvh) * (long)a.S_cap * DH +
                     (long)base0 * DH;
  const T* Kb = a.Kc + cbase;
  const T* Vb = a.Vc + cbase;

  frag_t<T> qf[QT][C::NKS];
  const T* Qb = a.Q + (((long)l * a.B + b) * a.Hq + hq) * (long)a.T_new * DH;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    int qi = qw0 + 32 * qt + r;
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks)
      qf[qt][ks] = qi < a.T_new ? ld_frag<T>(Qb + (long)qi * DH + 16 * ks + 8 * h) : zero_frag<T>();
  }
  // queries in log2 units: the MFMAs then give s' = q.k log2(e) / sqrt(d), and the
  // softmax weight of a slot is exp2(s' - m') with m' the row's running reference
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks)
#pragma unroll
      for (int i = 0; i < 8; ++i) qf[qt][ks][i] = from_f32<T>(to_f32(qf[qt][ks][i]) * cl2);

  // running state per query row (lanes r and r + 32 hold the same row): reference max,
  // partial row sum (each half-wave sums its own keys), and O^T
  float m[QT], lsum[QT];
  f32x16 o[C::NDT][QT];
  if (a.mask_paper) {
    const T* kd = a.Kd + ((long)c * a.Hkv + kvh) * DH;
    const T* vd = a.Vd + ((long)c * a.Hkv + kvh) * DH;
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float part = 0.f;
#pragma unroll
      for (int ks = 0; ks < C::NKS; ++ks)
#pragma unroll
        for (int i = 0; i < 8; ++i) part += to_f32(qf[qt][ks][i]) * to_f32(kd[16 * ks + 8 * h + i]);
      m[qt] = halves_sum(part);
      lsum[qt] = h == 0 ? 1.f : 0.f;
#pragma unroll
      for (int dt = 0; dt < C::NDT; ++dt)
#pragma unroll
        for (int q = 0; q < 16; ++q) o[dt][qt][q] = to_f32(vd[32 * dt + 8 * (q >> 2) + 4 * h + (q & 3)]);
    }
  } else {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      m[qt] = kNoRef;
      lsum[qt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < C::NDT; ++dt) o[dt][qt] = zero16();
    }
  }

  const int qlast = min(q0 + C::BQ, a.T_new) - 1;
  const int kend = min(ctxr + gs * qlast + incl, scap);    // slots the workgroup may see
  const int wq_last = min(qw0 + 32 * QT - 1, a.T_new - 1);
  const int wkend = wq_last >= qw0 ? ctxr + gs * wq_last + incl : 0;  // slots this wave may see
  // slots in [wlo_max, wfree) are visible to all its rows
  const int wfree = ctxr + gs * qw0 + incl;
  const int nblk = (kend + C::BKV - 1) / C::BKV;

  // staged next block: K fragments (row-major copy) and V fragments (row-major, bf16)
  // or V key pairs (transposed store, fp32)
  frag_t<T> kreg[C::KFR], vreg[C::VPT][C::VTR ? 1 : 2];
  // the (channel, sequence, KV head) slice through buffer views: slots at or past kend
  // read as zeros without a branch
  const __amdgpu_buffer_rsrc_t kview = make_view(Kb, (uint32_t)scap * DH * sizeof(T));
  const __amdgpu_buffer_rsrc_t vview = make_view(Vb, (uint32_t)scap * DH * sizeof(T));
  auto slot_off = [&](int s, int col) {
    return s < kend ? (uint32_t)(s * DH + col) * (uint32_t)sizeof(T) : kOffOob;
  };
  auto fetch = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::KFR; ++i) {
      int f = tid + C::NT * i, key = f / (DH / 8), dc = (f % (DH / 8)) * 8;
      kreg[i] = buf_frag<T>(kview, f < C::KIT ? slot_off(k0 + key, dc) : kOffOob);
    }
#pragma unroll
    for (int i = 0; i < C::VPT; ++i) {
      int it = tid + C::NT * i;
      bool ok = it < C::VIT;
      if constexpr (C::VTR) {
        int key = it / (DH / 8), dc = (it % (DH / 8)) * 8;
        vreg[i][0] = buf_frag<T>(vview, ok ? slot_off(k0 + key, dc) : kOffOob);
      } else {
        int kp = it % (C::BKV / 2), dg = it / (C::BKV / 2), s = k0 + 2 * kp;
        vreg[i][0] = buf_frag<T>(vview, ok ? slot_off(s, 8 * dg) : kOffOob);
        vreg[i][1] = buf_frag<T>(vview, ok ? slot_off(s + 1, 8 * dg) : kOffOob);
      }
    }
  };
  auto stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < C::KFR; ++i) {
      int f = tid + C::NT * i, key = f / (DH / 8), dc = (f % (DH / 8)) * 8;
      if (f < C::KIT) st_frag<T>(&Ks[buf][key * C::LDK + dc], kreg[i]);
    }
#pragma unroll
    for (int i = 0; i < C::VPT; ++i) {
      int it = tid + C::NT * i;
      if (it < C::VIT) {
        if constexpr (C::VTR) {
          int key = it / (DH / 8), dc = (it % (DH / 8)) * 8;
          st_frag<T>(&Vt[buf][key * C::LDV + dc], vreg[i][0]);
        } else {
          int kp = it % (C::BKV / 2), dg = it / (C::BKV / 2);
          st_pair_t(&Vt[buf][(8 * dg) * C::LDV + 2 * kp], C::LDV, vreg[i][0], vreg[i][1]);
        }
      }
    }
  };

  // fetch and stage run unconditionally (a block past kend reads zeros and lands in the
  // idle buffer), so the only branches in the loop are wave-uniform compute skips
  fetch(0);
  stage(0);
  __syncthreads();
  for (int j = 0; j < nblk; ++j) {
    const int k0 = j * C::BKV, buf = j & 1;
    fetch(k0 + C::BKV);
    if (k0 < wkend && k0 + C::BKV > wlo_min) {
      if (k0 + C::BKV > wfree || k0 < wlo_max)
        attend_block<T, DH, true>(Ks[buf], Vt[buf], qf, m, lsum, o, k0, wkend,
                                  ctxr + gs * qw0, gs, incl, dlo, h, r);
      else
        attend_block<T, DH, false>(Ks[buf], Vt[buf], qf, m, lsum, o, k0, wkend,
                                   ctxr + gs * qw0, gs, incl, dlo, h, r);
    }
    stage(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qi = qw0 + 32 * qt + r;
    const float lt = halves_sum(lsum[qt]);
    if (qi >= a.T_new) continue;
    const float inv = 1.0f / lt;
    T* dst = a.O + ((((long)l * a.B + b) * a.T_new + qi) * a.Hq + hq) * DH;
#pragma unroll
    for (int dt = 0; dt < C::NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = o[dt][qt][4 * g + i] * inv;
        store4(dst + 32 * dt + 8 * g + 4 * h, v);
      }
  }
}

// ---------------------------------------------- prefill, bf16, head dims 64 and 96
// K/V blocks of 64 slots are copied from HBM straight into LDS (no trip through
// registers), two barriers per block. A slot row is 2 DH bytes (8 or 12 chunks of 16 B);
// its chunk c sits at chunk c ^ pf_swz(row) of the LDS row. That makes both readers
// free of bank conflicts: the K fragment reads (16 rows, one chunk) and the transposing
// V reads (4 rows x 4 chunks per 32 lanes).
//
// Each wave owns QT tiles of 32 queries and walks its keys in 32-slot steps. Step i
// issues the MFMAs of S(i+1) = K Q^T and of O^T += V^T P(i-1)^T, and meanwhile computes
// the softmax weights P(i) of S(i) on the vector ALUs, so the matrix cores and the ALUs
// work on independent data. Every K or V fragment read from LDS feeds QT MFMAs.
// Workgroup shape: 4 waves of one 32-query tile each and rings of 3 blocks. Head dim
// 64: 48 KB of LDS and at most 168 registers per lane, so a CU holds three workgroups
// (3 waves per SIMD, each from a different workgroup, so no two waves of a SIMD wait at
// the same barrier). Measured on MI355X and slower: 8-wave workgroups (4 waves per
// SIMD, in lock-step pairs; 128 registers), and 2 query tiles per wave (2 waves per
// SIMD). Head dim 96: 72 KB and two workgroups per CU; a step has 12 MFMAs (6 for the
// scores, 6 for the output) against the same 16 exponentials per lane.
constexpr int kPfWaves = 4, kPfNs = 3, kPfQt = 1;
// work queue of the persistent kernel: one counter per XCD, 64 bytes apart
constexpr int kQueueStride = 16, kQueueWords = kNumXcd * kQueueStride;
static_assert(kQueueWords * 4 == kPrefillQueueBytes, "queue size");
template <int QT, int DH_> struct PfDma {
  static constexpr int NW = kPfWaves, NT = 64 * NW;
  static constexpr int BQ = 32 * QT * NW;              // queries per workgroup
  static constexpr int BKV = 64, DH = DH_;
  static constexpr int NKS = DH / 16;                  // k16 steps of S (= step groups)
  static constexpr int NDT = DH / 32;                  // 32-column tiles of O^T
  static constexpr int ROW_BYTES = DH * 2;             // one slot row of K or V
  static constexpr int CPR = ROW_BYTES / 16;           // 16-B chunks per row
  static constexpr int BLK_BYTES = BKV * ROW_BYTES;    // one K (or V) block
  static constexpr int RPW = BKV / NW;                 // block rows each wave copies
  static constexpr int NI = RPW * ROW_BYTES / 1024;    // ... in copy instructions of 1 KB
  // Two rings of NS blocks. While block j is processed, K of j and j+1 and V of j-1 and
  // j are read; K of j+2 and V of j+1 (and, with 4 blocks, K of j+3 and V of j+2) are
  // in flight.
  static constexpr int NS = kPfNs;
  static constexpr int V_BASE = NS * BLK_BYTES;        // K ring first, then the V ring
  static constexpr int SMEM_BYTES = 2 * NS * BLK_BYTES;
  static constexpr int WPE = DH == 64 ? 3 : 2;         // waves per SIMD
  static_assert((DH == 64 || DH == 96) && NI * 1024 == RPW * ROW_BYTES && (NS == 3 || NS == 4),
                "tile shapes");
  static_assert(SMEM_BYTES % (16 * NT) == 0, "the rings are zeroed in whole passes");
};

template <int QT, int DH> struct PfState {  // one wave's running softmax state (2 lanes per row)
  f32x16 o[DH / 32][QT];  // O^T per 32-column tile of the values and query tile
  bf16x8 pf[2][QT];       // P(i-1)^T fragments (keys 0-15, 16-31 of the step)
  f32x16 nb[QT];          // -m in every element: the start value of each step's scores
  float m[QT], lsum[QT];
};

// byte offsets of the K and V ring half blocks: ring stage u, half hf
template <int DH> constexpr uint32_t pf_kh(int u, int hf) {
  return u * 64 * 2 * DH + hf * 32 * 2 * DH;
}
template <int DH> constexpr uint32_t pf_vh(int u, int hf) {
  return kPfNs * 64 * 2 * DH + u * 64 * 2 * DH + hf * 32 * 2 * DH;
}

// S^T fragment rows of one step for one query tile: the 32 K slots of the half block
// at kh against the lane's query column, accumulated on top of acc.
template <int DH>
__device__ __forceinline__ f32x16 pf_scores(const char* sm, const PfLane<DH>& lo, uint32_t kh,
                                            const bf16x8 (&qf)[DH / 16], f32x16 acc) {
  bf16x8 kf[DH / 16];
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) kf[ks] = pf_ldk<DH>(sm, lo, kh, ks);
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) acc = mma32(acc, kf[ks], qf[ks]);
  return acc;
}

// Accumulator start for a recomputation of the scores of step i (the rescale path):
// -m (the row reference), or -1e30 for the slots a masked step hides from this lane's
// row (slot 32 i + 8(q/4) + 4h + q%4 is visible iff it is at least lo0, the row's
// document start, and below lim0, the row position + incl). -1e30 plus any score stays
// about -1e30, so the MFMAs that follow need no masking afterwards.
template <bool DOC>
__device__ __forceinline__ void pf_init(f32x16& v, float init, bool masked, int i, int lim0,
                                        int lo0, int lane) {
  if (masked) {
    const int base = 32 * i + 4 * (lane >> 5), lim = lim0 - base, lo = lo0 - base;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int off = 8 * (q >> 2) + (q & 3);
      v[q] = off >= lim || (DOC && off < lo) ? kNegBig : init;
    }
  } else {
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q] = init;
  }
}

// 4 bf16 at byte offset off of a buffer view (zeros out of range)
__device__ __forceinline__ bf16x4 buf_ld8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

// Hides the slots a masked step hides from this lane's row (see pf_init) in finished
// scores: they become -1e30, whose weight is 0.
template <bool DOC>
__device__ __forceinline__ void pf_mask(f32x16& v, int i, int lim0, int lo0, int lane) {
  const int base = 32 * i + 4 * (lane >> 5), lim = lim0 - base, lo = lo0 - base;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int off = 8 * (q >> 2) + (q & 3);
    v[q] = off >= lim || (DOC && off < lo) ? kNegBig : v[q];
  }
}

// Sum of the 16 bf16 weights of a lane, two dot products against (1, 1) per pair of
// fragments' halves: the normaliser then adds exactly the weights the PV products use.
__device__ __forceinline__ float pf_wsum(const bf16x8& a, const bf16x8& b) {
  const bf16x2 one = {(bf16)1.f, (bf16)1.f};
  float s0 = 0.f, s1 = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bf16x2 pa = {a[2 * e], a[2 * e + 1]}, pb = {b[2 * e], b[2 * e + 1]};
    s0 = __builtin_amdgcn_fdot2_f32_bf16(pa, one, s0, false);
    s1 = __builtin_amdgcn_fdot2_f32_bf16(pb, one, s1, false);
  }
  return s0 + s1;
}

// f(integral_constant<int, I>) for I = I0 .. N-1, in order.
template <int I0, int N, class F> __device__ __forceinline__ void static_for(F& f) {
  if constexpr (I0 < N) {
    f(std::integral_constant<int, I0>());
    static_for<I0 + 1, N>(f);
  }
}

// Sum of v[Q0 .. Q1) as a balanced tree.
template <int Q0, int Q1> __device__ __forceinline__ float tree_sum(const f32x16& v) {
  if constexpr (Q1 - Q0 == 1) return v[Q0];
  else {
    constexpr int QM = Q0 + (Q1 - Q0) / 2;
    return tree_sum<Q0, QM>(v) + tree_sum<QM, Q1>(v);
  }
}
template <int N, int I0 = 0> __device__ __forceinline__ float tree_sum_arr(const float* p) {
  if constexpr (N == 1) return p[I0];
  else return tree_sum_arr<N / 2, I0>(p) + tree_sum_arr<N - N / 2, I0 + N / 2>(p);
}

// One step (see above), the same straight-line code for every step: the MFMAs of
// PV(i-1) and S(i+1) and the exponentials of S(i) sit in one basic block, so they
// interleave. sc holds S(i) in log2 units minus the row reference m; a masked step hides
// its slots here, before the exponentials. sn leaves holding S(i+1): its first MFMA
// starts from st.nb (-m in every element), so no register is set per step. Two register
// sets alternate between consecutive steps, so no step waits on the MFMAs it has just
// issued. lim0 is the first tile's row limit; tile t's rows sit tstride (32 times the
// position stride between consecutive queries) further; dlo[t] is tile t's document start.
template <int QT, int DH, bool DOC>
__device__ __forceinline__ void pf_step(const char* sm, const PfLane<DH>& lo, uint32_t kh_cur,
                                        uint32_t kh_nxt, uint32_t vh_prv, int i,
                                        const bf16x8 (&qf)[QT][DH / 16], PfState<QT, DH>& st,
                                        f32x16 (&sc)[QT], f32x16 (&sn)[QT], int lane, int lim0,
                                        int tstride, const int (&dlo)[QT], bool mask_cur) {
  if (__builtin_expect(mask_cur, 0)) {
#pragma unroll
    for (int t = 0; t < QT; ++t) pf_mask<DOC>(sc[t], i, lim0 + tstride * t, dlo[t], lane);
  }
  // NG groups g, each: the MFMAs of PV(i-1) for keys 16(g / NDT).. and value tile
  // g % NDT and of S(i+1) for k16 step g, plus the weights of rows [q0(g), q0(g+1)) of
  // S(i). The fragments of V^T (step i-1; before the first step a zeroed stage) and K
  // (step i+1) are read one group ahead, and groups are not reordered, so at most two
  // groups' fragments are live.
  constexpr int NG = DH / 16, NDT = DH / 32;
  bf16x8 vf[2], kf[2];
  vf[0] = pf_ldv<DH>(sm, lo, vh_prv, 0, 0);
  kf[0] = pf_ldk<DH>(sm, lo, kh_nxt, 0);
  // weights against the current reference, in place (S(i) is not needed again unless
  // the rescale below runs, which recomputes it from the K block still in LDS)
  auto group = [&](auto gc) {
    constexpr int g = decltype(gc)::value;
    constexpr int q0 = (16 * g + NG - 1) / NG, q1 = (16 * (g + 1) + NG - 1) / NG;
    if constexpr (g + 1 < NG) {
      vf[(g + 1) & 1] = pf_ldv<DH>(sm, lo, vh_prv, (g + 1) / NDT, (g + 1) % NDT);
      kf[(g + 1) & 1] = pf_ldk<DH>(sm, lo, kh_nxt, g + 1);
    }
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      st.o[g % NDT][t] = mma32(st.o[g % NDT][t], vf[g & 1], st.pf[g / NDT][t]);
      sn[t] = mma32(g == 0 ? st.nb[t] : sn[t], kf[g & 1], qf[t][g]);
    }
#pragma unroll
    for (int t = 0; t < QT; ++t)
#pragma unroll
      for (int q = q0; q < q1; ++q) sc[t][q] = fast_exp2(sc[t][q]);
    __builtin_amdgcn_sched_barrier(0);
  };
  static_for<0, NG>(group);
#pragma unroll
  for (int t = 0; t < QT; ++t) {
#pragma unroll
    for (int q = 0; q < 16; ++q) st.pf[q >> 3][t][q & 7] = (bf16)sc[t][q];
    float ps = pf_wsum(st.pf[0][t], st.pf[1][t]);
    if (__builtin_expect(__any(!(ps <= kGrowSum) || st.m[t] == kNoRef), 0)) {
      // rare: move the reference up to the exact row max (never down, but from kNoRef
      // to it) and rescale the state; S(i+1) was started from the old reference, so it
      // moves too
      f32x16 sr;
      pf_init<DOC>(sr, -st.m[t], mask_cur, i, lim0 + tstride * t, dlo[t], lane);
      sr = pf_scores<DH>(sm, lo, kh_cur, qf[t], sr);
      float mx = sr[0];
#pragma unroll
      for (int q = 1; q < 16; ++q) mx = fmaxf(mx, sr[q]);
      mx = ref_growth(halves_max(mx), st.m[t]);
      const float alpha = ref_rescale(mx, st.m[t]);
      st.m[t] += mx;
      st.lsum[t] *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) st.o[dt][t] *= alpha;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        st.nb[t][q] = -st.m[t];
        sn[t][q] -= mx;
        st.pf[q >> 3][t][q & 7] = (bf16)fast_exp2(sr[q] - mx);
      }
      ps = pf_wsum(st.pf[0][t], st.pf[1][t]);
    }
    st.lsum[t] += ps;
  }
}

// One query tile of the persistent kernel below: 32 QT rows per wave of one (consumer,
// sequence, head). On entry every wave is past the previous tile (its copies have
// landed and its ring reads are done) and the rings hold finite values.
template <int QT, int DH, bool DOC, bool SPLIT>
__device__ __forceinline__ void pf_tile(const AttnArgs<bf16>& a, const int tile, const int split,
                                        char* smem, int* s_lo) {
  using P = PfDma<QT, DH>;
  constexpr int NKS = P::NKS, NDT = P::NDT;
  // Tile order: sequence, KV head, consumer (in channel order), query head of the KV
  // head's group, query tile (longest first). Consecutive tiles read one channel's K/V
  // slice: every query tile and grouped head of a consumer, then the next consumer of
  // the same channel, so an XCD's L2 serves a slice to all its readers.
  const int G = a.Hq / a.Hkv;
  const int qtile = a.n_qtiles - 1 - tile % a.n_qtiles;
  int y = tile / a.n_qtiles;
  const int hg = y % G;
  y /= G;
  const int li = y % a.L;
  y /= a.L;
  const int kvh = y % a.Hkv, b = y / a.Hkv;
  const int hq = kvh * G + hg, l = a.lord.v[li];
  const int c = a.chan.v[l];
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ctx = __builtin_amdgcn_readfirstlane(ctx_at(a.ctx_len, b, a.ctx_hi));
  const int incl = a.mask_paper ? 0 : 1;
  const int q0 = qtile * P::BQ, qw0 = q0 + 32 * QT * w;
  const float cl2 = a.scale_log2;
  const int gs = a.gs, pos0 = ctx + a.gq;  // query i sits at position pos0 + gs i

  // The queries and the dummy slot are loaded first and used only once the first copies
  // are issued, so their latency overlaps the copies'.
  // (buffer loads: rows past T_new, and the dummy when the mask has none, read as zeros)
  bf16x8 qf[QT][NKS];
  {
    const auto qview = make_view(a.Q + (((long)l * a.B + b) * a.Hq + hq) * (long)a.T_new * DH,
                                 (uint32_t)a.T_new * DH * 2u);
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      const int qi = qw0 + 32 * t + r;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
        qf[t][ks] = buf_frag<bf16>(qview, qi < a.T_new ? (uint32_t)(qi * DH + 16 * ks + 8 * h) * 2u
                                                      : kOffOob);
    }
  }
  bf16x8 kdv[NKS];      // the dummy's key at this lane's columns
  bf16x4 vdv[NDT][4];   // and its value at this lane's rows of O^T
  {
    const long dof = ((long)c * a.Hkv + kvh) * DH;
    const uint32_t dbytes = a.mask_paper ? DH * 2u : 0u;
    const auto kdview = make_view(a.mask_paper ? a.Kd + dof : nullptr, dbytes);
    const auto vdview = make_view(a.mask_paper ? a.Vd + dof : nullptr, dbytes);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) kdv[ks] = buf_frag<bf16>(kdview, (16 * ks + 8 * h) * 2u);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        vdv[dt][g4] = buf_ld8(vdview, (32 * dt + 8 * g4 + 4 * h) * 2u);
  }

  // Document mask: each row's first readable slot; the walk starts at the 64-slot block
  // holding the workgroup's least one (base0), and every slot index below is relative
  // to base0. Blocks a wave's rows partly cannot read are masked like the causal edge.
  // (A wave's steps below its own rows' document starts are masked, not skipped:
  // measured, skipping them and restarting the pipeline later is slower.)
  int dlo[QT], base0 = 0, wlo_max = 0;
  if constexpr (DOC) {
    int wmin = 0x7fffffff;
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      const int qi = qw0 + 32 * t + r;
      dlo[t] = qi < a.T_new ? doc_first(a.doc, b, a.T_new, qi, pos0 + gs * qi) : 0;
      wmin = min(wmin, qi < a.T_new ? dlo[t] : 0x7fffffff);
      wlo_max = max(wlo_max, dlo[t]);
    }
    wmin = __builtin_amdgcn_readfirstlane(wave_min_i(wmin));
    wlo_max = __builtin_amdgcn_readfirstlane(wave_max_i(wlo_max));
    if (lane == 0) s_lo[w] = wmin;
    __syncthreads();
    int gmin = s_lo[0];
#pragma unroll
    for (int k = 1; k < P::NW; ++k) gmin = min(gmin, s_lo[k]);
    base0 = __builtin_amdgcn_readfirstlane(gmin / P::BKV * P::BKV);
#pragma unroll
    for (int t = 0; t < QT; ++t) dlo[t] -= base0;  // rows past T_new go negative: no mask
    wlo_max -= base0;
  } else {
#pragma unroll
    for (int t = 0; t < QT; ++t) dlo[t] = 0;
    if constexpr (SPLIT) base0 = split * a.split_blk * P::BKV;  // a split walks from its first block
  }
  const int ctxr = pos0 - base0;  // the first new token's position relative to base0

  const long cbase = (((long)c * a.B + b) * a.Hkv + kvh) * (long)a.S_cap * DH +
                     (long)base0 * DH;
  const int qlast = min(q0 + P::BQ, a.T_new) - 1;
  const int scap = a.S_cap - base0;
  int kend = min(ctxr + gs * qlast + incl, scap);   // slots the workgroup may see
  if constexpr (SPLIT) {
    if (kend <= 0) {  // the tile's walk ends before this split: an empty partial state
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        const int qi = qw0 + 32 * t + r;
        if (qi < a.T_new && h == 0) {
          const long rows = (long)a.L * a.B * a.Hq * a.T_new;
          const long row = (((long)l * a.B + b) * a.Hq + hq) * a.T_new + qi;
          float* ml = a.part + rows * a.nsplit * DH + 2 * ((long)split * rows + row);
          ml[0] = kNoRef;
          ml[1] = 0.f;
        }
      }
      return;
    }
    kend = min(kend, a.split_blk * P::BKV);
  }
  const int nblk = (kend + P::BKV - 1) / P::BKV;
  const int wq_last = min(qw0 + 32 * QT - 1, a.T_new - 1);
  const int wkend = wq_last >= qw0 ? ctxr + gs * wq_last + incl : 0;  // slots this wave may see
  const int wfree = ctxr + gs * qw0 + incl;  // slots < wfree are visible to all its rows ...
  // ... and at or past wlo_max (the document starts); a step is masked unless both hold
  auto masked = [&](int i) { return 32 * i + 32 > wfree || (DOC && 32 * i < wlo_max); };
  int ilast = (wkend + 31) / 32 - 1;  // the wave's last 32-slot step (-1: none)
  int lim0 = ctxr + gs * (qw0 + r) + incl;
  const int tstride = 32 * gs;
  if constexpr (SPLIT) {
    // a split stops at its last block (the step after it only adds that block's PV, its
    // own slots hidden by the limit) and a wave that sees nothing in it takes no step
    ilast = ilast < 0 ? -2 : min(ilast, 2 * nblk - 1);
    lim0 = min(lim0, kend);
    static_assert(QT == 1, "one query tile per wave: lim0 is the row's only limit");
  }

  // copies: wave w moves slot rows RPW w .. RPW w + RPW-1 of each K and V block, 1 KB
  // (64 chunks of 16 B) per instruction; lane x of instruction n fills LDS chunk
  // 64 n + x of the wave's rows, i.e. row (64 n + x) / CPR, chunk (64 n + x) % CPR, with
  // the chunk of the slot row that the swizzle puts there
  // (the views end at slot kend, so rows past it read as zeros without a test per copy)
  const __amdgpu_buffer_rsrc_t kview = make_view(a.Kc + cbase, (uint32_t)kend * P::ROW_BYTES);
  const __amdgpu_buffer_rsrc_t vview = make_view(a.Vc + cbase, (uint32_t)kend * P::ROW_BYTES);
  uint32_t coff[P::NI];  // byte offset of the lane's chunk within block 0
#pragma unroll
  for (int n = 0; n < P::NI; ++n) {
    const int ch = 64 * n + lane, crow = P::RPW * w + ch / P::CPR;
    coff[n] = (uint32_t)crow * P::ROW_BYTES + 16u * (uint32_t)((ch % P::CPR) ^ pf_swz<DH>(crow));
  }
  const uint32_t smem_base = (uint32_t)(uintptr_t)smem;
  // NI copy instructions per wave move its rows of a K or V block; blocks past the
  // visible range are copied too (as zeros), so every wave issues the same sequence
  // (4-block rings: K0 K1 V0 K2 V1 | K3 V2 | K4 V3 | ..., 3-block rings: K0 K1 V0 |
  // K2 V1 | K3 V2 | ...) and one vmcnt fits every block
  auto issue = [&](int blk, bool v) {
#pragma unroll
    for (int n = 0; n < P::NI; ++n) {
      const uint32_t off = coff[n] + (uint32_t)blk * P::BLK_BYTES;
      const uint32_t lds = __builtin_amdgcn_readfirstlane(
          smem_base + (v ? P::V_BASE : 0) + (blk % P::NS) * P::BLK_BYTES +
          P::RPW * w * P::ROW_BYTES + 1024 * n);
      lds_dma16(lds, off, v ? vview : kview);
    }
  };

  constexpr int AHEAD = P::NS - 3;  // (K, V) pairs still in flight when block j starts
  issue(0, false);
  issue(1, false);
  issue(0, true);
  if (AHEAD) {
    issue(2, false);
    issue(1, true);
  }

  // queries in log2 units: the MFMAs then give s' = q.k log2(e) / sqrt(d)
#pragma unroll
  for (int t = 0; t < QT; ++t)
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int i = 0; i < 8; ++i) qf[t][ks][i] = (bf16)((float)qf[t][ks][i] * cl2);
  PfState<QT, DH> st;
  f32x16 sa[QT], sb[QT];  // score registers of even and odd steps
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    st.pf[0][t] = zero_frag<bf16>();
    st.pf[1][t] = zero_frag<bf16>();
    if (a.mask_paper && split == 0) {  // the dummy starts the first split's state
      float part = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
        for (int i = 0; i < 8; ++i) part += (float)qf[t][ks][i] * (float)kdv[ks][i];
      st.m[t] = halves_sum(part);
      st.lsum[t] = h == 0 ? 1.f : 0.f;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int q = 0; q < 16; ++q) st.o[dt][t][q] = (float)vdv[dt][q >> 2][q & 3];
    } else {
      st.m[t] = kNoRef;
      st.lsum[t] = 0.f;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) st.o[dt][t] = zero16();
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) st.nb[t][q] = -st.m[t];
  }
  // block 0's first step reads K(0) only (and the zeroed V stage before it)
  wait_vmcnt<P::NI * (2 + 2 * AHEAD)>();
  __syncthreads();
  PfLane<DH> lo = pf_lane<DH>(lane);
  // one block of the walk; u = j mod NS is a compile-time constant, so every ring
  // address below is a lane offset plus a constant the LDS instructions carry
  auto block = [&](const int j, auto uc) {
    constexpr int u = decltype(uc)::value;
    // keep the lane offsets as they are (not one precomputed address per use)
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) asm volatile("" : "+v"(lo.k[ks]));
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) asm volatile("" : "+v"(lo.v[dt][0]), "+v"(lo.v[dt][1]));
    // Two barriers per block. Here every wave is past block j-1, so the stages of K(j-1)
    // and V(j-2) are free; the first step reads only K(j) and V(j-1), which landed
    // before the previous block's second barrier. (Measured: waiting for K(j+1) here
    // instead, one barrier per block, is 2-6% slower.)
    __syncthreads();
    issue(j + P::NS - 1, false);
    issue(j + P::NS - 2, true);
    if (u == 0 && j == 0 && ilast >= 0) {
#pragma unroll
      for (int t = 0; t < QT; ++t) sa[t] = pf_scores<DH>(smem, lo, pf_kh<DH>(0, 0), qf[t], st.nb[t]);
    }
    // steps up to ilast + 1: the last one only adds PV(ilast) (its own slots are all
    // past the wave's rows, so its weights are 0)
    const int i = 2 * j;
    if (i <= ilast + 1)
      pf_step<QT, DH, DOC>(smem, lo, pf_kh<DH>(u, 0), pf_kh<DH>(u, 1),
                      pf_vh<DH>((u + P::NS - 1) % P::NS, 1), i, qf, st, sa, sb, lane, lim0,
                      tstride, dlo, masked(i));
    // the second step reads K(j+1) and V(j): only the copies issued above may still be
    // in flight
    wait_vmcnt<2 * P::NI * (1 + AHEAD)>();
    __syncthreads();
    if (i + 1 <= ilast + 1)
      pf_step<QT, DH, DOC>(smem, lo, pf_kh<DH>(u, 1), pf_kh<DH>((u + 1) % P::NS, 0),
                      pf_vh<DH>(u, 0), i + 1, qf, st, sb, sa, lane, lim0, tstride, dlo,
                      masked(i + 1));
  };
  for (int j = 0; j < nblk; j += P::NS) {
    block(j, std::integral_constant<int, 0>());
    if (j + 1 < nblk) block(j + 1, std::integral_constant<int, 1>());
    if (j + 2 < nblk) block(j + 2, std::integral_constant<int, 2>());
    if (P::NS == 4 && j + 3 < nblk) block(j + 3, std::integral_constant<int, 3 % P::NS>());
  }
  if (ilast + 1 == 2 * nblk) {
    const int u = nblk % P::NS;
    pf_step<QT, DH, DOC>(smem, lo, pf_kh<DH>(u, 0), pf_kh<DH>(u, 1),
                    pf_vh<DH>((u + P::NS - 1) % P::NS, 1), 2 * nblk, qf, st, sa, sb, lane, lim0,
                    tstride, dlo, true);
  }
  wait_vmcnt<0>();  // no copy may land after the workgroup ends

  if constexpr (SPLIT) {  // the partial state: O unnormalised, the reference and the weights' sum
    const long rows = (long)a.L * a.B * a.Hq * a.T_new;
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      const int qi = qw0 + 32 * t + r;
      const float lt = halves_sum(st.lsum[t]);
      if (qi < a.T_new) {
        const long row = (((long)l * a.B + b) * a.Hq + hq) * a.T_new + qi;
        float* po = a.part + ((long)split * rows + row) * DH;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            f32x4 v;
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = st.o[dt][t][4 * g + i];
            *(f32x4*)(po + 32 * dt + 8 * g + 4 * h) = v;
          }
        if (h == 0) {
          float* ml = a.part + rows * a.nsplit * DH + 2 * ((long)split * rows + row);
          ml[0] = st.m[t];
          ml[1] = lt;
        }
      }
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int qi = qw0 + 32 * t + r;
    const float lt = halves_sum(st.lsum[t]);
    if (qi < a.T_new) {
      const float inv = 1.0f / lt;
      bf16* dst = a.O + ((((long)l * a.B + b) * a.T_new + qi) * a.Hq + hq) * DH;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float v[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = st.o[dt][t][4 * g + i] * inv;
          store4(dst + 32 * dt + 8 * g + 4 * h, v);
        }
    }
  }
}

// Persistent form: a grid of as many workgroups as the CUs hold at once (3 per CU at head
// dim 64, 2 at 96), each taking query tiles from a work queue until it runs dry, so a
// workgroup's launch and set-up are paid once rather than per tile (measured: 64-step
// tiles in workgroups of their own ran 16% slower than the same tiles in persistent
// workgroups). Workgroup i serves queue i mod 8: workgroups are dispatched round-robin
// over the 8 XCDs, so each XCD's L2 sees one contiguous share of the tiles (in tile
// order, the query tiles of one head, longest first, then the next head), and taking
// them in that order keeps the heads being read by an XCD few and their K/V in its L2.
// The queue counters (queue[16 x], zeroed before the launch) hand out tile indices in
// order, so the slow (long) tiles start first and the last ones are the shortest. With
// queue null the grid has one workgroup per tile (tile order as above, XCD-aware).
// DOC: the document mask is on (a.doc is not null); the kernel without it keeps the
// step loop free of the document bookkeeping.
template <int QT, int DH, bool DOC, bool SPLIT = false>
__global__ __launch_bounds__(64 * kPfWaves) __attribute__((amdgpu_waves_per_eu(DH == 64 ? 3 : 2)))
void attend_prefill_dma_kernel(AttnArgs<bf16> a, uint32_t* queue) {
  using P = PfDma<QT, DH>;
  static_assert(P::NT == 64 * kPfWaves && P::WPE == (DH == 64 ? 3 : 2), "launch bounds");
  __shared__ __align__(16) char smem[P::SMEM_BYTES];
  __shared__ int s_lo[P::NW];
  __shared__ int s_tile;
  const int tid = threadIdx.x;
  // zero the rings once: "block -1" feeds a tile's first (weightless) PV, and slot rows
  // past the visible range get weight 0, so every stage must hold finite values (later
  // tiles find the previous tile's K/V there, which are finite)
  {
    const i32x4 z = {0, 0, 0, 0};
#pragma unroll
    for (int k = 0; k < P::SMEM_BYTES / (16 * P::NT); ++k)
      *(i32x4*)(smem + 16 * (tid + P::NT * k)) = z;
  }
  const int total = a.n_qtiles * a.Hq * a.B * a.L;
  if constexpr (SPLIT) {  // a workgroup per tile and split range (consecutive: one tile)
    __syncthreads();  // the zeroed rings are in place before any copy lands
    const int idx = xcd_tile(blockIdx.x, total * a.nsplit);
    pf_tile<QT, DH, DOC, true>(a, idx / a.nsplit, idx % a.nsplit, smem, s_lo);
    return;
  }
  if (!queue) {  // a grid of one workgroup per tile (grids the CUs hold at once)
    __syncthreads();  // the zeroed rings are in place before any copy lands
    pf_tile<QT, DH, DOC, false>(a, xcd_tile(blockIdx.x, total), 0, smem, s_lo);
    return;
  }
  const int nq = min((int)gridDim.x, kNumXcd), x = blockIdx.x % nq;
  const int per = total / nq, rem = total % nq;
  const int first = x * per + min(x, rem), count = per + (x < rem ? 1 : 0);
  uint32_t* ctr = queue + kQueueStride * x;
  if (tid == 0) s_tile = (int)atomicAdd(ctr, 1u);
  __syncthreads();  // also: the zeroed rings are in place before any copy lands
  int t = __builtin_amdgcn_readfirstlane(s_tile);
  while (t < count) {
    pf_tile<QT, DH, DOC, false>(a, first + t, 0, smem, s_lo);
    // every wave reads s_tile after this barrier and before the next tile's first one,
    // so thread 0 rewrites it only once all have read it
    if (tid == 0) s_tile = (int)atomicAdd(ctr, 1u);
    __syncthreads();
    t = __builtin_amdgcn_readfirstlane(s_tile);
  }
}

__global__ void queue_reset_kernel(uint32_t* queue) { queue[threadIdx.x] = 0u; }

int device_cus() {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Split slot ranges for small grids (bf16 kernel, no documents): when the query tiles
// fill at most a quarter of the workgroup slots the CUs hold at once, each tile's walk is
// cut into ranges of split_blk 64-slot blocks (at least 16) so that about one resident
// round of workgroups runs. Measured on the pass driver's group calls at the paper's
// shape: 2 ranges at 96 tiles, 11% faster; at 192 tiles any split was slower (the
// partial states' write and merge, 28 MB a call, cost more than the shorter walks save),
// as were ranges of 4-11 blocks.
// Returns the splits aimed at (an upper bound on *nsplit that grows with the slot range,
// which sizes the partial states).
static long prefill_split(const Shape& sh, long tiles, int* nsplit, int* split_blk) {
  const long resident = (long)device_cus() * (sh.d == 64 ? PfDma<kPfQt, 64>::WPE
                                                         : PfDma<kPfQt, 96>::WPE);
  const long kmax = (long)sh.ctx_max + sh.span();  // bound on any tile's visible slots
  const int max_blk = (int)std::max(1L, (kmax + 63) / 64);
  long n = 1;
  if (4 * tiles <= resident) n = std::min<long>((resident + tiles - 1) / tiles, max_blk / 16);
  if (n < 2) {
    *nsplit = 1;
    *split_blk = max_blk;
    return 1;
  }
  const int blk = (int)((max_blk + n - 1) / n);
  *nsplit = (max_blk + blk - 1) / blk;
  *split_blk = blk;
  return n;
}

static long prefill_tiles(const Shape& sh) {
  return (long)((sh.T_new + PfDma<kPfQt, 64>::BQ - 1) / PfDma<kPfQt, 64>::BQ) * sh.Hq * sh.B *
         sh.L;
}

size_t prefill_scratch_bytes(const Shape& sh) {
  if (sh.d != 64 && sh.d != 96) return kPrefillQueueBytes;
  int nsplit, blk;
  const long n = prefill_split(sh, prefill_tiles(sh), &nsplit, &blk);
  const size_t rows = (size_t)sh.L * sh.B * sh.Hq * sh.T_new;
  return n > 1 ? std::max(kPrefillQueueBytes, rows * n * (sh.d + 2) * sizeof(float))
               : kPrefillQueueBytes;
}

// The split ranges' partial states merged per row in split order: with M the largest
// reference among the ranges that saw a slot, O = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s
// (part: o [nsplit][rows][DH] unnormalised, then (m, l) [nsplit][rows][2]). A thread takes
// four columns of one row.
template <int DH>
__global__ __launch_bounds__(256) void attend_split_combine_kernel(const float* part, int nsplit,
                                                                   int T, int Hq, long rows,
                                                                   bf16* O) {
  constexpr int C4 = DH / 4;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= rows * C4) return;
  const long row = idx / C4;
  const int c = (int)(idx - row * C4);
  const float* ml = part + rows * nsplit * DH;
  float M = -3.0e38f;
  for (int s = 0; s < nsplit; ++s)
    if (ml[2 * (s * rows + row) + 1] > 0.f) M = fmaxf(M, ml[2 * (s * rows + row)]);
  float lsum = 0.f, acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < nsplit; ++s) {
    const float ls = ml[2 * (s * rows + row) + 1];
    if (ls > 0.f) {
      const float wgt = fast_exp2(ml[2 * (s * rows + row)] - M);
      const f32x4 o = *(const f32x4*)(part + (s * rows + row) * DH + 4 * c);
      lsum += ls * wgt;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] += o[i] * wgt;
    }
  }
  const float inv = 1.0f / lsum;
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] *= inv;
  // row = ((l B + b) Hq + hq) T + i  ->  O[(l B + b) T + i][hq DH + 4 c]
  const long i = row % T, lbh = row / T;
  const int hq = (int)(lbh % Hq);
  const long lb = lbh / Hq;
  store4(O + ((lb * T + i) * Hq + hq) * DH + 4 * c, acc);
}

template <typename T>
void launch_attend_prefill(const Shape& sh, const LayerTable& chan_map, const T* Q, const T* Kc,
                           const T* Vc, const T* Kd, const T* Vd, const int32_t* ctx_len,
                           const int32_t* doc, T* O, void* scratch, hipStream_t s) {
  if (sh.N() <= 0) return;
  constexpr int BQ = PrefillCfg<T, 64>::BQ, NT = PrefillCfg<T, 64>::NT;
  static_assert(BQ == PrefillCfg<T, 32>::BQ && NT == PrefillCfg<T, 32>::NT, "tile shapes");
  LayerTable lord{};  // consumers sorted by channel, stable
  for (int c = 0, n = 0; c < kMaxLayers && n < sh.L; ++c)
    for (int l = 0; l < sh.L; ++l)
      if (chan_map.v[l] == c) lord.v[n++] = l;
  AttnArgs<T> a{Q, Kc, Vc, Kd, Vd, ctx_len, doc, O, sh.B, sh.T_new, sh.L, sh.Hq, sh.Hkv, sh.S_cap,
                sh.mask_paper, (sh.T_new + BQ - 1) / BQ, sh.gs, sh.gq, sh.ctx_hi,
                kLog2e / sqrtf((float)sh.d), chan_map, lord, 1, 0, nullptr};
  dim3 grid(a.n_qtiles * sh.Hq * sh.B * sh.L);
  if (sizeof(T) == 2 && (sh.d == 64 || sh.d == 96)) {  // fp32 at d = 96 fails validation
    constexpr int BQD = PfDma<kPfQt, 64>::BQ;
    static_assert(BQD == PfDma<kPfQt, 96>::BQ && PfDma<kPfQt, 64>::NT == PfDma<kPfQt, 96>::NT,
                  "tile shapes");
    AttnArgs<T> ad = a;
    ad.n_qtiles = (sh.T_new + BQD - 1) / BQD;
    const long tiles = prefill_tiles(sh);
    const long resident = (long)device_cus() * (sh.d == 64 ? PfDma<kPfQt, 64>::WPE
                                                           : PfDma<kPfQt, 96>::WPE);
    // persistent only when the tiles outnumber what the CUs hold at once; smaller grids
    // start every tile at once and skip the queue (its reset launch and atomics), and the
    // smallest split their tiles' slot ranges
    const bool persistent = tiles > resident;
    if (!persistent && !doc) {
      prefill_split(sh, tiles, &ad.nsplit, &ad.split_blk);
      if (ad.nsplit > 1) ad.part = (float*)scratch;
    }
    uint32_t* queue = persistent ? (uint32_t*)scratch : nullptr;
    const AttnArgs<bf16>& ab = *reinterpret_cast<const AttnArgs<bf16>*>(&ad);
    const dim3 gd((unsigned)(persistent ? resident : tiles * ad.nsplit)),
        bd(PfDma<kPfQt, 64>::NT);
    if (persistent) hipLaunchKernelGGL(queue_reset_kernel, dim3(1), dim3(kQueueWords), 0, s, queue);
    if (sh.d == 64) {
      if (doc) hipLaunchKernelGGL((attend_prefill_dma_kernel<kPfQt, 64, true>), gd, bd, 0, s, ab, queue);
      else if (ad.nsplit > 1)
        hipLaunchKernelGGL((attend_prefill_dma_kernel<kPfQt, 64, false, true>), gd, bd, 0, s, ab, queue);
      else hipLaunchKernelGGL((attend_prefill_dma_kernel<kPfQt, 64, false>), gd, bd, 0, s, ab, queue);
    } else {
      if (doc) hipLaunchKernelGGL((attend_prefill_dma_kernel<kPfQt, 96, true>), gd, bd, 0, s, ab, queue);
      else if (ad.nsplit > 1)
        hipLaunchKernelGGL((attend_prefill_dma_kernel<kPfQt, 96, false, true>), gd, bd, 0, s, ab, queue);
      else hipLaunchKernelGGL((attend_prefill_dma_kernel<kPfQt, 96, false>), gd, bd, 0, s, ab, queue);
    }
    if (ad.nsplit > 1) {
      const long rows = (long)sh.L * sh.B * sh.Hq * sh.T_new;
      const unsigned nb = (unsigned)((rows * (sh.d / 4) + 255) / 256);
      if (sh.d == 64)
        hipLaunchKernelGGL(attend_split_combine_kernel<64>, dim3(nb), dim3(256), 0, s,
                           (const float*)ad.part, ad.nsplit, sh.T_new, sh.Hq, rows, (bf16*)O);
      else
        hipLaunchKernelGGL(attend_split_combine_kernel<96>, dim3(nb), dim3(256), 0, s,
                           (const float*)ad.part, ad.nsplit, sh.T_new, sh.Hq, rows, (bf16*)O);
    }
  } else if (sh.d == 64)
    hipLaunchKernelGGL((attend_prefill_kernel<T, 64>), grid, dim3(NT), 0, s, a);
  else
    hipLaunchKernelGGL((attend_prefill_kernel<T, 32>), grid, dim3(NT), 0, s, a);
}

// ------------------------------------------------------------------ decode
// Cache slots per split workgroup: long splits amortise a workgroup's set-up and its
// partial-state write; they are halved (down to 256) while the grid of splits x
// (channel, sequence, KV head) would hold fewer than kDecodeMinBlocks workgroups.
constexpr int kSplitMax = 4096, kSplitMin = 256;
constexpr long kDecodeMinBlocks = 4096;

int decode_split_len(const Shape& sh) {
  const long kend = (long)sh.ctx_max + sh.span();  // upper bound on visible slots
  const long slices = (long)sh.k * sh.B * sh.Hkv;
  int len = kSplitMax;
  while (len > kSplitMin && slices * ((kend + len - 1) / len) < kDecodeMinBlocks) len /= 2;
  return len;
}

int decode_splits(const Shape& sh) {
  const long kend = (long)sh.ctx_max + sh.span();
  const int len = decode_split_len(sh);
  int n = (int)((kend + len - 1) / len);
  return n < 1 ? 1 : n;
}

size_t decode_partials_bytes(const Shape& sh) {
  size_t rows = (size_t)sh.L * sh.B * sh.Hq * sh.T_new;
  return rows * decode_splits(sh) * (sh.d + 2) * sizeof(float);
}

template <typename T> struct DecodeArgs {
  const T *Q, *Kc, *Vc, *Kd, *Vd;
  const int32_t* ctx_len;
  const int32_t* doc;  // [B][T_new] first position of each token's document, or null
  float* part;  // [L][B][Hq][T_new][nsplit][d + 2]: unnormalised o, m, l
  T* O;
  int B, T_new, L, Hq, Hkv, S_cap, mask_paper, nsplit, split_len;
  int gs, gq, ctx_hi;  // query i of sequence b sits at position ctx_len[b] + gq + gs i
  float scale_log2;
  LayerTable chan;
  ChannelGroups cg;
};

// Merge online-softmax state (m2, l2, o2) into (m, l, o).
__device__ __forceinline__ void merge_state(float& m, float& l, float* o, float m2, float l2,
                                            const float* o2, int n, float c) {
  float M = fmaxf(m, m2);
  float a1 = fast_exp2((m - M) * c), a2 = fast_exp2((m2 - M) * c);
  l = l * a1 + l2 * a2;
  for (int i = 0; i < n; ++i) o[i] = o[i] * a1 + o2[i] * a2;
  m = M;
}

template <typename T, int DH, int NG>
__global__ __launch_bounds__(256) void attend_decode_kernel(DecodeArgs<T> a) {
  // A cache slot is read by CPS lanes of 8 elements each, in a group of LPS lanes (CPS
  // rounded up to a power of two, so the group's sums are butterflies); lanes c8 >= CPS
  // of a group load nothing and hold zeros (head dim 96: 12 of 16 lanes work).
  constexpr int CPS = DH / 8;
  constexpr int LPS = CPS <= 4 ? 4 : CPS <= 8 ? 8 : 16;
  static_assert(LPS >= CPS && DH % 8 == 0, "8-element chunks in a power-of-two group");
  constexpr int SPW = 64 / LPS;  // slots per wave per sweep step
  constexpr int U = NG <= 2 ? 2 : 1;  // sweep steps per batch (U slots per lane)
  constexpr int SPB = 4 * SPW * U;  // slots per batch of the 4 waves
  __shared__ float red[4][NG][DH + 2];

  const int split = blockIdx.x;
  int y = blockIdx.y;
  const int kvh = y % a.Hkv;
  y /= a.Hkv;
  const int b = y % a.B, c = y / a.B;
  const int off = a.cg.offsets[c], nmem = a.cg.offsets[c + 1] - off;
  if (nmem == 0) return;
  const int grp = a.Hq / a.Hkv;
  const int G = nmem * grp * a.T_new;
  // position of query i: pos0 + gs i (wave-uniform)
  const int pos0 = __builtin_amdgcn_readfirstlane(ctx_at(a.ctx_len, b, a.ctx_hi)) + a.gq;
  const int gs = a.gs;
  const int incl = a.mask_paper ? 0 : 1;
  const int kend = min(pos0 + gs * (a.T_new - 1) + incl, a.S_cap);
  const int s0 = split * a.split_len, s1 = min(s0 + a.split_len, kend);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int sg = lane / LPS, c8 = lane % LPS;
  const float cl2 = a.scale_log2;
  const float thresh = 8.0f / cl2;  // log2 headroom before a rescale

  const long cbase = (((long)c * a.B + b) * a.Hkv + kvh) * (long)a.S_cap * DH;
  // the slice through buffer views: slots at or past s1 read zeros without a branch
  const __amdgpu_buffer_rsrc_t kview = make_view(a.Kc + cbase, (uint32_t)a.S_cap * DH * sizeof(T));
  const __amdgpu_buffer_rsrc_t vview = make_view(a.Vc + cbase, (uint32_t)a.S_cap * DH * sizeof(T));
  const bool chunk = c8 < CPS;  // the lane holds 8 channels of the head
  auto slot_off = [&](int s) {
    return s < s1 && chunk ? (uint32_t)(s * DH + 8 * c8) * (uint32_t)sizeof(T) : kOffOob;
  };

  for (int g0 = 0; g0 < G; g0 += NG) {
    const int ng = min(NG, G - g0);
    float q[NG][8], m[NG], ls[NG], o[NG][8];
    int vis[NG], lov[NG];  // the row reads slots lov <= s < vis
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      m[gi] = kNegBig;
      ls[gi] = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[gi][i] = 0.f;
      if (gi < ng) {
        int g = g0 + gi;
        int i = g % a.T_new, gq = (g / a.T_new) % grp, mi = g / (a.T_new * grp);
        int l = a.cg.members[off + mi], hq = kvh * grp + gq;
        long rowid = (((long)l * a.B + b) * a.Hq + hq) * a.T_new + i;
        vis[gi] = pos0 + gs * i + incl;
        lov[gi] = doc_first(a.doc, b, a.T_new, i, pos0 + gs * i);
        if (chunk) load8(a.Q + rowid * DH + 8 * c8, q[gi]);
        else {
#pragma unroll
          for (int i = 0; i < 8; ++i) q[gi][i] = 0.f;
        }
      } else {
        vis[gi] = 0;
        lov[gi] = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) q[gi][i] = 0.f;
      }
    }

    // raw K/V fragments of a batch (U slots per lane), double-buffered across batches
    // (two batches per loop trip keep the buffer indices static)
    frag_t<T> kr0[U], vr0[U], kr1[U], vr1[U];
    auto fetch = [&](int sb, frag_t<T>* kr, frag_t<T>* vr) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t so = slot_off(sb + w * SPW * U + u * SPW + sg);
        kr[u] = buf_frag<T>(kview, so);
        vr[u] = buf_frag<T>(vview, so);
      }
    };
    auto consume = [&](int sb, const frag_t<T>* kr, const frag_t<T>* vr) {
      float p[U][NG];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int s = sb + w * SPW * U + u * SPW + sg;
#pragma unroll
        for (int gi = 0; gi < NG; ++gi) {
          float d = 0.f;
#pragma unroll
          for (int i = 0; i < 8; ++i) d += q[gi][i] * to_f32(kr[u][i]);
#pragma unroll
          for (int x = 1; x < LPS; x <<= 1) d += __shfl_xor(d, x, 64);
          p[u][gi] = s < s1 && s < vis[gi] && s >= lov[gi] ? d : kNegBig;
        }
      }
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        float mx = p[0][gi];
#pragma unroll
        for (int u = 1; u < U; ++u) mx = fmaxf(mx, p[u][gi]);
        if (mx > m[gi] + thresh) {  // lazy rescale (per lane; merged exactly below)
          const float al = fast_exp2((m[gi] - mx) * cl2);
          ls[gi] *= al;
#pragma unroll
          for (int i = 0; i < 8; ++i) o[gi][i] *= al;
          m[gi] = mx;
        }
        const float mc = m[gi] * cl2;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const float pe = p[u][gi] > 0.5f * kNegBig ? fast_exp2(p[u][gi] * cl2 - mc) : 0.f;
          ls[gi] += pe;
#pragma unroll
          for (int i = 0; i < 8; ++i) o[gi][i] += pe * to_f32(vr[u][i]);
        }
      }
    };
    // batches past the split read zeros (and are masked), so the loop runs in pairs
    fetch(s0, kr0, vr0);
    for (int sb = s0; sb < s1; sb += 2 * SPB) {
      fetch(sb + SPB, kr1, vr1);
      consume(sb, kr0, vr0);
      fetch(sb + 2 * SPB, kr0, vr0);
      consume(sb + SPB, kr1, vr1);
    }
    // merge the slot groups of the wave (lanes that share c8)
#pragma unroll
    for (int msk = LPS; msk < 64; msk <<= 1)
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        float m2 = __shfl_xor(m[gi], msk, 64), l2 = __shfl_xor(ls[gi], msk, 64), o2[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) o2[i] = __shfl_xor(o[gi][i], msk, 64);
        merge_state(m[gi], ls[gi], o[gi], m2, l2, o2, 8, cl2);
      }
    if (sg == 0 && chunk) {
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
#pragma unroll
        for (int i = 0; i < 8; ++i) red[w][gi][8 * c8 + i] = o[gi][i];
        if (c8 == 0) {
          red[w][gi][DH] = m[gi];
          red[w][gi][DH + 1] = ls[gi];
        }
      }
    }
    __syncthreads();
    for (int e = tid; e < ng * DH; e += 256) {
      int gi = e / DH, dd = e % DH;
      float M = kNegBig;
      for (int ww = 0; ww < 4; ++ww) M = fmaxf(M, red[ww][gi][DH]);
      float Lsum = 0.f, Osum = 0.f;
      for (int ww = 0; ww < 4; ++ww) {
        float sc = fast_exp2((red[ww][gi][DH] - M) * cl2);
        Lsum += red[ww][gi][DH + 1] * sc;
        Osum += red[ww][gi][dd] * sc;
      }
      // recompute the row id for gi (registers are per-lane; rows are uniform)
      int g = g0 + gi;
      int i = g % a.T_new, gq = (g / a.T_new) % grp, mi = g / (a.T_new * grp);
      int l = a.cg.members[off + mi], hq = kvh * grp + gq;
      long rid = (((long)l * a.B + b) * a.Hq + hq) * a.T_new + i;
      float* dst = a.part + (rid * a.nsplit + split) * (DH + 2);
      dst[dd] = Osum;
      if (dd == 0) {
        dst[DH] = M;
        dst[DH + 1] = Lsum;
      }
    }
    __syncthreads();
  }
}

// One wave per query row: fold the dummy slot and all split partials.
template <typename T, int DH>
__global__ __launch_bounds__(256) void attend_combine_kernel(DecodeArgs<T> a) {
  constexpr int EPL = (DH + 63) / 64;  // elements per lane: channel 64 e + lane
  const long rows = (long)a.L * a.B * a.Hq * a.T_new;
  const long rid = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (rid >= rows) return;
  long t = rid;
  const int i = (int)(t % a.T_new);
  t /= a.T_new;
  const int hq = (int)(t % a.Hq);
  t /= a.Hq;
  const int b = (int)(t % a.B), l = (int)(t / a.B);
  const int c = a.chan.v[l], kvh = hq / (a.Hq / a.Hkv);
  const float cl2 = a.scale_log2;

  float M, Lsum, o[EPL];
  auto active = [&](int e) { return 64 * e + lane < DH; };
  if (a.mask_paper) {
    const T* q = a.Q + rid * DH;
    const T* kd = a.Kd + ((long)c * a.Hkv + kvh) * DH;
    const T* vd = a.Vd + ((long)c * a.Hkv + kvh) * DH;
    float part = 0.f;
    for (int e = 0; e < EPL; ++e)
      if (active(e)) part += to_f32(q[64 * e + lane]) * to_f32(kd[64 * e + lane]);
    M = wave_sum(part);
    Lsum = 1.f;
    for (int e = 0; e < EPL; ++e) o[e] = active(e) ? to_f32(vd[64 * e + lane]) : 0.f;
  } else {
    M = kNegBig;
    Lsum = 0.f;
    for (int e = 0; e < EPL; ++e) o[e] = 0.f;
  }
  const float* src = a.part + rid * a.nsplit * (DH + 2);
  for (int sidx = 0; sidx < a.nsplit; ++sidx) {
    const float* ps = src + (long)sidx * (DH + 2);
    float o2[EPL];
    for (int e = 0; e < EPL; ++e) o2[e] = active(e) ? ps[64 * e + lane] : 0.f;
    merge_state(M, Lsum, o, ps[DH], ps[DH + 1], o2, EPL, cl2);
  }
  T* dst = a.O + ((((long)l * a.B + b) * a.T_new + i) * a.Hq + hq) * DH;
  for (int e = 0; e < EPL; ++e)
    if (active(e)) dst[64 * e + lane] = from_f32<T>(o[e] / Lsum);
}

template <typename T, int DH>
static void decode_dispatch(const DecodeArgs<T>& a, int G, dim3 grid, hipStream_t s) {
  if (G <= 1)
    hipLaunchKernelGGL((attend_decode_kernel<T, DH, 1>), grid, dim3(256), 0, s, a);
  else if (G <= 2)
    hipLaunchKernelGGL((attend_decode_kernel<T, DH, 2>), grid, dim3(256), 0, s, a);
  else if (G <= 4)
    hipLaunchKernelGGL((attend_decode_kernel<T, DH, 4>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((attend_decode_kernel<T, DH, 8>), grid, dim3(256), 0, s, a);
  long rows = (long)a.L * a.B * a.Hq * a.T_new;
  hipLaunchKernelGGL((attend_combine_kernel<T, DH>), dim3((unsigned)((rows + 3) / 4)), dim3(256),
                     0, s, a);
}

template <typename T>
void launch_attend_decode(const Shape& sh, const LayerTable& chan_map, const ChannelGroups& cg,
                          const T* Q, const T* Kc, const T* Vc, const T* Kd, const T* Vd,
                          const int32_t* ctx_len, const int32_t* doc, float* partials, T* O,
                          hipStream_t s) {
  if (sh.N() <= 0) return;
  DecodeArgs<T> a{Q, Kc, Vc, Kd, Vd, ctx_len, doc, partials, O, sh.B, sh.T_new, sh.L, sh.Hq, sh.Hkv,
                  sh.S_cap, sh.mask_paper, decode_splits(sh), decode_split_len(sh), sh.gs, sh.gq,
                  sh.ctx_hi, kLog2e / sqrtf((float)sh.d), chan_map, cg};
  int maxmem = 0;
  for (int c = 0; c < sh.k; ++c) {
    int n = cg.offsets[c + 1] - cg.offsets[c];
    if (n > maxmem) maxmem = n;
  }
  int G = maxmem * (sh.Hq / sh.Hkv) * sh.T_new;
  dim3 grid(a.nsplit, sh.Hkv * sh.B * sh.k);
  if (sh.d == 96) {
    if constexpr (sizeof(T) == 2) decode_dispatch<T, 96>(a, G, grid, s);
  } else if (sh.d == 64)
    decode_dispatch<T, 64>(a, G, grid, s);
  else
    decode_dispatch<T, 32>(a, G, grid, s);
}

// ------------------------------------------------------------ dense soft read
// Layer l's soft mix of the k channels (the dense read of Section 3.1 Step 3):
// Kl[l][b][h][s] = sum_c w[l][c] Kc[c][b][h][s], the same for V, over the slots the
// call's rows may see (below min(S_cap, ctx + span)), and the dummy slots
// Kdl[l][h] = sum_c w[l][c] Kd[c][h] (blockIdx.y = L B Hkv for those). Sums in fp32,
// one 8-element chunk per thread.
template <typename T>
__global__ __launch_bounds__(256) void soft_read_kernel(const T* __restrict__ Kc,
                                                        const T* __restrict__ Vc,
                                                        const T* __restrict__ Kd,
                                                        const T* __restrict__ Vd,
                                                        const float* __restrict__ w, int B,
                                                        int Hkv, int S_cap, int k, int d,
                                                        const int32_t* ctx_len, int ctx_hi,
                                                        long span, T* Kl, T* Vl, T* Kdl,
                                                        T* Vdl) {
  const int c8 = d / 8;
  const int y = blockIdx.y;  // (l, b, h) slice, or the dummies of layer l
  const long x = (long)blockIdx.x * 256 + threadIdx.x;
  const int L = gridDim.y / (B * Hkv + 1);  // the grid's rows: L B Hkv slices, L dummy rows
  if (y < L * B * Hkv) {
    const int h = y % Hkv, b = (y / Hkv) % B, l = y / (Hkv * B);
    const long lim = min((long)S_cap, (long)ctx_at(ctx_len, b, ctx_hi) + span);
    if (x >= lim * c8) return;
    const long s = x / c8, e = (x % c8) * 8;
    float ka[8] = {0, 0, 0, 0, 0, 0, 0, 0}, va[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int c = 0; c < k; ++c) {
      const float wc = w[(long)l * k + c];
      const long off = (((long)c * B + b) * Hkv + h) * S_cap * d + s * d + e;
      float kv[8], vv[8];
      load8(Kc + off, kv);
      load8(Vc + off, vv);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ka[i] += wc * kv[i];
        va[i] += wc * vv[i];
      }
    }
    const long o = (((long)l * B + b) * Hkv + h) * S_cap * d + s * d + e;
    store8(Kl + o, ka);
    store8(Vl + o, va);
  } else {
    const int l = y - L * B * Hkv;
    if (x >= (long)Hkv * c8) return;
    const long h = x / c8, e = (x % c8) * 8;
    float ka[8] = {0, 0, 0, 0, 0, 0, 0, 0}, va[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int c = 0; c < k; ++c) {
      const float wc = w[(long)l * k + c];
      float kv[8], vv[8];
      load8(Kd + ((long)c * Hkv + h) * d + e, kv);
      load8(Vd + ((long)c * Hkv + h) * d + e, vv);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ka[i] += wc * kv[i];
        va[i] += wc * vv[i];
      }
    }
    store8(Kdl + ((long)l * Hkv + h) * d + e, ka);
    store8(Vdl + ((long)l * Hkv + h) * d + e, va);
  }
}

template <typename T>
void launch_soft_read(const Shape& sh, const float* w, const T* Kc, const T* Vc, const T* Kd,
                      const T* Vd, const int32_t* ctx_len, T* Kl, T* Vl, T* Kdl, T* Vdl,
                      hipStream_t s) {
  const long incl = sh.mask_paper ? 0 : 1;
  const long span = sh.span() - 1 + incl;  // slots below ctx + span are visible to some row
  const long rows = min((long)sh.S_cap, (long)sh.ctx_max + span) * (sh.d / 8);
  const long n = max(rows, (long)sh.Hkv * (sh.d / 8));
  dim3 grid((unsigned)((n + 255) / 256), (unsigned)(sh.L * sh.B * sh.Hkv + sh.L));
  hipLaunchKernelGGL(soft_read_kernel<T>, grid, dim3(256), 0, s, Kc, Vc, Kd, Vd, w, sh.B, sh.Hkv,
                     sh.S_cap, sh.k, sh.d, ctx_len, sh.ctx_hi, span, Kl, Vl, Kdl, Vdl);
}

#define WM_INST(T)                                                                              \
  template void launch_attend_prefill<T>(const Shape&, const LayerTable&, const T*, const T*,   \
                                         const T*, const T*, const T*, const int32_t*,          \
                                         const int32_t*, T*, void*, hipStream_t);               \
  template void launch_attend_decode<T>(const Shape&, const LayerTable&, const ChannelGroups&,  \
                                        const T*, const T*, const T*, const T*, const T*,       \
                                        const int32_t*, const int32_t*, float*, T*, hipStream_t); \
  template void launch_soft_read<T>(const Shape&, const float*, const T*, const T*, const T*,   \
                                    const T*, const int32_t*, T*, T*, T*, T*, hipStream_t);
WM_INST(float)
WM_INST(bf16)
#undef WM_INST

}  // namespace wm
