// Gradients of the pool (Section 3.1 Steps 1-2) and of the consumer queries (Step 7):
// the backward pass through the norms, the router, the mix and the projections, which
// training runs through its gradient-carrying passes (Section 3.3). bf16 operands, fp32
// gradients.
//
//   grad_gemm_kernel       C (+)= A B for strided, batched operands (bf16 or fp32, staged
//                          to LDS as bf16), MFMA 32x32x16, fp32 accumulation: every
//                          projection and router gradient (dX = dY W, dW = dY^T X) and the
//                          recomputed pre-norm projections.
//   grad_norm_apply_kernel g x / rms(x) rows as bf16 (the normed operands the GEMMs need).
//   grad_head_kernel       per head: the transposed RoPE rotation, then the head RMSNorm's
//                          backward (query and key norms), with the gain gradient's partial
//                          sums.
//   grad_rms_kernel        RMSNorm backward over rows of D (input, pre-mix and mid norms),
//                          with the gain gradient's partial sums.
//   grad_mix_kernel        per token: dĥ_l = sum_j alpha_jl dh~_j and dalpha_jl =
//                          dh~_j . ĥ_l (fp32), then the softmax (or masking) backward into
//                          the router logits' gradient.
//   grad_sum_kernel        deterministic sums of partial rows (gain and bias gradients).
#include <algorithm>

#include "wm_device.hpp"
#include "wm_frag.hpp"
#include "wm_internal.hpp"

namespace wm {

// ------------------------------------------------------------------------ GEMM
// Tiles of BM x BN = (32 WM WGM) x (32 WN WGN) on WGM x WGN waves, each owning WM x WN
// blocks of 32 x 32, K-steps of 32 staged to LDS as bf16 (the next step's global loads in
// flight during this step's MFMAs, one barrier per step). 256 x 256 tiles on 8 waves for
// the large products (128 FLOP per staged byte), 128 x 128 on 4 waves when the large
// tiles would leave CUs idle. Each operand is staged in one of two layouts, chosen from
// its strides:
//   N (k contiguous in memory): LDS [BM rows][32 k], 64-byte rows with a chunk swizzle;
//     lane (h, r) reads row r, k 16 ks + 8 h .. + 7 as one 16-byte word.
//   T (rows contiguous, k strided: the transposed operands of dW = dY^T X and dX = dY W):
//     LDS [32 k][BM + 16], filled by 8-row vector loads along the rows; lane (h, r)
//     gathers the same fragment with two transposing reads (ds_read_b64_tr_b16).
// VEC: 16-byte vector loads of bf16 operands (the strides allow them); otherwise element
// by element (bf16 or fp32), kept out of the vector kernels since it needs many registers.
template <int WGM_, int WGN_, int WM_, int WN_> struct GemmCfg {
  static constexpr int WGM = WGM_, WGN = WGN_, WM = WM_, WN = WN_;
  static constexpr int NT = 64 * WGM * WGN;
  static constexpr int BM = 32 * WM * WGM, BN = 32 * WN * WGN;
  static constexpr int VA = BM * 4 / NT, VB = BN * 4 / NT;  // 16-byte chunks per thread
  static constexpr int LDTA = BM + 16, LDTB = BN + 16;      // T layout pitches (elements)
  // bytes per staged tile: the larger of the two layouts
  static constexpr int TA_BYTES = (BM * 64 > 32 * LDTA * 2) ? BM * 64 : 32 * LDTA * 2;
  static constexpr int TB_BYTES = (BN * 64 > 32 * LDTB * 2) ? BN * 64 : 32 * LDTB * 2;
};
typedef GemmCfg<2, 4, 4, 2> GemmBig;    // 256 x 256, 8 waves
typedef GemmCfg<2, 2, 2, 2> GemmSmall;  // 128 x 128, 4 waves
typedef GemmCfg<2, 2, 1, 1> GemmTiny;   // 64 x 64, 4 waves

__device__ __forceinline__ int grad_swz(int row) { return ((row >> 1) ^ (row >> 3)) & 3; }

// N layout: chunk v of this thread is row idx / 4, k = k0 + 8 (idx % 4) .. + 7 with
// idx = tid + NT v; elements with k < klo are zero.
template <int BM, int NT, int V, bool VEC>
__device__ __forceinline__ void gemm_load_n(const GemmOperand& o, long zoff, int row0, int k0,
                                            int nrows, int K, int klo, int tid, bf16x8 (&v)[V]) {
#pragma unroll
  for (int c = 0; c < V; ++c) {
    const int idx = tid + NT * c, row = row0 + (idx >> 2), k = k0 + 8 * (idx & 3);
    if constexpr (VEC) {  // bf16, k contiguous, rows 8-aligned; K rounded up to 8 readable
      const bool ok = row < nrows && k < K;
      v[c] = ok ? *(const bf16x8*)((const bf16*)o.p + zoff + (long)row * o.s_row + k)
                : zero_frag<bf16>();
      if (klo > k) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (k + e < klo) v[c][e] = (bf16)0.f;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x = 0.f;
        if (row < nrows && k + e < K && k + e >= klo) {
          const long off = zoff + (long)row * o.s_row + (long)(k + e) * o.s_k;
          x = o.f32 ? ((const float*)o.p)[off] : (float)((const bf16*)o.p)[off];
        }
        v[c][e] = (bf16)x;
      }
    }
  }
}

template <int NT, int V>
__device__ __forceinline__ void gemm_store_n(char* tile, int tid, const bf16x8 (&v)[V]) {
#pragma unroll
  for (int c = 0; c < V; ++c) {
    const int idx = tid + NT * c, r = idx >> 2;
    *(bf16x8*)(tile + r * 64 + 16 * ((idx & 3) ^ grad_swz(r))) = v[c];
  }
}

// T layout: chunk v of this thread is k = k0 + idx / (BM / 8), rows row0 + 8 (idx % (BM / 8))
// .. + 7 with idx = tid + NT v.
template <int BM, int NT, int V, bool VEC>
__device__ __forceinline__ void gemm_load_t(const GemmOperand& o, long zoff, int row0, int k0,
                                            int nrows, int K, int klo, int tid, bf16x8 (&v)[V]) {
  constexpr int RC = BM / 8;  // row chunks per k row
#pragma unroll
  for (int c = 0; c < V; ++c) {
    const int idx = tid + NT * c, k = k0 + idx / RC, row = row0 + 8 * (idx % RC);
    const bool kok = k < K && k >= klo;
    if constexpr (VEC) {  // bf16, rows contiguous and readable in whole groups of 8
      const bool ok = kok && row < nrows;
      v[c] = ok ? *(const bf16x8*)((const bf16*)o.p + zoff + (long)k * o.s_k + row)
                : zero_frag<bf16>();
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x = 0.f;
        if (kok && row + e < nrows) {
          const long off = zoff + (long)(row + e) * o.s_row + (long)k * o.s_k;
          x = o.f32 ? ((const float*)o.p)[off] : (float)((const bf16*)o.p)[off];
        }
        v[c][e] = (bf16)x;
      }
    }
  }
}

template <int BM, int NT, int V>
__device__ __forceinline__ void gemm_store_t(char* tile, int tid, const bf16x8 (&v)[V]) {
  constexpr int RC = BM / 8, LDT = BM + 16;
#pragma unroll
  for (int c = 0; c < V; ++c) {
    const int idx = tid + NT * c;
    *(bf16x8*)(tile + ((idx / RC) * LDT + 8 * (idx % RC)) * 2) = v[c];
  }
}

// Fragment of rows rb .. rb + 31 (lane row r), k 16 ks + 8 h .. + 7, from either layout.
// T layout: within a 16-lane group, lane j addresses k row 16 ks + 8 h + 4 s + j / 4 and
// rows rb + 16 (group & 1) + 4 (j % 4) .. + 3; the transposing read hands lane i the four
// k values of row rb + 16 (group & 1) + i, so s = 0, 1 give k 8 h + 0..3 and 4..7.
template <bool T, int LDT>
__device__ __forceinline__ bf16x8 gemm_frag(const char* tile, int rb, int ks, int lane) {
  if constexpr (T) {
    const int j = lane & 15, grp = lane >> 4, h = lane >> 5;
    const char* p =
        tile + ((16 * ks + 8 * h + (j >> 2)) * LDT + rb + 16 * (grp & 1) + 4 * (j & 3)) * 2;
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
    const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * LDT * 2));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
  } else {
    const int h = lane >> 5, row = rb + (lane & 31);
    return *(const bf16x8*)(tile + row * 64 + 16 * ((2 * ks + h) ^ grad_swz(row)));
  }
}

// The tile's results into C (or a split's partial rows): lane (h, r) holds column
// n0 + 32 (WN wn + j) + r, rows m0 + 32 (WM wm + i) + 8 (q / 4) + 4 h + q % 4. When adding
// into C, the 16 old values of a 32 x 32 block are all loaded before any is stored, so
// those loads wait on memory together rather than one round trip per element.
template <class C>
__device__ __forceinline__ void gemm_store(const f32x16 (&acc)[C::WM][C::WN], float* Cz,
                                           long crow, long ccol, int M, int N, int mlo,
                                           int acc_in, int m0, int n0, int wm, int wn, int h,
                                           int r) {
#pragma unroll
  for (int j = 0; j < C::WN; ++j) {
    const int n = n0 + 32 * (C::WN * wn + j) + r;
    if (n >= N) continue;
    float* col = Cz + (long)n * ccol;
    if (acc_in) {
#pragma unroll
      for (int i = 0; i < C::WM; ++i) {
        float old[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int m = m0 + 32 * (C::WM * wm + i) + 8 * (q >> 2) + 4 * h + (q & 3);
          old[q] = m < M && m >= mlo ? col[(long)m * crow] : 0.f;
        }
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int m = m0 + 32 * (C::WM * wm + i) + 8 * (q >> 2) + 4 * h + (q & 3);
          if (m < M && m >= mlo) col[(long)m * crow] = old[q] + acc[i][j][q];
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < C::WM; ++i)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int m = m0 + 32 * (C::WM * wm + i) + 8 * (q >> 2) + 4 * h + (q & 3);
          if (m < M && m >= mlo) col[(long)m * crow] = acc[i][j][q];
        }
    }
  }
}

template <class C, bool TA, bool TB, bool VEC>
__global__ __launch_bounds__(C::NT) void grad_gemm_kernel(GemmArgs a) {
  __shared__ __align__(16) char smem[2][C::TA_BYTES + C::TB_BYTES];  // [buffer][A | B]
  const int tm = (a.M + C::BM - 1) / C::BM, tn = (a.N + C::BN - 1) / C::BN;
  const int tile = xcd_tile(blockIdx.x, (int)gridDim.x);
  const int zs = tile / (tm * tn), t = tile % (tm * tn);
  const int z = zs / a.splits, slice = zs % a.splits;
  const int m0 = (t / tn) * C::BM, n0 = (t % tn) * C::BN;
  const int kbeg = slice * a.kchunk, kend = min(a.K, kbeg + a.kchunk);
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = tid >> 6, wm = w % C::WGM, wn = w / C::WGM;
  const long za = (long)z * a.A.s_z, zb = (long)z * a.B.s_z;
  const int klo = (int)(a.k_lo0 + a.k_lo_dz * z);
  f32x16 acc[C::WM][C::WN];
#pragma unroll
  for (int i = 0; i < C::WM; ++i)
#pragma unroll
    for (int j = 0; j < C::WN; ++j) acc[i][j] = zero16();
  bf16x8 va[C::VA], vb[C::VB];
  const int nk = (kend - kbeg + 31) / 32;
  auto load = [&](int k0) {
    if constexpr (TA) gemm_load_t<C::BM, C::NT, C::VA, VEC>(a.A, za, m0, k0, a.M, a.K, 0, tid, va);
    else gemm_load_n<C::BM, C::NT, C::VA, VEC>(a.A, za, m0, k0, a.M, a.K, 0, tid, va);
    if constexpr (TB) gemm_load_t<C::BN, C::NT, C::VB, VEC>(a.B, zb, n0, k0, a.N, a.K, klo, tid, vb);
    else gemm_load_n<C::BN, C::NT, C::VB, VEC>(a.B, zb, n0, k0, a.N, a.K, klo, tid, vb);
  };
  load(kbeg);
  for (int kt = 0; kt < nk; ++kt) {
    char* sa = smem[kt & 1];
    char* sb = sa + C::TA_BYTES;
    if constexpr (TA) gemm_store_t<C::BM, C::NT, C::VA>(sa, tid, va);
    else gemm_store_n<C::NT, C::VA>(sa, tid, va);
    if constexpr (TB) gemm_store_t<C::BN, C::NT, C::VB>(sb, tid, vb);
    else gemm_store_n<C::NT, C::VB>(sb, tid, vb);
    __syncthreads();  // tile kt in LDS; every wave is done with tile kt - 1
    if (kt + 1 < nk) load(kbeg + 32 * (kt + 1));
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 fa[C::WM], fb[C::WN];
#pragma unroll
      for (int i = 0; i < C::WM; ++i)
        fa[i] = gemm_frag<TA, C::LDTA>(sa, 32 * (C::WM * wm + i), ks, lane);
#pragma unroll
      for (int j = 0; j < C::WN; ++j)
        fb[j] = gemm_frag<TB, C::LDTB>(sb, 32 * (C::WN * wn + j), ks, lane);
#pragma unroll
      for (int i = 0; i < C::WM; ++i)
#pragma unroll
        for (int j = 0; j < C::WN; ++j) acc[i][j] = mma32(acc[i][j], fa[i], fb[j]);
    }
  }
  // lane (h, r): column n0 + 32 (WN wn + j) + r, rows m0 + 32 (WM wm + i) + 8 (q / 4) + 4 h + q % 4
  // (split K: the slice's partial tile goes to part[z][slice] as M x N rows, written)
  const bool split = a.splits > 1;
  float* Cz = split ? a.part + ((long)z * a.splits + slice) * a.M * a.N : a.C + (long)z * a.c_z;
  const long crow = split ? a.N : a.c_row, ccol = split ? 1 : a.c_col;
  const int mlo = split ? 0 : (int)(a.m_lo0 + a.m_lo_dz * z);
  const int acc_in = split ? 0 : a.accumulate;
  gemm_store<C>(acc, Cz, crow, ccol, a.M, a.N, mlo, acc_in, m0, n0, wm, wn, h, r);
}

// ---- the same product with LDS DMA: every tile goes from memory straight into LDS
// (buffer_load ... lds, no registers), kGemmStages K-steps in flight. Layouts as above,
// except that the k-major (T) tile has no padding: k row kk holds its BM rows as 16-byte
// chunks, chunk c at position c ^ 2 (kk mod 4), so the four k rows one transposing read
// touches fall in disjoint banks. Each wave issues the same number of copies per stage
// (BM / 16 per operand over the workgroup), which the vmcnt waits rely on.
constexpr int kGemmStages = 3;

// this lane's copy n of a tile: LDS chunk q = 64 (NI w + n) + lane; returns the byte offset
// of the chunk it fetches within the batch's view (kOffOob: zeros)
template <bool T, int BM>
__device__ __forceinline__ uint32_t dma_src(const GemmOperand& o, int q, int row0, int k0, int nrows,
                                            int K, int klo) {
  if constexpr (T) {
    const int kk = q / (BM / 8), c = (q % (BM / 8)) ^ (2 * (kk & 3));
    const int k = k0 + kk, row = row0 + 8 * c;
    const bool ok = k < K && k >= klo && row < nrows;
    return ok ? (uint32_t)(((long)k * o.s_k + row) * 2) : kOffOob;
  } else {
    const int r = q >> 2, c = (q & 3) ^ grad_swz(r);
    const int row = row0 + r, k = k0 + 8 * c;
    const bool ok = row < nrows && k < K;
    return ok ? (uint32_t)(((long)row * o.s_row + k) * 2) : kOffOob;
  }
}

// fragment of rows rb .. rb + 31, k 16 ks + 8 h .. + 7 from a DMA-staged tile
template <bool T, int BM>
__device__ __forceinline__ bf16x8 gemm_frag_dma(const char* tile, int rb, int ks, int lane) {
  if constexpr (T) {
    const int j = lane & 15, grp = lane >> 4, h = lane >> 5;
    const int row = rb + 16 * (grp & 1) + 4 * (j & 3), c = row >> 3, within = row & 7;
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    i16x4 v[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int kk = 16 * ks + 8 * h + 4 * s + (j >> 2);
      const char* p = tile + kk * BM * 2 + 16 * (c ^ (2 * (kk & 3))) + 2 * within;
      v[s] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
    }
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(v[0], v[1], 0, 1, 2, 3, 4, 5, 6, 7));
  } else {
    const int h = lane >> 5, row = rb + (lane & 31);
    return *(const bf16x8*)(tile + row * 64 + 16 * ((2 * ks + h) ^ grad_swz(row)));
  }
}

template <class C, bool TA, bool TB>
__global__ __launch_bounds__(C::NT) void grad_gemm_dma_kernel(GemmArgs a) {
  constexpr int S = kGemmStages, AB = C::BM * 64, BB = C::BN * 64;
  constexpr int NIA = C::BM / 16 / (C::NT / 64), NIB = C::BN / 16 / (C::NT / 64);
  static_assert(NIA * (C::NT / 64) * 16 == C::BM && NIB * (C::NT / 64) * 16 == C::BN,
                "whole copies per wave");
  static_assert((S - 2) * (NIA + NIB) < 16, "vmcnt range");
  __shared__ __align__(16) char smem[S][AB + BB];
  const int tm = (a.M + C::BM - 1) / C::BM, tn = (a.N + C::BN - 1) / C::BN;
  const int tile = xcd_tile(blockIdx.x, (int)gridDim.x);
  const int zs = tile / (tm * tn), t = tile % (tm * tn);
  const int z = zs / a.splits, slice = zs % a.splits;
  const int m0 = (t / tn) * C::BM, n0 = (t % tn) * C::BN;
  const int kbeg = slice * a.kchunk, kend = min(a.K, kbeg + a.kchunk);
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), wm = w % C::WGM, wn = w / C::WGM;
  const int klo = (int)(a.k_lo0 + a.k_lo_dz * z);
  const auto va = make_view((const bf16*)a.A.p + (long)z * a.A.s_z, (uint32_t)a.A.span);
  const auto vb = make_view((const bf16*)a.B.p + (long)z * a.B.s_z, (uint32_t)a.B.span);
  const uint32_t lbase = (uint32_t)(uintptr_t)&smem[0][0];
  const int nk = (kend - kbeg + 31) / 32;
  auto issue = [&](int kt) {
    const int k0 = kbeg + 32 * kt;
    const uint32_t st = lbase + (uint32_t)(kt % S) * (AB + BB);
#pragma unroll
    for (int n = 0; n < NIA; ++n) {
      const int q = 64 * (NIA * w + n) + lane;
      lds_dma16(__builtin_amdgcn_readfirstlane(st + 1024u * (NIA * w + n)),
                dma_src<TA, C::BM>(a.A, q, m0, k0, a.M, a.K, 0), va);
    }
#pragma unroll
    for (int n = 0; n < NIB; ++n) {
      const int q = 64 * (NIB * w + n) + lane;
      lds_dma16(__builtin_amdgcn_readfirstlane(st + AB + 1024u * (NIB * w + n)),
                dma_src<TB, C::BN>(a.B, q, n0, k0, a.N, a.K, klo), vb);
    }
  };
  f32x16 acc[C::WM][C::WN];
#pragma unroll
  for (int i = 0; i < C::WM; ++i)
#pragma unroll
    for (int j = 0; j < C::WN; ++j) acc[i][j] = zero16();
#pragma unroll
  for (int st = 0; st < S - 1; ++st)
    if (st < nk) issue(st);
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + S - 2 < nk) wait_vmcnt<(S - 2) * (NIA + NIB)>();
    else wait_vmcnt<0>();
    __syncthreads();  // stage kt in LDS; every wave is done with stage kt - 1
    if (kt + S - 1 < nk) issue(kt + S - 1);
    const char* sa = smem[kt % S];
    const char* sb = sa + AB;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 fa[C::WM], fb[C::WN];
#pragma unroll
      for (int i = 0; i < C::WM; ++i) fa[i] = gemm_frag_dma<TA, C::BM>(sa, 32 * (C::WM * wm + i), ks, lane);
#pragma unroll
      for (int j = 0; j < C::WN; ++j) fb[j] = gemm_frag_dma<TB, C::BN>(sb, 32 * (C::WN * wn + j), ks, lane);
#pragma unroll
      for (int i = 0; i < C::WM; ++i)
#pragma unroll
        for (int j = 0; j < C::WN; ++j) acc[i][j] = mma32(acc[i][j], fa[i], fb[j]);
    }
  }
  const bool split = a.splits > 1;
  float* Cz = split ? a.part + ((long)z * a.splits + slice) * a.M * a.N : a.C + (long)z * a.c_z;
  const long crow = split ? a.N : a.c_row, ccol = split ? 1 : a.c_col;
  const int mlo = split ? 0 : (int)(a.m_lo0 + a.m_lo_dz * z);
  const int acc_in = split ? 0 : a.accumulate;
  gemm_store<C>(acc, Cz, crow, ccol, a.M, a.N, mlo, acc_in, m0, n0, wm, wn, h, r);
}

static bool operand_t(const GemmOperand& o) { return o.s_row == 1 && o.s_k != 1; }

// Vector loads need bf16, 16-byte alignment and strides in whole 8-element groups, with
// the last group of rows (T) or of k (N) readable in full (a multiple of 8, or pad8).
static bool operand_vec(const GemmOperand& o, int nrows, int K) {
  if (o.f32 || (uintptr_t)o.p % 16 != 0 || o.s_z % 8 != 0) return false;
  if (operand_t(o)) return o.s_k % 8 == 0 && (nrows % 8 == 0 || o.pad8);
  return o.s_k == 1 && o.s_row % 8 == 0 && (K % 8 == 0 || o.pad8);
}

// C[z] (+)= sum over slices of part[z][slice], in slice order; rows below the batch's
// m_lo untouched.
__global__ __launch_bounds__(256) void grad_split_sum_kernel(GemmArgs a) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long mn = (long)a.M * a.N;
  const int z = blockIdx.y;
  if (idx >= mn) return;
  const int m = (int)(idx / a.N), n = (int)(idx % a.N);
  if (m < a.m_lo0 + a.m_lo_dz * z) return;
  const float* p = a.part + (long)z * a.splits * mn + idx;
  float v = 0.f;
  for (int sl = 0; sl < a.splits; ++sl) v += p[sl * mn];
  float* c = a.C + (long)z * a.c_z + (long)m * a.c_row + (long)n * a.c_col;
  *c = a.accumulate ? *c + v : v;
}

// bytes a batch's tile loads may reach (vector rows / k rounded up to 8)
static long operand_span(const GemmOperand& o, int nrows, int K) {
  const long r8 = (nrows + 7) / 8 * 8, k8 = ((long)K + 7) / 8 * 8;
  if (operand_t(o)) return ((long)(K - 1) * o.s_k + r8) * 2;
  return ((long)(nrows - 1) * o.s_row + k8) * 2;
}

template <class C, bool TA, bool TB>
static void launch_gemm_dma(const GemmArgs& a, int batches, hipStream_t s) {
  const long tiles = (long)((a.M + C::BM - 1) / C::BM) * ((a.N + C::BN - 1) / C::BN) * batches *
                     a.splits;
  hipLaunchKernelGGL((grad_gemm_dma_kernel<C, TA, TB>), dim3((unsigned)tiles), dim3(C::NT), 0, s, a);
}

template <class C, bool TA, bool TB, bool VEC>
static void launch_gemm_cfg(const GemmArgs& a, int batches, hipStream_t s) {
  const long tiles = (long)((a.M + C::BM - 1) / C::BM) * ((a.N + C::BN - 1) / C::BN) * batches *
                     a.splits;
  hipLaunchKernelGGL((grad_gemm_kernel<C, TA, TB, VEC>), dim3((unsigned)tiles), dim3(C::NT), 0, s,
                     a);
}

template <bool TA, bool TB>
static void launch_gemm_t(GemmArgs a, int batches, bool vec, hipStream_t s) {
  // the large tiles (vector operands only) when they still give every CU at least two, the
  // 64 x 64 ones when the 128 x 128 ones would leave CUs idle; LDS DMA when both operands'
  // batch spans fit a buffer view and no k-contiguous B operand carries a k limit (its
  // copies are whole 8-element chunks)
  const long big = (long)((a.M + 255) / 256) * ((a.N + 255) / 256) * batches;
  a.A.span = operand_span(a.A, a.M, a.K);
  a.B.span = operand_span(a.B, a.N, a.K);
  const bool dma = vec && a.A.span < (1L << 31) && a.B.span < (1L << 31) &&
                   (TB || (a.k_lo0 == 0 && a.k_lo_dz == 0));
  const long small = (long)((a.M + 127) / 128) * ((a.N + 127) / 128) * batches * a.splits;
  if (dma && big >= 2L * device_cus()) launch_gemm_dma<GemmBig, TA, TB>(a, batches, s);
  else if (dma && small < device_cus()) launch_gemm_dma<GemmTiny, TA, TB>(a, batches, s);
  else if (dma) launch_gemm_dma<GemmSmall, TA, TB>(a, batches, s);
  else if (vec && big >= 2L * device_cus()) launch_gemm_cfg<GemmBig, TA, TB, true>(a, batches, s);
  else if (vec) launch_gemm_cfg<GemmSmall, TA, TB, true>(a, batches, s);
  else launch_gemm_cfg<GemmSmall, TA, TB, false>(a, batches, s);
}

void launch_grad_gemm(GemmArgs a, int batches, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0 || batches <= 0) return;
  const bool vec = operand_vec(a.A, a.M, a.K) && operand_vec(a.B, a.N, a.K);
  const bool ta = operand_t(a.A), tb = operand_t(a.B);
  // split K when the 128 x 128 tiles number under two per CU and K spans >= 64 K-steps
  a.splits = 1;
  a.kchunk = ((a.K + 31) / 32) * 32;
  const long tiles = (long)((a.M + 127) / 128) * ((a.N + 127) / 128) * batches;
  const long mnb = (long)a.M * a.N * batches;
  if (vec && a.part && a.K >= 2048 && tiles < 2L * device_cus()) {
    long sp = std::min<long>((2L * device_cus() + tiles - 1) / tiles, a.K / 1024);
    sp = std::min<long>(sp, a.part_elems / std::max(mnb, 1L));
    if (sp > 1) {
      a.kchunk = (int)(((a.K + sp - 1) / sp + 31) / 32 * 32);
      a.splits = (a.K + a.kchunk - 1) / a.kchunk;
    }
  }
  if (ta && tb) launch_gemm_t<true, true>(a, batches, vec, s);
  else if (ta) launch_gemm_t<true, false>(a, batches, vec, s);
  else if (tb) launch_gemm_t<false, true>(a, batches, vec, s);
  else launch_gemm_t<false, false>(a, batches, vec, s);
  if (a.splits > 1) {
    const long mn = (long)a.M * a.N;
    hipLaunchKernelGGL(grad_split_sum_kernel, dim3((unsigned)((mn + 255) / 256), batches),
                       dim3(256), 0, s, a);
  }
}

// --------------------------------------------------------------- row kernels
// out[r][e] = g[(r / gdiv) % gmod][e] * x[r][e] * rinv[r], as bf16; one block per row,
// eight elements per thread (D is a multiple of 32, rows 16-byte aligned).
__global__ __launch_bounds__(256) void grad_norm_apply_kernel(const bf16* x, const bf16* g,
                                                              const float* rinv, long gdiv,
                                                              int gmod, int D, bf16* out) {
  const long r = blockIdx.x;
  const bf16* gr = g + ((r / gdiv) % gmod) * (long)D;
  const float ri = rinv[r];
  for (int e = 8 * threadIdx.x; e < D; e += 2048) {
    const bf16x8 xv = *(const bf16x8*)(x + r * D + e), gv = *(const bf16x8*)(gr + e);
    bf16x8 o;
#pragma unroll
    for (int u = 0; u < 8; ++u) o[u] = (bf16)((float)gv[u] * (float)xv[u] * ri);
    *(bf16x8*)(out + r * D + e) = o;
  }
}

void launch_grad_norm_apply(const bf16* x, const bf16* g, const float* rinv, long rows, long gdiv,
                            int gmod, int D, bf16* out, hipStream_t s) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(grad_norm_apply_kernel, dim3((unsigned)rows), dim3(256), 0, s, x, g, rinv,
                     gdiv, gmod, D, out);
}

// Head RMSNorm + RoPE backward. Row (z, b, h, i): the gradient dR of the rotated output at
// src[z][b][h][slot] (slot = i, or ctx_len[b] + i for the cache; rows of d floats), the
// pre-norm values y at y[z][b T + i][h d] (fp32), the gain g[z][d] and the angle table
// tab[b T + i][d / 2] (cos, sin) of the forward; writes dy (the gradient of y, y's layout)
// and adds each row's dg contribution into the workgroup's partial row
// dgp[z][blockIdx.x % chunks][d]. One wave per row.
template <int DH>
__global__ __launch_bounds__(256) void grad_head_kernel(HeadArgs a) {
  constexpr int PER = (DH + 63) / 64;
  const int chunk = blockIdx.x % a.chunks, z = blockIdx.x / a.chunks;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const long rows = (long)a.B * a.H * a.T;  // rows of one z
  const long r0 = rows * chunk / a.chunks, r1 = rows * (chunk + 1) / a.chunks;
  float dg[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) dg[q] = 0.f;
  const bf16* g = a.g + (long)z * DH;
  // row rr = (b H + hh) T + i, stepped by 4 without divisions in the loop
  long rr = r0 + w;
  int i = (int)(rr % a.T), hh = (int)(rr / a.T % a.H), b = (int)(rr / ((long)a.T * a.H));
  for (; rr < r1; rr += 4) {
    const int slot = a.slot_ctx ? ctx_at(a.ctx_len, b, a.ctx_hi) + a.gq + a.gs * i : i;
    const float* src = a.src + ((long)z * a.sZ + (long)b * a.sB + (long)hh * a.sH + slot) * DH;
    const long yrow = ((long)z * a.B * a.T + (long)b * a.T + i) * a.H * DH + (long)hh * DH;
    const float* tab = a.tab + ((long)b * a.T + i) * DH;  // DH / 2 (cos, sin) pairs
    // RoPE^T: (da, db) = (c dx_m + s dx_{m+d/2}, -s dx_m + c dx_{m+d/2})
    float yv[PER], gy[PER], dr[PER];
    float ss = 0.f;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = lane + 64 * q;
      yv[q] = gy[q] = dr[q] = 0.f;
      if (e < DH) {
        const int m = e < DH / 2 ? e : e - DH / 2;
        const float cs = tab[2 * m], sn = tab[2 * m + 1];
        const float dx = src[e], dp = src[e < DH / 2 ? e + DH / 2 : e - DH / 2];
        dr[q] = e < DH / 2 ? cs * dx + sn * dp : cs * dx - sn * dp;
        yv[q] = a.y[yrow + e];
        gy[q] = (float)g[e] * dr[q];
        ss += yv[q] * yv[q];
      }
    }
    ss = wave_sum(ss);
    const float ri = 1.0f / sqrtf(ss / DH + a.eps);
    float dot = 0.f;
#pragma unroll
    for (int q = 0; q < PER; ++q) dot += gy[q] * yv[q];
    dot = wave_sum(dot);
    const float c2 = ri * ri * dot / DH;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = lane + 64 * q;
      if (e < DH) {
        a.dy[yrow + e] = (bf16)(ri * (gy[q] - yv[q] * c2));
        dg[q] += dr[q] * yv[q] * ri;
      }
    }
    i += 4;
    while (i >= a.T) {
      i -= a.T;
      if (++hh == a.H) {
        hh = 0;
        ++b;
      }
    }
  }
  __shared__ float s_dg[4][DH];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = lane + 64 * q;
    if (e < DH) s_dg[w][e] = dg[q];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < DH; e += 256)
    a.dgp[((long)z * a.chunks + chunk) * DH + e] =
        (s_dg[0][e] + s_dg[1][e]) + (s_dg[2][e] + s_dg[3][e]);
}

void launch_grad_head(const HeadArgs& a, int Z, int d, hipStream_t s) {
  if (Z <= 0 || (long)a.B * a.H * a.T == 0) return;
  const dim3 grid(Z * a.chunks);
  if (d == 64) hipLaunchKernelGGL(grad_head_kernel<64>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(grad_head_kernel<96>, grid, dim3(256), 0, s, a);
}

// RMSNorm backward over rows of D: row (o, i) for gain row o (0 <= o < nouter) and
// i < ninner; tensors addressed as base + (o s_o + i s_i) D. With y = g x / rms(x):
// dx = rinv (g dy - x rinv^2 (g dy . x) / D), dg += dy x rinv. dx is added into out (or
// written when accumulate is 0); dg partial rows per workgroup.
__global__ __launch_bounds__(256) void grad_rms_kernel(RmsArgs a) {
  constexpr int MAXP = 18;  // D <= 4608
  const int chunk = blockIdx.x % a.chunks, o = blockIdx.x / a.chunks;
  const long i0 = (long)a.ninner * chunk / a.chunks, i1 = (long)a.ninner * (chunk + 1) / a.chunks;
  const int tid = threadIdx.x;
  __shared__ float s_red[2][4];
  float dg[MAXP];
#pragma unroll
  for (int q = 0; q < MAXP; ++q) dg[q] = 0.f;
  const bf16* g = a.g + (long)o * a.D;
  int par = 0;
  for (long i = i0; i < i1; ++i, par ^= 1) {
    const float* dy = a.dy + ((long)o * a.dy_o + i * a.dy_i) * a.D;
    const bf16* x = a.x + ((long)o * a.x_o + i * a.x_i) * a.D;
    float* out = a.out + ((long)o * a.out_o + i * a.out_i) * a.D;
    const float ri = a.rinv[(long)o * a.r_o + i * a.r_i];
    float dv[MAXP], xv[MAXP], dot = 0.f;
#pragma unroll
    for (int q = 0; q < MAXP; ++q) {
      const int e = tid + 256 * q;
      dv[q] = xv[q] = 0.f;
      if (e < a.D) {
        dv[q] = dy[e];
        xv[q] = (float)x[e];
        dot += (float)g[e] * dv[q] * xv[q];
      }
    }
    dot = wave_sum(dot);
    if ((tid & 63) == 0) s_red[par][tid >> 6] = dot;
    __syncthreads();  // (alternating halves of s_red: one barrier per row)
    dot = (s_red[par][0] + s_red[par][1]) + (s_red[par][2] + s_red[par][3]);
    const float c2 = ri * ri * dot / a.D;
#pragma unroll
    for (int q = 0; q < MAXP; ++q) {
      const int e = tid + 256 * q;
      if (e < a.D) {
        const float dx = ri * ((float)g[e] * dv[q] - xv[q] * c2);
        out[e] = a.accumulate ? out[e] + dx : dx;
        dg[q] += dv[q] * xv[q] * ri;
      }
    }
  }
#pragma unroll
  for (int q = 0; q < MAXP; ++q) {
    const int e = tid + 256 * q;
    if (e < a.D) a.dgp[((long)o * a.chunks + chunk) * a.D + e] = dg[q];
  }
}

// The same with one wave per row (no workgroup barrier between rows, four rows in flight
// per workgroup): lane t takes elements 4 t + 256 q .. + 3 (q < PER / 4), so D <= 64 PER;
// the waves' gain partials are added in wave order at the end.
template <int PER>
__global__ __launch_bounds__(256) void grad_rms_wave_kernel(RmsArgs a) {
  constexpr int NV = PER / 4;
  const int chunk = blockIdx.x % a.chunks, o = blockIdx.x / a.chunks;
  const long i0 = (long)a.ninner * chunk / a.chunks, i1 = (long)a.ninner * (chunk + 1) / a.chunks;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, D = a.D;
  __shared__ float s_dg[64 * PER];  // the gain partials, summed over the waves
  const bf16* g = a.g + (long)o * D;
  float gv[PER], dg[PER];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int e = 4 * lane + 256 * v;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      gv[4 * v + u] = e + u < D ? (float)g[e + u] : 0.f;
      dg[4 * v + u] = 0.f;
    }
  }
  for (long i = i0 + w; i < i1; i += 4) {
    const float* dy = a.dy + ((long)o * a.dy_o + i * a.dy_i) * D;
    const bf16* x = a.x + ((long)o * a.x_o + i * a.x_i) * D;
    float* out = a.out + ((long)o * a.out_o + i * a.out_i) * D;
    const float ri = a.rinv[(long)o * a.r_o + i * a.r_i];
    float dv[PER], xv[PER], dot = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int e = 4 * lane + 256 * v;
      if (e < D) {  // D is a multiple of 32: a lane's four elements are all in or all out
        const f32x4 d4 = *(const f32x4*)(dy + e);
        const bf16x4 x4 = *(const bf16x4*)(x + e);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          dv[4 * v + u] = d4[u];
          xv[4 * v + u] = (float)x4[u];
          dot += gv[4 * v + u] * d4[u] * xv[4 * v + u];
        }
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) dv[4 * v + u] = xv[4 * v + u] = 0.f;
      }
    }
    dot = wave_sum(dot);
    const float c2 = ri * ri * dot / D;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int e = 4 * lane + 256 * v;
      if (e < D) {
        f32x4 r4;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int q = 4 * v + u;
          r4[u] = ri * (gv[q] * dv[q] - xv[q] * c2);
          dg[q] += dv[q] * xv[q] * ri;
        }
        if (a.accumulate) r4 += *(const f32x4*)(out + e);
        *(f32x4*)(out + e) = r4;
      }
    }
  }
  for (int ww = 0; ww < 4; ++ww) {
    if (w == ww) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int e = 4 * lane + 256 * v;
        if (e < D)
#pragma unroll
          for (int u = 0; u < 4; ++u)
            s_dg[e + u] = ww == 0 ? dg[4 * v + u] : s_dg[e + u] + dg[4 * v + u];
      }
    }
    __syncthreads();
  }
  for (int e = tid; e < D; e += 256) a.dgp[((long)o * a.chunks + chunk) * D + e] = s_dg[e];
}

static bool rms_wave_ok(const RmsArgs& a) {
  // vector access: row bases and the tensors 16-byte (fp32) / 8-byte (bf16) aligned
  const long rows[] = {a.dy_o, a.dy_i, a.out_o, a.out_i, a.x_o, a.x_i};
  for (long r : rows)
    if ((r * a.D) % 4 != 0) return false;
  return (uintptr_t)a.dy % 16 == 0 && (uintptr_t)a.out % 16 == 0 && (uintptr_t)a.x % 8 == 0;
}

void launch_grad_rms(const RmsArgs& a, int nouter, hipStream_t s) {
  if (nouter <= 0 || a.ninner <= 0) return;
  const dim3 grid(nouter * a.chunks), blk(256);
  if (rms_wave_ok(a) && a.D <= 512) hipLaunchKernelGGL(grad_rms_wave_kernel<8>, grid, blk, 0, s, a);
  else if (rms_wave_ok(a) && a.D <= 1024)
    hipLaunchKernelGGL(grad_rms_wave_kernel<16>, grid, blk, 0, s, a);
  else if (rms_wave_ok(a) && a.D <= 2048)
    hipLaunchKernelGGL(grad_rms_wave_kernel<32>, grid, blk, 0, s, a);
  else hipLaunchKernelGGL(grad_rms_kernel, grid, blk, 0, s, a);
}

// out[o][e] (+)= scale * sum over c < chunks of part[(o chunks + c) n + e], in a fixed
// order: with many chunks, first groups of kSumGroup chunks (each group's sum written over
// its first row, read only by the thread that writes it), then the groups' sums in order.
constexpr int kSumGroup = 32;

// v + p[0] + p[stride] + ... over cnt rows, added in row order; the loads are issued eight
// at a time before their adds, so a thread waits for memory once per eight rows
__device__ __forceinline__ float sum_rows(float v, const float* p, long stride, int cnt) {
  int c = 0;
  for (; c + 8 <= cnt; c += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = p[(c + u) * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u) v += t[u];
  }
  for (; c < cnt; ++c) v += p[c * stride];
  return v;
}

__global__ __launch_bounds__(256) void grad_sum_group_kernel(float* part, int chunks, long n) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const int ngr = (chunks + kSumGroup - 1) / kSumGroup;
  const long o = blockIdx.y / ngr;
  const int g = blockIdx.y % ngr;
  if (idx >= n) return;
  const int c0 = g * kSumGroup, c1 = min(chunks, c0 + kSumGroup);
  float* p = part + (o * chunks + c0) * n + idx;
  const float v = sum_rows(0.f, p, n, c1 - c0);
  *p = v;
}

__global__ __launch_bounds__(256) void grad_sum_kernel(const float* part, int chunks, int step,
                                                       long n, float* out, float scale,
                                                       int accumulate) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long o = blockIdx.y;
  if (idx >= n) return;
  const float v = sum_rows(0.f, part + o * chunks * n + idx, (long)step * n,
                           (chunks + step - 1) / step);
  out[o * n + idx] = accumulate ? out[o * n + idx] + v * scale : v * scale;
}

void launch_grad_sum(float* part, int outer, int chunks, long n, float* out, float scale,
                     int accumulate, hipStream_t s) {
  if (outer <= 0 || n <= 0) return;
  const unsigned bx = (unsigned)((n + 255) / 256);
  int step = 1;
  if (chunks > 2 * kSumGroup) {
    const int ngr = (chunks + kSumGroup - 1) / kSumGroup;
    hipLaunchKernelGGL(grad_sum_group_kernel, dim3(bx, outer * ngr), dim3(256), 0, s, part,
                       chunks, n);
    step = kSumGroup;
  }
  hipLaunchKernelGGL(grad_sum_kernel, dim3(bx, outer), dim3(256), 0, s, (const float*)part,
                     chunks, step, n, out, scale, accumulate);
}

// Per token and branch, with hn[l] = g[l] h[l] / rms(h[l]) recomputed in fp32 from the
// bf16 states H [N][L][D], the branch's gains g [L][D] and rinv [N][L] (as the forward mix
// computes them), the channels' gradient dmix [k][N][D] (fp32) and the final mixing
// weights alpha [N][k][L]:
//   dhn[n][l][e] = sum_j alpha[j][l] dmix[j][e]   (written, fp32): each thread takes whole
//     columns e, holding the k values dmix[.][e] in registers against alpha^T in LDS;
//   dalpha[j][l] = dmix[j] . hn[l]: a k x L product over the D columns on the fp32 matrix
//     cores (32 x 32 x 2 steps, the four waves taking every fourth 16-column step, their
//     partial tiles summed in a fixed order). It stays fp32 because dalpha[j][l] is a
//     small difference when one source dominates a channel (the mid norm's gradient is
//     orthogonal to the mixed channel), which bf16 operands would swamp;
// then the softmax-over-depth backward (or the mask of the sources a channel may not mix)
// gives the router logits' gradient dlog [N][k L]. MAXK >= k (16, 32 or 64).
template <int MAXK>
__global__ __launch_bounds__(256) void grad_mix_kernel(MixGradArgs a) {
  extern __shared__ __align__(16) unsigned char gsm[];
  const int L = a.L, k = a.k, D = a.D;
  const int KP = (k + 3) & ~3;
  const long n = blockIdx.x;
  float* alT = (float*)gsm;        // [L][KP] alpha transposed, zero-padded
  float* al = alT + L * KP;        // [k][L]
  float* da = al + k * L;          // [k][L]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int e = tid; e < L * KP; e += 256) {
    const int l = e / KP, j = e % KP;
    alT[e] = j < k ? a.alpha[(n * k + j) * L + l] : 0.f;
  }
  for (int e = tid; e < k * L; e += 256) al[e] = a.alpha[n * k * L + e];
  __syncthreads();
  // dhn, one column per thread at a time
  for (int c = tid; c < D; c += 256) {
    float dm[MAXK];
#pragma unroll
    for (int j = 0; j < MAXK; ++j) dm[j] = j < k ? a.dmix[((long)j * a.N + n) * D + c] : 0.f;
    float* out = a.dhn + n * L * D + c;
    for (int l = 0; l < L; ++l) {
      const float* ar = alT + l * KP;
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < MAXK; j += 4) {
        if (j < KP) {
          const f32x4 av = *(const f32x4*)(ar + j);
          s += av[0] * dm[j] + av[1] * dm[j + 1] + av[2] * dm[j + 2] + av[3] * dm[j + 3];
        }
      }
      out[(long)l * D] = s;
    }
  }
  // dalpha on the fp32 matrix cores: tile (tj, tl) rows j = 32 tj + .., columns l = 32 tl + ..
  // lane (h, r) supplies columns 16 s + 8 h .. + 7 of row r of both operands
  constexpr int TJ = MAXK > 32 ? 2 : 1;
  const int tj_n = (k + 31) / 32, tl_n = (L + 31) / 32;
  const int h = lane >> 5, r = lane & 31;
  f32x16 acc[TJ][2];
#pragma unroll
  for (int tj = 0; tj < TJ; ++tj)
#pragma unroll
    for (int tl = 0; tl < 2; ++tl) acc[tj][tl] = zero16();
  const float* rinv = a.rinv + n * L;
  for (int st = w; st < D / 16; st += 4) {
    const int c0 = 16 * st + 8 * h;
    f32x8 av[TJ], bv[2];
#pragma unroll
    for (int tj = 0; tj < TJ; ++tj) {
      const int j = 32 * tj + r;
      if (tj < tj_n && j < k) {
        const float* p = a.dmix + ((long)j * a.N + n) * D + c0;
        const f32x4 x = *(const f32x4*)p, y = *(const f32x4*)(p + 4);
        av[tj] = f32x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
      } else {
        av[tj] = f32x8{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int tl = 0; tl < 2; ++tl) {
      const int l = 32 * tl + r;
      if (tl < tl_n && l < L) {
        const bf16x8 hv = *(const bf16x8*)(a.H + (n * L + l) * D + c0);
        const bf16x8 gv = *(const bf16x8*)(a.g + (long)l * D + c0);
        const float ri = rinv[l];
#pragma unroll
        for (int i = 0; i < 8; ++i) bv[tl][i] = (float)gv[i] * (float)hv[i] * ri;
      } else {
        bv[tl] = f32x8{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int tj = 0; tj < TJ; ++tj)
#pragma unroll
      for (int tl = 0; tl < 2; ++tl)
        if (tj < tj_n && tl < tl_n) acc[tj][tl] = mma32(acc[tj][tl], av[tj], bv[tl]);
  }
  // the four waves' partial tiles, added in wave order
  for (int ww = 0; ww < 4; ++ww) {
    if (w == ww) {
#pragma unroll
      for (int tj = 0; tj < TJ; ++tj)
#pragma unroll
        for (int tl = 0; tl < 2; ++tl)
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const int j = 32 * tj + 8 * (q >> 2) + 4 * h + (q & 3), l = 32 * tl + r;
            if (tj < tj_n && tl < tl_n && j < k && l < L)
              da[j * L + l] = ww == 0 ? acc[tj][tl][q] : da[j * L + l] + acc[tj][tl][q];
          }
    }
    __syncthreads();
  }
  // logits' gradient per channel row (fp32, and a bf16 copy padded to kLp for the GEMMs)
  for (int j = tid; j < k; j += 256) {
    const int nl = a.nofeedback ? j + 1 : L;
    float dot = 0.f;
    if (a.softmax)
      for (int l = 0; l < nl; ++l) dot += al[j * L + l] * da[j * L + l];
    for (int l = 0; l < L; ++l) {
      float v = 0.f;
      if (l < nl) v = a.softmax ? al[j * L + l] * (da[j * L + l] - dot) : da[j * L + l];
      a.dlog[n * k * L + j * L + l] = v;
      a.dlogb[n * a.kLp + j * L + l] = (bf16)v;
    }
  }
  for (int e = k * L + tid; e < a.kLp; e += 256) a.dlogb[n * a.kLp + e] = (bf16)0.f;
}

size_t grad_mix_smem(int L, int k, int D) {
  (void)D;
  return ((size_t)L * ((k + 3) & ~3) + (size_t)2 * k * L) * 4;
}

void launch_grad_mix(const MixGradArgs& a, hipStream_t s) {
  if (a.N <= 0) return;
  const dim3 grid((unsigned)a.N), blk(256);
  const size_t sm = grad_mix_smem(a.L, a.k, a.D);
  if (a.k <= 16) hipLaunchKernelGGL(grad_mix_kernel<16>, grid, blk, sm, s, a);
  else if (a.k <= 32) hipLaunchKernelGGL(grad_mix_kernel<32>, grid, blk, sm, s, a);
  else hipLaunchKernelGGL(grad_mix_kernel<64>, grid, blk, sm, s, a);
}

// dst[j][b T + i][h d + e] = src[j][b][h][ctx_len[b] + gq + gs i][e]: the call's slots' rows
// of a cache-layout gradient, token-major for the projection GEMMs.
__global__ __launch_bounds__(256) void grad_gather_kernel(const float* src, int k, int B, int H,
                                                          int T, int S_cap, int d,
                                                          const int32_t* ctx_len, int ctx_hi,
                                                          int gs, int gq, bf16* dst) {
  // four consecutive elements per thread (d is a multiple of 4); the group count fits 31 bits
  const unsigned n4 = (unsigned)((long)k * B * T * H * d / 4);
  const unsigned idx = blockIdx.x * 256u + threadIdx.x;
  if (idx >= n4) return;
  const unsigned d4 = (unsigned)d / 4, e = 4 * (idx % d4), hh = idx / d4 % (unsigned)H;
  const unsigned t = idx / (d4 * (unsigned)H);  // (j, b, i)
  const unsigned i = t % (unsigned)T, b = t / (unsigned)T % (unsigned)B, j = t / ((unsigned)T * B);
  const int slot = ctx_at(ctx_len, (int)b, ctx_hi) + gq + gs * (int)i;
  const f32x4 v = *(const f32x4*)(src + ((((long)j * B + b) * H + hh) * S_cap + slot) * d + e);
  bf16x4 o;
#pragma unroll
  for (int u = 0; u < 4; ++u) o[u] = (bf16)v[u];
  *(bf16x4*)(dst + (long)idx * 4) = o;
}

void launch_grad_gather(const float* src, int k, int B, int H, int T, int S_cap, int d,
                        const int32_t* ctx_len, int ctx_hi, int gs, int gq, bf16* dst,
                        hipStream_t s) {
  const long n4 = (long)k * B * T * H * d / 4;
  if (n4 <= 0) return;
  hipLaunchKernelGGL(grad_gather_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s,
                     src, k, B, H, T, S_cap, d, ctx_len, ctx_hi, gs, gq, dst);
}

// part[c][o] = sum over rows r in chunk c of x[r][o] (x [rows][n]); chunks = gridDim.y.
__global__ __launch_bounds__(256) void grad_colsum_kernel(const float* x, long rows, int n,
                                                          float* part) {
  const int o = blockIdx.x * 256 + threadIdx.x, c = blockIdx.y, nc = gridDim.y;
  if (o >= n) return;
  const long r0 = rows * c / nc, r1 = rows * (c + 1) / nc;
  float v = 0.f;
  for (long r = r0; r < r1; ++r) v += x[r * n + o];
  part[(long)c * n + o] = v;
}

void launch_grad_colsum(const float* x, long rows, int n, int chunks, float* part, hipStream_t s) {
  if (n <= 0) return;
  hipLaunchKernelGGL(grad_colsum_kernel, dim3((n + 255) / 256, chunks), dim3(256), 0, s, x, rows,
                     n, part);
}

// ------------------------------------------------- small elementwise helpers
__global__ __launch_bounds__(256) void grad_fill_kernel(float* p, long n, float v) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}
void launch_grad_fill(float* p, long n, float v, hipStream_t s) {
  if (n > 0)
    hipLaunchKernelGGL(grad_fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n,
                       v);
}

__global__ __launch_bounds__(256) void grad_cast_kernel(const float* src, bf16* dst, long n) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = (bf16)src[i];
}
void launch_grad_cast(const float* src, bf16* dst, long n, hipStream_t s) {
  if (n > 0)
    hipLaunchKernelGGL(grad_cast_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src,
                       dst, n);
}

// dst[r * dst_stride + e] += sum over l < nsrc of src[r * src_stride + l * D + e] (rows of D)
__global__ __launch_bounds__(256) void grad_add_rows_kernel(float* dst, long dst_stride,
                                                            const float* src, long rows, int D,
                                                            long src_stride, int nsrc) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * D) return;
  const long r = i / D;
  const int e = (int)(i % D);
  float v = 0.f;
  for (int l = 0; l < nsrc; ++l) v += src[r * src_stride + (long)l * D + e];
  dst[r * dst_stride + e] += v;
}
void launch_grad_add_rows(float* dst, long dst_stride, const float* src, long rows, int D,
                          long src_stride, int nsrc, hipStream_t s) {
  const long n = rows * D;
  if (n > 0)
    hipLaunchKernelGGL(grad_add_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       dst, dst_stride, src, rows, D, src_stride, nsrc);
}

// The slots q + g i (i < Tg) of every row of S_cap slots of the caches K and V, copied to
// (restore = 0) or back from (restore = 1) compact [rows][Tg][d] arrays, 8 elements a
// thread; on the way back the slots' fp32 gradients dK, dV are cleared when given.
__global__ __launch_bounds__(256) void grad_slots_kernel(bf16* K, bf16* V, bf16* Kg, bf16* Vg,
                                                         float* dK, float* dV, long rows, int Tg,
                                                         int g, int q, int S_cap, int d,
                                                         int restore) {
  const int dv = d / 8;
  const long n = (long)blockIdx.x * 256 + threadIdx.x;
  if (n >= rows * Tg * dv) return;
  const long ri = n / dv;  // r Tg + i
  const int v = (int)(n - ri * dv), i = (int)(ri % Tg);
  const long r = ri / Tg;
  const long full = (r * S_cap + q + (long)g * i) * d + 8 * v, comp = ri * d + 8 * v;
  if (!restore) {
    *(uint4*)(Kg + comp) = *(const uint4*)(K + full);
    *(uint4*)(Vg + comp) = *(const uint4*)(V + full);
    return;
  }
  *(uint4*)(K + full) = *(const uint4*)(Kg + comp);
  *(uint4*)(V + full) = *(const uint4*)(Vg + comp);
  if (dK) {
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    *(float4*)(dK + full) = z;
    *(float4*)(dK + full + 4) = z;
    *(float4*)(dV + full) = z;
    *(float4*)(dV + full + 4) = z;
  }
}
void launch_grad_slots(bf16* K, bf16* V, bf16* Kg, bf16* Vg, float* dK, float* dV, long rows,
                       int Tg, int g, int q, int S_cap, int d, bool restore, hipStream_t s) {
  const long n = rows * Tg * (d / 8);
  if (n > 0)
    hipLaunchKernelGGL(grad_slots_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, K,
                       V, Kg, Vg, dK, dV, rows, Tg, g, q, S_cap, d, restore ? 1 : 0);
}

// dst[r][e] = src[r * src_stride + e] (bf16 rows of D)
__global__ __launch_bounds__(256) void grad_copy_rows_kernel(const bf16* src, long src_stride,
                                                             bf16* dst, long rows, int D) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * D) return;
  dst[i] = src[(i / D) * src_stride + i % D];
}
void launch_grad_copy_rows(const bf16* src, long src_stride, bf16* dst, long rows, int D,
                           hipStream_t s) {
  const long n = rows * D;
  if (n > 0)
    hipLaunchKernelGGL(grad_copy_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       src, src_stride, dst, rows, D);
}

// Zeroes the router weight entries (o, m) whose source layer sel[m] lies above channel
// o / L (the no-feedback ablation's mask): W [kL][Lp D] rows, in place (bf16 or fp32).
template <typename T>
__global__ __launch_bounds__(256) void grad_mask_kernel(T* W, int kL, int L, int Lp, int D,
                                                        LayerTable sel) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long n = (long)kL * Lp * D;
  if (idx >= n) return;
  const int o = (int)(idx / ((long)Lp * D)), m = (int)(idx / D % Lp);
  if (sel.v[m] > o / L) W[idx] = (T)0.f;
}

template <typename T>
void launch_grad_mask(T* W, int kL, int L, int Lp, int D, const LayerTable& sel, hipStream_t s) {
  const long n = (long)kL * Lp * D;
  if (n <= 0) return;
  hipLaunchKernelGGL(grad_mask_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, W,
                     kL, L, Lp, D, sel);
}
template void launch_grad_mask<bf16>(bf16*, int, int, int, int, const LayerTable&, hipStream_t);
template void launch_grad_mask<float>(float*, int, int, int, int, const LayerTable&, hipStream_t);

}  // namespace wm
