// Grouped "NT" GEMM on the matrix cores: C_g[m][o] = sum_k A_g[m][k] * W_g[o][k].
// Both operands are K-contiguous (activations row-major, weights [out][in]),
// which is how the router, the per-channel K/V projections and the per-layer
// Q projections store them. blockIdx.z selects the group g.
//
// The A operand is produced on the fly by an ALoad functor (it applies the
// RMSNorm gain and row scale and rounds once to the operand type), the B
// operand is copied from the weights, and an Epi functor consumes the fp32
// C tile from LDS (bias, per-head norm, RoPE, cache store ...).
//
// Tile: 128 x 128 x 32, 256 threads = 4 waves in a 2 x 2 grid, each wave
// owning 64 x 64 = 2 x 2 MFMA 32x32 tiles. The next K slice is fetched into
// registers while the current one is multiplied.
#pragma once
#include "wm_device.hpp"

namespace wm {

template <typename T> struct GemmCfg {
  static constexpr int BM = 128, BN = 128, BK = 32;
  static constexpr int PAD = sizeof(T) == 2 ? 8 : 4;  // keeps 16-B row alignment
  static constexpr int LDA = BK + PAD;                 // LDS row stride (elements)
  static constexpr int LDC = BN + 4;                   // fp32 C tile row stride
  static constexpr int AB_BYTES = 2 * BM * LDA * (int)sizeof(T);
  static constexpr int C_BYTES = BM * LDC * 4;
  static constexpr int SMEM = AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES;
};

// ALoad: void operator()(int g, int row, int k, float* out16) const   (16 elements)
// BLoad: const T* operator()(int g, int o) const  -> row o of W_g (nullptr if o >= Nout)
// Epi:   void operator()(int g, int m0, int n0, const float* C, int ldc, int tid) const
template <typename T, class ALoad, class BLoad, class Epi>
__global__ __launch_bounds__(256) void gemm_nt_kernel(int M, int Nout, int K, ALoad aload,
                                                      BLoad bload, Epi epi) {
  using C = GemmCfg<T>;
  __shared__ __align__(16) unsigned char smem[C::SMEM];
  T* As = (T*)smem;
  T* Bs = As + C::BM * C::LDA;
  float* Cs = (float*)smem;

  const int g = blockIdx.z;
  const int m0 = blockIdx.y * C::BM, n0 = blockIdx.x * C::BN;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 1, wn = w & 1, h = lane >> 5, r = lane & 31;

  // each thread moves 16 consecutive k-elements of one A row and one B row
  const int lrow = tid >> 1, lk = (tid & 1) * 16;
  const bool arow_ok = m0 + lrow < M;
  const T* brow = bload(g, n0 + lrow);

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = zero16();

  float av[16];
  frag_t<T> bv0, bv1;
  auto fetch = [&](int k0) {
    if (arow_ok) {
      aload(g, m0 + lrow, k0 + lk, av);
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) av[i] = 0.f;
    }
    if (brow) {
      bv0 = ld_frag<T>(brow + k0 + lk);
      bv1 = ld_frag<T>(brow + k0 + lk + 8);
    } else {
      bv0 = zero_frag<T>();
      bv1 = zero_frag<T>();
    }
  };

  fetch(0);
  for (int k0 = 0; k0 < K; k0 += C::BK) {
    __syncthreads();
    {
      frag_t<T> a0, a1;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        a0[i] = from_f32<T>(av[i]);
        a1[i] = from_f32<T>(av[8 + i]);
      }
      st_frag<T>(As + lrow * C::LDA + lk, a0);
      st_frag<T>(As + lrow * C::LDA + lk + 8, a1);
      st_frag<T>(Bs + lrow * C::LDA + lk, bv0);
      st_frag<T>(Bs + lrow * C::LDA + lk + 8, bv1);
    }
    __syncthreads();
    if (k0 + C::BK < K) fetch(k0 + C::BK);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      frag_t<T> a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = ld_frag<T>(As + (64 * wm + 32 * i + r) * C::LDA + 16 * ks + 8 * h);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = ld_frag<T>(Bs + (64 * wn + 32 * j + r) * C::LDA + 16 * ks + 8 * h);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mma32(acc[i][j], a[i], b[j]);
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        int row = 64 * wm + 32 * i + 8 * (q >> 2) + 4 * h + (q & 3);
        int col = 64 * wn + 32 * j + r;
        Cs[row * C::LDC + col] = acc[i][j][q];
      }
  __syncthreads();
  epi(g, m0, n0, Cs, C::LDC, tid);
}

}  // namespace wm
