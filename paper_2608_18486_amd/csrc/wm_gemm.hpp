// Grouped "NT" GEMM on the matrix cores: C_g[m][o] = sum_k A_g[m][k] * W_g[o][k].
// Both operands are K-contiguous (activations row-major, weights [out][in]),
// which is how the router, the per-channel K/V projections and the per-layer
// Q projections store them. blockIdx.z selects the group g.
//
// An ALoad functor produces the A operand fragments (a plain copy, or the
// router's normed states), a BLoad functor points at weight rows, and an Epi
// functor consumes the fp32 C tile from LDS (bias, row scale, per-head norm,
// RoPE, cache store ...).
//
// K must be a multiple of 32; a last half slice (bf16) is zero-filled.
// Tile 128 x 128 x BK (BK = 64 for bf16, 32 for fp32), 256 threads = 4 waves
// in a 2 x 2 grid, each wave owning 64 x 64 = 2 x 2 MFMA 32x32 tiles. LDS is
// double-buffered: the next K slice is fetched into registers while the
// current one is multiplied, then stored to the other buffer, with one
// barrier per K slice. A ring of PIPE register stages keeps the global loads of
// later slices in flight while the current one is multiplied.
#pragma once
#include "wm_device.hpp"

namespace wm {

// A group's weight matrix [Nout][K] seen through a buffer resource.
template <typename T> struct WeightView {
  __amdgpu_buffer_rsrc_t rsrc;
};

template <typename T> struct GemmCfg {
  static constexpr int BM = 128, BN = 128;
  static constexpr int BK = sizeof(T) == 2 ? 64 : 32;
  static constexpr int PAD = sizeof(T) == 2 ? 8 : 4;  // keeps 16-B row alignment
  static constexpr int LDA = BK + PAD;                 // LDS row stride (elements)
  static constexpr int LDC = BN + 4;                   // fp32 C tile row stride
  static constexpr int FR = BM * BK / 8 / 256;         // operand fragments per thread per slice
  static constexpr int TPR = BK / (8 * FR);            // threads per tile row
  static constexpr int STAGE = 2 * BM * LDA;           // elements per stage (A and B)
  static constexpr int AB_BYTES = 2 * STAGE * (int)sizeof(T);
  static constexpr int C_BYTES = BM * LDC * 4;
  static constexpr int SMEM = AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES;
  static constexpr int PIPE = 3;                       // K slices held in registers
};

// ALoad: State begin(int g) const;
//        void load(const State&, int row, int k, bool ok, frag_t<T>* out) const
//          (FR consecutive frags of row `row` from column k; zeros when !ok)
// BLoad: WeightView<T> view(int g) const  -> the group's [Nout][K] weights
// Epi:   void operator()(int g, int m0, int n0, const float* C, int ldc, int tid) const
// Launched on a 1-D grid of groups x row tiles x column tiles blocks; the tile
// order is (group, row tile, column tile) and is spread over the XCDs so the
// column tiles of a row block share one L2.
template <typename T, class ALoad, class BLoad, class Epi>
__global__ __launch_bounds__(256) void gemm_nt_kernel(int M, int Nout, int K, int groups,
                                                      ALoad aload, BLoad bload, Epi epi) {
  using C = GemmCfg<T>;
  __shared__ __align__(16) unsigned char smem[C::SMEM];
  T* stage0 = (T*)smem;
  float* Cs = (float*)smem;

  const int nt = (Nout + C::BN - 1) / C::BN, mt = (M + C::BM - 1) / C::BM;
  const int tile = xcd_tile(blockIdx.x, groups * mt * nt);
  const int g = tile / (mt * nt);
  const int m0 = (tile / nt % mt) * C::BM, n0 = (tile % nt) * C::BN;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 1, wn = w & 1, h = lane >> 5, r = lane & 31;

  // each thread moves FR consecutive fragments of one A row and one B row per slice
  const int lrow = tid / C::TPR, lk = (tid % C::TPR) * 8 * C::FR;
  const bool arow_ok = m0 + lrow < M;
  const auto ast = aload.begin(g);
  const auto wv = bload.view(g);
  const bool brow_ok = n0 + lrow < Nout;
  const uint32_t brow_off = (uint32_t)((n0 + lrow) * K) * (uint32_t)sizeof(T);

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = zero16();

  // K slices in flight: slice kb + P is fetched while slice kb is multiplied, so each
  // slice's global loads have P - 1 slices of matrix-core work to land.
  constexpr int P = C::PIPE;
  frag_t<T> av[P][C::FR], bv[P][C::FR];
  auto fetch = [&](int k0, frag_t<T>* a_out, frag_t<T>* b_out) {
    const bool kin = k0 + lk < K;  // the thread's chunk lies wholly inside or outside K
    aload.load(ast, m0 + lrow, k0 + lk, arow_ok && kin, a_out);
    const uint32_t off = brow_ok && kin ? brow_off + (uint32_t)(k0 + lk) * sizeof(T) : kOffOob;
#pragma unroll
    for (int i = 0; i < C::FR; ++i) b_out[i] = buf_frag<T>(wv.rsrc, off + 8 * i * sizeof(T));
  };
  auto stage = [&](int buf, const frag_t<T>* a_in, const frag_t<T>* b_in) {
    T* As = stage0 + buf * C::STAGE;
    T* Bs = As + C::BM * C::LDA;
#pragma unroll
    for (int i = 0; i < C::FR; ++i) {
      st_frag<T>(As + lrow * C::LDA + lk + 8 * i, a_in[i]);
      st_frag<T>(Bs + lrow * C::LDA + lk + 8 * i, b_in[i]);
    }
  };
  auto compute = [&](int buf) {
    const T* As = stage0 + buf * C::STAGE;
    const T* Bs = As + C::BM * C::LDA;
#pragma unroll
    for (int ks = 0; ks < C::BK / 16; ++ks) {
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
  };

  // The slice count is padded to a multiple of P; padded slices read zeros through the
  // out-of-range offset, so the loop body has no branch and every load's wait count
  // stays exact.
  const int nk = (K + C::BK - 1) / C::BK;
  const int nkp = (nk + P - 1) / P * P;
#pragma unroll
  for (int u = 0; u < P; ++u) fetch(u * C::BK, av[u], bv[u]);
  stage(0, av[0], bv[0]);
  __syncthreads();
  for (int kb0 = 0; kb0 < nkp; kb0 += P) {
#pragma unroll
    for (int u = 0; u < P; ++u) {
      const int kb = kb0 + u;  // slot u held slice kb, already staged into buffer kb & 1
      fetch((kb + P) * C::BK, av[u], bv[u]);
      compute(kb & 1);
      stage((kb + 1) & 1, av[(u + 1) % P], bv[(u + 1) % P]);
      __syncthreads();
    }
  }
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
