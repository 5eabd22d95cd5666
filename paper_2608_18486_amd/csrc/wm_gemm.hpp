// Grouped projection GEMM on the matrix cores, computed transposed:
//   C_g^T[o][n] = sum_k W_g[o][k] * X_g[n][k]
// W_g is a group's weight matrix [Nout][K] and X_g its activations (one row of
// K per token), both K-contiguous. Computing C^T puts one token in each lane of
// an MFMA result: lane (h, r) of a 32x32 block holds token r and output channels
// 8*(q/4) + 4h + q%4, q = 0..15. A head of d channels therefore lives in one
// token's lane pair (h = 0, 1): its RMS norm needs a single cross-half swap,
// the rotate-half RoPE pairs (m, m + d/2) sit in the same lane, and 4
// consecutive channels leave as one vector store. The epilogue runs on the
// accumulators in registers; there is no C tile in LDS.
//
// Macro tile OT x NTOK (channels x tokens) = (32 WO WGO) x (32 WN WGN) with
// WGO x WGN waves, each owning WO x WN blocks of 32 x 32. Per K slice of BK the
// W and X tiles are fetched into registers PIPE slices ahead (buffer loads:
// rows past the matrix and padded slices read zeros, so the loop has no
// divergent branch and keeps exact wait counts), stored to the other half of a
// double-buffered LDS stage, and multiplied with one barrier per slice.
#pragma once
#include <type_traits>

#include "wm_device.hpp"

namespace wm {

// LDS an epilogue may use once the main loop is done (one with kUsesLds set, in the
// LDS-staged kernel): 32 x 32 WO elements of T per wave, at p + wave * that.
struct EpiLds {
  char* p;   // the block's LDS (free once the K loop is done)
  int wave;  // this wave's index in the block
  int n0;    // the block's first token
};

// Epilogues with kTabLds copy the block's rows of a per-token table into LDS before
// finish() (stage_tab, all threads, then a barrier), so the waves that share tokens read
// it there instead of each reading it from memory.
template <class Epi, class = void> struct TabLds { static constexpr bool value = false; };
template <class Epi>
struct TabLds<Epi, std::void_t<decltype(Epi::kTabLds)>> {
  static constexpr bool value = Epi::kTabLds;
};

template <typename T, int BK_, int WGO_, int WGN_, int WO_, int WN_> struct ProjCfg {
  static constexpr int BK = BK_, WGO = WGO_, WGN = WGN_, WO = WO_, WN = WN_;
  static constexpr int NT = 64 * WGO * WGN;                 // threads
  static constexpr int OT = 32 * WO * WGO, NTOK = 32 * WN * WGN;
  // bf16 with BK = 32: 64-B LDS rows whose four 16-B chunks are XOR-swizzled (chunk c of
  // row r at c ^ swz(r)), so that a fragment read -- 16 lanes reading one chunk of 16
  // consecutive rows, served 256 B per LDS cycle -- hits 16 distinct 16-B bank groups;
  // the same holds 8 rows at a time at 128 B per cycle. Otherwise rows are padded.
  static constexpr bool SWZ = sizeof(T) == 2 && BK == 32;
  static constexpr int PAD = SWZ ? 0 : sizeof(T) == 2 ? 8 : 4;  // keeps 16-B row alignment
  static constexpr int LDA = BK + PAD;                       // LDS row stride (elements)
  static constexpr int CPR = BK / 8;                         // fragments per tile row
  __device__ static int swz(int row) { return ((row >> 1) ^ (row >> 3)) & 3; }
  // element offset of 8-element chunk ch of tile row row
  __device__ static int chunk_at(int row, int ch) {
    return row * LDA + 8 * (SWZ ? ch ^ swz(row) : ch);
  }
  static constexpr int FW = (OT * CPR + NT - 1) / NT;        // W fragments per thread
  static constexpr int FX = (NTOK * CPR + NT - 1) / NT;      // X fragments per thread
  static constexpr int STAGE = (OT + NTOK) * LDA;            // elements per LDS stage
#ifndef WM_PROJ_PIPE
#define WM_PROJ_PIPE 2
#endif
  static constexpr int PIPE = WM_PROJ_PIPE;                  // K slices held in registers
  static_assert(BK % 16 == 0, "K slices hold whole k16 steps");
};

// A group's row-major matrix seen through a buffer resource: rows of row_bytes;
// the loader's slice(k0) gives the byte offset of column k0 within a row.
struct RowsView {
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t row_bytes;
};

// XLoad / WLoad: RowsView view(int g) const; uint32_t slice(int k0) const
//   (activations [M][..] and weights [Nout][..]; slice() is uniform over the block)
// kspan: 0, or the K range of each group for split K: group g then covers
//   columns [g kspan, min(K, (g+1) kspan)) of one shared matrix pair.
// Epi:   struct State;
//        template <class C> void begin(int g, int nw0, int lane, State&) const
//        template <class C> void segment(int g, int seg, int nw0,
//                                        f32x16 (&acc)[C::WO][C::WN], int lane, State&) const
//          (entering K segment seg, i.e. slice seg * seg_len; the router rescales there)
//        template <class C> void finish(int g, int ow0, int nw0,
//                                       f32x16 (&acc)[C::WO][C::WN], int lane, State&) const
//          (ow0 / nw0: the wave's first channel / token)
// Launched on a 1-D grid of groups x token tiles x channel tiles; the tile order
// (group, token tile, channel tile) is spread over the XCDs so the channel tiles
// of a token block share one L2.
template <class C, typename T, class XLoad, class WLoad, class Epi>
__global__ __launch_bounds__(C::NT) void proj_gemm_kernel(int M, int Nout, int K, int groups,
                                                          int seg_len, int kspan, XLoad xl,
                                                          WLoad wl, Epi epi) {
  __shared__ __align__(16) T smem[2 * C::STAGE];

  const int ot = (Nout + C::OT - 1) / C::OT, mt = (M + C::NTOK - 1) / C::NTOK;
  const int tile = xcd_tile(blockIdx.x, groups * mt * ot);
  const int g = tile / (mt * ot);
  const int n0 = (tile / ot % mt) * C::NTOK, o0 = (tile % ot) * C::OT;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wo = w % C::WGO, wn = w / C::WGO;
  const int h = lane >> 5, r = lane & 31;

  const RowsView xv = xl.view(g), wv = wl.view(g);
  // fragment f of this thread: tile row idx / CPR, 8-element chunk idx % CPR
  uint32_t xoff[C::FX], woff[C::FW];
#pragma unroll
  for (int f = 0; f < C::FX; ++f) {
    const int idx = tid + f * C::NT, row = idx / C::CPR, ch = idx % C::CPR;
    const bool ok = idx < C::NTOK * C::CPR && n0 + row < M;
    xoff[f] = ok ? (uint32_t)(n0 + row) * xv.row_bytes + ch * 8 * (uint32_t)sizeof(T) : kOffOob;
  }
#pragma unroll
  for (int f = 0; f < C::FW; ++f) {
    const int idx = tid + f * C::NT, row = idx / C::CPR, ch = idx % C::CPR;
    const bool ok = idx < C::OT * C::CPR && o0 + row < Nout;
    woff[f] = ok ? (uint32_t)(o0 + row) * wv.row_bytes + ch * 8 * (uint32_t)sizeof(T) : kOffOob;
  }

  f32x16 acc[C::WO][C::WN];
#pragma unroll
  for (int i = 0; i < C::WO; ++i)
#pragma unroll
    for (int j = 0; j < C::WN; ++j) acc[i][j] = zero16();

  constexpr int P = C::PIPE;
  frag_t<T> xr[P][C::FX], wr[P][C::FW];
  // Rows past the matrix keep the out-of-range offset whatever the slice adds
  // (every view spans less than 2 GiB).
  const int kbeg = kspan > 0 ? g * kspan : 0;
  const int kend = kspan > 0 ? min(K, kbeg + kspan) : K;
  auto fetch = [&](int k0, frag_t<T>* x_out, frag_t<T>* w_out) {
    const bool kin = k0 < kend;
    const uint32_t xs = kin ? xl.slice(k0) : 0u, ws = kin ? wl.slice(k0) : 0u;
#pragma unroll
    for (int f = 0; f < C::FX; ++f) x_out[f] = buf_frag<T>(xv.rsrc, kin ? xoff[f] + xs : kOffOob);
#pragma unroll
    for (int f = 0; f < C::FW; ++f) w_out[f] = buf_frag<T>(wv.rsrc, kin ? woff[f] + ws : kOffOob);
  };
  auto stage = [&](int buf, const frag_t<T>* x_in, const frag_t<T>* w_in) {
    T* Ws = smem + buf * C::STAGE;
    T* Xs = Ws + C::OT * C::LDA;
#pragma unroll
    for (int f = 0; f < C::FX; ++f) {
      const int idx = tid + f * C::NT;
      if (C::NTOK * C::CPR % C::NT == 0 || idx < C::NTOK * C::CPR)
        st_frag<T>(Xs + C::chunk_at(idx / C::CPR, idx % C::CPR), x_in[f]);
    }
#pragma unroll
    for (int f = 0; f < C::FW; ++f) {
      const int idx = tid + f * C::NT;
      if (C::OT * C::CPR % C::NT == 0 || idx < C::OT * C::CPR)
        st_frag<T>(Ws + C::chunk_at(idx / C::CPR, idx % C::CPR), w_in[f]);
    }
  };
  auto compute = [&](int buf) {
    const T* Ws = smem + buf * C::STAGE;
    const T* Xs = Ws + C::OT * C::LDA;
#pragma unroll
    for (int ks = 0; ks < C::BK / 16; ++ks) {
      frag_t<T> a[C::WO], b[C::WN];
#pragma unroll
      for (int i = 0; i < C::WO; ++i)
        a[i] = ld_frag<T>(Ws + C::chunk_at(32 * (wo * C::WO + i) + r, 2 * ks + h));
#pragma unroll
      for (int j = 0; j < C::WN; ++j)
        b[j] = ld_frag<T>(Xs + C::chunk_at(32 * (wn * C::WN + j) + r, 2 * ks + h));
#pragma unroll
      for (int i = 0; i < C::WO; ++i)
#pragma unroll
        for (int j = 0; j < C::WN; ++j) acc[i][j] = mma32(acc[i][j], a[i], b[j]);
    }
  };

  const int ow0 = o0 + 32 * C::WO * wo, nw0 = n0 + 32 * C::WN * wn;
  typename Epi::State est;
  epi.template begin<C>(g, nw0, lane, est);

  // The slice count is padded to a multiple of P; padded slices read zeros through the
  // out-of-range offset, so the loop body has no divergent branch.
  // Slices are counted from kbeg (a multiple of BK); kb below is the absolute slice.
  const int kb_beg = kbeg / C::BK, kb_end = (kend + C::BK - 1) / C::BK;
  const int nkp = (kb_end - kb_beg + P - 1) / P * P;
#pragma unroll
  for (int u = 0; u < P; ++u) fetch((kb_beg + u) * C::BK, xr[u], wr[u]);
  stage(0, xr[0], wr[0]);
  __syncthreads();
  for (int i0 = 0; i0 < nkp; i0 += P) {
#pragma unroll
    for (int u = 0; u < P; ++u) {
      const int i = i0 + u, kb = kb_beg + i;  // slot u held slice kb, staged into buffer i & 1
      fetch((kb + P) * C::BK, xr[u], wr[u]);
      compute(i & 1);
      if ((kb + 1) % seg_len == 0 && kb + 1 < kb_end)
        epi.template segment<C>(g, (kb + 1) / seg_len, nw0, acc, lane, est);
      stage((i + 1) & 1, xr[(u + 1) % P], wr[(u + 1) % P]);
      __syncthreads();
    }
  }
  if constexpr (TabLds<Epi>::value) {  // the loop ended at a barrier: the stages are free
    static_assert(Epi::template tab_end<C>() <= sizeof(smem), "the table fits the stages");
    epi.template stage_tab<C>(g, n0, (char*)smem, tid);
    __syncthreads();
  }
  epi.template finish<C>(g, ow0, nw0, acc, lane, est, EpiLds{(char*)smem, w, n0});
}

// bf16 variant whose K slices travel straight from memory into LDS
// (buffer_load ... lds: each wave instruction fills 1 KB of LDS, lane l's 16 bytes
// at 16 l), so nothing is staged in registers and the prefetch runs two slices
// ahead through three LDS stages. A stage holds the W and X tiles as 64-byte rows
// in the swizzled chunk order of ProjCfg::chunk_at; a lane of the instruction that
// fills rows R .. R+15 fetches row R + l/4, logical chunk (l%4) ^ swizzle, so the
// copy lands already swizzled. Loads past the matrix or past K read zeros.
// The loads are issued from inline asm and waited for with an explicit vmcnt:
// the compiler, seeing LDS DMA in flight, would otherwise wait for every
// outstanding load (the prefetched slices too) before each barrier.
template <class C> struct DmaCfg {
  static constexpr int NS = 3;                              // LDS stages
  static constexpr int ROWS = C::OT + C::NTOK;              // tile rows per stage
  static constexpr int NW = C::NT / 64;
  static constexpr int NI = (ROWS / 16 + NW - 1) / NW;      // 16-row instructions per wave
  // Every wave issues exactly NI loads per slice (so one vmcnt fits all waves); blocks
  // past the tile rows load zeros into padding rows that are never read.
  static constexpr int ROWS_PAD = 16 * NW * NI;
  static constexpr int STAGE_BYTES = ROWS_PAD * 64;
  static_assert(C::SWZ && C::LDA == 32, "64-byte swizzled rows");
  static_assert(C::OT % 16 == 0 && C::NTOK % 16 == 0, "16-row instruction blocks");
  static_assert(NI <= 15, "vmcnt encodes at most 15 here");
};

template <class C, typename T, class XLoad, class WLoad, class Epi>
__global__ __launch_bounds__(C::NT) void proj_gemm_dma_kernel(int M, int Nout, int K, int groups,
                                                              int seg_len, int kspan, XLoad xl,
                                                              WLoad wl, Epi epi) {
  using D = DmaCfg<C>;
  __shared__ __align__(16) T smem[D::NS * D::ROWS_PAD * 32];

  const int ot = (Nout + C::OT - 1) / C::OT, mt = (M + C::NTOK - 1) / C::NTOK;
  const int tile = xcd_tile(blockIdx.x, groups * mt * ot);
  const int g = tile / (mt * ot);
  const int n0 = (tile / ot % mt) * C::NTOK, o0 = (tile % ot) * C::OT;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, held in an SGPR
  const int wo = w % C::WGO, wn = w / C::WGO;
  const int h = lane >> 5, r = lane & 31;

  const RowsView xv = xl.view(g), wv = wl.view(g);
  const int kbeg = kspan > 0 ? g * kspan : 0;
  const int kend = kspan > 0 ? min(K, kbeg + kspan) : K;

  // this lane's row offset (k = 0) and chunk for each of the wave's instructions;
  // rows 0 .. OT-1 of a stage are W rows, the rest X rows
  uint32_t roff[D::NI];
#pragma unroll
  for (int i = 0; i < D::NI; ++i) {
    const int blk = w * D::NI + i, row = 16 * blk + lane / 4;
    const int c = (lane & 3) ^ C::swz(row);
    bool ok;
    uint32_t off;
    if (row < C::OT) {
      ok = o0 + row < Nout;
      off = (uint32_t)(o0 + row) * wv.row_bytes;
    } else {
      ok = n0 + (row - C::OT) < M;
      off = (uint32_t)(n0 + row - C::OT) * xv.row_bytes;
    }
    ok = ok && blk < D::ROWS / 16;
    roff[i] = ok ? off + 16u * c : kOffOob;
  }
  const uint32_t smem_base = (uint32_t)(uintptr_t)smem;
  auto issue = [&](int kb, int stage) {  // slice kb into LDS stage `stage`
    const int k0 = kb * C::BK;
    const bool kin = k0 < kend;
    const uint32_t xs = kin ? xl.slice(k0) : 0u, ws = kin ? wl.slice(k0) : 0u;
#pragma unroll
    for (int i = 0; i < D::NI; ++i) {
      const int blk = w * D::NI + i;  // wave-uniform
      const bool wrow = 16 * blk < C::OT;
      const uint32_t lds = __builtin_amdgcn_readfirstlane(smem_base + stage * D::STAGE_BYTES +
                                                          blk * 1024);
      const uint32_t off = kin && roff[i] != kOffOob ? roff[i] + (wrow ? ws : xs) : kOffOob;
      lds_dma16(lds, off, wrow ? wv.rsrc : xv.rsrc);
    }
  };

  f32x16 acc[C::WO][C::WN];
#pragma unroll
  for (int i = 0; i < C::WO; ++i)
#pragma unroll
    for (int j = 0; j < C::WN; ++j) acc[i][j] = zero16();

  auto compute = [&](int stage) {
    const T* Ws = smem + stage * D::ROWS_PAD * 32;
    const T* Xs = Ws + C::OT * 32;
#pragma unroll
    for (int ks = 0; ks < C::BK / 16; ++ks) {
      frag_t<T> a[C::WO], b[C::WN];
#pragma unroll
      for (int i = 0; i < C::WO; ++i)
        a[i] = ld_frag<T>(Ws + C::chunk_at(32 * (wo * C::WO + i) + r, 2 * ks + h));
#pragma unroll
      for (int j = 0; j < C::WN; ++j)
        b[j] = ld_frag<T>(Xs + C::chunk_at(32 * (wn * C::WN + j) + r, 2 * ks + h));
#pragma unroll
      for (int i = 0; i < C::WO; ++i)
#pragma unroll
        for (int j = 0; j < C::WN; ++j) acc[i][j] = mma32(acc[i][j], a[i], b[j]);
    }
  };

  const int ow0 = o0 + 32 * C::WO * wo, nw0 = n0 + 32 * C::WN * wn;
  typename Epi::State est;
  epi.template begin<C>(g, nw0, lane, est);

  const int kb_beg = kbeg / C::BK, kb_end = (kend + C::BK - 1) / C::BK;
  issue(kb_beg, 0);
  issue(kb_beg + 1, 1);
  for (int kb = kb_beg, st = 0; kb < kb_end; ++kb, st = st == D::NS - 1 ? 0 : st + 1) {
    // this wave's loads of slice kb are done once only the next slice's remain
    wait_vmcnt<D::NI>();
    __syncthreads();  // every wave's slice kb is in LDS, and slice kb-1 is consumed
    issue(kb + 2, st == 0 ? 2 : st - 1);  // into the stage slice kb-1 used
    compute(st);
    if ((kb + 1) % seg_len == 0 && kb + 1 < kb_end)
      epi.template segment<C>(g, (kb + 1) / seg_len, nw0, acc, lane, est);
  }
  wait_vmcnt<0>();  // the trailing prefetches (zeros) land before the block ends
  // an epilogue that stages its stores through the ring waits until every wave is past
  // its last read of it
  if constexpr (Epi::kUsesLds || TabLds<Epi>::value) {
    static_assert(!Epi::kUsesLds ||
                      sizeof(smem) >= (size_t)(C::NT / 64) * 32 * 32 * C::WO * sizeof(T),
                  "the epilogue's staging fits the ring");
    __syncthreads();
  }
  if constexpr (TabLds<Epi>::value) {
    static_assert(Epi::template tab_end<C>() <= sizeof(smem), "the table fits the ring");
    epi.template stage_tab<C>(g, n0, (char*)smem, tid);
    __syncthreads();
  }
  epi.template finish<C>(g, ow0, nw0, acc, lane, est, EpiLds{(char*)smem, w, n0});
}

}  // namespace wm
