// Cross-layer KV pool kernels (paper Section 3.1, Steps 1 and 2).
//
//   row_rms      1 / RMS of every (token, layer) state (the pre-mix and the
//                consumer input norms share it; only the gains differ)
//   rope_table   (cos, sin) of pos * theta^(-2m/d) per new token, in fp64
//   router       alpha logits = W_alpha xi + b_alpha on the matrix cores; xi is
//                the stack of normed states of layers {L-1-p*m}
//   mix          (optional softmax over source layers) and the per-token mix
//                h~_j = sum_l alpha[j][l] h^_l, plus 1 / RMS of each channel
//   kv_project   per-channel W^K_j / W^V_j on the matrix cores; the mid
//                RMSNorm gain is folded into a per-call copy of the weights and
//                its 1/RMS, the key norm, RoPE and the channel-major cache
//                store happen in the epilogue
//   q_project    the consumer's query (input norm, W^Q_l, q norm, RoPE), built
//                the same way
#include <algorithm>

#include "wm_gemm.hpp"
#include "wm_internal.hpp"

namespace wm {

// ----------------------------------------------------------------- row rms
// Row r of length D starts at X + r * xs; its 1/RMS goes to rinv[r * os].
// One wave per row, any D.
template <typename T>
__global__ __launch_bounds__(256) void row_rms_loop_kernel(const T* X, long rows, int D, long xs,
                                                           long os, float eps, float* rinv) {
  const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const T* x = X + row * xs;
  float ss = 0.f;
  for (int e = lane * 8; e < D; e += 512) {
    float v[8];
    load8(x + e, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += v[i] * v[i];
  }
  ss = wave_sum(ss);
  if (lane == 0) rinv[row * os] = 1.0f / sqrtf(ss / (float)D + eps);
}

// One wave per R rows of at most 512 NC elements; a lane loads its NC chunks of 8 from
// each of them before any arithmetic, so a wave has R NC loads in flight (one row of
// 1-1.5 KB per wave left the HBM read stream short of loads in flight).
template <typename T, int R, int NC>
__global__ __launch_bounds__(256) void row_rms_kernel(const T* X, long rows, int D, long xs,
                                                      long os, float eps, float* rinv) {
  const long row0 = ((long)blockIdx.x * 4 + (threadIdx.x >> 6)) * R;
  const int lane = threadIdx.x & 63;
  if (row0 >= rows) return;
  float v[R][NC][8];
#pragma unroll
  for (int q = 0; q < R; ++q)
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int e = lane * 8 + 512 * c;
      if (row0 + q < rows && e < D) load8(X + (row0 + q) * xs + e, v[q][c]);
      else
#pragma unroll
        for (int i = 0; i < 8; ++i) v[q][c][i] = 0.f;
    }
#pragma unroll
  for (int q = 0; q < R; ++q) {
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int i = 0; i < 8; ++i) ss += v[q][c][i] * v[q][c][i];
    ss = wave_sum(ss);
    if (lane == 0 && row0 + q < rows) rinv[(row0 + q) * os] = 1.0f / sqrtf(ss / (float)D + eps);
  }
}

#ifndef WM_RMS_ROWS
#define WM_RMS_ROWS 2
#endif
template <typename T, int NC>
static void launch_row_rms_nc(const T* X, long rows, int D, long xs, long os, float eps,
                              float* rinv, hipStream_t s) {
  constexpr int R = WM_RMS_ROWS;
  hipLaunchKernelGGL((row_rms_kernel<T, R, NC>), dim3((unsigned)((rows + 4 * R - 1) / (4 * R))),
                     dim3(256), 0, s, X, rows, D, xs, os, eps, rinv);
}

template <typename T>
void launch_row_rms_strided(const T* X, long rows, int D, long xs, long os, float eps,
                            float* rinv, hipStream_t s) {
  if (rows <= 0) return;
  const int nc = (D + 511) / 512;  // chunks of 8 per lane (D is a multiple of 8)
  if (nc <= 1) launch_row_rms_nc<T, 1>(X, rows, D, xs, os, eps, rinv, s);
  else if (nc == 2) launch_row_rms_nc<T, 2>(X, rows, D, xs, os, eps, rinv, s);
  else if (nc <= 4) launch_row_rms_nc<T, 4>(X, rows, D, xs, os, eps, rinv, s);
  else
    hipLaunchKernelGGL(row_rms_loop_kernel<T>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s,
                       X, rows, D, xs, os, eps, rinv);
}

template <typename T>
void launch_row_rms(const T* X, long rows, int D, float eps, float* rinv, hipStream_t s) {
  launch_row_rms_strided<T>(X, rows, D, D, 1, eps, rinv, s);
}

// -------------------------------------------------------------- rope table
// tab[n][m] = (cos, sin)(pos(n) theta^(-2m/d)). The frequencies (one per m) are computed
// once per block in double; each angle is formed and reduced modulo 2 pi in double, so
// the float sincos that follows sees |r| <= pi and keeps float accuracy at any position.
__global__ __launch_bounds__(256) void rope_table_kernel(const int32_t* ctx_len, int B,
                                                         int T_new, int d, int gs, int gq,
                                                         int ctx_hi, double theta, float* tab) {
  __shared__ double freq[kMaxHeadDim / 2];
  const int half = d / 2;
  for (int m = threadIdx.x; m < half; m += blockDim.x)
    freq[m] = pow(theta, -2.0 * (double)m / (double)d);
  __syncthreads();
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)B * T_new * half) return;
  const int m = (int)(idx % half);
  const long n = idx / half;
  const int b = (int)(n / T_new), i = (int)(n % T_new);
  const long pos = (long)ctx_at(ctx_len, b, ctx_hi) + gq + (long)gs * i;
  const double ang = (double)pos * freq[m];
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  const float r = (float)(ang - kTwoPi * rint(ang / kTwoPi));
  float sn, cs;
  sincosf(r, &sn, &cs);
  tab[2 * idx] = cs;
  tab[2 * idx + 1] = sn;
}

void launch_rope_table(const Shape& sh, const int32_t* ctx_len, float* tab, hipStream_t s) {
  long total = (long)sh.N() * (sh.d / 2);
  if (total <= 0) return;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     ctx_len, sh.B, sh.T_new, sh.d, sh.gs, sh.gq, sh.ctx_hi,
                     (double)sh.rope_theta, tab);
}

// -------------------------------------------------------- GEMM operands
// Plain rows: X[g * gstride + row * rstride + k], rows < rows (weights or activations).
template <typename T> struct PlainRows {
  const T* X;
  long gstride, rstride;
  int rows;
  __device__ RowsView view(int g) const {
    return {make_view(X + (long)g * gstride, (uint32_t)((long)rows * rstride * sizeof(T))),
            (uint32_t)(rstride * sizeof(T))};
  }
  __device__ uint32_t slice(int k0) const { return (uint32_t)k0 * (uint32_t)sizeof(T); }
};

// Router operand: token n's row is the stack of the selected layers' raw states,
// column k = m * D + e reading H[n][sel[m]][e] (the 1/RMS is applied to the
// accumulators, the gain is folded into the weights).
// The stacked layers are affine in m: sel[m] = s0 + p m (every p-th layer counting down
// from L-1, in ascending order), so a slice's offset needs no table read; with p = 1 the
// stack is the whole row.
template <typename T> struct StackedRows {
  const T* H;
  int s0, p, L, D, M;
  __device__ RowsView view(int) const {
    return {make_view(H, (uint32_t)((long)M * L * D * sizeof(T))),
            (uint32_t)((long)L * D * sizeof(T))};
  }
  __device__ uint32_t slice(int k0) const {
    if (p == 1) return (uint32_t)(s0 * D + k0) * (uint32_t)sizeof(T);
    const int m = k0 / D, e = k0 - m * D;
    return (uint32_t)((s0 + p * m) * D + e) * (uint32_t)sizeof(T);
  }
};

// ------------------------------------------------------ head epilogue
// The K/V and Q projections end in the same per-head work on the transposed
// accumulators. For token n (lane r of block column jn) and a head of DH
// channels held by the wave, value v = 0 .. DH/2-1 of the lane sits in block
// v / 16, register v % 16, i.e. at channel m(v) = 32 (v/16) + 8 ((v%16)/4) +
// 4h + v%4; the other half of the head is in the partner lane (h ^ 1).
//   scale by the row's 1/RMS; then either store (V) or RMS-normalise over the
//   head (one cross-half sum), apply the gain and rotate: value v < DH/4 pairs
//   with v + DH/4 (channels m and m + DH/2), at angle index m(v).
template <int DH> __device__ __forceinline__ int head_chan(int v, int h) {
  return 32 * (v >> 4) + 8 * ((v & 15) >> 2) + 4 * h + (v & 3);
}

// Chunk swizzle of the RoPE rows staged in LDS (see stage_rope_rows).
template <int DH> __device__ __forceinline__ int rope_row_swz(int t) {
  return DH == 64 ? (t & 15) : ((t >> 1) & 7);
}

// STAGE (bf16): stores go through the wave's LDS area so that each store instruction
// writes whole head rows (measured faster for the cache writes of the K/V projection,
// not for the query workspace).
// Memory order: every load the epilogue needs for a column block (row scales, the
// slot base of each token, the RoPE table entries) is issued before the previous
// block's stores, and every store is issued whether or not its lane has a row to
// write (lanes without one write to a small trash area of the workspace). So each
// wave issues a fixed sequence of memory operations, and waiting for a load leaves
// the earlier blocks' stores in flight instead of draining them.
//   scale_at(n) -> float   the row's 1/RMS
//   aux_at(n)   -> int     a per-token value the destination needs (or 0)
//   dst_at(n, head, aux) -> T*   the row's destination, nullptr when there is none
//   tab, tab_n0: the RoPE table rows of tokens tab_n0 .. : with TABLDS the block's rows
//   in LDS, laid out by stage_rope_rows; else the whole table in memory (tab_n0 = 0)
template <typename T, int DH, int WO, int WN, bool STAGE, bool TABLDS, class ScaleAt,
          class AuxAt, class DstAt>
__device__ __forceinline__ void head_epilogue(f32x16 (&acc)[WO][WN], int ow0, int nw0, int lane,
                                              int M, bool rotate, const T* gain,
                                              const float* tab, int tab_n0, float eps,
                                              ScaleAt scale_at,
                                              AuxAt aux_at, DstAt dst_at, T* trash,
                                              const EpiLds& lds) {
  constexpr int NV = DH / 2;          // values of one head per lane
  constexpr int HPW = 32 * WO / DH;   // heads per wave
  static_assert(HPW * DH == 32 * WO, "a wave holds whole heads");
  const int h = lane >> 5, r = lane & 31;
  float gv[NV];
  if (rotate) {
#pragma unroll
    for (int c = 0; c < NV / 4; ++c) {
      const T* gp = gain + head_chan<DH>(4 * c, h);
#pragma unroll
      for (int t = 0; t < 4; ++t) gv[4 * c + t] = to_f32(gp[t]);
    }
  }
  int nn[WN];
  bool in[WN];
  float sc[WN];
  int aux[WN];
#pragma unroll
  for (int jn = 0; jn < WN; ++jn) {
    const int n = nw0 + 32 * jn + r;
    in[jn] = n < M;
    nn[jn] = in[jn] ? n : M - 1;
    sc[jn] = scale_at(nn[jn]);
    aux[jn] = aux_at(nn[jn]);
  }
  f32x4 tb[DH / 16][2];  // (cos, sin) of angle indices 8g + 4h + t, t = 0..3
  auto load_tab = [&](int jn) {
#pragma unroll
    for (int g = 0; g < DH / 16; ++g) {
      const int t = nn[jn] - tab_n0, sw = TABLDS ? rope_row_swz<DH>(t) : 0;
      const float* tp = tab + (long)t * DH;
      tb[g][0] = *(const f32x4*)(tp + 4 * ((4 * g + 2 * h) ^ sw));
      tb[g][1] = *(const f32x4*)(tp + 4 * ((4 * g + 2 * h + 1) ^ sw));
    }
  };
  if (rotate) load_tab(0);
#pragma unroll
  for (int jn = 0; jn < WN; ++jn) {
    float c[HPW][NV];
#pragma unroll
    for (int hw = 0; hw < HPW; ++hw) {
#pragma unroll
      for (int v = 0; v < NV; ++v) c[hw][v] = acc[hw * (DH / 32) + (v >> 4)][jn][v & 15] * sc[jn];
      if (rotate) {
        float ss = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v) ss += c[hw][v] * c[hw][v];
        ss = halves_sum(ss);
        const float rs = 1.0f / sqrtf(ss / (float)DH + eps);
#pragma unroll
        for (int v = 0; v < NV; ++v) c[hw][v] *= rs * gv[v];
#pragma unroll
        for (int v = 0; v < NV / 2; ++v) {
          const int t = v & 3;
          const float cs = tb[v >> 2][t >> 1][2 * (t & 1)], sn = tb[v >> 2][t >> 1][2 * (t & 1) + 1];
          const float x1 = c[hw][v], x2 = c[hw][v + NV / 2];
          c[hw][v] = x1 * cs - x2 * sn;
          c[hw][v + NV / 2] = x2 * cs + x1 * sn;
        }
      }
    }
    // the next block's table entries, ahead of this block's stores
    if (rotate && jn + 1 < WN) load_tab(jn + 1);
    if constexpr (sizeof(T) == 2 && STAGE) {
      // Stage the block (32 tokens x HPW heads, one head row of DH channels per token)
      // in the wave's LDS area, then store it row by row: each store instruction writes
      // whole head rows (CPR lanes of 16 bytes per row) instead of 32-byte pieces of 32
      // rows. 16-byte chunk c of row t sits at chunk c ^ ((t / 2) mod CPR).
      constexpr int CPR = DH / 8, RPI = 64 / CPR, ROWS = 32 * HPW;
      char* reg = lds.p + lds.wave * (ROWS * DH * 2);
#pragma unroll
      for (int hw = 0; hw < HPW; ++hw) {
        const int row = 32 * hw + r;
        // chunks 2p, 2p+1 (channels m0 + 4h + 0..3 and m0 + 8 + 4h + 0..3): one swap of
        // the middle quarters gives lane h the 8 contiguous channels m0 + 8h .. m0 + 8h + 7
#pragma unroll
        for (int p = 0; p < NV / 8; ++p) {
          uint32_t a[2], b[2];
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            bf16x2 x = {(bf16)c[hw][8 * p + 2 * i], (bf16)c[hw][8 * p + 2 * i + 1]};
            bf16x2 y = {(bf16)c[hw][8 * p + 4 + 2 * i], (bf16)c[hw][8 * p + 4 + 2 * i + 1]};
            a[i] = __builtin_bit_cast(uint32_t, x);
            b[i] = __builtin_bit_cast(uint32_t, y);
            auto sw = __builtin_amdgcn_permlane32_swap(a[i], b[i], false, false);
            a[i] = sw[0];
            b[i] = sw[1];
          }
          const int ch = 4 * (p >> 1) + 2 * (p & 1) + h;  // 16-byte chunk of the row
          const i32x4 o = {(int)a[0], (int)a[1], (int)b[0], (int)b[1]};
          *(i32x4*)(reg + row * DH * 2 + 16 * (ch ^ ((row >> 1) & (CPR - 1)))) = o;
        }
      }
      const int cl = lane % CPR;
#pragma unroll
      for (int it = 0; it < ROWS / RPI; ++it) {
        const int row = RPI * it + lane / CPR, t = row & 31, hw = row >> 5;
        const i32x4 o = *(const i32x4*)(reg + row * DH * 2 + 16 * (cl ^ ((row >> 1) & (CPR - 1))));
        const int n = nw0 + 32 * jn + t;
        const int ax = __shfl(aux[jn], t, 64);
        T* dst = dst_at(n < M ? n : M - 1, (ow0 + hw * DH) / DH, ax);
        if (!(n < M && dst != nullptr)) dst = trash;
        *(i32x4*)(dst + 8 * cl) = o;
      }
    } else if constexpr (sizeof(T) == 2) {
      // direct: each store writes 32 bytes of each of the block's 32 rows
#pragma unroll
      for (int hw = 0; hw < HPW; ++hw) {
        T* dst = dst_at(nn[jn], (ow0 + hw * DH) / DH, aux[jn]);
        if (!(in[jn] && dst != nullptr)) dst = trash;
#pragma unroll
        for (int p = 0; p < NV / 8; ++p) {
          uint32_t a[2], b[2];
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            bf16x2 x = {(bf16)c[hw][8 * p + 2 * i], (bf16)c[hw][8 * p + 2 * i + 1]};
            bf16x2 y = {(bf16)c[hw][8 * p + 4 + 2 * i], (bf16)c[hw][8 * p + 4 + 2 * i + 1]};
            a[i] = __builtin_bit_cast(uint32_t, x);
            b[i] = __builtin_bit_cast(uint32_t, y);
            auto sw = __builtin_amdgcn_permlane32_swap(a[i], b[i], false, false);
            a[i] = sw[0];
            b[i] = sw[1];
          }
          i32x4 o = {(int)a[0], (int)a[1], (int)b[0], (int)b[1]};
          *(i32x4*)(dst + 32 * (p >> 1) + 16 * (p & 1) + 8 * h) = o;
        }
      }
    } else {
#pragma unroll
      for (int hw = 0; hw < HPW; ++hw) {
        T* dst = dst_at(nn[jn], (ow0 + hw * DH) / DH, aux[jn]);
        if (!(in[jn] && dst != nullptr)) dst = trash;
#pragma unroll
        for (int q = 0; q < NV / 4; ++q) {
          f32x4 o = {c[hw][4 * q], c[hw][4 * q + 1], c[hw][4 * q + 2], c[hw][4 * q + 3]};
          *(f32x4*)(dst + head_chan<DH>(4 * q, h)) = o;
        }
      }
    }
  }
}

// Workspace elements (of T) after the folded weights that lanes without a row write
// to: the staged bf16 stores reach 64 elements past the pointer, the others DH.
constexpr size_t kTrashElems = 512;

struct NoState {};

// The block's rows [n0, n0 + NTOK) of the RoPE table (DH floats per token; rows past the
// last token repeat it) copied into LDS at byte offset `off`, 16 bytes per thread and step.
// 16-byte chunk c of row t sits at chunk c ^ rope_row_swz(t), so the 16 lanes of a read,
// one token each, hit 16 distinct bank groups (the rows are 128, 256 or 384 bytes).
template <class C, int DH>
__device__ __forceinline__ void stage_rope_rows(const float* tab, int M, int n0, char* lds,
                                                size_t off, int tid) {
  static_assert(DH == 32 || DH == 64 || DH == 96, "swizzle shapes");
  constexpr int CH = DH / 4, N = C::NTOK * CH;
  float* dst = (float*)(lds + off);
  for (int i = tid; i < N; i += C::NT) {
    const int t = i / CH, c = i - t * CH, n = min(n0 + t, M - 1);
    *(f32x4*)(dst + t * DH + 4 * (c ^ rope_row_swz<DH>(t))) =
        *(const f32x4*)(tab + (long)n * DH + 4 * c);
  }
}

template <typename T, int DH> struct KVEpi {
  // bf16 stages the cache writes when a head row is a power-of-two count of 16-B chunks
  // (head dims 32 and 64); head dim 96 stores directly
  static constexpr bool kUsesLds = sizeof(T) == 2 && ((DH / 8) & (DH / 8 - 1)) == 0;
  // the key blocks' RoPE rows go to LDS after the output staging area (head dims 32 and
  // 64; measured slower at 96, whose blocks read the table from memory)
  static constexpr bool kTabLds = DH != 96;
  template <class C> static constexpr size_t tab_off() {
    return kUsesLds ? (size_t)(C::NT / 64) * 32 * 32 * C::WO * sizeof(T) : 0;
  }
  template <class C> static constexpr size_t tab_end() {
    return tab_off<C>() + (size_t)C::NTOK * DH * sizeof(float);
  }
  T *Kc, *Vc;
  T* trash;  // kTrashElems elements of workspace
  const float* rs;  // [2k][M] 1 / RMS of each mixed channel row (the mid RMSNorm)
  const T* g_knorm;
  const float* tab;
  const int32_t* ctx_len;
  int M, T_new, B, Hkv, S_cap, k;
  int gs, gq, ctx_hi;  // token i of sequence b goes to slot ctx_len[b] + gq + gs i
  float eps;
  using State = NoState;
  template <class C> __device__ void begin(int, int, int, State&) const {}
  template <class C>
  __device__ void segment(int, int, int, f32x16 (&)[C::WO][C::WN], int, State&) const {}
  template <class C> __device__ void stage_tab(int g, int n0, char* lds, int tid) const {
    if (g < k) stage_rope_rows<C, DH>(tab, M, n0, lds, tab_off<C>(), tid);  // key branch
  }
  template <class C>
  __device__ void finish(int g, int ow0, int nw0, f32x16 (&acc)[C::WO][C::WN], int lane,
                         State&, const EpiLds& lds) const {
    const int br = g / k, j = g - br * k;
    const bool key = br == 0;
    T* base = key ? Kc : Vc;
    head_epilogue<T, DH, C::WO, C::WN, kUsesLds, kTabLds>(
        acc, ow0, nw0, lane, M, key, g_knorm + (long)j * DH,
        kTabLds ? (const float*)(lds.p + tab_off<C>()) : tab, kTabLds ? lds.n0 : 0, eps,
        [&](int n) { return rs[(long)g * M + n]; },
        [&](int n) { return ctx_at(ctx_len, n / T_new, ctx_hi) + gq; },
        [&](int n, int head, int pos0) -> T* {
          if (head >= Hkv) return nullptr;
          const int b = n / T_new, i = n - b * T_new;
          const long slot = (long)pos0 + (long)gs * i;
          if (slot < 0 || slot >= S_cap) return nullptr;
          return base + ((((long)j * B + b) * Hkv + head) * S_cap + slot) * DH;
        },
        trash, lds);
  }
};

template <typename T, int DH> struct QEpi {
  static constexpr bool kUsesLds = false;
  static constexpr bool kTabLds = DH != 96;  // RoPE rows in LDS (as for the keys)
  template <class C> static constexpr size_t tab_end() {
    return (size_t)C::NTOK * DH * sizeof(float);
  }
  template <class C> __device__ void stage_tab(int, int n0, char* lds, int tid) const {
    stage_rope_rows<C, DH>(tab, M, n0, lds, 0, tid);
  }
  T* Q;
  T* trash;  // kTrashElems elements of workspace
  const float* rs;  // [M][L] 1 / RMS of each consumer's input state (the input RMSNorm)
  const T* g_qnorm;
  const float* tab;
  int M, T_new, B, Hq, L;
  int l0;  // group g of the launch is consumer layer l0 + g; Q holds the launch's layers
  float eps;
  using State = NoState;
  template <class C> __device__ void begin(int, int, int, State&) const {}
  template <class C>
  __device__ void segment(int, int, int, f32x16 (&)[C::WO][C::WN], int, State&) const {}
  template <class C>
  __device__ void finish(int l, int ow0, int nw0, f32x16 (&acc)[C::WO][C::WN], int lane,
                         State&, const EpiLds& lds) const {
    head_epilogue<T, DH, C::WO, C::WN, false, kTabLds>(
        acc, ow0, nw0, lane, M, true, g_qnorm + (long)(l0 + l) * DH,
        kTabLds ? (const float*)lds.p : tab, kTabLds ? lds.n0 : 0, eps,
        [&](int n) { return rs[(long)n * L + l0 + l]; }, [](int) { return 0; },
        [&](int n, int head, int) -> T* {
          if (head >= Hq) return nullptr;
          const int b = n / T_new, i = n - b * T_new;
          return Q + ((((long)l * B + b) * Hq + head) * T_new + i) * DH;
        },
        trash, lds);
  }
};

// Router epilogue. Column block m of the stacked operand is layer sel[m]'s raw
// state; its 1/RMS is a per-token factor, so the accumulators are kept in units
// of the current layer's 1/RMS: at a layer boundary they are multiplied by
// rinv(previous) / rinv(next), and by rinv(last) at the end. With split K a
// block covers the layers [s * per, ...) and writes a partial sum for the
// reduction; without it the bias is added and the logits are stored directly.
template <typename T> struct RouterEpi {
  static constexpr bool kUsesLds = false;
  float* out;        // splits == 1: logits [2][M][kL]; else partials [splits][M][2kL]
  const T* bias;     // [2kL]
  const float* rinv; // [M][L]
  LayerTable sel;
  int M, Nout, kL, L, Lp, seg_per_split, splits;
  struct State {
    float cur[4], nxt[4];
  };
  __device__ float rinv_at(int n, int m) const {
    return rinv[(long)n * L + sel.v[min(m, Lp - 1)]];
  }
  template <class C> __device__ void begin(int s, int nw0, int lane, State& st) const {
    static_assert(C::WN <= 4, "router state holds 4 token blocks");
    const int m0 = s * seg_per_split;
#pragma unroll
    for (int jn = 0; jn < C::WN; ++jn) {
      const int n = min(nw0 + 32 * jn + (lane & 31), M - 1);
      st.cur[jn] = rinv_at(n, m0);
      st.nxt[jn] = rinv_at(n, m0 + 1);
    }
  }
  template <class C>
  __device__ void segment(int, int seg, int nw0, f32x16 (&acc)[C::WO][C::WN], int lane,
                          State& st) const {
#pragma unroll
    for (int jn = 0; jn < C::WN; ++jn) {
      const float f = st.cur[jn] / st.nxt[jn];
#pragma unroll
      for (int i = 0; i < C::WO; ++i)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[i][jn][q] *= f;
      st.cur[jn] = st.nxt[jn];
      const int n = min(nw0 + 32 * jn + (lane & 31), M - 1);
      st.nxt[jn] = rinv_at(n, seg + 1);
    }
  }
  template <class C>
  __device__ void finish(int s, int ow0, int nw0, f32x16 (&acc)[C::WO][C::WN], int lane,
                         State& st, const EpiLds&) const {
    const int h = lane >> 5, r = lane & 31;
#pragma unroll
    for (int jn = 0; jn < C::WN; ++jn) {
      const int n = nw0 + 32 * jn + r;
      if (n >= M) continue;
#pragma unroll
      for (int i = 0; i < C::WO; ++i)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int o = ow0 + 32 * i + 8 * (q >> 2) + 4 * h + (q & 3);
          if (o >= Nout) continue;
          const float v = acc[i][jn][q] * st.cur[jn];
          if (splits == 1) {
            const int br = o >= kL, oo = o - br * kL;
            out[((long)br * M + n) * kL + oo] = v + to_f32(bias[o]);
          } else {
            out[((long)s * M + n) * Nout + o] = v;
          }
        }
    }
  }
};

// logits[br][n][o'] = sum_s part[s][n][br kL + o'] + bias[br kL + o']
template <typename T>
__global__ __launch_bounds__(256) void router_reduce_kernel(const float* part, const T* bias,
                                                            float* logits, int M, int kL,
                                                            int splits) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x, total = (long)M * 2 * kL;
  if (idx >= total) return;
  const int n = (int)(idx / (2 * kL)), o = (int)(idx - (long)n * 2 * kL);
  float v = to_f32(bias[o]);
  for (int s = 0; s < splits; ++s) v += part[(long)s * total + idx];
  const int br = o >= kL, oo = o - br * kL;
  logits[((long)br * M + n) * kL + oo] = v;
}

// Router weights with the pre-mix gain folded in: Wf[o][m D + e] =
// W_alpha[o][m D + e] * g_pre[o / kL][sel[m]][e], o over both branches.
// Without feedback (nofb), the row of channel j = (o mod kL) / L reads only the stacked
// blocks of layers <= j: the other blocks of its folded weights are zero.
template <typename T>
__global__ __launch_bounds__(256) void router_fold_kernel(const T* W, const T* g_pre,
                                                          LayerTable sel, int kL, int L, int Lp,
                                                          int D, int nofb, T* Wf) {
  const long idx = ((long)blockIdx.x * 256 + threadIdx.x) * 8;
  const long K = (long)Lp * D, total = 2 * kL * K;
  if (idx >= total) return;
  const int o = (int)(idx / K);
  const long kk = idx - o * K;
  const int m = (int)(kk / D), e = (int)(kk - (long)m * D);
  float wv[8], gv[8];
  load8(W + idx, wv);
  load8(g_pre + ((long)(o / kL) * L + sel.v[m]) * D + e, gv);
  const float keep = nofb && sel.v[m] > (o % kL) / L ? 0.f : 1.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) wv[i] *= gv[i] * keep;
  store8(Wf + idx, wv);
}

// Static mixing weights: logits[br][n][o] = b_alpha[br][o] for every token.
template <typename T>
__global__ __launch_bounds__(256) void alpha_static_kernel(const T* b_alpha, int N, int kL,
                                                           float* logits) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= 2L * N * kL) return;
  const int o = (int)(idx % kL), br = (int)(idx / ((long)N * kL));
  logits[idx] = to_f32(b_alpha[(long)br * kL + o]);
}

template <class C> static unsigned proj_blocks(int M, int Nout, int groups) {
  return (unsigned)(groups * ((M + C::NTOK - 1) / C::NTOK) * ((Nout + C::OT - 1) / C::OT));
}

template <class C, typename T, class XL, class WL, class Epi>
static void launch_proj(int M, int Nout, int K, int groups, int seg_len, int kspan,
                        const XL& xl, const WL& wl, const Epi& e, hipStream_t s) {
  if constexpr (C::SWZ) {
    hipLaunchKernelGGL((proj_gemm_dma_kernel<C, T, XL, WL, Epi>),
                       dim3(proj_blocks<C>(M, Nout, groups)), dim3(C::NT), 0, s, M, Nout, K,
                       groups, seg_len, kspan, xl, wl, e);
  } else {
    hipLaunchKernelGGL((proj_gemm_kernel<C, T, XL, WL, Epi>), dim3(proj_blocks<C>(M, Nout, groups)),
                       dim3(C::NT), 0, s, M, Nout, K, groups, seg_len, kspan, xl, wl, e);
  }
}
constexpr int kNoSegments = 1 << 30;

// Tile shapes. Large token counts: 256 channels x 256 tokens per block of 8 waves,
// 64 x 128 per wave (bf16). Few tokens (decode): 128 x 64. fp32: 128 x 128, 4 waves.
template <typename T, bool FEW> struct ProjShape;
#ifndef WM_PROJ_BF16
#define WM_PROJ_BF16 32, 4, 2, 2, 4
#endif
template <> struct ProjShape<bf16, false> { using C = ProjCfg<bf16, WM_PROJ_BF16>; };
template <> struct ProjShape<bf16, true> { using C = ProjCfg<bf16, 32, 2, 2, 2, 1>; };
template <> struct ProjShape<float, false> { using C = ProjCfg<float, 32, 2, 2, 2, 2>; };
template <> struct ProjShape<float, true> { using C = ProjCfg<float, 32, 2, 2, 2, 1>; };
// Head dim 96 (bf16): a wave holds one head (96 channels) of 64 tokens. K/V: 288
// channels x 128 tokens per block of 6 waves, i.e. one projection of 3 KV heads (64
// tokens for few tokens). Q: 192 x 256 per block of 8 waves (measured 15% faster than
// 288 x 128 for 6 query heads; 20% slower for the K/V projections).
template <typename T, bool FEW, int DH, bool Q> struct ProjShapeD {
  using C = typename ProjShape<T, FEW>::C;
};
template <bool Q> struct ProjShapeD<bf16, false, 96, Q> {
  using C = ProjCfg<bf16, 32, Q ? 2 : 3, Q ? 4 : 2, 3, 2>;
};
template <bool Q> struct ProjShapeD<bf16, true, 96, Q> { using C = ProjCfg<bf16, 32, 3, 2, 3, 1>; };
// Router: 288 channels x 128 tokens per bf16 block on 6 waves, 96 x 64 per wave (the
// channel count 2kL is small: 288 for L = k = 12, so a block covers all of it and the
// stacked states are read once; measured 10% faster than 96-channel blocks at L = 24).
// Long K (the stacked states of many wide layers, L' D >= kRouterWideK) in bf16: 288 x 256
// on 12 waves, 3 per SIMD (the 6-wave block leaves two of the four SIMDs one wave each),
// its grid filled by splitting K. Measured: 21% faster at L = 24, D = 1024; no change at
// L = 12, D = 768; 12% slower at the paper's L' = 8, D = 512 (a short K, whose split
// doubles the fixed costs), so the 6-wave block stays there.
template <typename T, bool FEW, bool WIDE = false> struct RouterShape;
#ifndef WM_ROUTER_BF16
#define WM_ROUTER_BF16 32, 3, 2, 3, 2
#endif
template <> struct RouterShape<bf16, false> { using C = ProjCfg<bf16, WM_ROUTER_BF16>; };
template <> struct RouterShape<bf16, false, true> { using C = ProjCfg<bf16, 32, 3, 4, 3, 2>; };
template <> struct RouterShape<bf16, true> { using C = ProjCfg<bf16, 32, 1, 2, 3, 1>; };
template <> struct RouterShape<float, false> { using C = ProjCfg<float, 32, 1, 4, 3, 1>; };
template <> struct RouterShape<float, false, true> { using C = ProjCfg<float, 32, 1, 4, 3, 1>; };
template <> struct RouterShape<float, true> { using C = ProjCfg<float, 32, 1, 2, 3, 1>; };

constexpr int kFewTokens = 64;
constexpr int kRouterWideK = 16384;
static bool router_wide(const Shape& sh) {
  return sh.N() > kFewTokens && (long)sh.Lp * sh.D >= kRouterWideK;
}

// ------------------------------------------------------------------ router
size_t router_fold_elems(const Shape& sh) { return 2ul * sh.k * sh.L * sh.Lp * sh.D; }

// Layers per K split: enough blocks to cover the chip (one per CU), splitting K at layer
// boundaries when the token and channel tiles alone give fewer. (Aiming at two blocks per
// CU measured 6-21% slower: the extra partial sums cost more than the occupancy gains.)
#ifndef WM_ROUTER_MIN_BLOCKS
#define WM_ROUTER_MIN_BLOCKS 256
#endif
static int router_layers_per_split(const Shape& sh) {
  using CF = RouterShape<bf16, false>::C;
  using CW = RouterShape<bf16, false, true>::C;
  using CD = RouterShape<bf16, true>::C;
  const bool few = sh.N() <= kFewTokens, wide = router_wide(sh);
  const int tok = few ? CD::NTOK : wide ? CW::NTOK : CF::NTOK;
  const int och = few ? CD::OT : wide ? CW::OT : CF::OT;
  const long blocks = (long)((sh.N() + tok - 1) / tok) * ((2 * sh.k * sh.L + och - 1) / och);
  int s = 1;
  while (s < sh.Lp && blocks * s < WM_ROUTER_MIN_BLOCKS) s *= 2;
  return (sh.Lp + s - 1) / s;
}

static int router_splits(const Shape& sh) {  // every split covers at least one layer
  const int per = router_layers_per_split(sh);
  return (sh.Lp + per - 1) / per;
}

size_t router_partials_bytes(const Shape& sh) {
  const int s = router_splits(sh);
  return s > 1 ? (size_t)s * sh.N() * 2 * sh.k * sh.L * sizeof(float) : 0;
}

template <typename T, bool FEW, bool WIDE>
static void router_gemm(const Shape& sh, const LayerTable& sel, const T* H, const float* rinv,
                        const T* wf, const T* b_alpha, float* logits, float* part,
                        hipStream_t s) {
  using C = typename RouterShape<T, FEW, WIDE>::C;
  const int M = sh.N(), kL = sh.k * sh.L, Nout = 2 * kL, K = sh.Lp * sh.D;
  const int seg = sh.D / C::BK, splits = router_splits(sh);
  const int per = router_layers_per_split(sh);
  StackedRows<T> x{H, sel.v[0], sh.p, sh.L, sh.D, M};
  PlainRows<T> w{wf, 0, K, Nout};
  RouterEpi<T> e{splits > 1 ? part : logits, b_alpha, rinv, sel, M, Nout, kL, sh.L, sh.Lp, per,
                 splits};
  // the split index plays the group: split s covers layers [s per, (s+1) per)
  launch_proj<C, T>(M, Nout, K, splits, seg, per * sh.D, x, w, e, s);
  if (splits > 1) {
    const long total = (long)M * Nout;
    hipLaunchKernelGGL(router_reduce_kernel<T>, dim3((unsigned)((total + 255) / 256)), dim3(256),
                       0, s, part, b_alpha, logits, M, kL, splits);
  }
}

template <typename T>
void launch_router_fold(const Shape& sh, const LayerTable& sel, const T* g_pre, const T* W_alpha,
                        T* wfold, hipStream_t s) {
  if (sh.router_mode == 1) return;  // static weights: no router
  const long total = (long)router_fold_elems(sh) / 8;
  hipLaunchKernelGGL(router_fold_kernel<T>, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                     s, W_alpha, g_pre, sel, sh.k * sh.L, sh.L, sh.Lp, sh.D,
                     sh.router_mode == 2 ? 1 : 0, wfold);
}

template <typename T>
void launch_router(const Shape& sh, const LayerTable& sel, const T* H, const float* rinv,
                   const T* g_pre, const T* W_alpha, const T* b_alpha, float* logits, T* wfold,
                   float* part, hipStream_t s, bool prefolded) {
  const int M = sh.N();
  if (M <= 0) return;
  if (sh.router_mode == 1) {  // static weights: no router, the logits are the bias
    const long n = 2L * M * sh.k * sh.L;
    hipLaunchKernelGGL(alpha_static_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       b_alpha, M, sh.k * sh.L, logits);
    return;
  }
  if (!prefolded) launch_router_fold<T>(sh, sel, g_pre, W_alpha, wfold, s);
  if (M <= kFewTokens)
    router_gemm<T, true, false>(sh, sel, H, rinv, wfold, b_alpha, logits, part, s);
  else if (router_wide(sh))
    router_gemm<T, false, true>(sh, sel, H, rinv, wfold, b_alpha, logits, part, s);
  else
    router_gemm<T, false, false>(sh, sel, H, rinv, wfold, b_alpha, logits, part, s);
}

// --------------------------------------------------------------------- mix
// One block per token; each thread owns 8 consecutive columns. LDS holds the
// token's L states and the coefficients alpha[j][l] / RMS(h_l), stored layer-
// major with the channel count padded to JC (zeros), so a thread reads JC
// coefficients of one layer with JC/4 broadcast loads. For each branch the
// thread scales a layer's 8 columns by the gain once and accumulates them into
// all JC channels, then stores the channels and their sums of squares.
constexpr int kMixBatch = 12;

template <typename T, int JC>
__global__ __launch_bounds__(128) void mix_kernel(Shape sh, const T* __restrict__ H,
                                                  const float* __restrict__ rinv,
                                                  const T* __restrict__ g_pre, float* alpha,
                                                  T* __restrict__ mixed, float* rinv_mid) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int L = sh.L, k = sh.k, D = sh.D, N = sh.N();
  const int kp = (k + JC - 1) / JC * JC;  // padded channel count
  const long n = blockIdx.x;
  T* hs = (T*)smem;
  float* coef = (float*)(smem + ((size_t)L * D * sizeof(T) + 15) / 16 * 16);  // [2][L][kp]
  float* part = coef + 2 * L * kp;                                             // [2 waves][2k]
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

  // The token's L states go to LDS in batches of kMixBatch loads per thread, all in
  // flight together (past the row they read zeros through the buffer view).
  const auto hv = make_view(H + n * L * D, (uint32_t)((long)L * D * sizeof(T)));
  for (int e0 = tid * 8; e0 < L * D; e0 += 128 * 8 * kMixBatch) {
    frag_t<T> v[kMixBatch];
#pragma unroll
    for (int b = 0; b < kMixBatch; ++b) {
      const int e = e0 + b * 128 * 8;
      v[b] = buf_frag<T>(hv, e < L * D ? (uint32_t)e * (uint32_t)sizeof(T) : kOffOob);
    }
#pragma unroll
    for (int b = 0; b < kMixBatch; ++b) {
      const int e = e0 + b * 128 * 8;
      if (e < L * D) st_frag<T>(hs + e, v[b]);
    }
  }
  for (int e = tid; e < 2 * L * kp; e += 128) coef[e] = 0.f;
  __syncthreads();
  if (tid < 2 * k) {
    int br = tid / k, j = tid - br * k;
    const float* row = alpha + ((long)br * N + n) * k * L + (long)j * L;  // final weights
    for (int l = 0; l < L; ++l) coef[((long)br * L + l) * kp + j] = row[l] * rinv[n * L + l];
  }
  __syncthreads();

  const int ncg = D / 8;
  for (int br = 0; br < 2; ++br) {
    for (int j0 = 0; j0 < k; j0 += JC) {
      float ss[JC];
#pragma unroll
      for (int jj = 0; jj < JC; ++jj) ss[jj] = 0.f;
      for (int cg = tid; cg < ncg; cg += 128) {
        float acc[JC][8];
#pragma unroll
        for (int jj = 0; jj < JC; ++jj)
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[jj][i] = 0.f;
        // the next layer's gains are fetched one layer ahead (clamped, so unconditionally)
        const T* gbase = g_pre + (long)br * L * D + cg * 8;
        frag_t<T> gnext = ld_frag<T>(gbase);
        for (int l = 0; l < L; ++l) {
          const frag_t<T> gcur = gnext;
          gnext = ld_frag<T>(gbase + (long)min(l + 1, L - 1) * D);
          float xv[8];
          load8(hs + l * D + cg * 8, xv);
#pragma unroll
          for (int i = 0; i < 8; ++i) xv[i] *= to_f32(gcur[i]);
          const float* cl = coef + ((long)br * L + l) * kp + j0;
#pragma unroll
          for (int jq = 0; jq < JC; jq += 4) {
            f32x4 c4 = *(const f32x4*)(cl + jq);
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
              for (int i = 0; i < 8; ++i) acc[jq + t][i] += c4[t] * xv[i];
          }
        }
#pragma unroll
        for (int jj = 0; jj < JC; ++jj) {
          if (j0 + jj < k) {
            store8(mixed + (((long)br * k + j0 + jj) * N + n) * D + cg * 8, acc[jj]);
#pragma unroll
            for (int i = 0; i < 8; ++i) ss[jj] += acc[jj][i] * acc[jj][i];
          }
        }
      }
#pragma unroll
      for (int jj = 0; jj < JC; ++jj) {
        float v = wave_sum(ss[jj]);
        if (lane == 0 && j0 + jj < k) part[wv * 2 * k + br * k + j0 + jj] = v;
      }
    }
  }
  __syncthreads();
  if (tid < 2 * k) {
    float v = part[tid] + part[2 * k + tid];
    int br = tid / k, j = tid - br * k;
    rinv_mid[((long)br * k + j) * N + n] = 1.0f / sqrtf(v / (float)D + sh.eps);
  }
}

// Channels per pass of the VALU mix: 4 keeps the accumulators small enough for
// several blocks per SIMD (the kernel waits on memory more than it computes).
static int mix_chunk(int) { return 4; }

size_t mix_smem_bytes(int L, int k, int D, size_t es) {
  int jc = mix_chunk(k), kp = (k + jc - 1) / jc * jc;
  return ((size_t)L * D * es + 15) / 16 * 16 + sizeof(float) * (2 * (size_t)L * kp + 4 * k);
}

// ---------------------------------------------------------- mix (MFMA)
// The bf16 mix as a batch of small matrix products on the matrix cores: for
// token n and branch br, mixed^T[e][j] = sum_l Hh[l][e] C[j][l] with
// Hh = g_pre[br] * h_n (rounded to bf16 once, staged in LDS row-major, one row
// per layer) and C[j][l] = alpha[br][n][j][l] / RMS(h_l), split into bf16 hi + lo
// parts so the coefficients keep about 16 significant bits. One 16x16x16 MFMA
// covers 16 states e, 16 channels j and 16 layers; lane group g of its operand
// takes layers 4g .. 4g+3 of its state column, which one transposing LDS read
// (ds_read_b64_tr_b16) gathers from the row-major tile. The staged tile has L
// rows plus one row of zeros that stands in for the layers past L.
// A block of NT threads walks up to kMixTok consecutive tokens; the next token's
// states and coefficients are fetched while the current token's second branch is
// multiplied. NT is 256 when a token's states are at most 1536 chunks of 8 (six per
// thread), else 512, which keeps the registers a thread holds for the prefetch low
// enough for two or more blocks per CU (measured best for L12 D768 and L24 D1024). In softmax mode alpha is normalised beforehand
// (softmax_rows_kernel).
constexpr int kMixTok = 8;
constexpr int kMixCoefMax = 1024;  // coefficient entries 2kL per token at most

__host__ __device__ static int mix_threads(int L, int D) { return L * (D / 8) <= 1536 ? 256 : 512; }

__host__ __device__ static int mix_mfma_ldh(int D) { return D + 16; }  // staged row stride
__host__ __device__ static int mix_coef_ld(int LT) { return 16 * LT + 4; }
static size_t mix_mfma_smem(const Shape& sh) {
  const int JT = (sh.k + 15) / 16, LT = (sh.L + 15) / 16;
  return (size_t)(sh.L + 1) * mix_mfma_ldh(sh.D) * 2 + 2 * 2 * 16 * JT * mix_coef_ld(LT) * 2 +
         (mix_threads(sh.L, sh.D) / 64) * 2 * 16 * JT * 4;
}
static bool mix_mfma_fits(const Shape& sh) {
  // (the kernel stores through a buffer view per branch, which must span under 2 GiB)
  return sh.L <= 32 && sh.k <= 32 && 2 * sh.k * sh.L <= kMixCoefMax && sh.D % 16 == 0 &&
         (long)sh.k * sh.N() * sh.D * 2 < (1L << 31) &&
         mix_mfma_smem(sh) <= 65536;
}

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// EB: column blocks of 16 states per wave and branch (D = 16 waves EB), or 0 for a runtime
// count. With EB fixed every wave issues the same, static sequence of memory operations
// per token (all stores go through buffer views, out-of-range lanes to an offset past
// the view), so the waits for the next token's loads leave the current token's stores
// in flight instead of draining them.
template <int JT, int LT, int NCH, int EB, int NT>
__global__ __launch_bounds__(NT) void mix_mfma_kernel(Shape sh, const bf16* __restrict__ H,
                                                       const float* __restrict__ rinv,
                                                       const bf16* __restrict__ g_pre,
                                                       float* alpha, bf16* __restrict__ mixed,
                                                       float* __restrict__ rinv_mid, int tpb) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int kMixThreads = NT, kMixWaves = NT / 64, kMixCoefPer = kMixCoefMax / NT;
  const int L = sh.L, k = sh.k, D = sh.D, N = sh.N(), kL = k * L;
  const int LDH = mix_mfma_ldh(D), DG = D / 8, chunks = L * DG;
  constexpr int CLD = 16 * LT + 4;
  bf16* Hs = (bf16*)smem;                                     // [L + 1][LDH], row L zero
  bf16* Cs = Hs + (size_t)(L + 1) * LDH;                      // [2 br][2 hi/lo][16 JT][CLD]
  float* part = (float*)(Cs + 2 * 2 * 16 * JT * CLD);         // [waves][2 br][16 JT]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, jj = lane & 15;
  const int n_beg = blockIdx.x * tpb, n_end = min(N, n_beg + tpb);

  // coefficient rows j >= k and slots l >= L, and the zero state row, stay zero
  for (int e = tid; e < 2 * 2 * 16 * JT * CLD; e += kMixThreads) Cs[e] = (bf16)0.f;
  for (int e = tid; e < LDH; e += kMixThreads) Hs[L * LDH + e] = (bf16)0.f;

  // this thread's chunks: c = tid + kMixThreads i -> layer c / DG, states 8 (c % DG) .. + 7
  frag_t<bf16> hv[NCH], gv[NCH];
  uint32_t coff[NCH];  // byte offset of chunk i in an [L][D] array (past the end: out of range)
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    const int c = tid + kMixThreads * i;
    const int l = c / DG, eg = c - l * DG;
    coff[i] = c < chunks ? (uint32_t)(l * D + 8 * eg) * 2u : kOffOob;
  }
  // coefficient entries x = tid + kMixThreads i -> (br, j, l); their LDS slot is fixed
  float av[kMixCoefPer], rv[kMixCoefPer];
  int xin[kMixCoefPer], xcs[kMixCoefPer], xl[kMixCoefPer];
#pragma unroll
  for (int i = 0; i < kMixCoefPer; ++i) {
    const int x = min(tid + kMixThreads * i, 2 * kL - 1);
    const int br = x / kL, jl = x - br * kL, j = jl / L, l = jl - j * L;
    xin[i] = br * N * kL + jl;  // + n * kL
    xcs[i] = ((br * 2) * 16 * JT + j) * CLD + l;
    xl[i] = l;
  }
  const auto gview0 = make_view(g_pre, (uint32_t)((long)L * D * 2));
  const auto gview1 = make_view(g_pre + (long)L * D, (uint32_t)((long)L * D * 2));
  auto fetch = [&](long n) {  // the states and coefficients of token n
    const auto view = make_view(H + n * L * D, (uint32_t)((long)L * D * 2));
#pragma unroll
    for (int i = 0; i < NCH; ++i) hv[i] = buf_frag<bf16>(view, coff[i]);
#pragma unroll
    for (int i = 0; i < kMixCoefPer; ++i) {
      av[i] = alpha[(long)xin[i] + n * kL];
      rv[i] = rinv[n * L + xl[i]];
    }
  };
  auto fetch_gain = [&](const __amdgpu_buffer_rsrc_t& gview) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) gv[i] = buf_frag<bf16>(gview, coff[i]);
  };
  // stage g * h as bf16; chunks past the end land in row 0's padding (columns D .. D+7,
  // never read)
  auto stage = [&]() {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + kMixThreads * i;
      const int l = c / DG, eg = c - l * DG;
      bf16x8 v;
#pragma unroll
      for (int t = 0; t < 8; ++t) v[t] = (bf16)((float)hv[i][t] * (float)gv[i][t]);
      *(bf16x8*)(Hs + (c < chunks ? l * LDH + 8 * eg : D)) = v;
    }
  };
  if (n_beg < n_end) {
    fetch(n_beg);
    fetch_gain(gview0);
  }
  __syncthreads();

  // per-lane LDS byte address of the transposing read: lane j of each 16-lane group
  // addresses layer 16 lt + 4g + j/4 (the zero row past L) at states 4 (j % 4) .. + 3
  // of the block's 16 columns
  uint32_t tr_base[LT];
#pragma unroll
  for (int lt = 0; lt < LT; ++lt) {
    const int row = min(16 * lt + 4 * g + (jj >> 2), L);
    tr_base[lt] = (uint32_t)(uintptr_t)(Hs + row * LDH + 4 * (jj & 3));
  }
  // output views: mixed[br] ([k][N][D]) and rinv_mid; lane rows j >= k store out of range
  const auto mview0 = make_view(mixed, (uint32_t)((long)k * N * D * 2));
  const auto mview1 = make_view(mixed + (long)k * N * D, (uint32_t)((long)k * N * D * 2));
  const auto rview = make_view(rinv_mid, (uint32_t)(2L * k * N * 4));

  // One branch: O[j][e] = sum_l C[j][l] (g h)[l][e] on the matrix cores, stored as bf16,
  // and the wave's sums of squares per channel into part.
  auto branch = [&](const int br, const long n) {
    bf16x4 bh[JT][LT], bl[JT][LT];
    float ss[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
#pragma unroll
      for (int lt = 0; lt < LT; ++lt) {
        const bf16* crow = Cs + ((br * 2) * 16 * JT + 16 * jt + jj) * CLD + 16 * lt + 4 * g;
        bh[jt][lt] = *(const bf16x4*)crow;
        bl[jt][lt] = *(const bf16x4*)(crow + 16 * JT * CLD);
      }
      ss[jt] = 0.f;
    }
    uint32_t moff[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      const int j = 16 * jt + jj;
      moff[jt] = j < k ? (uint32_t)(((long)j * N + n) * D + 4 * g) * 2u : kOffOob;
    }
    auto column = [&](const int eb) {
      bf16x4 a[LT];
#pragma unroll
      for (int lt = 0; lt < LT; ++lt) {
        typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
        const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4*)(uintptr_t)(tr_base[lt] + (uint32_t)(16 * eb) * 2u));
        a[lt] = __builtin_bit_cast(bf16x4, v);
      }
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int lt = 0; lt < LT; ++lt) {
          acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, a[lt]),
                                                         __builtin_bit_cast(i16x4_t, bh[jt][lt]),
                                                         acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, a[lt]),
                                                         __builtin_bit_cast(i16x4_t, bl[jt][lt]),
                                                         acc, 0, 0, 0);
        }
        // acc[t]: state 16 eb + 4 g + t of channel 16 jt + jj
        bf16x4 o;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          o[t] = (bf16)acc[t];
          ss[jt] += acc[t] * acc[t];
        }
        typedef int i32x2_t __attribute__((ext_vector_type(2)));
        __builtin_amdgcn_raw_buffer_store_b64(
            __builtin_bit_cast(i32x2_t, o), br ? mview1 : mview0,
            moff[jt] == kOffOob ? kOffOob : moff[jt] + (uint32_t)(16 * eb) * 2u, 0, 0);
      }
    };
    if constexpr (EB > 0) {
#pragma unroll
      for (int e = 0; e < EB; ++e) {
        column(w + kMixWaves * e);
        // with 8 waves, keep the columns in order (fewer values live at once)
        if constexpr (NT == 512) __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      for (int eb = w; eb < D / 16; eb += kMixWaves) column(eb);
    }
    // sum of squares of channel j over the wave's states: the 4 lane groups hold parts
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      float v = ss[jt];
      v += __shfl_xor(v, 16, 64);
      v += __shfl_xor(v, 32, 64);
      if (g == 0) part[(w * 2 + br) * 16 * JT + 16 * jt + jj] = v;
    }
  };

  for (int n = n_beg; n < n_end; ++n) {
    // coefficients of both branches (alpha is already normalised in softmax mode)
#pragma unroll
    for (int i = 0; i < kMixCoefPer; ++i) {
      if (tid + kMixThreads * i < 2 * kL) {
        const float c = av[i] * rv[i];
        const bf16 ch = (bf16)c;
        Cs[xcs[i]] = ch;
        Cs[xcs[i] + 16 * JT * CLD] = (bf16)(c - (float)ch);
      }
    }
    stage();             // branch 0 (waits for this token's states and the branch-0 gains)
    fetch_gain(gview1);  // issued before branch 0's stores, so its wait leaves them in flight
    __syncthreads();
    branch(0, n);
    __syncthreads();     // Hs is rewritten next
    stage();             // branch 1
    if (n + 1 < n_end) {  // next token's states and branch-0 gains, ahead of branch 1's stores
      fetch(n + 1);
      fetch_gain(gview0);
    }
    __syncthreads();
    branch(1, n);
    __syncthreads();     // Hs is rewritten next; part is complete
    {
      const int br = tid / k, j = tid - br * k;
      float v = 0.f;
      if (tid < 2 * k) {
#pragma unroll
        for (int ww = 0; ww < kMixWaves; ++ww) v += part[(ww * 2 + br) * 16 * JT + j];
      }
      __builtin_amdgcn_raw_buffer_store_b32(
          __float_as_uint(1.0f / sqrtf(v / (float)D + sh.eps)), rview,
          tid < 2 * k ? (uint32_t)(((long)br * k + j) * N + n) * 4u : kOffOob, 0, 0);
    }
  }
}

// Mixing weights from the router logits, per channel row alpha[r][0..L) (r = (br N + n) k
// + j), in place: without feedback the row keeps layers 0..j only (the rest set to 0);
// in softmax mode the kept entries are normalised by a softmax.
__global__ __launch_bounds__(256) void alpha_rows_kernel(float* alpha, long rows, int k, int L,
                                                         int softmax, int nofb) {
  const long r = (long)blockIdx.x * 256 + threadIdx.x;
  if (r >= rows) return;
  float* row = alpha + r * L;
  const int nl = nofb ? (int)(r % k) + 1 : L;
  if (softmax) {
    float mx = row[0];
    for (int l = 1; l < nl; ++l) mx = fmaxf(mx, row[l]);
    float z = 0.f;
    for (int l = 0; l < nl; ++l) z += expf(row[l] - mx);
    const float iz = 1.0f / z;
    for (int l = 0; l < nl; ++l) row[l] = expf(row[l] - mx) * iz;
  }
  for (int l = nl; l < L; ++l) row[l] = 0.f;
}

// The weights the mix applies, from the router output (see alpha_rows_kernel).
static void finish_alpha(const Shape& sh, float* alpha, hipStream_t s) {
  const bool nofb = sh.router_mode == 2;
  if (!sh.mix_softmax && !nofb) return;
  const long rows = 2L * sh.N() * sh.k;
  hipLaunchKernelGGL(alpha_rows_kernel, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s,
                     alpha, rows, sh.k, sh.L, sh.mix_softmax, nofb ? 1 : 0);
}

template <int JT, int LT>
static void mix_mfma_launch(const Shape& sh, const bf16* H, const float* rinv, const bf16* g_pre,
                            float* alpha, bf16* mixed, float* rinv_mid, hipStream_t s) {
  const int nt = mix_threads(sh.L, sh.D);
  const int nch = (sh.L * (sh.D / 8) + nt - 1) / nt;
  // tokens per block: up to kMixTok, fewer when that would leave under ~2048 blocks
  const int tpb = std::max(1, std::min(kMixTok, sh.N() / 2048));
  const dim3 grid((sh.N() + tpb - 1) / tpb), block(nt);
  const size_t smem = mix_mfma_smem(sh);
#define WM_MIX_GO(NC, NT)                                                                      \
  do {                                                                                         \
    if (sh.D == 768)                                                                           \
      hipLaunchKernelGGL((mix_mfma_kernel<JT, LT, NC, 768 / 16 / (NT / 64), NT>), grid, block,  \
                         smem, s, sh, H, rinv, g_pre, alpha, mixed, rinv_mid, tpb);            \
    else if (sh.D == 1024)                                                                     \
      hipLaunchKernelGGL((mix_mfma_kernel<JT, LT, NC, 1024 / 16 / (NT / 64), NT>), grid, block, \
                         smem, s, sh, H, rinv, g_pre, alpha, mixed, rinv_mid, tpb);            \
    else                                                                                       \
      hipLaunchKernelGGL((mix_mfma_kernel<JT, LT, NC, 0, NT>), grid, block, smem, s, sh, H,    \
                         rinv, g_pre, alpha, mixed, rinv_mid, tpb);                            \
  } while (0)
  if (nt == 256) {  // at most 6 chunks per thread
    if (nch <= 2) WM_MIX_GO(2, 256);
    else if (nch <= 4) WM_MIX_GO(4, 256);
    else WM_MIX_GO(6, 256);
  } else {
    if (nch <= 4) WM_MIX_GO(4, 512);
    else if (nch <= 6) WM_MIX_GO(6, 512);
    else if (nch <= 8) WM_MIX_GO(8, 512);
    else if (nch <= 12) WM_MIX_GO(12, 512);
    else WM_MIX_GO(16, 512);
  }
#undef WM_MIX_GO
}

template <typename T>
void launch_mix(const Shape& sh, const T* H, const float* rinv, const T* g_pre, float* alpha,
                T* mixed, float* rinv_mid, hipStream_t s) {
  if (sh.N() <= 0) return;
  finish_alpha(sh, alpha, s);
  if constexpr (sizeof(T) == 2) {
    if (mix_mfma_fits(sh)) {
      const bool jt1 = sh.k <= 16, lt1 = sh.L <= 16;
      if (jt1 && lt1) mix_mfma_launch<1, 1>(sh, H, rinv, g_pre, alpha, mixed, rinv_mid, s);
      else if (jt1) mix_mfma_launch<1, 2>(sh, H, rinv, g_pre, alpha, mixed, rinv_mid, s);
      else if (lt1) mix_mfma_launch<2, 1>(sh, H, rinv, g_pre, alpha, mixed, rinv_mid, s);
      else mix_mfma_launch<2, 2>(sh, H, rinv, g_pre, alpha, mixed, rinv_mid, s);
      return;
    }
  }
  size_t smem = mix_smem_bytes(sh.L, sh.k, sh.D, sizeof(T));
  dim3 grid(sh.N()), block(128);
  switch (mix_chunk(sh.k)) {
    case 4: hipLaunchKernelGGL((mix_kernel<T, 4>), grid, block, smem, s, sh, H, rinv, g_pre, alpha, mixed, rinv_mid); break;
    case 8: hipLaunchKernelGGL((mix_kernel<T, 8>), grid, block, smem, s, sh, H, rinv, g_pre, alpha, mixed, rinv_mid); break;
    case 12: hipLaunchKernelGGL((mix_kernel<T, 12>), grid, block, smem, s, sh, H, rinv, g_pre, alpha, mixed, rinv_mid); break;
    default: hipLaunchKernelGGL((mix_kernel<T, 16>), grid, block, smem, s, sh, H, rinv, g_pre, alpha, mixed, rinv_mid); break;
  }
}

// ------------------------------------------------------------- projections
// Fold an RMSNorm gain into the weights that consume the normed vector:
// Wf[grp][o][e] = W[grp][o][e] * gain[grp][e]; the row's 1/RMS is applied in the
// GEMM epilogue. The K/V projections take two source tensors (groups [0, split)
// from W0 = W^K, the rest from W1 = W^V).
template <typename T>
__global__ __launch_bounds__(256) void fold_gain_kernel(const T* W0, const T* W1, int split,
                                                        const T* gain, T* Wf, int Nout, int K) {
  // one group per grid row; 32-bit offsets within it (a group holds under 2^31 elements)
  const int grp = blockIdx.y;
  const uint32_t per = (uint32_t)Nout * (uint32_t)K;
  const uint32_t idx = (blockIdx.x * 256u + threadIdx.x) * 8u;
  if (idx >= per) return;
  const uint32_t e = idx % (uint32_t)K;
  const T* src = grp < split ? W0 + (long)grp * per : W1 + (long)(grp - split) * per;
  float wv[8], gv[8];
  load8(src + idx, wv);
  load8(gain + (long)grp * K + e, gv);
#pragma unroll
  for (int i = 0; i < 8; ++i) wv[i] *= gv[i];
  store8(Wf + (long)grp * per + idx, wv);
}

template <typename T>
static void fold_gain(const T* W0, const T* W1, int split, const T* gain, T* Wf, int groups,
                      int Nout, int K, hipStream_t s) {
  const long per = (long)Nout * K;  // K is a multiple of 8
  if (per <= 0 || groups <= 0) return;
  hipLaunchKernelGGL(fold_gain_kernel<T>, dim3((unsigned)((per / 8 + 255) / 256), (unsigned)groups),
                     dim3(256), 0, s, W0, W1, split, gain, Wf, Nout, K);
}

// folded weights, then the epilogue's trash area
size_t kv_fold_elems(const Shape& sh) { return 2ul * sh.k * sh.Hkv * sh.d * sh.D + kTrashElems; }
size_t q_fold_elems(const Shape& sh) { return (size_t)sh.L * sh.Hq * sh.d * sh.D + kTrashElems; }

template <typename T, int DH, bool FEW>
static void kv_gemm(const Shape& sh, const T* mixed, const float* rinv_mid, const T* wfold,
                    const T* g_knorm, const float* rope_tab, const int32_t* ctx_len, T* Kc, T* Vc,
                    hipStream_t s) {
  using C = typename ProjShapeD<T, FEW, DH, false>::C;
  const int M = sh.N(), Nout = sh.Hkv * DH, K = sh.D;
  PlainRows<T> x{mixed, (long)M * K, K, M};
  PlainRows<T> w{wfold, (long)Nout * K, K, Nout};
  T* trash = const_cast<T*>(wfold) + (kv_fold_elems(sh) - kTrashElems);
  KVEpi<T, DH> e{Kc, Vc, trash, rinv_mid, g_knorm, rope_tab, ctx_len, M, sh.T_new, sh.B,
                 sh.Hkv, sh.S_cap, sh.k, sh.gs, sh.gq, sh.ctx_hi, sh.eps};
  launch_proj<C, T>(M, Nout, K, 2 * sh.k, kNoSegments, 0, x, w, e, s);
}

template <typename T>
void launch_kv_fold(const Shape& sh, const T* g_mid, const T* Wk, const T* Wv, T* wfold,
                    hipStream_t s) {
  fold_gain<T>(Wk, Wv, sh.k, g_mid, wfold, 2 * sh.k, sh.Hkv * sh.d, sh.D, s);
}

template <typename T>
void launch_kv_project(const Shape& sh, const T* mixed, const float* rinv_mid, const T* g_mid,
                       const T* Wk, const T* Wv, const T* g_knorm, const float* rope_tab,
                       const int32_t* ctx_len, T* Kc, T* Vc, T* wfold, hipStream_t s,
                       bool prefolded) {
  const int M = sh.N();
  if (M <= 0) return;
  if (!prefolded) launch_kv_fold<T>(sh, g_mid, Wk, Wv, wfold, s);
  const bool few = M <= kFewTokens;
  if (sh.d == 96) {
    if constexpr (sizeof(T) == 2) {  // fp32 at d = 96 is rejected by validation
      if (few) kv_gemm<T, 96, true>(sh, mixed, rinv_mid, wfold, g_knorm, rope_tab, ctx_len, Kc, Vc, s);
      else kv_gemm<T, 96, false>(sh, mixed, rinv_mid, wfold, g_knorm, rope_tab, ctx_len, Kc, Vc, s);
    }
  } else if (sh.d == 64) {
    if (few) kv_gemm<T, 64, true>(sh, mixed, rinv_mid, wfold, g_knorm, rope_tab, ctx_len, Kc, Vc, s);
    else kv_gemm<T, 64, false>(sh, mixed, rinv_mid, wfold, g_knorm, rope_tab, ctx_len, Kc, Vc, s);
  } else {
    if (few) kv_gemm<T, 32, true>(sh, mixed, rinv_mid, wfold, g_knorm, rope_tab, ctx_len, Kc, Vc, s);
    else kv_gemm<T, 32, false>(sh, mixed, rinv_mid, wfold, g_knorm, rope_tab, ctx_len, Kc, Vc, s);
  }
}

// Layers l0 .. l0 + nl - 1; wfold holds the folded weights of all L layers (layer l at
// l * Hq d * D) followed by the trash area; Q receives [nl][B][Hq][T_new][d].
template <typename T, int DH, bool FEW>
static void q_gemm(const Shape& sh, const T* H, const float* rinv, const T* wfold,
                   const T* g_qnorm, const float* rope_tab, T* Q, int l0, int nl, hipStream_t s) {
  using C = typename ProjShapeD<T, FEW, DH, true>::C;
  const int M = sh.N(), Nout = sh.Hq * DH, K = sh.D;
  PlainRows<T> x{H + (long)l0 * K, K, (long)sh.L * K, M};
  PlainRows<T> w{wfold + (long)l0 * Nout * K, (long)Nout * K, K, Nout};
  T* trash = const_cast<T*>(wfold) + (q_fold_elems(sh) - kTrashElems);
  QEpi<T, DH> e{Q, trash, rinv, g_qnorm, rope_tab, M, sh.T_new, sh.B, sh.Hq, sh.L, l0, sh.eps};
  launch_proj<C, T>(M, Nout, K, nl, kNoSegments, 0, x, w, e, s);
}

template <typename T>
void launch_q_fold(const Shape& sh, const T* g_in, const T* Wq, T* wfold, int l0, int nl,
                   hipStream_t s) {
  const long per = (long)sh.Hq * sh.d * sh.D;
  fold_gain<T>(Wq + l0 * per, Wq + l0 * per, nl, g_in + (long)l0 * sh.D, wfold + l0 * per, nl,
               sh.Hq * sh.d, sh.D, s);
}

template <typename T>
void launch_q_layers(const Shape& sh, const T* H, const float* rinv, const T* g_qnorm,
                     const float* rope_tab, T* Q, const T* wfold, int l0, int nl,
                     hipStream_t s) {
  const int M = sh.N();
  if (M <= 0 || nl <= 0) return;
  // few tokens, or a grid of large tiles that would not cover the chip: small tiles
  using CL = typename ProjShape<T, false>::C;
  const long big = (long)nl * ((M + CL::NTOK - 1) / CL::NTOK) *
                   ((sh.Hq * sh.d + CL::OT - 1) / CL::OT);
  const bool few = M <= kFewTokens || big < 128;
  if (sh.d == 96) {
    if constexpr (sizeof(T) == 2) {
      if (few) q_gemm<T, 96, true>(sh, H, rinv, wfold, g_qnorm, rope_tab, Q, l0, nl, s);
      else q_gemm<T, 96, false>(sh, H, rinv, wfold, g_qnorm, rope_tab, Q, l0, nl, s);
    }
  } else if (sh.d == 64) {
    if (few) q_gemm<T, 64, true>(sh, H, rinv, wfold, g_qnorm, rope_tab, Q, l0, nl, s);
    else q_gemm<T, 64, false>(sh, H, rinv, wfold, g_qnorm, rope_tab, Q, l0, nl, s);
  } else {
    if (few) q_gemm<T, 32, true>(sh, H, rinv, wfold, g_qnorm, rope_tab, Q, l0, nl, s);
    else q_gemm<T, 32, false>(sh, H, rinv, wfold, g_qnorm, rope_tab, Q, l0, nl, s);
  }
}

template <typename T>
void launch_q_project(const Shape& sh, const T* H, const float* rinv, const T* g_in,
                      const T* Wq, const T* g_qnorm, const float* rope_tab, T* Q, T* wfold,
                      hipStream_t s) {
  if (sh.N() <= 0) return;
  launch_q_fold<T>(sh, g_in, Wq, wfold, 0, sh.L, s);
  launch_q_layers<T>(sh, H, rinv, g_qnorm, rope_tab, Q, wfold, 0, sh.L, s);
}

// ------------------------------------------------- pass driver (Section 3.3)
// The stand-in for the rest of a decoder block: h_{l+1} = h_l + W_o[l] o_l (output
// projection and residual of the attention sublayer). GEMM C^T = W_o o_l^T; lane (h, r)
// of a 32 x 32 block holds token n and output channels o = 32 i + 8 (q/4) + 4h + q%4,
// 4 consecutive channels per register quad, added to h_l and stored 4 at a time.
template <typename T> __device__ __forceinline__ void load4(const T* p, float* out);
template <> __device__ __forceinline__ void load4<bf16>(const bf16* p, float* out) {
  const bf16x4 v = *(const bf16x4*)p;
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = (float)v[i];
}
template <> __device__ __forceinline__ void load4<float>(const float* p, float* out) {
  const f32x4 v = *(const f32x4*)p;
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = v[i];
}

template <typename T> struct ResidEpi {
  static constexpr bool kUsesLds = false;
  const T* h;   // h_l, row n at h + n * hs
  T* out;       // h_{l+1}, row n at out + n * os
  long hs, os;
  int M, Nout;
  using State = NoState;
  template <class C> __device__ void begin(int, int, int, State&) const {}
  template <class C>
  __device__ void segment(int, int, int, f32x16 (&)[C::WO][C::WN], int, State&) const {}
  template <class C>
  __device__ void finish(int, int ow0, int nw0, f32x16 (&acc)[C::WO][C::WN], int lane, State&,
                         const EpiLds&) const {
    const int hh = lane >> 5, r = lane & 31;
#pragma unroll
    for (int jn = 0; jn < C::WN; ++jn) {
      const int n = nw0 + 32 * jn + r;
      if (n >= M) continue;
#pragma unroll
      for (int i = 0; i < C::WO; ++i)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int o = ow0 + 32 * i + 8 * q4 + 4 * hh;
          if (o >= Nout) continue;
          float v[4];
          load4<T>(h + (long)n * hs + o, v);
#pragma unroll
          for (int t = 0; t < 4; ++t) v[t] += acc[i][jn][4 * q4 + t];
          store4(out + (long)n * os + o, v);
        }
    }
  }
};

template <typename T>
void launch_block_residual(int M, int D, int HD, const T* o_l, const T* W, const T* h, long hs,
                           T* out, long os, hipStream_t s) {
  if (M <= 0) return;
  PlainRows<T> x{o_l, 0, HD, M};
  PlainRows<T> w{W, 0, HD, D};
  ResidEpi<T> e{h, out, hs, os, M, D};
  using CL = typename ProjShape<T, false>::C;
  using CS = typename ProjShape<T, true>::C;
  const long big = (long)((M + CL::NTOK - 1) / CL::NTOK) * ((D + CL::OT - 1) / CL::OT);
  if (big >= 128) launch_proj<CL, T>(M, D, HD, 1, kNoSegments, 0, x, w, e, s);
  else launch_proj<CS, T>(M, D, HD, 1, kNoSegments, 0, x, w, e, s);
}

// The pass driver keeps the states of a group contiguous: Hg[q][b][m][l][e] is the state
// entering layer l at position i = q + g m of sequence b (T a multiple of g, Tg = T / g).
// gather: Hg[q][b][m][l] = X[b][i] for every layer l (H^(0): each token's embedding).
template <typename T>
__global__ __launch_bounds__(256) void group_gather_kernel(const T* X, T* Hg, int B, int T_len,
                                                           int g, int L, int D) {
  const int Tg = T_len / g, c8 = D / 8;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)B * T_len * L * c8) return;
  long r = idx;
  const int e = (int)(r % c8) * 8;
  r /= c8;
  r /= L;  // the layer: every layer gets the same state
  const int m = (int)(r % Tg);
  r /= Tg;
  const int b = (int)(r % B), q = (int)(r / B);
  st_frag<T>(Hg + idx * 8, ld_frag<T>(X + ((long)b * T_len + q + (long)g * m) * D + e));
}
// scatter: Y[b][i][row] = Yg[q][b][m][row] for rows of R * D elements (R = L for the
// states, 1 for the top states).
template <typename T>
__global__ __launch_bounds__(256) void group_scatter_kernel(const T* Yg, T* Y, int B, int T_len,
                                                            int g, long row) {
  const int Tg = T_len / g;
  const long c8 = row / 8;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)B * T_len * c8) return;
  long r = idx;
  const long e = (r % c8) * 8;
  r /= c8;
  const int m = (int)(r % Tg);
  r /= Tg;
  const int b = (int)(r % B), q = (int)(r / B);
  st_frag<T>(Y + ((long)b * T_len + q + (long)g * m) * row + e, ld_frag<T>(Yg + idx * 8));
}

template <typename T>
void launch_group_gather(const T* X, T* Hg, int B, int T_len, int g, int L, int D,
                         hipStream_t s) {
  const long n = (long)B * T_len * L * (D / 8);
  if (n <= 0) return;
  hipLaunchKernelGGL(group_gather_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     X, Hg, B, T_len, g, L, D);
}
template <typename T>
void launch_group_scatter(const T* Yg, T* Y, int B, int T_len, int g, long row, hipStream_t s) {
  const long n = (long)B * T_len * (row / 8);
  if (n <= 0) return;
  hipLaunchKernelGGL(group_scatter_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     Yg, Y, B, T_len, g, row);
}

#define WM_INST(T)                                                                             \
  template void launch_row_rms<T>(const T*, long, int, float, float*, hipStream_t);            \
  template void launch_row_rms_strided<T>(const T*, long, int, long, long, float, float*,      \
                                          hipStream_t);                                        \
  template void launch_router_fold<T>(const Shape&, const LayerTable&, const T*, const T*, T*, \
                                      hipStream_t);                                            \
  template void launch_router<T>(const Shape&, const LayerTable&, const T*, const float*,      \
                                 const T*, const T*, const T*, float*, T*, float*,             \
                                 hipStream_t, bool);                                           \
  template void launch_mix<T>(const Shape&, const T*, const float*, const T*, float*, T*,      \
                              float*, hipStream_t);                                            \
  template void launch_kv_fold<T>(const Shape&, const T*, const T*, const T*, T*, hipStream_t); \
  template void launch_kv_project<T>(const Shape&, const T*, const float*, const T*, const T*, \
                                     const T*, const T*, const float*, const int32_t*, T*, T*, \
                                     T*, hipStream_t, bool);                                   \
  template void launch_q_fold<T>(const Shape&, const T*, const T*, T*, int, int, hipStream_t); \
  template void launch_q_layers<T>(const Shape&, const T*, const float*, const T*,             \
                                   const float*, T*, const T*, int, int, hipStream_t);         \
  template void launch_q_project<T>(const Shape&, const T*, const float*, const T*, const T*,  \
                                    const T*, const float*, T*, T*, hipStream_t);              \
  template void launch_block_residual<T>(int, int, int, const T*, const T*, const T*, long,    \
                                         T*, long, hipStream_t);                               \
  template void launch_group_gather<T>(const T*, T*, int, int, int, int, int, hipStream_t);    \
  template void launch_group_scatter<T>(const T*, T*, int, int, int, long, hipStream_t);
WM_INST(float)
WM_INST(bf16)
#undef WM_INST

}  // namespace wm
