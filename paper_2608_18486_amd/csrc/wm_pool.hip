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
#include "wm_gemm.hpp"
#include "wm_internal.hpp"

namespace wm {

// ----------------------------------------------------------------- row rms
template <typename T>
__global__ __launch_bounds__(256) void row_rms_kernel(const T* X, long rows, int D, float eps,
                                                      float* rinv) {
  long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const T* x = X + row * D;
  float ss = 0.f;
  for (int e = lane * 8; e < D; e += 512) {
    float v[8];
    load8(x + e, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += v[i] * v[i];
  }
  ss = wave_sum(ss);
  if (lane == 0) rinv[row] = 1.0f / sqrtf(ss / (float)D + eps);
}

template <typename T>
void launch_row_rms(const T* X, long rows, int D, float eps, float* rinv, hipStream_t s) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(row_rms_kernel<T>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, X,
                     rows, D, eps, rinv);
}

// -------------------------------------------------------------- rope table
__global__ __launch_bounds__(256) void rope_table_kernel(const int32_t* ctx_len, int B,
                                                         int T_new, int d, double theta,
                                                         float* tab) {
  int half = d / 2;
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)B * T_new * half) return;
  int m = (int)(idx % half);
  long n = idx / half;
  int b = (int)(n / T_new), i = (int)(n % T_new);
  double pos = (double)((ctx_len ? ctx_len[b] : 0) + i);
  double freq = pow(theta, -2.0 * (double)m / (double)d);
  double sn, cs;
  sincos(pos * freq, &sn, &cs);
  tab[2 * idx] = (float)cs;
  tab[2 * idx + 1] = (float)sn;
}

void launch_rope_table(const Shape& sh, const int32_t* ctx_len, float* tab, hipStream_t s) {
  long total = (long)sh.N() * (sh.d / 2);
  if (total <= 0) return;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     ctx_len, sh.B, sh.T_new, sh.d, (double)sh.rope_theta, tab);
}

static unsigned gemm_blocks(int M, int Nout, int groups) {
  return (unsigned)(groups * ((M + 127) / 128) * ((Nout + 127) / 128));
}

// -------------------------------------------------------- GEMM functors
// Weight matrices W + g * group_stride, [Nout][K] each.
template <typename T> struct WeightRows {
  const T* W;
  long group_stride;
  int Nout, K;
  __device__ WeightView<T> view(int g) const {
    return {make_view(W + (long)g * group_stride, (uint32_t)((long)Nout * K * sizeof(T)))};
  }
};

// Router operand: the stacked normed states xi (gain and 1/RMS applied, one rounding).
// Rows past M read zeros (their 1/RMS index is clamped to a valid row).
template <typename T> struct RouterA {
  const T* H;
  const float* rinv;
  const T* g_pre;
  LayerTable sel;
  int L, D, M;
  struct State {
    __amdgpu_buffer_rsrc_t h;
    const T* g;
  };
  __device__ State begin(int br) const {
    return {make_view(H, (uint32_t)((long)M * L * D * sizeof(T))), g_pre + (long)br * L * D};
  }
  __device__ void load(const State& st, int n, int k, bool ok, frag_t<T>* out) const {
    const int m = k / D, e = k - m * D, layer = sel.v[m];
    const uint32_t off = ok ? (uint32_t)(((long)n * L + layer) * D + e) * sizeof(T) : kOffOob;
    const T* g = st.g + (long)layer * D + e;
    const float rs = rinv[(long)min(n, M - 1) * L + layer];
#pragma unroll
    for (int f = 0; f < GemmCfg<T>::FR; ++f) {
      frag_t<T> x = buf_frag<T>(st.h, off + 8 * f * sizeof(T));
      float gv[8];
      load8(g + 8 * f, gv);
#pragma unroll
      for (int i = 0; i < 8; ++i) out[f][i] = from_f32<T>(to_f32(x[i]) * gv[i] * rs);
    }
  }
};

// Plain operand rows: X[g * gstride + row * rstride + k] for rows < M (scales live elsewhere).
template <typename T> struct CopyRowsA {
  const T* X;
  long gstride, rstride;
  int M;
  __device__ __amdgpu_buffer_rsrc_t begin(int g) const {
    return make_view(X + (long)g * gstride, (uint32_t)((long)M * rstride * sizeof(T)));
  }
  __device__ void load(const __amdgpu_buffer_rsrc_t& r, int row, int k, bool ok,
                       frag_t<T>* out) const {
    const uint32_t off = ok ? (uint32_t)((long)row * rstride + k) * sizeof(T) : kOffOob;
#pragma unroll
    for (int f = 0; f < GemmCfg<T>::FR; ++f) out[f] = buf_frag<T>(r, off + 8 * f * sizeof(T));
  }
};

template <typename T> struct RouterEpi {
  float* logits;
  const T* bias;
  int M, Nout;
  __device__ void operator()(int br, int m0, int n0, const float* C, int ldc, int tid) const {
    int col = tid & 127, o = n0 + col;
    if (o >= Nout) return;
    float b = to_f32(bias[(long)br * Nout + o]);
    for (int row = tid >> 7; row < 128; row += 2) {
      int n = m0 + row;
      if (n >= M) break;
      logits[((long)br * M + n) * Nout + o] = C[row * ldc + col] + b;
    }
  }
};

// Head-wise epilogue shared by the K/V and Q projections. A C tile row holds
// 128 / d heads; d / 8 consecutive lanes own one (row, head) item, 8 contiguous
// elements each, so a lane group reads its row from LDS without bank conflicts
// and writes the whole d-element head row (one 128-B line for d = 64) at once.
// Per item: scale by the row's 1/RMS, then either store (V) or RMS-normalise
// over the head, apply the gain and rotate the pairs (m, m + d/2) (K, Q); the
// partner of element m lives d/16 lanes away.
template <typename T, int DH> struct HeadItems {
  static constexpr int LPI = DH / 8;          // lanes per item
  static constexpr int IPP = 256 / LPI;       // items per pass of 256 threads
  static constexpr int ITEMS = 128 * (128 / DH);
};

template <int LPI>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int x = 1; x < LPI; x <<= 1) v += __shfl_xor(v, x, 64);
  return v;
}

// c: this lane's 8 fp32 values; sc: row scale; normalise+rotate when gain != nullptr.
template <typename T, int DH>
__device__ __forceinline__ void head_chunk(float* c, float sc, const T* gain, const float* tabrow,
                                           int lane_c, float eps, T* dst) {
  constexpr int LPI = DH / 8;
#pragma unroll
  for (int i = 0; i < 8; ++i) c[i] *= sc;
  if (gain) {
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += c[i] * c[i];
    ss = group_sum<LPI>(ss);
    const float rs = 1.0f / sqrtf(ss / (float)DH + eps);
    float gv[8];
    load8(gain + 8 * lane_c, gv);
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] *= rs * gv[i];
    // pair (m, m + DH/2): lanes c < LPI/2 hold m, lanes c >= LPI/2 hold m + DH/2
    const bool lo = lane_c < LPI / 2;
    const int mc = lo ? lane_c : lane_c - LPI / 2;  // which 8 pairs
    float cs[8], sn[8];
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      f32x4 t = *(const f32x4*)(tabrow + 2 * (8 * mc + i));
      cs[i] = t[0];
      sn[i] = t[1];
      cs[i + 1] = t[2];
      sn[i + 1] = t[3];
    }
    float y[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float other = __shfl_xor(c[i], LPI / 2, 64);
      // lo: x1 = c, x2 = other -> x1 cos - x2 sin;  hi: x2 = c, x1 = other -> x2 cos + x1 sin
      y[i] = lo ? c[i] * cs[i] - other * sn[i] : c[i] * cs[i] + other * sn[i];
    }
    store8(dst, y);
  } else {
    store8(dst, c);
  }
}

template <typename T> struct KVEpi {
  T *Kc, *Vc;
  const float* rs;  // [2k][M] 1 / RMS of each mixed channel row (the mid RMSNorm)
  const T* g_knorm;
  const float* tab;
  const int32_t* ctx_len;
  int M, Nout, d, T_new, B, Hkv, S_cap, k;
  float eps;
  template <int DH>
  __device__ void run(int g, int m0, int n0, const float* C, int ldc, int tid) const {
    using HI = HeadItems<T, DH>;
    const int br = g / k, j = g - br * k;
    const int lane_c = tid % HI::LPI;
    for (int it = tid / HI::LPI; it < HI::ITEMS; it += HI::IPP) {
      const int row = it & 127, hh = it >> 7;
      const int n = m0 + row, col0 = n0 + hh * DH;
      if (n >= M || col0 >= Nout) continue;
      const int b = n / T_new, i = n - b * T_new;
      const long slot = (long)(ctx_len ? ctx_len[b] : 0) + i;
      if (slot < 0 || slot >= S_cap) continue;
      const int head = col0 / DH;
      const long off = ((((long)j * B + b) * Hkv + head) * S_cap + slot) * DH + 8 * lane_c;
      float c[8];
      const float* src = C + row * ldc + hh * DH + 8 * lane_c;
      *(f32x4*)c = *(const f32x4*)src;
      *(f32x4*)(c + 4) = *(const f32x4*)(src + 4);
      head_chunk<T, DH>(c, rs[(long)g * M + n], br == 0 ? g_knorm + (long)j * DH : nullptr,
                        tab + (long)n * DH, lane_c, eps, (br == 0 ? Kc : Vc) + off);
    }
  }
  __device__ void operator()(int g, int m0, int n0, const float* C, int ldc, int tid) const {
    if (d == 64) run<64>(g, m0, n0, C, ldc, tid);
    else run<32>(g, m0, n0, C, ldc, tid);
  }
};

template <typename T> struct QEpi {
  T* Q;
  const float* rs;  // [M][L] 1 / RMS of each consumer's input state (the input RMSNorm)
  const T* g_qnorm;
  const float* tab;
  int M, Nout, d, T_new, B, Hq, L;
  float eps;
  template <int DH>
  __device__ void run(int l, int m0, int n0, const float* C, int ldc, int tid) const {
    using HI = HeadItems<T, DH>;
    const int lane_c = tid % HI::LPI;
    for (int it = tid / HI::LPI; it < HI::ITEMS; it += HI::IPP) {
      const int row = it & 127, hh = it >> 7;
      const int n = m0 + row, col0 = n0 + hh * DH;
      if (n >= M || col0 >= Nout) continue;
      const int b = n / T_new, i = n - b * T_new, head = col0 / DH;
      const long off = ((((long)l * B + b) * Hq + head) * T_new + i) * DH + 8 * lane_c;
      float c[8];
      const float* src = C + row * ldc + hh * DH + 8 * lane_c;
      *(f32x4*)c = *(const f32x4*)src;
      *(f32x4*)(c + 4) = *(const f32x4*)(src + 4);
      head_chunk<T, DH>(c, rs[(long)n * L + l], g_qnorm + (long)l * DH, tab + (long)n * DH,
                        lane_c, eps, Q + off);
    }
  }
  __device__ void operator()(int l, int m0, int n0, const float* C, int ldc, int tid) const {
    if (d == 64) run<64>(l, m0, n0, C, ldc, tid);
    else run<32>(l, m0, n0, C, ldc, tid);
  }
};

// ------------------------------------------------------------------ router
template <typename T>
void launch_router(const Shape& sh, const LayerTable& sel, const T* H, const float* rinv,
                   const T* g_pre, const T* W_alpha, const T* b_alpha, float* logits,
                   hipStream_t s) {
  int M = sh.N(), Nout = sh.k * sh.L, K = sh.Lp * sh.D;
  if (M <= 0) return;
  RouterA<T> a{H, rinv, g_pre, sel, sh.L, sh.D, M};
  WeightRows<T> w{W_alpha, (long)Nout * K, Nout, K};
  RouterEpi<T> e{logits, b_alpha, M, Nout};
  hipLaunchKernelGGL((gemm_nt_kernel<T, RouterA<T>, WeightRows<T>, RouterEpi<T>>),
                     dim3(gemm_blocks(M, Nout, 2)), dim3(256), 0, s, M, Nout, K, 2, a, w, e);
}

// --------------------------------------------------------------------- mix
// One block per token; each thread owns 8 consecutive columns. LDS holds the
// token's L states and the coefficients alpha[j][l] / RMS(h_l), stored layer-
// major with the channel count padded to JC (zeros), so a thread reads JC
// coefficients of one layer with JC/4 broadcast loads. For each branch the
// thread scales a layer's 8 columns by the gain once and accumulates them into
// all JC channels, then stores the channels and their sums of squares.
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

  const T* hsrc = H + n * L * D;
  for (int e = tid * 8; e < L * D; e += 128 * 8) st_frag<T>(hs + e, ld_frag<T>(hsrc + e));
  for (int e = tid; e < 2 * L * kp; e += 128) coef[e] = 0.f;
  __syncthreads();
  if (tid < 2 * k) {
    int br = tid / k, j = tid - br * k;
    float* row = alpha + ((long)br * N + n) * k * L + (long)j * L;
    if (sh.mix_softmax) {
      float mx = row[0];
      for (int l = 1; l < L; ++l) mx = fmaxf(mx, row[l]);
      float z = 0.f;
      for (int l = 0; l < L; ++l) z += expf(row[l] - mx);
      float iz = 1.0f / z;
      for (int l = 0; l < L; ++l) row[l] = expf(row[l] - mx) * iz;
    }
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

static int mix_chunk(int k) { return k <= 4 ? 4 : k <= 8 ? 8 : k <= 12 ? 12 : 16; }

size_t mix_smem_bytes(int L, int k, int D, size_t es) {
  int jc = mix_chunk(k), kp = (k + jc - 1) / jc * jc;
  return ((size_t)L * D * es + 15) / 16 * 16 + sizeof(float) * (2 * (size_t)L * kp + 4 * k);
}

template <typename T>
void launch_mix(const Shape& sh, const T* H, const float* rinv, const T* g_pre, float* alpha,
                T* mixed, float* rinv_mid, hipStream_t s) {
  if (sh.N() <= 0) return;
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
                                                        const T* gain, T* Wf, int groups,
                                                        int Nout, int K) {
  long idx = ((long)blockIdx.x * 256 + threadIdx.x) * 8;
  long per = (long)Nout * K;
  if (idx >= per * groups) return;
  int grp = (int)(idx / per);
  long rem = idx - (long)grp * per;
  int e = (int)(rem % K);
  const T* src = grp < split ? W0 + (long)grp * per + rem : W1 + (long)(grp - split) * per + rem;
  float wv[8], gv[8];
  load8(src, wv);
  load8(gain + (long)grp * K + e, gv);
#pragma unroll
  for (int i = 0; i < 8; ++i) wv[i] *= gv[i];
  store8(Wf + idx, wv);
}

template <typename T>
static void fold_gain(const T* W0, const T* W1, int split, const T* gain, T* Wf, int groups,
                      int Nout, int K, hipStream_t s) {
  long total = (long)groups * Nout * K / 8;
  hipLaunchKernelGGL(fold_gain_kernel<T>, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     W0, W1, split, gain, Wf, groups, Nout, K);
}

size_t kv_fold_elems(const Shape& sh) { return 2ul * sh.k * sh.Hkv * sh.d * sh.D; }
size_t q_fold_elems(const Shape& sh) { return (size_t)sh.L * sh.Hq * sh.d * sh.D; }

template <typename T>
void launch_kv_project(const Shape& sh, const T* mixed, const float* rinv_mid, const T* g_mid,
                       const T* Wk, const T* Wv, const T* g_knorm, const float* rope_tab,
                       const int32_t* ctx_len, T* Kc, T* Vc, T* wfold, hipStream_t s) {
  int M = sh.N(), Nout = sh.Hkv * sh.d, K = sh.D;
  if (M <= 0) return;
  fold_gain<T>(Wk, Wv, sh.k, g_mid, wfold, 2 * sh.k, Nout, K, s);
  CopyRowsA<T> a{mixed, (long)M * K, K, M};
  WeightRows<T> w{wfold, (long)Nout * K, Nout, K};
  KVEpi<T> e{Kc, Vc, rinv_mid, g_knorm, rope_tab, ctx_len, M, Nout, sh.d, sh.T_new, sh.B,
             sh.Hkv, sh.S_cap, sh.k, sh.eps};
  hipLaunchKernelGGL((gemm_nt_kernel<T, CopyRowsA<T>, WeightRows<T>, KVEpi<T>>),
                     dim3(gemm_blocks(M, Nout, 2 * sh.k)), dim3(256), 0, s, M, Nout, K, 2 * sh.k,
                     a, w, e);
}

template <typename T>
void launch_q_project(const Shape& sh, const T* H, const float* rinv, const T* g_in,
                      const T* Wq, const T* g_qnorm, const float* rope_tab, T* Q, T* wfold,
                      hipStream_t s) {
  int M = sh.N(), Nout = sh.Hq * sh.d, K = sh.D;
  if (M <= 0) return;
  fold_gain<T>(Wq, Wq, sh.L, g_in, wfold, sh.L, Nout, K, s);
  CopyRowsA<T> a{H, K, (long)sh.L * K, M};
  WeightRows<T> w{wfold, (long)Nout * K, Nout, K};
  QEpi<T> e{Q, rinv, g_qnorm, rope_tab, M, Nout, sh.d, sh.T_new, sh.B, sh.Hq, sh.L, sh.eps};
  hipLaunchKernelGGL((gemm_nt_kernel<T, CopyRowsA<T>, WeightRows<T>, QEpi<T>>),
                     dim3(gemm_blocks(M, Nout, sh.L)), dim3(256), 0, s, M, Nout, K, sh.L, a, w, e);
}

#define WM_INST(T)                                                                             \
  template void launch_row_rms<T>(const T*, long, int, float, float*, hipStream_t);            \
  template void launch_router<T>(const Shape&, const LayerTable&, const T*, const float*,      \
                                 const T*, const T*, const T*, float*, hipStream_t);           \
  template void launch_mix<T>(const Shape&, const T*, const float*, const T*, float*, T*,      \
                              float*, hipStream_t);                                            \
  template void launch_kv_project<T>(const Shape&, const T*, const float*, const T*, const T*, \
                                     const T*, const T*, const float*, const int32_t*, T*, T*, \
                                     T*, hipStream_t);                                         \
  template void launch_q_project<T>(const Shape&, const T*, const float*, const T*, const T*,  \
                                    const T*, const float*, T*, T*, hipStream_t);
WM_INST(float)
WM_INST(bf16)
#undef WM_INST

}  // namespace wm
