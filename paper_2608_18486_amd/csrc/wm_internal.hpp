// Internal launch interface between the C-ABI host layer and the kernels.
// All launches are asynchronous on the given stream; shapes are validated by
// the caller (wm_api.cpp) before any launch.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace wm {

typedef __bf16 bf16;
constexpr int kMaxLayers = 64;  // L limit (kernel-argument tables are sized by it)
constexpr int kMaxHeadDim = 96;  // head dims 32 and 64 (fp32, bf16) and 96 (bf16)

struct Shape {
  int B, T_new, L, k, D, Hq, Hkv, d, p, Lp, S_cap;
  int mix_softmax;   // 1: softmax over source layers per channel row
  int mask_paper;    // 1: dummy slot + strictly earlier slots; 0: slots <= own position
  int router_mode;   // 0 content-dependent router, 1 static weights (alpha = b), 2 no feedback
  float eps, rope_theta;
  int ctx_max;       // host-side bound on ctx_len[b] (sizes the attention grid)
  // Token i of sequence b sits at position ctx_len[b] + gq + gs * i (a strided token
  // group of Section 3.3: gs = g groups, gq = q; contiguous tokens: gs = 1, gq = 0).
  int gs, gq;
  int ctx_hi;        // device clamp of ctx_len[b]: S_cap minus the positions the call spans
  __host__ __device__ int N() const { return B * T_new; }
  // positions covered by one sequence's new tokens: gq + gs (T_new - 1) + 1
  __host__ __device__ long span() const { return T_new > 0 ? (long)gq + (long)gs * (T_new - 1) + 1 : 0; }
};

struct LayerTable {  // small per-call integer tables, passed by value
  int v[kMaxLayers];
};

// -- pool side (Steps 1 and 2) ------------------------------------------------
// rinv[r] = 1 / sqrt(mean(X[r][:]^2) + eps) for rows of length D.
template <typename T>
void launch_row_rms(const T* X, long rows, int D, float eps, float* rinv, hipStream_t s);
// rows at X + r * xs, results at rinv[r * os]
template <typename T>
void launch_row_rms_strided(const T* X, long rows, int D, long xs, long os, float eps,
                            float* rinv, hipStream_t s);

// tab[n][m] = (cos, sin)(pos(n) * theta^(-2m/d)), pos(n) = ctx_len[b] + gq + gs i, in fp64.
void launch_rope_table(const Shape& sh, const int32_t* ctx_len, float* tab, hipStream_t s);

// logits[br][n][o] = sum over stacked layers of W_alpha[br][o] . normed state + b_alpha[br][o]
// wfold: router_fold_elems(sh) elements (weights with the pre-mix gain folded in);
// part: router_partials_bytes(sh) bytes of split-K partial sums (may be 0).
size_t router_fold_elems(const Shape& sh);
size_t router_partials_bytes(const Shape& sh);
// prefolded: wfold already holds launch_router_fold's output for these weights
template <typename T>
void launch_router_fold(const Shape& sh, const LayerTable& sel, const T* g_pre, const T* W_alpha,
                        T* wfold, hipStream_t s);
template <typename T>
void launch_router(const Shape& sh, const LayerTable& sel, const T* H, const float* rinv,
                   const T* g_pre, const T* W_alpha, const T* b_alpha, float* logits, T* wfold,
                   float* part, hipStream_t s, bool prefolded = false);

// alpha (in: logits [2][N][k*L], out: mixing weights) -> mixed[2][k][N][D], rinv_mid[2][k][N]
size_t mix_smem_bytes(int L, int k, int D, size_t elem_bytes);
template <typename T>
void launch_mix(const Shape& sh, const T* H, const float* rinv, const T* g_pre, float* alpha,
                T* mixed, float* rinv_mid, hipStream_t s);

// mixed -> K (mid norm, W^K_j, key norm, RoPE) and V (mid norm, W^V_j) at slot pos(n).
// wfold: workspace for the gain-folded weights, kv_fold_elems(sh) elements.
size_t kv_fold_elems(const Shape& sh);
template <typename T>
void launch_kv_fold(const Shape& sh, const T* g_mid, const T* Wk, const T* Wv, T* wfold,
                    hipStream_t s);
template <typename T>
void launch_kv_project(const Shape& sh, const T* mixed, const float* rinv_mid, const T* g_mid,
                       const T* Wk, const T* Wv, const T* g_knorm, const float* rope_tab,
                       const int32_t* ctx_len, T* Kc, T* Vc, T* wfold, hipStream_t s,
                       bool prefolded = false);

// H -> Q[L][B][Hq][T_new][d] (input norm, W^Q_l, q norm, RoPE); wfold: q_fold_elems(sh).
size_t q_fold_elems(const Shape& sh);
template <typename T>
void launch_q_project(const Shape& sh, const T* H, const float* rinv, const T* g_in,
                      const T* Wq, const T* g_qnorm, const float* rope_tab, T* Q, T* wfold,
                      hipStream_t s);
// the same in two parts: fold the input-norm gains of layers l0 .. l0 + nl - 1 into their
// slots of wfold (layer l at l Hq d D), then project layers l0 .. l0 + nl - 1 into
// Q[nl][B][Hq][T_new][d]
template <typename T>
void launch_q_fold(const Shape& sh, const T* g_in, const T* Wq, T* wfold, int l0, int nl,
                   hipStream_t s);
template <typename T>
void launch_q_layers(const Shape& sh, const T* H, const float* rinv, const T* g_qnorm,
                     const float* rope_tab, T* Q, const T* wfold, int l0, int nl, hipStream_t s);

// -- pass driver (Section 3.3) --------------------------------------------------
// The stand-in decoder block: out[n] = h[n] + W o_l[n] (W [D][HD], o_l [M][HD]); rows of h
// and out strided by hs and os elements.
template <typename T>
void launch_block_residual(int M, int D, int HD, const T* o_l, const T* W, const T* h, long hs,
                           T* out, long os, hipStream_t s);
// Group-major states: Hg[q][b][m][l][e] for position q + g m (T a multiple of g).
template <typename T>
void launch_group_gather(const T* X, T* Hg, int B, int T_len, int g, int L, int D,
                         hipStream_t s);
template <typename T>
void launch_group_scatter(const T* Yg, T* Y, int B, int T_len, int g, long row, hipStream_t s);

// -- consumer side (Step 3) ---------------------------------------------------
struct ChannelGroups {       // CSR inverse of the consumer -> channel map
  int offsets[kMaxLayers + 1];
  int members[kMaxLayers];
};

// scratch: prefill_scratch_bytes(sh) of device memory (at least kPrefillQueueBytes): the
// work queue the bf16 kernel's persistent grid takes its tiles from (reset on the stream
// before each launch), or the partial states of its split slot ranges on small grids;
// other paths ignore it.
constexpr size_t kPrefillQueueBytes = 512;
size_t prefill_scratch_bytes(const Shape& sh);
template <typename T>
void launch_attend_prefill(const Shape& sh, const LayerTable& chan_map, const T* Q,
                           const T* Kc, const T* Vc, const T* Kd, const T* Vd,
                           const int32_t* ctx_len, const int32_t* doc, T* O, void* scratch,
                           hipStream_t s);

// Gradients of the full-sequence channel attention (bf16, head dims 64 and 96): dQ
// [L][B][Hq][T][d], dKc / dVc [k][B][Hkv][S_cap][d] (slots below ctx_len[b] + T written),
// dKd / dVd [k][Hkv][d], all fp32; rows: attend_backward_rows_bytes of workspace.
size_t attend_backward_rows_bytes(const Shape& sh);
void launch_attend_backward(const Shape& sh, const LayerTable& chan_map,
                            const ChannelGroups& groups, const bf16* Q, const bf16* Kc,
                            const bf16* Vc, const bf16* Kd, const bf16* Vd, const bf16* O,
                            const bf16* dO, const int32_t* ctx_len, float* dQ, float* dKc,
                            float* dVc, float* dKd, float* dVd, float* rows, hipStream_t s,
                            bool accumulate = false);

// compute units of the current device (cached per device)
int device_cus();

// -- gradients of the pool and the queries (wm_grad.hip) ----------------------
// Operand element (row, k) of batch z at p + z s_z + row s_row + k s_k (bf16 or fp32).
struct GemmOperand {
  const void* p;
  long s_row, s_k, s_z;
  int f32;
  int pad8;  // the operand's memory extends to a whole group of 8 past its last row (rows
             // contiguous) or k (k contiguous), zero-filled: vector loads may read it
  long span; // set by launch_grad_gemm: bytes one batch's tile loads may reach
};
// C[z][m][n] (+)= sum_k A(m, k) B(n, k) over batches z; C at C + z c_z + m c_row + n c_col.
// Batch z uses only k >= k_lo0 + k_lo_dz z of B and stores only rows m >= m_lo0 + m_lo_dz z
// (the no-feedback router's triangular weights); zero both for a plain GEMM.
// part / part_elems (optional): fp32 scratch for split K. When the tiles would leave CUs
// idle and K is long, each tile's K range is cut into slices computed by separate
// workgroups into part, then summed in slice order into C (the same sum on any device).
struct GemmArgs {
  GemmOperand A, B;
  float* C;
  long c_row, c_col, c_z;
  int M, N, K, accumulate;
  long k_lo0, k_lo_dz, m_lo0, m_lo_dz;
  float* part;
  long part_elems;
  int splits;   // set by launch_grad_gemm
  int kchunk;   // set by launch_grad_gemm: K per slice, a multiple of 32
};
void launch_grad_gemm(GemmArgs a, int batches, hipStream_t s);
// out[r] = g[(r / gdiv) % gmod] * x[r] * rinv[r] (bf16 rows of D)
void launch_grad_norm_apply(const bf16* x, const bf16* g, const float* rinv, long rows, long gdiv,
                            int gmod, int D, bf16* out, hipStream_t s);
struct HeadArgs {
  const float* src;       // rotated output's gradient, rows of d at (z sZ + b sB + h sH + slot)
  long sZ, sB, sH;
  int slot_ctx;           // slot = ctx_len[b] + gq + gs i (cache layout) or i
  int gs, gq;
  const int32_t* ctx_len;
  int ctx_hi;
  const float* y;         // pre-norm values [Z][B T][H d]
  bf16* dy;               // their gradient, same layout (bf16: the GEMMs' operand)
  const bf16* g;          // [Z][d]
  const float* tab;       // RoPE table [B T][d / 2] (cos, sin)
  float* dgp;             // gain gradient partials [Z][chunks][d]
  int B, H, T, chunks;
  float eps;
};
void launch_grad_head(const HeadArgs& a, int Z, int d, hipStream_t s);
struct RmsArgs {           // rows (o, i); offsets in rows of D
  const float* dy;
  long dy_o, dy_i;
  const bf16* x;
  long x_o, x_i;
  float* out;
  long out_o, out_i;
  const float* rinv;       // per row, at o r_o + i r_i
  long r_o, r_i;
  const bf16* g;           // [nouter][D]
  float* dgp;              // [nouter][chunks][D]
  int D, ninner, chunks, accumulate;
};
void launch_grad_rms(const RmsArgs& a, int nouter, hipStream_t s);
// out[o][e] (+)= scale * sum_c part[(o chunks + c) n + e] (part is overwritten)
void launch_grad_sum(float* part, int outer, int chunks, long n, float* out, float scale,
                     int accumulate, hipStream_t s);
void launch_grad_colsum(const float* x, long rows, int n, int chunks, float* part, hipStream_t s);
void launch_grad_gather(const float* src, int k, int B, int H, int T, int S_cap, int d,
                        const int32_t* ctx_len, int ctx_hi, int gs, int gq, bf16* dst,
                        hipStream_t s);
struct MixGradArgs {
  const bf16* H;           // [N][L][D] states
  const bf16* g;           // [L][D] the branch's pre-mix gains
  const float* rinv;       // [N][L] 1 / rms of each state
  const float* dmix;       // [k][N][D] gradient of that branch's mixed channels
  const float* alpha;      // [N][k][L] final mixing weights
  float* dhn;              // [N][L][D]
  float* dlog;             // [N][k L] gradient of the router logits
  bf16* dlogb;             // [N][kLp] the same in bf16, rows padded with zeros to kLp
  int N, L, k, D, softmax, nofeedback, kLp;
};
size_t grad_mix_smem(int L, int k, int D);
void launch_grad_mix(const MixGradArgs& a, hipStream_t s);
template <typename T>
void launch_grad_mask(T* W, int kL, int L, int Lp, int D, const LayerTable& sel, hipStream_t s);

void launch_grad_fill(float* p, long n, float v, hipStream_t s);
void launch_grad_cast(const float* src, bf16* dst, long n, hipStream_t s);
// dst[r dst_stride + e] += sum over l < nsrc of src[r src_stride + l D + e]
void launch_grad_add_rows(float* dst, long dst_stride, const float* src, long rows, int D,
                          long src_stride, int nsrc, hipStream_t s);
// slots q + g i (i < Tg) of the [rows][S_cap][d] caches to (restore false) or back from
// (restore true) compact [rows][Tg][d] copies; restoring clears dK, dV there when given
void launch_grad_slots(bf16* K, bf16* V, bf16* Kg, bf16* Vg, float* dK, float* dV, long rows,
                       int Tg, int g, int q, int S_cap, int d, bool restore, hipStream_t s);
void launch_grad_copy_rows(const bf16* src, long src_stride, bf16* dst, long rows, int D,
                           hipStream_t s);

// Split-S decode for small T_new; partials live in the workspace.
size_t decode_partials_bytes(const Shape& sh);
int decode_splits(const Shape& sh);
template <typename T>
void launch_attend_decode(const Shape& sh, const LayerTable& chan_map, const ChannelGroups& cg,
                          const T* Q, const T* Kc, const T* Vc, const T* Kd, const T* Vd,
                          const int32_t* ctx_len, const int32_t* doc, float* partials, T* O,
                          hipStream_t s);

// The dense soft read: Kl/Vl[l][B][Hkv][S_cap][d] = sum_c w[l][c] Kc/Vc[c], over the slots the
// call's rows may see, and Kdl/Vdl[l][Hkv][d] from the dummies.
template <typename T>
void launch_soft_read(const Shape& sh, const float* w, const T* Kc, const T* Vc, const T* Kd,
                      const T* Vd, const int32_t* ctx_len, T* Kl, T* Vl, T* Kdl, T* Vdl,
                      hipStream_t s);

// -- measurement helper ---------------------------------------------------------
// blocks x 4 waves, each issuing 8 * iters independent 32x32x16 bf16 MFMAs on small
// constant operands, or (random) on hashed operands that change from one MFMA to the next.
void launch_mfma_loop(int blocks, int iters, bool random, float* sink, hipStream_t s);
// Reads n16 16-byte chunks of buf once.
void launch_read_loop(const void* buf, long n16, float* sink, hipStream_t s);

}  // namespace wm
