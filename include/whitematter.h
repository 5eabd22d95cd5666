/*
 * whitematter.h -- C ABI of libwhitematter.so, the MI355X (gfx950) hot path of
 * WhiteMatter ("WhiteMatter: All-to-All Cross-Layer Connections via KV
 * Mixing"): the cross-layer KV pool of Section 3.1 and the per-layer channel
 * attention of Section 3.1 Step 3 / Section 3.2.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 *  - Tensors are caller-owned, contiguous, row-major, in the layouts given
 *    below. "Device" pointers must point to GPU memory of the current HIP
 *    device and be 16-byte aligned; "host" pointers are ordinary memory.
 *  - Element type: every tensor named "in dtype" is fp32 (WM_F32) or bf16
 *    (WM_BF16) as dims->dtype says; mixing weights and workspaces are fp32.
 *  - The library never allocates device memory. Scratch comes from the
 *    caller: ws points to at least wm_workspace_size(dims, op) bytes of device
 *    memory, 256-byte aligned, and ws_bytes states its size.
 *  - Every call validates on the host first and launches nothing on error.
 *    Work is enqueued asynchronously on `stream` (NULL = the null stream);
 *    nothing synchronises. Calls keep no state between them, so concurrent
 *    calls are safe as long as their output and workspace buffers differ.
 *  - Return value: WM_OK or one of the WM_ERR_* codes; wm_last_error() gives
 *    a message for the calling thread's last failure.
 *  - N = B * T_new new tokens; token n = b * T_new + i of sequence b sits at
 *    position pos(b, i) = ctx_len[b] + q + g * i and is cached at that slot, where
 *    g = dims->groups and q = dims->group select a strided token group of Section
 *    3.3 (G_q = positions congruent to q mod g); g = 1, q = 0 (or g = 0) are
 *    contiguous new tokens, pos(b, i) = ctx_len[b] + i.
 *  - ctx_len (device, int32 [B], NULL = all zero) must lie in [0, ctx_max];
 *    ctx_max + q + g * (T_new - 1) + 1 <= S_cap is checked on the host. The
 *    kernels clamp each entry into [0, S_cap - (q + g * (T_new - 1) + 1)], so an
 *    entry outside [0, ctx_max] leaves that sequence's outputs unspecified but
 *    never causes an access outside the given buffers.
 */
#ifndef WHITEMATTER_H
#define WHITEMATTER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *wm_stream_t; /* a hipStream_t */

enum wm_status {
  WM_OK = 0,
  WM_ERR_ARG = 1,         /* null, misaligned or negative argument */
  WM_ERR_SHAPE = 2,       /* inconsistent or unsupported dimensions */
  WM_ERR_DTYPE = 3,       /* unknown dtype / mode value */
  WM_ERR_MAP = 4,         /* consumer->channel map entry outside [0, k) */
  WM_ERR_CAPACITY = 5,    /* ctx_max + positions of the new tokens > S_cap */
  WM_ERR_WORKSPACE = 6,   /* ws NULL, misaligned or smaller than required */
  WM_ERR_LAUNCH = 7       /* the HIP runtime rejected a launch */
};

enum wm_dtype { WM_F32 = 0, WM_BF16 = 1 };

/* Mixing weights: the paper's signed linear router (Section 3.1 Step 1), or
 * additionally normalised by a softmax over the L source layers of each
 * channel row (weights positive, summing to 1). */
enum wm_mix_mode { WM_MIX_LINEAR = 0, WM_MIX_SOFTMAX = 1 };

/* Attention mask: the paper's (Section 3.2) -- a learned dummy slot plus the
 * cached slots strictly before the query's own position, so a token never
 * reads its own channels -- or standard causal (slots <= own position, no
 * dummy). */
enum wm_mask_mode { WM_MASK_PAPER = 0, WM_MASK_INCLUSIVE = 1 };

/* Where the mixing weights come from (the ablations of Section 5.3):
 *   WM_ROUTER_DYNAMIC    the paper's content-dependent router (Section 3.1 Step 1)
 *   WM_ROUTER_STATIC     static learnable weights, no router: alpha[j][l] = b_alpha[j*L + l]
 *                        for every token (W_alpha is not read)
 *   WM_ROUTER_NOFEEDBACK no deep-to-shallow feedback: requires k = L; channel j mixes
 *                        source layers 0..j only (weights on deeper layers are 0, or left
 *                        out of the softmax), and its router reads only the stacked states
 *                        of layers <= j (W_alpha entries on deeper layers are not used). */
enum wm_router_mode { WM_ROUTER_DYNAMIC = 0, WM_ROUTER_STATIC = 1, WM_ROUTER_NOFEEDBACK = 2 };

enum wm_op {
  WM_OP_ROUTER_MIX = 0,
  WM_OP_KV_PROJECT = 1,
  WM_OP_Q_PROJECT = 2,
  WM_OP_CHANNEL_ATTEND = 3,
  WM_OP_LAYER_STEP = 4,
  WM_OP_POOL = 5,          /* wm_pool */
  WM_OP_LAYER_ATTEND = 6,  /* wm_layer_attend */
  WM_OP_PASSES = 7,        /* wm_prefill_passes */
  WM_OP_DENSE_ATTEND = 8,  /* wm_channel_attend_dense */
  WM_OP_ATTEND_BACKWARD = 9, /* wm_channel_attend_backward */
  WM_OP_Q_BACKWARD = 10,      /* wm_q_project_backward */
  WM_OP_POOL_BACKWARD = 11,   /* wm_pool_backward */
  WM_OP_STEP_BACKWARD = 12,   /* wm_layer_step_backward */
  WM_OP_PASSES_BACKWARD = 13  /* wm_prefill_passes_backward (size: see
                                 wm_passes_backward_workspace) */
};

/* Problem dimensions (paper notation). Supported: 1 <= L <= 64, 1 <= k <= L,
 * D a multiple of 32, Hq a multiple of Hkv, d in {32, 64} (either dtype) or d = 96
 * (WM_BF16 only), 1 <= p <= L, and a token's L states plus its mixing coefficients
 * within 64 KiB of LDS: L * D * sizeof(dtype) (rounded up to 16) + 8 * L * k4 + 16 * k
 * bytes with k4 = k rounded up to a multiple of 4, e.g. L <= 31 at D = 1024 in bf16,
 * L <= 15 in fp32. */
typedef struct wm_dims {
  int32_t B;         /* sequences */
  int32_t T_new;     /* new tokens per sequence in this call */
  int32_t L;         /* decoder layers = source layers = consumer layers */
  int32_t k;         /* KV channels */
  int32_t D;         /* hidden width */
  int32_t Hq;        /* query heads */
  int32_t Hkv;       /* KV heads; query head h reads KV head h / (Hq / Hkv) */
  int32_t d;         /* head dimension */
  int32_t p;         /* router reads every p-th source layer counting down from L-1 */
  int32_t S_cap;     /* cache slots per (channel, sequence, KV head) */
  int32_t ctx_max;   /* upper bound on ctx_len[b] */
  int32_t dtype;     /* enum wm_dtype */
  int32_t mix_mode;  /* enum wm_mix_mode */
  int32_t mask_mode; /* enum wm_mask_mode */
  int32_t router_mode; /* enum wm_router_mode */
  float eps;         /* RMSNorm epsilon (e.g. 1e-6) */
  float rope_theta;  /* RoPE base (e.g. 1e6) */
  int32_t groups;    /* g of Section 3.3: the call's tokens are the strided group q of a
                        pass split into g groups (token i at position ctx_len[b] + q + g i);
                        0 or 1: contiguous tokens */
  int32_t group;     /* q, 0 <= q < max(g, 1) */
} wm_dims;

/* Parameters, device pointers, in dtype, row-major. L' = ceil(L / p). */
typedef struct wm_params {
  const void *g_pre;   /* [2][L][D]        pre-mix RMSNorm gains, key then value branch */
  const void *W_alpha; /* [2][k*L][L'*D]   router weights; input = normed states of layers
                                           {L-1-p*m}, stacked in ascending layer order */
  const void *b_alpha; /* [2][k*L]         router bias; alpha[j][l] = out[j*L + l] */
  const void *g_mid;   /* [2][k][D]        mid RMSNorm gains per channel */
  const void *Wk;      /* [k][Hkv*d][D]    key projection per channel */
  const void *Wv;      /* [k][Hkv*d][D]    value projection per channel */
  const void *g_knorm; /* [k][d]           key-norm gain per channel (shared by KV heads) */
  const void *Kd;      /* [k][Hkv][d]      learned dummy key (used as stored, no RoPE) */
  const void *Vd;      /* [k][Hkv][d]      learned dummy value */
  const void *g_in;    /* [L][D]           consumer input RMSNorm gains */
  const void *Wq;      /* [L][Hq*d][D]     consumer query projections */
  const void *g_qnorm; /* [L][d]           consumer q-norm gains (shared by query heads) */
} wm_params;

/* Gradients of the parameters, device fp32 pointers in the shapes and layouts of the
 * wm_params entries of the same names (4-byte aligned). The backward entry points ADD
 * their contribution, so that the gradient passes of a training step (Section 3.3) sum
 * into one set: zero the buffers before the first call. Each entry point names the
 * entries it uses; the others may be NULL. */
typedef struct wm_grads {
  float *g_pre, *W_alpha, *b_alpha, *g_mid, *Wk, *Wv, *g_knorm, *Kd, *Vd, *g_in, *Wq, *g_qnorm;
} wm_grads;

/* Section 3.1 Step 1 (mix L states into k channels), both branches.
 *   H         device [B][T_new][L][D] in dtype: state entering each layer
 *   alpha_out device [2][N][k][L] fp32 or NULL: mixing weights per token
 *             (linear router output, or its softmax over l in WM_MIX_SOFTMAX)
 *   mixed_out device [2][k][N][D] in dtype: h~_j = sum_l alpha[j][l] RMSNorm(h_l)
 * Uses g_pre, W_alpha, b_alpha. */
int wm_router_mix(const wm_dims *dims, const wm_params *params, const void *H,
                  float *alpha_out, void *mixed_out, void *ws, size_t ws_bytes,
                  wm_stream_t stream);

/* Section 3.1 Step 2 (KV projections and cache storage).
 *   mixed   device [2][k][N][D] in dtype: mixed channels (key branch, value branch)
 *   ctx_len device int32 [B] or NULL
 *   Kc, Vc  device [k][B][Hkv][S_cap][d] in dtype: channel-major cache. Slot
 *           ctx_len[b] + i receives RoPE(knorm(W^K_j RMSNorm(h~^K_j))) and
 *           W^V_j RMSNorm(h~^V_j); no other slot is written.
 * Uses g_mid, Wk, Wv, g_knorm. */
int wm_kv_project(const wm_dims *dims, const wm_params *params, const void *mixed,
                  const int32_t *ctx_len, void *Kc, void *Vc, void *ws, size_t ws_bytes,
                  wm_stream_t stream);

/* The consumer's query (the unchanged Qwen3 block, Section 4.1):
 * Q_l = RoPE(qnorm(W^Q_l RMSNorm_in(h_l))) at the token's position.
 *   H       device [B][T_new][L][D] in dtype
 *   ctx_len device int32 [B] or NULL
 *   Q       device [L][B][Hq][T_new][d] in dtype
 * Uses g_in, Wq, g_qnorm. */
int wm_q_project(const wm_dims *dims, const wm_params *params, const void *H,
                 const int32_t *ctx_len, void *Q, void *ws, size_t ws_bytes,
                 wm_stream_t stream);

/* Section 3.1 Step 3 and Section 3.2: consumer l attends channel chan_map[l].
 *   Q        device [L][B][Hq][T_new][d] in dtype (after q-norm and RoPE)
 *   chan_map host int32 [L], entries in [0, k) (the paper's choice is l mod k)
 *   ctx_len  device int32 [B] or NULL
 *   Kc, Vc   device [k][B][Hkv][S_cap][d] in dtype (read only)
 *   O        device [L][B][T_new][Hq*d] in dtype: softmax(q K^T / sqrt(d)) V over
 *            the visible slots of the mask mode (dummy Kd/Vd of the channel
 *            included in WM_MASK_PAPER)
 * Uses Kd, Vd. T_new <= 4 takes the split-S decode kernels (their partial sums go to the
 * workspace); longer calls take the full-sequence kernels, whose workgroups take query tiles
 * from a 512-byte work queue in the workspace, reset on `stream` before each launch, or,
 * when the query tiles are few against long slot ranges (bf16, no document mask), walk
 * split ranges of each tile's slots whose partial softmax states go to the workspace and are
 * merged in a fixed order. */
int wm_channel_attend(const wm_dims *dims, const wm_params *params, const void *Q,
                      const int32_t *chan_map, const int32_t *ctx_len, const void *Kc,
                      const void *Vc, void *O, void *ws, size_t ws_bytes,
                      wm_stream_t stream);

/* The fused step: pool the T_new new tokens of every sequence into their cache
 * slots pos(b, i) (Steps 1-2), project the consumer queries, then every consumer
 * attends its channel (Step 3). With ctx_len = 0 and T_new = T this is one
 * full-sequence (Jacobi) pass, Section 3.3; with T_new = 1 it is a decode step,
 * Section 3.2. Every kernel runs on `stream`, in order; the call keeps no state
 * between calls (calls on different streams with their own buffers may overlap,
 * and the step may be captured into a graph).
 *   H        device [B][T_new][L][D] in dtype
 *   chan_map host int32 [L]
 *   ctx_len  device int32 [B] or NULL
 *   Kc, Vc   device [k][B][Hkv][S_cap][d] in dtype (slots < ctx_len[b] read, new
 *            slots written)
 *   O        device [L][B][T_new][Hq*d] in dtype */
int wm_layer_step(const wm_dims *dims, const wm_params *params, const void *H,
                  const int32_t *chan_map, const int32_t *ctx_len, void *Kc, void *Vc,
                  void *O, void *ws, size_t ws_bytes, wm_stream_t stream);

/* The dense soft read of Section 3.1 Step 3, the variant the paper contrasts with its
 * fixed selection: every consumer reads all k channels, mixed with its own weights,
 * K^_l[s] = sum_c read_w[l][c] K~_c[s] and V^_l[s] = sum_c read_w[l][c] V_c[s] (the dummy
 * slot likewise), then attends them as wm_channel_attend does. The fixed selection is
 * the one-hot row read_w[l][c] = (c == chan_map[l]).
 *   read_w  device float [L][k], 16-byte aligned: the weights as given (apply a softmax
 *           beforehand for a soft assignment)
 *   other arguments as wm_channel_attend (no chan_map)
 * The mixed channels go to the workspace first (2 L B Hkv S_cap d elements in dtype, the
 * mix summed in fp32 and rounded to dtype): each consumer streams the k channels' slots it
 * may see, k times the bytes of the fixed selection, which is the cost the paper names. */
int wm_channel_attend_dense(const wm_dims *dims, const wm_params *params, const float *read_w,
                            const void *Q, const int32_t *ctx_len, const void *Kc,
                            const void *Vc, void *O, void *ws, size_t ws_bytes,
                            wm_stream_t stream);

/* Gradients of wm_channel_attend (Section 3.1 Step 3 with the dummy slot of Section 3.2),
 * the attention part of the backward pass that training runs through its last n_g passes
 * (Section 3.3, truncated backpropagation). For the loss gradient dO of the output, with
 * scores s_j = q.k_j / sqrt(d) over a row's visible slots and the dummy, P = softmax(s),
 * dS_j = P_j (dO.v_j - dO.O): dQ = sum_j dS_j k_j / sqrt(d); every slot's dK sums
 * dS_j q / sqrt(d) and its dV sums P_j dO over all rows that read it (every consumer of
 * its channel and every query head of its KV head); the dummy's likewise.
 * bf16 only, head dims 64 and 96, full-sequence calls (T_new > 4) of contiguous tokens or
 * of one strided group (dims.groups, dims.group), no document mask.
 *   Q, chan_map, ctx_len, Kc, Vc  as wm_channel_attend
 *   O        device [L][B][T_new][Hq*d] bf16: that call's output
 *   dO       device [L][B][T_new][Hq*d] bf16: the gradient of the loss in O
 *   dQ       device float [L][B][Hq][T_new][d]
 *   dKc, dVc device float [k][B][Hkv][S_cap][d]: slots below ctx_len[b] + span of every
 *            (channel, sequence, KV head) are written (zero where no row reads the slot),
 *            span = T_new for contiguous tokens, q + g (T_new - 1) + 1 for group q of g;
 *            the others are left as they are
 *   dKd, dVd device float [k][Hkv][d] (written; zero in WM_MASK_INCLUSIVE)
 * Workspace: wm_workspace_size(dims, WM_OP_ATTEND_BACKWARD) bytes (four floats per query
 * row: the row's log-sum-exp, dO.O and the dummy's weight and dS). Errors: WM_ERR_DTYPE for
 * fp32, WM_ERR_SHAPE for other head dims or T_new <= 4, WM_ERR_ARG for a NULL pointer,
 * otherwise as wm_channel_attend. */
int wm_channel_attend_backward(const wm_dims *dims, const wm_params *params, const void *Q,
                               const int32_t *chan_map, const int32_t *ctx_len, const void *Kc,
                               const void *Vc, const void *O, const void *dO, float *dQ,
                               float *dKc, float *dVc, float *dKd, float *dVd, void *ws,
                               size_t ws_bytes, wm_stream_t stream);

/* Gradients of the consumer queries (wm_q_project) for a loss gradient dQ in the
 * queries: back through RoPE (the transposed rotation), the q norm, W^Q_l and the input
 * norm, with the forward's intermediate values recomputed from H.
 * bf16, head dims 64 and 96, contiguous tokens or one strided group, D <= 4608.
 *   H        device [B][T_new][L][D] bf16, ctx_len device int32 [B] or NULL: as the forward
 *   dQ       device float [L][B][Hq][T_new][d]
 *   dH       device float [B][T_new][L][D]: the gradient in H is ADDED
 *   grads    g_in, Wq, g_qnorm: ADDED
 * Workspace: wm_workspace_size(dims, WM_OP_Q_BACKWARD). Errors as wm_q_project, plus
 * WM_ERR_DTYPE for fp32 and WM_ERR_SHAPE / WM_ERR_ARG for what the gradients do not support
 * or a NULL gradient pointer. */
int wm_q_project_backward(const wm_dims *dims, const wm_params *params, const void *H,
                          const int32_t *ctx_len, const float *dQ, float *dH,
                          const wm_grads *grads, void *ws, size_t ws_bytes, wm_stream_t stream);

/* Gradients of the pool (wm_pool, Section 3.1 Steps 1-2) for loss gradients in the cache
 * rows the call wrote: back through RoPE and the key norm (key branch), W^K_j / W^V_j, the
 * mid norm, the mix (dh_l gets sum_j alpha_jl dh~_j; the weights' gradient dh~_j . h_l goes
 * through the softmax over depth, or the no-feedback mask, to the router's logits), the
 * router (W_alpha, b_alpha) and the pre-mix norm. The router, mix and norms of the forward
 * are recomputed from H with the forward's kernels.
 * bf16, head dims 64 and 96, contiguous tokens or one strided group, D <= 4608; every
 * router mode and mix mode.
 *   H, ctx_len  as wm_pool
 *   dKc, dVc device float [k][B][Hkv][S_cap][d], 16-byte aligned: the slot of token i,
 *            ctx_len[b] + i (ctx_len[b] + q + g i in group q of g), of every (channel,
 *            sequence, KV head) is read (the call's new rows); no other slot is read
 *   dH       device float [B][T_new][L][D]: ADDED
 *   grads    g_pre, W_alpha (not with WM_ROUTER_STATIC), b_alpha, g_mid, Wk, Wv, g_knorm:
 *            ADDED. Without feedback the router entries a channel never reads get nothing.
 * Workspace: wm_workspace_size(dims, WM_OP_POOL_BACKWARD). Errors as wm_q_project_backward. */
int wm_pool_backward(const wm_dims *dims, const wm_params *params, const void *H,
                     const int32_t *ctx_len, const float *dKc, const float *dVc, float *dH,
                     const wm_grads *grads, void *ws, size_t ws_bytes, wm_stream_t stream);

/* Gradients of the fused step (wm_layer_step) for a loss gradient dO in its output and,
 * optionally, gradients already reaching its cache rows: the step's backward that training
 * runs in each gradient-carrying pass (Section 3.3). Recomputes the queries, then runs
 * wm_channel_attend_backward (its slot and dummy gradients ADDED into dKc, dVc and
 * grads->Kd, grads->Vd), wm_q_project_backward and wm_pool_backward on the new slots'
 * total gradient.
 *   H, chan_map, ctx_len  as wm_layer_step
 *   Kc, Vc   device [k][B][Hkv][S_cap][d] bf16: the caches as the forward step left them
 *   O        device [L][B][T_new][Hq*d] bf16: the forward step's output
 *   dO       device [L][B][T_new][Hq*d] bf16
 *   dKc, dVc device float [k][B][Hkv][S_cap][d], 16-byte aligned, in/out: on entry the
 *            gradient that reaches the caches from elsewhere (zero if none); the attention's
 *            gradient is added to slots below ctx_len[b] + span (as in
 *            wm_channel_attend_backward), and the new slots' total is what the pool's
 *            backward receives. On return the other slots hold the gradient for the steps
 *            that wrote them.
 *   dH       device float [B][T_new][L][D]: ADDED
 *   grads    every entry (Kd, Vd only with WM_MASK_PAPER; W_alpha not with static
 *            weights): ADDED
 * Workspace: wm_workspace_size(dims, WM_OP_STEP_BACKWARD). Errors as
 * wm_channel_attend_backward and wm_pool_backward. */
int wm_layer_step_backward(const wm_dims *dims, const wm_params *params, const void *H,
                           const int32_t *chan_map, const int32_t *ctx_len, const void *Kc,
                           const void *Vc, const void *O, const void *dO, float *dKc,
                           float *dVc, float *dH, const wm_grads *grads, void *ws,
                           size_t ws_bytes, wm_stream_t stream);

/* wm_channel_attend for callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): no workspace argument. Its only
 * scratch, the split-S decode partials (T_new <= 4), the full-sequence kernels' 512-byte
 * work queue or, on grids of few query tiles, the partial states of their split slot
 * ranges, lives in a fixed array of 64 MiB of device memory inside the library; each
 * device holds its own copy until the process ends. The call itself allocates nothing. Calls on one
 * device share that array, so calls that overlap on one device race; serialise them (one
 * stream, or events). A call needing more scratch than the array holds (its
 * wm_workspace_size(dims, WM_OP_CHANNEL_ATTEND)) fails with WM_ERR_WORKSPACE before any
 * launch. Arguments, results and errors otherwise as wm_channel_attend. */
int wm_channel_attend_static(const wm_dims *dims, const wm_params *params, const void *Q,
                             const int32_t *chan_map, const int32_t *ctx_len, const void *Kc,
                             const void *Vc, void *O, wm_stream_t stream);

/* Document mask (Section 4.1: sequences packed from several documents, attention
 * confined to each document). Same as wm_channel_attend / wm_layer_step, plus
 *   doc_start device int32 [B][T_new], 4-byte aligned, not NULL: the position of
 *             the first token of the document that holds token i of sequence b
 *             (positions count from the start of the sequence, so token i sits at
 *             ctx_len[b] + i). Nondecreasing in i within a sequence (documents are
 *             contiguous). The row reads only cached slots at or after doc_start
 *             (and below its own position, as the mask mode says); the dummy slot
 *             stays visible in WM_MASK_PAPER. Values outside [0, position] are
 *             clamped into it; a decreasing array gives unspecified rows but no
 *             access outside the cache. */
int wm_channel_attend_doc(const wm_dims *dims, const wm_params *params, const void *Q,
                          const int32_t *chan_map, const int32_t *ctx_len,
                          const int32_t *doc_start, const void *Kc, const void *Vc, void *O,
                          void *ws, size_t ws_bytes, wm_stream_t stream);
int wm_layer_step_doc(const wm_dims *dims, const wm_params *params, const void *H,
                      const int32_t *chan_map, const int32_t *ctx_len, const int32_t *doc_start,
                      void *Kc, void *Vc, void *O, void *ws, size_t ws_bytes,
                      wm_stream_t stream);

/* Section 3.1 Steps 1-2 fused: the pool of the call's tokens into their cache slots
 * pos(b, i) (row norms, router, mix, mid norm, K/V projection, key norm, RoPE), with
 * the mixed channels kept in the workspace. The same cache writes as wm_layer_step.
 *   H        device [B][T_new][L][D] in dtype
 *   ctx_len  device int32 [B] or NULL
 *   Kc, Vc   device [k][B][Hkv][S_cap][d] in dtype (only the new slots are written)
 * Uses g_pre, W_alpha (not with WM_ROUTER_STATIC), b_alpha, g_mid, Wk, Wv, g_knorm. */
int wm_pool(const wm_dims *dims, const wm_params *params, const void *H, const int32_t *ctx_len,
            void *Kc, void *Vc, void *ws, size_t ws_bytes, wm_stream_t stream);

/* One consumer layer of Section 3.1 Step 3 on its own, as a depth-sequential decoder
 * runs it (Sections 3.2, 3.3): the query of `layer` from h_layer = H[b][i][layer][:]
 * (input norm, W^Q, q norm, RoPE at pos(b, i)), then attention over channel
 * chan_map[layer] in the mask mode (dummy + slots < pos, or slots <= pos).
 *   layer    0 <= layer < L
 *   H        device [B][T_new][L][D] in dtype (only layer `layer` is read)
 *   chan_map host int32 [L]
 *   ctx_len  device int32 [B] or NULL
 *   Kc, Vc   device [k][B][Hkv][S_cap][d] in dtype (read only)
 *   O_l      device [B][T_new][Hq*d] in dtype
 * Uses g_in, Wq, g_qnorm and (paper mask) Kd, Vd. */
int wm_layer_attend(const wm_dims *dims, const wm_params *params, int32_t layer, const void *H,
                    const int32_t *chan_map, const int32_t *ctx_len, const void *Kc,
                    const void *Vc, void *O_l, void *ws, size_t ws_bytes, wm_stream_t stream);

/* The fixed-point passes of Section 3.3 over sequences that start empty: P = Pool(H),
 * H = States(X; P), solved by cyclic Gauss-Seidel iteration over g = dims->groups strided
 * groups G_q = {i : i mod g = q} (g = 1: Jacobi iteration; g = T: one pass is exact
 * left-to-right evaluation). H^(0) takes every layer's state to be the token's embedding
 * and the cache starts as Pool(H^(0)); each pass evaluates G_0 .. G_{g-1} in order, and
 * group q first recomputes the states of all its positions, layer by layer, from the
 * cache as it stands (current-pass slots of groups < q, previous-pass slots of the rest),
 * then pools them into its slots. States needs the rest of each decoder block, which the
 * method leaves unchanged; a stand-in takes its place: h_{l+1} = h_l + W_o[l] o_l, the
 * attention sublayer's output projection and residual, o_l = layer l's channel attention
 * (wm_layer_attend), no MLP.
 *   dims     T_new = T, the sequence length, a multiple of groups; group = 0; ctx_max = 0;
 *            S_cap >= T. Every mode of dims applies (mask, mix, router).
 *   W_o      device [L][D][Hq*d] in dtype: the stand-in block's output projections
 *   X        device [B][T][D] in dtype: the state entering layer 0 (the embedding)
 *   chan_map host int32 [L]
 *   passes   >= 1
 *   Kc, Vc   device [k][B][Hkv][S_cap][d] in dtype: slots [0, T) are written; at return
 *            they hold Pool(H) of the returned states
 *   H        device [B][T][L][D] in dtype: the states entering every layer after the passes
 *   h_top    device [B][T][D] in dtype or NULL: the state leaving the top layer
 * The workspace (wm_workspace_size(dims, WM_OP_PASSES)) holds the states group by group,
 * B T L D elements, plus one group's scratch. Only the paper's mask has an exact
 * left-to-right solution: with WM_MASK_INCLUSIVE a position reads its own slot. */
int wm_prefill_passes(const wm_dims *dims, const wm_params *params, const void *W_o,
                      const void *X, const int32_t *chan_map, int32_t passes, void *Kc,
                      void *Vc, void *H, void *h_top, void *ws, size_t ws_bytes,
                      wm_stream_t stream);

/* A training step's passes with truncated backpropagation (Section 3.3): the passes of
 * wm_prefill_passes over g = dims->groups strided groups (g = 1: Jacobi iteration), then
 * the gradients of the loss through the last n_grad of them only. The cache starts as
 * Pool(H^(0)) with H^(0) = X in every layer; in each pass group q recomputes the states of
 * its positions from X and the cache as it stands (the stand-in block
 * h_{l+1} = h_l + W_o[l] o_l), then pools them into its slots. The cache entering pass
 * passes - n_grad + 1 is held fixed (no gradient flows into it or the passes before),
 * except with n_grad = passes, where the initial pool's gradient goes to X. Each window
 * step (one group of one pass) is differentiated whole: its pool (the router, mix,
 * projections and norms that wrote its slots), then every layer from the top down (the
 * block's W_o, the consumer's attention over its channel with the dummy, its query), the
 * residual stream carrying the gradient down to X. The window's group states, per-layer
 * attention outputs and the cache slots each step overwrote are kept in the workspace; the
 * queries are recomputed.
 * bf16, head dims 64 and 96, T_new = T with T / g > 4, D <= 4608, every mask, mix and
 * router mode.
 *   dims, params, W_o, X, chan_map, passes  as wm_prefill_passes
 *   n_grad   1 <= n_grad <= passes: the passes that carry gradients
 *   dh_top   device float [B][T][D]: the loss gradient in the state leaving the top layer
 *            after the last pass
 *   h_top    device [B][T][D] bf16 or NULL: that state (the forward's output)
 *   dX       device float [B][T][D]: ADDED
 *   dW_o     device float [L][D][Hq*d]: ADDED
 *   grads    every entry (Kd, Vd only with WM_MASK_PAPER; W_alpha not with static
 *            weights): ADDED
 * Workspace: wm_passes_backward_workspace(dims, n_grad) bytes, 256-byte aligned (it grows
 * with n_grad: per window pass the states, the attention outputs and two caches' worth of
 * the T written slots). Errors as wm_prefill_passes and wm_layer_step_backward;
 * WM_ERR_SHAPE for T / g <= 4, WM_ERR_ARG for n_grad outside [1, passes]. */
int wm_prefill_passes_backward(const wm_dims *dims, const wm_params *params, const void *W_o,
                               const void *X, const int32_t *chan_map, int32_t passes,
                               int32_t n_grad, const float *dh_top, void *h_top, float *dX,
                               float *dW_o, const wm_grads *grads, void *ws, size_t ws_bytes,
                               wm_stream_t stream);
/* Bytes of workspace wm_prefill_passes_backward needs for a window of n_grad passes; 0 when
 * dims are invalid (see wm_validate) or n_grad < 1. */
size_t wm_passes_backward_workspace(const wm_dims *dims, int32_t n_grad);

/* Measurement helper: wm_layer_step (doc_start NULL) or wm_layer_step_doc
 * (doc_start not NULL) that also records caller-created HIP events (hipEvent_t,
 * passed as void*) on `stream` at its phase boundaries, for per-phase timing of
 * the fused step: events[0] before the row norms, [1] before the router, [2]
 * before the mix, [3] before the K/V projection, [4] before the Q projection,
 * [5] before the channel attention, [6] after it. The array holds
 * WM_PROFILE_EVENTS non-NULL handles, owned by the caller. Results and errors
 * are those of the step it runs. */
#define WM_PROFILE_EVENTS 7
int wm_layer_step_profiled(const wm_dims *dims, const wm_params *params, const void *H,
                           const int32_t *chan_map, const int32_t *ctx_len,
                           const int32_t *doc_start, void *Kc, void *Vc, void *O, void *ws,
                           size_t ws_bytes, wm_stream_t stream, void *const *events);

/* Bytes of device workspace the op needs for these dims (0 if dims invalid). */
size_t wm_workspace_size(const wm_dims *dims, int op);

/* Host-only validation of dims for op (and of chan_map when non-NULL). */
int wm_validate(const wm_dims *dims, int op, const int32_t *chan_map);

/* Host helpers (no GPU work). */
/* Inverse of chan_map (Section 3.1 Step 3): channel c is read by layers
 * members[offsets[c] .. offsets[c+1]) in ascending order. offsets has k+1
 * entries, members L. */
int wm_channel_groups(int32_t L, int32_t k, const int32_t *chan_map, int32_t *offsets,
                      int32_t *members);
/* The paper's fixed selection: map[l] = l mod k. */
int wm_default_map(int32_t L, int32_t k, int32_t *chan_map);
/* The paper's router bias initialisation (Section 3.1, Router initialization):
 * k = 1 top layer; 1 < k < L layer l -> channel l mod k; k = L channel j <-
 * layer min(j+1, L-1). b has k*L floats, alpha[j][l] = b[j*L + l]. */
int wm_init_bias(int32_t L, int32_t k, float *b);

const char *wm_last_error(void);
const char *wm_version(void);

/* Measurement helper, not part of the method: launches `blocks` workgroups of 4
 * waves on `stream`, each wave issuing 8 * iters independent 32x32x16 bf16 MFMAs
 * (blocks * iters * 1048576 flop in all), so that a caller timing it with events
 * reads the matrix-core ceiling of the device. operands: 0 = small constants, the same
 * for every MFMA (the unthrottled issue rate); 1 = pseudo-random values in [-1, 1) that
 * change from one MFMA to the next, as real data does (the matrix cores then draw more
 * power and the clock may drop). sink: device float, caller-owned; written only in a case
 * that does not occur, kept so the loop is not removed.
 * WM_ERR_ARG for blocks or iters <= 0 (or above 2^20 / 2^24), operands not 0 or 1, or a
 * NULL sink. */
int wm_calibrate_mfma(int32_t blocks, int32_t iters, int32_t operands, float *sink,
                      wm_stream_t stream);

/* Measurement helper, not part of the method: reads `bytes` of the device buffer buf
 * once on `stream` (the HBM read ceiling when timed with events). buf: caller-owned,
 * 16-byte aligned, bytes a positive multiple of 16; sink as above. WM_ERR_ARG
 * otherwise. */
int wm_calibrate_read(const void *buf, size_t bytes, float *sink, wm_stream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* WHITEMATTER_H */
