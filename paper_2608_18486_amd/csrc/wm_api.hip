// Host layer of libwhitematter.so: the C ABI declared in include/whitematter.h.
// Validates every argument on the host before anything is enqueued, lays out
// the caller's workspace, builds the channel -> consumers table and launches
// the kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <climits>
#include <cstring>
#include <mutex>

#include "whitematter.h"
#include "wm_internal.hpp"

using wm::bf16;

// Scratch of wm_channel_attend_static, for callers that cannot allocate: the decode
// kernels' split partials live in this array instead of a caller workspace. Every device
// the library runs on holds its own copy until the process ends; calls that overlap on
// one device share it and race.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }
size_t elem_size(const wm_dims& d) { return d.dtype == WM_BF16 ? 2 : 4; }
bool decode_path(const wm_dims& d) { return d.T_new <= 4; }

struct Layout {
  size_t rinv = 0, alpha = 0, mixed = 0, rinv_mid = 0, tab = 0, q = 0, part = 0, wkv = 0, wq = 0,
         wa = 0, rpart = 0, hg = 0, topg = 0, ol = 0, kl = 0, vl = 0, kdl = 0, vdl = 0, total = 0;
  // gradients: dQ, gain partial rows, dummy scratch, the Q side's normed input, pre-norm
  // projection and its gradient, the pool side's normed states, mid-normed channels,
  // K/V pre-norm values and gradients, channel gradients, state gradients, logit gradients
  size_t dq = 0, dgp = 0, gkd = 0, x = 0, yq = 0, dyq = 0, dx = 0, hn = 0, u = 0, ydy = 0,
         dyb = 0, du = 0, dhn = 0, dlog = 0, dlogb = 0, split = 0;
};

int group_stride(const wm_dims& d) { return d.groups > 1 ? d.groups : 1; }
// positions covered by one sequence's new tokens (group + groups (T_new - 1) + 1)
long long call_span(const wm_dims& d) {
  return d.T_new > 0 ? (long long)d.group + (long long)group_stride(d) * (d.T_new - 1) + 1 : 0;
}

wm::Shape make_shape(const wm_dims& d) {
  wm::Shape s;
  s.B = d.B;
  s.T_new = d.T_new;
  s.L = d.L;
  s.k = d.k;
  s.D = d.D;
  s.Hq = d.Hq;
  s.Hkv = d.Hkv;
  s.d = d.d;
  s.p = d.p;
  s.Lp = (d.L + d.p - 1) / d.p;
  s.S_cap = d.S_cap;
  s.mix_softmax = d.mix_mode == WM_MIX_SOFTMAX;
  s.mask_paper = d.mask_mode == WM_MASK_PAPER;
  s.router_mode = d.router_mode;
  s.eps = d.eps;
  s.rope_theta = d.rope_theta;
  s.ctx_max = d.ctx_max;
  s.gs = group_stride(d);
  s.gq = d.group;
  // the device clamps ctx_len[b] into [0, ctx_hi]; without a cache (S_cap unused) only
  // the lower bound applies
  const long long hi = d.S_cap > 0 ? (long long)d.S_cap - call_span(d) : INT_MAX;
  s.ctx_hi = (int)std::min<long long>(std::max<long long>(hi, 0), INT_MAX);
  return s;
}

// The dims of one strided group of a pass-driver call (T_new = T / g tokens per sequence).
wm_dims group_dims(const wm_dims& d, int q) {
  wm_dims dg = d;
  dg.T_new = d.T_new / group_stride(d);
  dg.groups = group_stride(d);
  dg.group = q;
  dg.ctx_max = 0;
  return dg;
}

// The shape of one consumer's attention: a single layer reading channel map[l].
wm::Shape one_layer(wm::Shape sh) {
  sh.L = 1;
  return sh;
}

// The dense soft read attends L mixed channels, one per consumer layer.
wm::Shape dense_shape(wm::Shape sh) {
  sh.k = sh.L;
  return sh;
}

// Partial rows per gain or bias gradient: fixed, so every sum has one order on any device.
constexpr int kGradChunks = 64;
// fp32 scratch of the split-K weight-gradient GEMMs (K = the call's tokens)
constexpr size_t kSplitElems = (size_t)8 << 20;
// Partial rows of a gain gradient with `outer` gain rows: kGradChunks per row, more when
// that would leave fewer than ~1024 workgroups (one layer at a time).
int red_chunks(int outer) {
  return std::max(kGradChunks, std::min(1024, (1024 + outer - 1) / std::max(outer, 1)));
}
// Floats of partial rows the gradient ops need at most: outer red_chunks(outer) rows of the
// gain width for the gains (L or k rows of D, of d), kGradChunks rows of kL for the bias.
size_t dgp_elems(const wm_dims& d) {
  size_t m = (size_t)kGradChunks * d.k * d.L;
  for (int outer : {d.L, d.k})
    m = std::max(m, (size_t)outer * red_chunks(outer) * std::max(d.D, d.d));
  return m;
}

// Workspace of the backward ops. The step's backward recomputes Q into q, takes the
// attention gradients (dQ into dq), then runs the Q side and the pool side one after the
// other in the same region: both start at the offset after the shared rows.
Layout grad_layout(const wm_dims& d, int op) {
  Layout Ly;
  const size_t N = (size_t)d.B * d.T_new, L = d.L, k = d.k, D = d.D;
  const size_t HQ = (size_t)d.Hq * d.d, HK = (size_t)d.Hkv * d.d;
  const wm::Shape sh = make_shape(d);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += al256(bytes);
    return at;
  };
  if (op == WM_OP_STEP_BACKWARD) {
    Ly.q = take(L * N * HQ * 2);
    Ly.dq = take(L * N * HQ * 4);
    Ly.part = take(wm::attend_backward_rows_bytes(sh));
    Ly.gkd = take(2 * k * HK * 4);
    Ly.wq = take(wm::q_fold_elems(sh) * 2);
  }
  Ly.rinv = take(N * L * 4);
  Ly.tab = take(N * d.d * 4);
  Ly.dgp = take(dgp_elems(d) * 4);
  Ly.split = take(kSplitElems * 4);
  const size_t base = off;
  size_t end = off;
  if (op == WM_OP_Q_BACKWARD || op == WM_OP_STEP_BACKWARD) {
    Ly.x = take(N * L * D * 2);
    Ly.yq = take(L * N * HQ * 4);
    Ly.dyq = take(L * N * HQ * 2);
    Ly.dx = take(N * L * D * 4);
    end = std::max(end, off);
    off = base;
  }
  if (op == WM_OP_POOL_BACKWARD || op == WM_OP_STEP_BACKWARD) {
    Ly.alpha = take(2 * N * k * L * 4);
    Ly.mixed = take(2 * k * N * D * 2);
    Ly.rinv_mid = take(2 * k * N * 4);
    Ly.wa = take(wm::router_fold_elems(sh) * 2);
    Ly.rpart = take(wm::router_partials_bytes(sh));
    Ly.hn = take(N * L * D * 2);
    Ly.u = take(k * N * D * 2);
    Ly.ydy = take(k * N * HK * 4);
    Ly.dyb = take(k * N * HK * 2);
    Ly.du = take(k * N * D * 4);
    Ly.dhn = take(N * L * D * 4);
    Ly.dlog = take(N * k * L * 4);
    Ly.dlogb = take(N * ((k * L + 7) & ~(size_t)7) * 2);
    end = std::max(end, off);
  }
  Ly.total = N == 0 ? 0 : end;
  return Ly;
}

// Workspace regions for an op (offsets in bytes, each 256-byte aligned).
struct PassBwdLayout {
  size_t fw = 0, kv = 0, hs = 0, undo = 0, op = 0, gcur = 0, gb = 0, dof = 0, dob = 0, dql = 0,
         h1 = 0, rows = 0, gkd = 0, dpk = 0, dpv = 0, dhn = 0, split = 0, sub = 0, total = 0;
  // bytes of one cache, and per window step: one group's states, its slots of one cache,
  // its layers' attention outputs
  size_t cache = 0, state = 0, slots = 0, outs = 0;
};

PassBwdLayout passes_bwd_layout(const wm_dims& d, int n_grad);

Layout layout(const wm_dims& dd, int op) {
  if (op == WM_OP_Q_BACKWARD || op == WM_OP_POOL_BACKWARD || op == WM_OP_STEP_BACKWARD)
    return grad_layout(dd, op);
  if (op == WM_OP_PASSES_BACKWARD) {  // the size with a one-pass window
    Layout Ly;
    Ly.total = passes_bwd_layout(dd, 1).total;
    return Ly;
  }
  Layout Ly;
  const bool passes = op == WM_OP_PASSES;
  // the pass driver works on one group at a time: its scratch is sized by a group (the
  // last one, whose positions reach furthest: the decode partials grow with them)
  const wm_dims d = passes ? group_dims(dd, group_stride(dd) - 1) : dd;
  const size_t N = (size_t)d.B * d.T_new, es = elem_size(d);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += al256(bytes);
    return at;
  };
  const bool all = op == WM_OP_LAYER_STEP;
  const bool pool = op == WM_OP_POOL || passes;  // the fused Steps 1-2
  const bool layer = op == WM_OP_LAYER_ATTEND || passes;  // one consumer at a time
  if (passes) {
    Ly.hg = take((size_t)dd.B * dd.T_new * d.L * d.D * es);
    Ly.topg = take((size_t)dd.B * dd.T_new * d.D * es);
    Ly.ol = take(N * d.Hq * d.d * es);
  }
  if (op == WM_OP_ROUTER_MIX || op == WM_OP_Q_PROJECT || all || pool || layer)
    Ly.rinv = take(N * d.L * 4);
  if (op == WM_OP_ROUTER_MIX || all || pool) Ly.alpha = take(2 * N * d.k * d.L * 4);
  if (all || pool) Ly.mixed = take(2 * (size_t)d.k * N * d.D * es);
  if (op == WM_OP_ROUTER_MIX || op == WM_OP_KV_PROJECT || all || pool)
    Ly.rinv_mid = take(2 * (size_t)d.k * N * 4);
  if (op == WM_OP_KV_PROJECT || op == WM_OP_Q_PROJECT || all || pool || layer)
    Ly.tab = take(N * d.d * 4);
  if (all) Ly.q = take((size_t)d.L * N * d.Hq * d.d * es);
  if (layer) Ly.q = take(N * d.Hq * d.d * es);
  if ((op == WM_OP_CHANNEL_ATTEND || all) && decode_path(d))
    Ly.part = take(wm::decode_partials_bytes(make_shape(d)));
  if (op == WM_OP_DENSE_ATTEND) {
    const size_t cache = (size_t)d.L * d.B * d.Hkv * d.S_cap * d.d * es;
    Ly.kl = take(cache);
    Ly.vl = take(cache);
    Ly.kdl = take((size_t)d.L * d.Hkv * d.d * es);
    Ly.vdl = take((size_t)d.L * d.Hkv * d.d * es);
    if (decode_path(d)) Ly.part = take(wm::decode_partials_bytes(dense_shape(make_shape(d))));
  }
  if (layer && decode_path(d)) Ly.part = take(wm::decode_partials_bytes(one_layer(make_shape(d))));
  if (op == WM_OP_ATTEND_BACKWARD) Ly.part = take(wm::attend_backward_rows_bytes(make_shape(d)));
  // the full-sequence attention's work queue (or its split ranges' partial states) takes
  // the decode partials' place
  if (!decode_path(d) && (op == WM_OP_CHANNEL_ATTEND || all || layer || op == WM_OP_DENSE_ATTEND)) {
    const wm::Shape sp = layer ? one_layer(make_shape(d))
                               : op == WM_OP_DENSE_ATTEND ? dense_shape(make_shape(d)) : make_shape(d);
    Ly.part = take(wm::prefill_scratch_bytes(sp));
  }
  if (op == WM_OP_KV_PROJECT || all || pool) Ly.wkv = take(wm::kv_fold_elems(make_shape(d)) * es);
  if (op == WM_OP_Q_PROJECT || all || layer) Ly.wq = take(wm::q_fold_elems(make_shape(d)) * es);
  if (op == WM_OP_ROUTER_MIX || all || pool) {
    Ly.wa = take(wm::router_fold_elems(make_shape(d)) * es);
    Ly.rpart = take(wm::router_partials_bytes(make_shape(d)));
  }
  Ly.total = N == 0 ? 0 : off;
  return Ly;
}

bool uses_cache(int op) {
  return op == WM_OP_KV_PROJECT || op == WM_OP_CHANNEL_ATTEND || op == WM_OP_LAYER_STEP ||
         op == WM_OP_POOL || op == WM_OP_LAYER_ATTEND || op == WM_OP_PASSES ||
         op == WM_OP_DENSE_ATTEND || op == WM_OP_ATTEND_BACKWARD || op == WM_OP_POOL_BACKWARD ||
         op == WM_OP_STEP_BACKWARD || op == WM_OP_PASSES_BACKWARD;
}

int validate_dims(const wm_dims* dp, int op, const int32_t* chan_map) {
  if (!dp) return fail(WM_ERR_ARG, "dims is NULL");
  const wm_dims& d = *dp;
  if (op < WM_OP_ROUTER_MIX || op > WM_OP_PASSES_BACKWARD) return fail(WM_ERR_ARG, "unknown op %d", op);
  if (d.dtype != WM_F32 && d.dtype != WM_BF16) return fail(WM_ERR_DTYPE, "unknown dtype %d", d.dtype);
  if (d.mix_mode != WM_MIX_LINEAR && d.mix_mode != WM_MIX_SOFTMAX)
    return fail(WM_ERR_DTYPE, "unknown mix_mode %d", d.mix_mode);
  if (d.mask_mode != WM_MASK_PAPER && d.mask_mode != WM_MASK_INCLUSIVE)
    return fail(WM_ERR_DTYPE, "unknown mask_mode %d", d.mask_mode);
  if (d.router_mode < WM_ROUTER_DYNAMIC || d.router_mode > WM_ROUTER_NOFEEDBACK)
    return fail(WM_ERR_DTYPE, "unknown router_mode %d", d.router_mode);
  if (d.B < 0 || d.T_new < 0) return fail(WM_ERR_ARG, "B and T_new must be >= 0");
  if (d.L < 1 || d.L > wm::kMaxLayers) return fail(WM_ERR_SHAPE, "L must be in [1, %d]", wm::kMaxLayers);
  if (d.k < 1 || d.k > d.L) return fail(WM_ERR_SHAPE, "k must be in [1, L]");
  if (d.router_mode == WM_ROUTER_NOFEEDBACK && d.k != d.L)
    return fail(WM_ERR_SHAPE, "router_mode WM_ROUTER_NOFEEDBACK needs k = L");
  if (d.D < 32 || d.D % 32 != 0) return fail(WM_ERR_SHAPE, "D must be a positive multiple of 32");
  if (d.Hq < 1 || d.Hkv < 1 || d.Hq % d.Hkv != 0)
    return fail(WM_ERR_SHAPE, "Hq must be a positive multiple of Hkv");
  if (d.d != 32 && d.d != 64 && d.d != 96)
    return fail(WM_ERR_SHAPE, "head dim d must be 32, 64 or 96");
  if (d.d == 96 && d.dtype != WM_BF16)
    return fail(WM_ERR_SHAPE, "head dim 96 is supported in bf16 only");
  if (d.p < 1 || d.p > d.L) return fail(WM_ERR_SHAPE, "p must be in [1, L]");
  if (!(d.eps > 0.f) || !std::isfinite(d.eps)) return fail(WM_ERR_ARG, "eps must be positive");
  if (!(d.rope_theta > 0.f) || !std::isfinite(d.rope_theta))
    return fail(WM_ERR_ARG, "rope_theta must be positive");
  if (d.ctx_max < 0) return fail(WM_ERR_ARG, "ctx_max must be >= 0");
  if (d.groups < 0) return fail(WM_ERR_ARG, "groups must be >= 0");
  if (d.group < 0 || d.group >= group_stride(d))
    return fail(WM_ERR_ARG, "group must be in [0, groups)");
  // positions the call covers: the pass driver's T_new is the whole sequence, the other
  // calls place their tokens at group + groups i
  const bool pass_op = op == WM_OP_PASSES || op == WM_OP_PASSES_BACKWARD;
  const long long span = pass_op ? (long long)d.T_new : call_span(d);
  if ((long long)d.ctx_max + span > INT_MAX / 2)
    return fail(WM_ERR_SHAPE, "positions past the 32-bit range");
  if (uses_cache(op)) {
    if (d.S_cap < 1) return fail(WM_ERR_SHAPE, "S_cap must be >= 1");
    if ((long long)d.ctx_max + span > d.S_cap)
      return fail(WM_ERR_CAPACITY, "ctx_max + the positions of the new tokens = %lld exceeds "
                  "S_cap = %d", (long long)d.ctx_max + span, d.S_cap);
  }
  const long long N = (long long)d.B * d.T_new;
  if (N > (1LL << 30)) return fail(WM_ERR_SHAPE, "B * T_new too large");
  if ((N + 127) / 128 > 65535) return fail(WM_ERR_SHAPE, "B * T_new exceeds the grid limit");
  if ((long long)d.Hq * d.B * d.L > 65535 || (long long)d.Hkv * d.B * d.k > 65535)
    return fail(WM_ERR_SHAPE, "heads x sequences x layers exceeds the grid limit");
  if (op == WM_OP_DENSE_ATTEND && (long long)d.L * d.B * d.Hkv > 65535)
    return fail(WM_ERR_SHAPE, "layers x sequences x KV heads exceeds the grid limit");
  {
    // tiles are read through 32-bit buffer views: every operand view must span < 2 GiB
    const double es = (double)elem_size(d), lim = 2147483647.0;
    const double views[] = {(double)N * d.L * d.D * es,            // H
                            (double)N * d.D * es,                  // one mixed channel
                            (double)d.S_cap * d.d * es,            // one cache slice
                            (double)d.Hq * d.d * d.D * es,         // one Q projection
                            (double)d.Hkv * d.d * d.D * es,        // one K/V projection
                            2.0 * d.k * d.L * ((d.L + d.p - 1) / d.p) * d.D * es};  // router
    for (double v : views)
      if (v >= lim) return fail(WM_ERR_SHAPE, "an operand spans more than 2 GiB (%.0f B)", v);
  }
  if (pass_op) {
    if (d.group != 0) return fail(WM_ERR_ARG, "the pass driver runs every group: group must be 0");
    if (d.T_new % group_stride(d) != 0)
      return fail(WM_ERR_SHAPE, "the pass driver needs T_new a multiple of groups");
    if (d.ctx_max != 0) return fail(WM_ERR_ARG, "the pass driver starts empty sequences: ctx_max 0");
  }
  if (op == WM_OP_ROUTER_MIX || op == WM_OP_LAYER_STEP || op == WM_OP_POOL ||
      op == WM_OP_PASSES || op == WM_OP_POOL_BACKWARD || op == WM_OP_STEP_BACKWARD ||
      op == WM_OP_PASSES_BACKWARD) {
    size_t lds = wm::mix_smem_bytes(d.L, d.k, d.D, elem_size(d));
    if (lds > 65536) return fail(WM_ERR_SHAPE, "L * D too large for the mix kernel (%zu B of LDS)", lds);
  }
  if (chan_map) {
    for (int l = 0; l < d.L; ++l)
      if (chan_map[l] < 0 || chan_map[l] >= d.k)
        return fail(WM_ERR_MAP, "chan_map[%d] = %d is outside [0, %d)", l, chan_map[l], d.k);
  }
  return WM_OK;
}

int need_ptr(const void* p, const char* name) {
  if (!p) return fail(WM_ERR_ARG, "%s is NULL", name);
  if ((uintptr_t)p % 16 != 0) return fail(WM_ERR_ARG, "%s is not 16-byte aligned", name);
  return WM_OK;
}

int check_ws(const wm_dims& d, int op, void* ws, size_t ws_bytes) {
  size_t need = layout(d, op).total;
  if (need == 0) return WM_OK;
  if (!ws) return fail(WM_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if ((uintptr_t)ws % 256 != 0) return fail(WM_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (ws_bytes < need) return fail(WM_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  return WM_OK;
}

int launched() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(WM_ERR_LAUNCH, "launch failed: %s", hipGetErrorString(e));
  return WM_OK;
}

#define WM_TRY(x)              \
  do {                         \
    int _rc = (x);             \
    if (_rc != WM_OK) return _rc; \
  } while (0)

wm::LayerTable router_layers(const wm_dims& d) {
  wm::LayerTable t{};
  int Lp = (d.L + d.p - 1) / d.p;
  for (int m = 0; m < Lp; ++m) t.v[Lp - 1 - m] = d.L - 1 - d.p * m;
  return t;
}

wm::LayerTable map_table(const wm_dims& d, const int32_t* chan_map) {
  wm::LayerTable t{};
  for (int l = 0; l < d.L; ++l) t.v[l] = chan_map[l];
  return t;
}

wm::ChannelGroups groups(const wm_dims& d, const int32_t* chan_map) {
  wm::ChannelGroups g{};
  wm_channel_groups(d.L, d.k, chan_map, g.offsets, g.members);
  return g;
}

char* at(void* ws, size_t off) { return (char*)ws + off; }

// ----------------------------------------------------------------- ops
template <typename T>
void run_router_mix(const wm_dims& d, const wm_params& P, const T* H, float* alpha_out, T* mixed,
                    void* ws, hipStream_t s) {
  wm::Shape sh = make_shape(d);
  Layout Ly = layout(d, WM_OP_ROUTER_MIX);
  float* rinv = (float*)at(ws, Ly.rinv);
  float* alpha = alpha_out ? alpha_out : (float*)at(ws, Ly.alpha);
  wm::launch_row_rms<T>(H, (long)sh.N() * sh.L, sh.D, sh.eps, rinv, s);
  wm::launch_router<T>(sh, router_layers(d), H, rinv, (const T*)P.g_pre, (const T*)P.W_alpha,
                       (const T*)P.b_alpha, alpha, (T*)at(ws, Ly.wa), (float*)at(ws, Ly.rpart),
                       s);
  wm::launch_mix<T>(sh, H, rinv, (const T*)P.g_pre, alpha, mixed, (float*)at(ws, Ly.rinv_mid), s);
}

template <typename T>
void run_kv_project(const wm_dims& d, const wm_params& P, const T* mixed, const int32_t* ctx_len,
                    T* Kc, T* Vc, void* ws, hipStream_t s) {
  wm::Shape sh = make_shape(d);
  Layout Ly = layout(d, WM_OP_KV_PROJECT);
  float* rinv_mid = (float*)at(ws, Ly.rinv_mid);
  float* tab = (float*)at(ws, Ly.tab);
  wm::launch_row_rms<T>(mixed, 2L * sh.k * sh.N(), sh.D, sh.eps, rinv_mid, s);
  wm::launch_rope_table(sh, ctx_len, tab, s);
  wm::launch_kv_project<T>(sh, mixed, rinv_mid, (const T*)P.g_mid, (const T*)P.Wk,
                           (const T*)P.Wv, (const T*)P.g_knorm, tab, ctx_len, Kc, Vc,
                           (T*)at(ws, Ly.wkv), s);
}

template <typename T>
void run_q_project(const wm_dims& d, const wm_params& P, const T* H, const int32_t* ctx_len, T* Q,
                   void* ws, hipStream_t s) {
  wm::Shape sh = make_shape(d);
  Layout Ly = layout(d, WM_OP_Q_PROJECT);
  float* rinv = (float*)at(ws, Ly.rinv);
  float* tab = (float*)at(ws, Ly.tab);
  wm::launch_row_rms<T>(H, (long)sh.N() * sh.L, sh.D, sh.eps, rinv, s);
  wm::launch_rope_table(sh, ctx_len, tab, s);
  wm::launch_q_project<T>(sh, H, rinv, (const T*)P.g_in, (const T*)P.Wq, (const T*)P.g_qnorm,
                          tab, Q, (T*)at(ws, Ly.wq), s);
}

template <typename T>
void run_attend(const wm_dims& d, const wm_params& P, const T* Q, const int32_t* chan_map,
                const int32_t* ctx_len, const int32_t* doc, const T* Kc, const T* Vc, T* O,
                float* part, hipStream_t s) {
  wm::Shape sh = make_shape(d);
  wm::LayerTable mt = map_table(d, chan_map);
  if (decode_path(d))
    wm::launch_attend_decode<T>(sh, mt, groups(d, chan_map), Q, Kc, Vc, (const T*)P.Kd,
                                (const T*)P.Vd, ctx_len, doc, part, O, s);
  else
    wm::launch_attend_prefill<T>(sh, mt, Q, Kc, Vc, (const T*)P.Kd, (const T*)P.Vd, ctx_len, doc,
                                 O, (uint32_t*)part, s);
}

template <typename T>
int run_layer_step(const wm_dims& d, const wm_params& P, const T* H, const int32_t* chan_map,
                   const int32_t* ctx_len, const int32_t* doc, T* Kc, T* Vc, T* O, void* ws,
                   hipStream_t s, void* const* events) {
  auto mark = [&](int i) {
    if (events) (void)hipEventRecord((hipEvent_t)events[i], s);
  };
  wm::Shape sh = make_shape(d);
  Layout Ly = layout(d, WM_OP_LAYER_STEP);
  float* rinv = (float*)at(ws, Ly.rinv);
  float* alpha = (float*)at(ws, Ly.alpha);
  T* mixed = (T*)at(ws, Ly.mixed);
  float* rinv_mid = (float*)at(ws, Ly.rinv_mid);
  float* tab = (float*)at(ws, Ly.tab);
  T* Q = (T*)at(ws, Ly.q);
  mark(0);
  wm::launch_row_rms<T>(H, (long)sh.N() * sh.L, sh.D, sh.eps, rinv, s);
  wm::launch_rope_table(sh, ctx_len, tab, s);
  mark(1);
  wm::launch_router<T>(sh, router_layers(d), H, rinv, (const T*)P.g_pre, (const T*)P.W_alpha,
                       (const T*)P.b_alpha, alpha, (T*)at(ws, Ly.wa), (float*)at(ws, Ly.rpart),
                       s);
  mark(2);
  wm::launch_mix<T>(sh, H, rinv, (const T*)P.g_pre, alpha, mixed, rinv_mid, s);
  mark(3);
  wm::launch_kv_project<T>(sh, mixed, rinv_mid, (const T*)P.g_mid, (const T*)P.Wk,
                           (const T*)P.Wv, (const T*)P.g_knorm, tab, ctx_len, Kc, Vc,
                           (T*)at(ws, Ly.wkv), s);
  mark(4);
  wm::launch_q_project<T>(sh, H, rinv, (const T*)P.g_in, (const T*)P.Wq, (const T*)P.g_qnorm,
                          tab, Q, (T*)at(ws, Ly.wq), s);
  mark(5);
  run_attend<T>(d, P, Q, chan_map, ctx_len, doc, Kc, Vc, O, (float*)at(ws, Ly.part), s);
  mark(6);
  return WM_OK;
}

// Steps 1-2 for the call's tokens: row norms (unless have_rinv), angle table (unless
// have_tab), router, mix, K/V projection into the cache. prefolded: the workspace already
// holds the gain-folded router and K/V weights.
template <typename T>
void run_pool(const wm_dims& d, const wm_params& P, const T* H, const int32_t* ctx_len, T* Kc,
              T* Vc, const Layout& Ly, void* ws, hipStream_t s, bool have_rinv, bool have_tab,
              bool prefolded) {
  wm::Shape sh = make_shape(d);
  float* rinv = (float*)at(ws, Ly.rinv);
  float* alpha = (float*)at(ws, Ly.alpha);
  T* mixed = (T*)at(ws, Ly.mixed);
  float* rinv_mid = (float*)at(ws, Ly.rinv_mid);
  float* tab = (float*)at(ws, Ly.tab);
  if (!have_rinv) wm::launch_row_rms<T>(H, (long)sh.N() * sh.L, sh.D, sh.eps, rinv, s);
  if (!have_tab) wm::launch_rope_table(sh, ctx_len, tab, s);
  wm::launch_router<T>(sh, router_layers(d), H, rinv, (const T*)P.g_pre, (const T*)P.W_alpha,
                       (const T*)P.b_alpha, alpha, (T*)at(ws, Ly.wa), (float*)at(ws, Ly.rpart),
                       s, prefolded);
  wm::launch_mix<T>(sh, H, rinv, (const T*)P.g_pre, alpha, mixed, rinv_mid, s);
  wm::launch_kv_project<T>(sh, mixed, rinv_mid, (const T*)P.g_mid, (const T*)P.Wk,
                           (const T*)P.Wv, (const T*)P.g_knorm, tab, ctx_len, Kc, Vc,
                           (T*)at(ws, Ly.wkv), s, prefolded);
}

// Consumer l alone: input norm of h_l = H[..][l][..], W^Q_l, q norm, RoPE (angle table
// unless have_tab), then attention over channel chan_map[l] into O_l [B][T_new][Hq d].
// q_prefolded: the workspace already holds the gain-folded query weights of every layer.
template <typename T>
void run_layer_attend(const wm_dims& d, const wm_params& P, int l, const T* H,
                      const int32_t* chan_map, const int32_t* ctx_len, const T* Kc, const T* Vc,
                      T* O_l, const Layout& Ly, void* ws, hipStream_t s, bool have_tab,
                      bool q_prefolded) {
  wm::Shape sh = make_shape(d);
  float* rinv = (float*)at(ws, Ly.rinv);
  float* tab = (float*)at(ws, Ly.tab);
  T* Q = (T*)at(ws, Ly.q);
  T* wq = (T*)at(ws, Ly.wq);
  wm::launch_row_rms_strided<T>(H + (long)l * sh.D, sh.N(), sh.D, (long)sh.L * sh.D, sh.L, sh.eps,
                                rinv + l, s);
  if (!have_tab) wm::launch_rope_table(sh, ctx_len, tab, s);
  if (!q_prefolded) wm::launch_q_fold<T>(sh, (const T*)P.g_in, (const T*)P.Wq, wq, l, 1, s);
  wm::launch_q_layers<T>(sh, H, rinv, (const T*)P.g_qnorm, tab, Q, wq, l, 1, s);
  const wm::Shape sh1 = one_layer(sh);
  wm::LayerTable mt{};
  mt.v[0] = chan_map[l];
  if (decode_path(d)) {
    wm::ChannelGroups cg{};
    wm_channel_groups(1, d.k, &chan_map[l], cg.offsets, cg.members);
    wm::launch_attend_decode<T>(sh1, mt, cg, Q, Kc, Vc, (const T*)P.Kd, (const T*)P.Vd, ctx_len,
                                nullptr, (float*)at(ws, Ly.part), O_l, s);
  } else {
    wm::launch_attend_prefill<T>(sh1, mt, Q, Kc, Vc, (const T*)P.Kd, (const T*)P.Vd, ctx_len,
                                 nullptr, O_l, (uint32_t*)at(ws, Ly.part), s);
  }
}

// Section 3.3: the cache starts as Pool(H^(0)) (every layer's state the embedding X);
// each pass runs the g strided groups in order, and group q first recomputes the states
// of its positions layer by layer (its consumers' attention over the cache as it stands,
// then the stand-in block h_{l+1} = h_l + W_o[l] o_l), then pools them into its slots.
template <typename T>
void run_passes(const wm_dims& d, const wm_params& P, const T* W_o, const T* X,
                const int32_t* chan_map, int passes, T* Kc, T* Vc, T* H, T* h_top, void* ws,
                hipStream_t s) {
  const int g = group_stride(d), Tg = d.T_new / g, L = d.L, D = d.D, HD = d.Hq * d.d;
  const Layout Ly = layout(d, WM_OP_PASSES);
  const wm::Shape sh0 = make_shape(group_dims(d, 0));
  T* Hg = (T*)at(ws, Ly.hg);
  T* topg = (T*)at(ws, Ly.topg);
  T* Ol = (T*)at(ws, Ly.ol);
  const long gsz = (long)d.B * Tg * L * D;  // one group's states
  wm::launch_router_fold<T>(sh0, router_layers(d), (const T*)P.g_pre, (const T*)P.W_alpha,
                            (T*)at(ws, Ly.wa), s);
  wm::launch_kv_fold<T>(sh0, (const T*)P.g_mid, (const T*)P.Wk, (const T*)P.Wv,
                        (T*)at(ws, Ly.wkv), s);
  wm::launch_q_fold<T>(sh0, (const T*)P.g_in, (const T*)P.Wq, (T*)at(ws, Ly.wq), 0, L, s);
  wm::launch_group_gather<T>(X, Hg, d.B, d.T_new, g, L, D, s);
  for (int q = 0; q < g; ++q)
    run_pool<T>(group_dims(d, q), P, Hg + q * gsz, nullptr, Kc, Vc, Ly, ws, s, false, false,
                true);
  for (int t = 0; t < passes; ++t) {
    for (int q = 0; q < g; ++q) {
      const wm_dims dq = group_dims(d, q);
      T* Hq = Hg + q * gsz;
      wm::launch_rope_table(make_shape(dq), nullptr, (float*)at(ws, Ly.tab), s);
      for (int l = 0; l < L; ++l) {
        run_layer_attend<T>(dq, P, l, Hq, chan_map, nullptr, Kc, Vc, Ol, Ly, ws, s, true, true);
        const bool last = l + 1 == L;
        wm::launch_block_residual<T>(d.B * Tg, D, HD, Ol, W_o + (long)l * D * HD,
                                     Hq + (long)l * D, (long)L * D,
                                     last ? topg + (long)q * d.B * Tg * D : Hq + (long)(l + 1) * D,
                                     last ? D : (long)L * D, s);
      }
      // every layer's row norms are already current: only the pool remains
      run_pool<T>(dq, P, Hq, nullptr, Kc, Vc, Ly, ws, s, true, true, true);
    }
  }
  wm::launch_group_scatter<T>(Hg, H, d.B, d.T_new, g, (long)L * D, s);
  if (h_top) wm::launch_group_scatter<T>(topg, h_top, d.B, d.T_new, g, D, s);
}

// The dense soft read: every consumer's mix of the k channels into the workspace, then the
// attention of L consumers over L mixed channels (consumer l reads its own).
template <typename T>
void run_attend_dense(const wm_dims& d, const wm_params& P, const float* read_w, const T* Q,
                      const int32_t* ctx_len, const T* Kc, const T* Vc, T* O, void* ws,
                      hipStream_t s) {
  const Layout Ly = layout(d, WM_OP_DENSE_ATTEND);
  const wm::Shape sh = make_shape(d);
  T* Kl = (T*)at(ws, Ly.kl);
  T* Vl = (T*)at(ws, Ly.vl);
  T* Kdl = (T*)at(ws, Ly.kdl);
  T* Vdl = (T*)at(ws, Ly.vdl);
  wm::launch_soft_read<T>(sh, read_w, Kc, Vc, (const T*)P.Kd, (const T*)P.Vd, ctx_len, Kl, Vl,
                          Kdl, Vdl, s);
  const wm::Shape shd = dense_shape(sh);
  wm::LayerTable ident{};
  for (int l = 0; l < d.L; ++l) ident.v[l] = l;
  if (decode_path(d)) {
    wm::ChannelGroups cg{};
    int32_t map[wm::kMaxLayers];
    for (int l = 0; l < d.L; ++l) map[l] = l;
    wm_channel_groups(d.L, d.L, map, cg.offsets, cg.members);
    wm::launch_attend_decode<T>(shd, ident, cg, Q, Kl, Vl, Kdl, Vdl, ctx_len, nullptr,
                                (float*)at(ws, Ly.part), O, s);
  } else {
    wm::launch_attend_prefill<T>(shd, ident, Q, Kl, Vl, Kdl, Vdl, ctx_len, nullptr, O,
                                 (uint32_t*)at(ws, Ly.part), s);
  }
}

int check_params(const wm_params* P, std::initializer_list<int> which) {
  if (!P) return fail(WM_ERR_ARG, "params is NULL");
  static const char* names[] = {"g_pre", "W_alpha", "b_alpha", "g_mid", "Wk", "Wv",
                                "g_knorm", "Kd", "Vd", "g_in", "Wq", "g_qnorm"};
  const void* ptrs[] = {P->g_pre, P->W_alpha, P->b_alpha, P->g_mid, P->Wk, P->Wv,
                        P->g_knorm, P->Kd, P->Vd, P->g_in, P->Wq, P->g_qnorm};
  for (int i : which) {
    if (!ptrs[i]) return fail(WM_ERR_ARG, "params->%s is NULL", names[i]);
    if ((uintptr_t)ptrs[i] % 16 != 0)
      return fail(WM_ERR_ARG, "params->%s is not 16-byte aligned", names[i]);
  }
  return WM_OK;
}

enum { P_GPRE, P_WA, P_BA, P_GMID, P_WK, P_WV, P_GKN, P_KD, P_VD, P_GIN, P_WQ, P_GQN };

// The array's device address, looked up once per device with that device current (in host
// code the array's name is only a stand-in, never a device address).
constexpr int kMaxDevices = 64;
struct ScratchAddr {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t rc = hipSuccess;
};
ScratchAddr g_scratch_addr[kMaxDevices];

int static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(WM_ERR_LAUNCH, "no current HIP device below %d", kMaxDevices);
  ScratchAddr& a = g_scratch_addr[dev];
  std::call_once(a.once, [&] { a.rc = hipGetSymbolAddress(&a.ptr, HIP_SYMBOL(scratch)); });
  if (a.rc != hipSuccess || !a.ptr)
    return fail(WM_ERR_LAUNCH, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                hipGetErrorString(a.rc));
  *out = a.ptr;
  return WM_OK;
}


// ------------------------------------------------------------------ gradients
wm::GemmOperand opnd(const void* p, long s_row, long s_k, long s_z, bool f32, bool pad8 = false) {
  return wm::GemmOperand{p, s_row, s_k, s_z, f32 ? 1 : 0, pad8 ? 1 : 0, 0};
}

// C[z] (+)= A[z] B[z]^T over `batches`; see GemmArgs for the k / row limits.
// part: kSplitElems floats of split-K scratch (or NULL: no split)
void gemm(const wm::GemmOperand& A, const wm::GemmOperand& B, float* C, long c_row, long c_col,
          long c_z, int M, int N, int K, int batches, bool acc, hipStream_t s, long klo0 = 0,
          long klo_dz = 0, long mlo0 = 0, long mlo_dz = 0, float* part = nullptr) {
  wm::GemmArgs g{A, B, C, c_row, c_col, c_z, M, N, K, acc ? 1 : 0, klo0, klo_dz, mlo0, mlo_dz,
                 part, part ? (long)kSplitElems : 0, 1, 0};
  wm::launch_grad_gemm(g, batches, s);
}

// RMSNorm backward over rows (o, i) of D, gain rows o < nouter; dg partials in dgp.
void rms_backward(const float* dy, long dy_o, long dy_i, const bf16* x, long x_o, long x_i,
                  float* out, long out_o, long out_i, const float* rinv, long r_o, long r_i,
                  const bf16* g, int D, int nouter, int ninner, bool acc, float* dgp,
                  hipStream_t s, int* chunks) {
  wm::RmsArgs a;
  a.dy = dy, a.dy_o = dy_o, a.dy_i = dy_i;
  a.x = x, a.x_o = x_o, a.x_i = x_i;
  a.out = out, a.out_o = out_o, a.out_i = out_i;
  a.rinv = rinv, a.r_o = r_o, a.r_i = r_i;
  a.g = g, a.dgp = dgp;
  a.D = D, a.ninner = ninner, a.chunks = red_chunks(nouter), a.accumulate = acc ? 1 : 0;
  *chunks = a.chunks;
  wm::launch_grad_rms(a, nouter, s);
}

int grad_ptr(const float* p, const char* name) {
  if (!p) return fail(WM_ERR_ARG, "grads->%s is NULL", name);
  if ((uintptr_t)p % 4 != 0) return fail(WM_ERR_ARG, "grads->%s is not 4-byte aligned", name);
  return WM_OK;
}

// What every gradient op supports: bf16, head dims 64 and 96, rows of at most 4608 for the
// norms' backward, and the mix gradient's LDS.
int check_backward(const wm_dims& d) {
  if (d.dtype != WM_BF16) return fail(WM_ERR_DTYPE, "the gradients are built for bf16");
  if (d.d != 64 && d.d != 96) return fail(WM_ERR_SHAPE, "the gradients support head dims 64 and 96");
  if (d.D > 4608) return fail(WM_ERR_SHAPE, "the gradients support D <= 4608");
  if (wm::grad_mix_smem(d.L, d.k, d.D) > 65536)
    return fail(WM_ERR_SHAPE, "L and k too large for the mix gradient's LDS");
  return WM_OK;
}

// Gradients of the queries (input norm, W^Q, q norm, RoPE) for dQ [L][B][Hq][T][d]: into
// dH [N][L][D] and the gradients of g_in, Wq, g_qnorm (all added).
void run_q_backward(const wm_dims& d, const wm_params& P, const bf16* H, const int32_t* ctx_len,
                    const float* dQ, float* dH, const wm_grads& G, const Layout& Ly, void* ws,
                    hipStream_t s) {
  const wm::Shape sh = make_shape(d);
  const int N = sh.N(), L = d.L, D = d.D, HQ = d.Hq * d.d;
  float* rinv = (float*)at(ws, Ly.rinv);
  float* tab = (float*)at(ws, Ly.tab);
  float* dgp = (float*)at(ws, Ly.dgp);
  bf16* x = (bf16*)at(ws, Ly.x);
  float* yq = (float*)at(ws, Ly.yq);
  bf16* dyq = (bf16*)at(ws, Ly.dyq);
  float* dx = (float*)at(ws, Ly.dx);
  const bf16* Wq = (const bf16*)P.Wq;
  wm::launch_row_rms<bf16>(H, (long)N * L, D, sh.eps, rinv, s);
  wm::launch_rope_table(sh, ctx_len, tab, s);
  // x[n][l] = g_in[l] h[n][l] / rms (bf16), then y_l = x_l Wq_l^T [N][HQ] per layer
  wm::launch_grad_norm_apply(H, (const bf16*)P.g_in, rinv, (long)N * L, 1, L, D, x, s);
  gemm(opnd(x, (long)L * D, 1, D, false), opnd(Wq, D, 1, (long)HQ * D, false), yq, HQ, 1,
       (long)N * HQ, N, HQ, D, L, false, s);
  // RoPE and q norm backward: y's gradient (bf16)
  wm::HeadArgs h{};
  h.src = dQ, h.sZ = (long)d.B * d.Hq * d.T_new, h.sB = (long)d.Hq * d.T_new, h.sH = d.T_new;
  h.slot_ctx = 0, h.ctx_len = ctx_len, h.ctx_hi = sh.ctx_hi, h.gs = 1, h.gq = 0;
  h.y = yq, h.dy = dyq, h.g = (const bf16*)P.g_qnorm, h.tab = tab, h.dgp = dgp;
  h.B = d.B, h.H = d.Hq, h.T = d.T_new, h.chunks = red_chunks(L), h.eps = d.eps;
  wm::launch_grad_head(h, L, d.d, s);
  wm::launch_grad_sum(dgp, L, h.chunks, d.d, G.g_qnorm, 1.f, 1, s);
  // dx_l = dy_l Wq_l [N][D] (into [N][L][D]); dWq_l += dy_l^T x_l [HQ][D]
  gemm(opnd(dyq, HQ, 1, (long)N * HQ, false), opnd(Wq, 1, D, (long)HQ * D, false), dx,
       (long)L * D, 1, D, N, D, HQ, L, false, s);
  gemm(opnd(dyq, 1, HQ, (long)N * HQ, false), opnd(x, 1, (long)L * D, D, false), G.Wq, D, 1,
       (long)HQ * D, HQ, D, N, L, true, s, 0, 0, 0, 0, (float*)at(ws, Ly.split));
  // input norm backward: rows (l, n) at n L + l
  int nch = 0;
  rms_backward(dx, 1, L, H, 1, L, dH, 1, L, rinv, 1, L, (const bf16*)P.g_in, D, L, N, true, dgp,
               s, &nch);
  wm::launch_grad_sum(dgp, L, nch, D, G.g_in, 1.f, 1, s);
}

// Gradients of the pool (Steps 1-2) for the gradients of the call's new cache slots
// (dKc, dVc at slot ctx_len[b] + i): into dH and the gradients of g_pre, W_alpha (not with
// static weights), b_alpha, g_mid, Wk, Wv, g_knorm (all added). The forward's router, mix
// and norms are recomputed with the forward kernels.
void run_pool_backward(const wm_dims& d, const wm_params& P, const bf16* H,
                       const int32_t* ctx_len, const float* dKc, const float* dVc, float* dH,
                       const wm_grads& G, const Layout& Ly, void* ws, hipStream_t s) {
  const wm::Shape sh = make_shape(d);
  const int N = sh.N(), L = d.L, k = d.k, D = d.D, HK = d.Hkv * d.d, Lp = sh.Lp;
  const int kL = k * L;
  float* rinv = (float*)at(ws, Ly.rinv);
  float* tab = (float*)at(ws, Ly.tab);
  float* dgp = (float*)at(ws, Ly.dgp);
  float* alpha = (float*)at(ws, Ly.alpha);
  bf16* mixed = (bf16*)at(ws, Ly.mixed);
  float* rinv_mid = (float*)at(ws, Ly.rinv_mid);
  bf16* hn = (bf16*)at(ws, Ly.hn);
  bf16* u = (bf16*)at(ws, Ly.u);
  float* ydy = (float*)at(ws, Ly.ydy);
  bf16* dyb = (bf16*)at(ws, Ly.dyb);
  float* du = (float*)at(ws, Ly.du);
  float* dhn = (float*)at(ws, Ly.dhn);
  float* dlog = (float*)at(ws, Ly.dlog);
  bf16* dlogb = (bf16*)at(ws, Ly.dlogb);
  const int kLp = (kL + 7) & ~7;
  const wm::LayerTable sel = router_layers(d);
  const bool dynamic = d.router_mode != WM_ROUTER_STATIC;
  const bool nofb = d.router_mode == WM_ROUTER_NOFEEDBACK;
  wm::launch_row_rms<bf16>(H, (long)N * L, D, sh.eps, rinv, s);
  wm::launch_rope_table(sh, ctx_len, tab, s);
  wm::launch_router<bf16>(sh, sel, H, rinv, (const bf16*)P.g_pre, (const bf16*)P.W_alpha,
                          (const bf16*)P.b_alpha, alpha, (bf16*)at(ws, Ly.wa),
                          (float*)at(ws, Ly.rpart), s);
  wm::launch_mix<bf16>(sh, H, rinv, (const bf16*)P.g_pre, alpha, mixed, rinv_mid, s);
  for (int br = 0; br < 2; ++br) {
    const bf16* gpre = (const bf16*)P.g_pre + (long)br * L * D;
    const bf16* gmid = (const bf16*)P.g_mid + (long)br * k * D;
    const bf16* W = (const bf16*)(br ? P.Wv : P.Wk);
    const bf16* mix_b = mixed + (long)br * k * N * D;
    const float* rmid = rinv_mid + (long)br * k * N;
    // u_j = g_mid[j] mixed_j / rms (bf16 [k][N][D])
    wm::launch_grad_norm_apply(mix_b, gmid, rmid, (long)k * N, N, k, D, u, s);
    if (br == 0) {
      // y_j = u_j Wk_j^T [N][HK], then RoPE and key norm backward (y's gradient, bf16)
      gemm(opnd(u, D, 1, (long)N * D, false), opnd(W, D, 1, (long)HK * D, false), ydy, HK, 1,
           (long)N * HK, N, HK, D, k, false, s);
      wm::HeadArgs h{};
      h.src = dKc, h.sZ = (long)d.B * d.Hkv * d.S_cap, h.sB = (long)d.Hkv * d.S_cap;
      h.sH = d.S_cap, h.slot_ctx = 1, h.ctx_len = ctx_len, h.ctx_hi = sh.ctx_hi;
      h.gs = sh.gs, h.gq = sh.gq;
      h.y = ydy, h.dy = dyb, h.g = (const bf16*)P.g_knorm, h.tab = tab, h.dgp = dgp;
      h.B = d.B, h.H = d.Hkv, h.T = d.T_new, h.chunks = red_chunks(k), h.eps = d.eps;
      wm::launch_grad_head(h, k, d.d, s);
      wm::launch_grad_sum(dgp, k, h.chunks, d.d, G.g_knorm, 1.f, 1, s);
    } else {
      wm::launch_grad_gather(dVc, k, d.B, d.Hkv, d.T_new, d.S_cap, d.d, ctx_len, sh.ctx_hi, sh.gs,
                             sh.gq, dyb, s);
    }
    // du_j = dy_j W_j [N][D]; dW_j += dy_j^T u_j [HK][D]
    gemm(opnd(dyb, HK, 1, (long)N * HK, false), opnd(W, 1, D, (long)HK * D, false), du, D, 1,
         (long)N * D, N, D, HK, k, false, s);
    gemm(opnd(dyb, 1, HK, (long)N * HK, false), opnd(u, 1, D, (long)N * D, false),
         br ? G.Wv : G.Wk, D, 1, (long)HK * D, HK, D, N, k, true, s, 0, 0, 0, 0,
         (float*)at(ws, Ly.split));
    // mid norm backward in place: du becomes the mixed channels' gradient
    int nch = 0;
    rms_backward(du, N, 1, mix_b, N, 1, du, N, 1, rmid, N, 1, gmid, D, k, N, false, dgp, s, &nch);
    wm::launch_grad_sum(dgp, k, nch, D, G.g_mid + (long)br * k * D, 1.f, 1, s);
    // mix backward: dhn (written) and the logits' gradient
    wm::MixGradArgs m{H, gpre, rinv, du, alpha + (long)br * N * kL, dhn, dlog, dlogb, N, L, k,
                      D, d.mix_mode == WM_MIX_SOFTMAX ? 1 : 0, nofb ? 1 : 0, kLp};
    wm::launch_grad_mix(m, s);
    wm::launch_grad_colsum(dlog, N, kL, kGradChunks, dgp, s);
    wm::launch_grad_sum(dgp, 1, kGradChunks, kL, G.b_alpha + (long)br * kL, 1.f, 1, s);
    if (dynamic) {
      wm::launch_grad_norm_apply(H, gpre, rinv, (long)N * L, 1, L, D, hn, s);
      // stacked source m is layer sel[m] = sel[0] + p m. dhn[n][sel[m]] += dlog[n] W_alpha[:, m]
      // and dW_alpha[:, m] += dlog^T hn[:, sel[m]], batched over m; without feedback, router
      // row o reads source m only when sel[m] <= o / L
      const bf16* Wa = (const bf16*)P.W_alpha + (long)br * kL * Lp * D;
      const long s0 = sel.v[0];
      const long klo0 = nofb ? (long)L * s0 : 0, klo_dz = nofb ? (long)L * d.p : 0;
      gemm(opnd(dlogb, kLp, 1, 0, false, true), opnd(Wa, 1, (long)Lp * D, D, false),
           dhn + s0 * D, (long)L * D, 1, (long)d.p * D, N, D, kL, Lp, true, s, klo0, klo_dz);
      gemm(opnd(dlogb, 1, kLp, 0, false, true),
           opnd(hn + s0 * D, 1, (long)L * D, (long)d.p * D, false),
           G.W_alpha + (long)br * kL * Lp * D, (long)Lp * D, 1, D, kL, D, N, Lp, true, s, 0, 0,
           klo0, klo_dz, (float*)at(ws, Ly.split));
    }
    // pre-mix norm backward into dH: rows (l, n) at n L + l
    rms_backward(dhn, 1, L, H, 1, L, dH, 1, L, rinv, 1, L, gpre, D, L, N, true, dgp, s, &nch);
    wm::launch_grad_sum(dgp, L, nch, D, G.g_pre + (long)br * L * D, 1.f, 1, s);
  }
}


// ------------------------------------------- Section 3.3: truncated backpropagation
// Workspace of wm_prefill_passes_backward: the forward's scratch, what the gradient
// window keeps of its passes (the states H^(t) for t = passes - n_grad .. passes, the
// caches and the per-layer attention outputs of the window's passes), and the backward's
// scratch (the Q-side and pool-side gradient workspaces share one region).

wm_dims one_consumer(const wm_dims& d) {
  wm_dims d1 = d;
  d1.L = 1;
  d1.k = 1;
  d1.p = 1;
  return d1;
}

PassBwdLayout passes_bwd_layout(const wm_dims& d, int n_grad) {
  PassBwdLayout Ly;
  const int g = group_stride(d);
  const size_t Ng = (size_t)d.B * (d.T_new / g), L = d.L, D = d.D, HQ = (size_t)d.Hq * d.d;
  const size_t steps = (size_t)n_grad * g;
  Ly.cache = (size_t)d.k * d.B * d.Hkv * d.S_cap * d.d * 2;
  Ly.state = al256(Ng * L * D * 2);
  Ly.slots = al256((size_t)d.k * d.B * d.Hkv * (d.T_new / g) * d.d * 2);
  Ly.outs = al256(L * Ng * HQ * 2);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += al256(bytes);
    return at;
  };
  Ly.fw = take(layout(d, WM_OP_PASSES).total);
  Ly.kv = take(al256(Ly.cache) * 2);
  Ly.hs = take(Ly.state * steps);
  Ly.undo = take(Ly.slots * 2 * steps);
  Ly.op = take(Ly.outs * steps);
  Ly.gcur = take(Ng * D * 4);
  Ly.gb = take(Ng * D * 2);
  Ly.dof = take(Ng * HQ * 4);
  Ly.dob = take(Ng * HQ * 2);
  Ly.dql = take(Ng * HQ * 4);
  Ly.h1 = take(Ng * D * 2);
  Ly.rows = take(wm::attend_backward_rows_bytes(make_shape(one_consumer(group_dims(d, 0)))));
  Ly.gkd = take(2 * (size_t)d.Hkv * d.d * 4);
  Ly.dpk = take(Ly.cache * 2);
  Ly.dpv = take(Ly.cache * 2);
  Ly.dhn = take(Ng * L * D * 4);
  Ly.split = take(kSplitElems * 4);
  wm_dims dq = group_dims(d, 0);
  dq.L = 1;
  Ly.sub = take(std::max(layout(dq, WM_OP_Q_BACKWARD).total,
                         layout(group_dims(d, 0), WM_OP_POOL_BACKWARD).total));
  Ly.total = Ng == 0 ? 0 : off;
  return Ly;
}

// The passes of Section 3.3 over g strided groups (g = 1: Jacobi iteration), as
// wm_prefill_passes runs them: the cache starts as Pool(H^(0) = X in every layer); each
// pass runs the groups in order, group q recomputing the states of its positions layer by
// layer from the cache as it stands, then pooling them into its slots. The passes before
// the gradient window run in scratch; each window step (pass t, group q) keeps its group's
// states, its layers' attention outputs and the slots its pool overwrote. The last step's
// pool is left out: nothing reads the slots it would write.
// The backward walks the window's steps from the last. It holds the loss gradient in the
// whole cache (dK, dV) as the forward left it at that point: the step's pool sends the
// gradient at its slots to its states, and those slots are then given back the values the
// step read (their gradient cleared); its layers from the top down (the stand-in blocks,
// the consumers' attention over the restored cache, whose gradient joins dK, dV, and
// their queries) carry the residual stream's gradient down to X. The cache entering the
// window is held fixed unless the window starts at the initial pool, whose gradient goes
// to X through every layer.
void run_passes_backward(const wm_dims& d, const wm_params& P, const bf16* W_o, const bf16* X,
                         const int32_t* chan_map, int passes, int n_grad, const float* dh_top,
                         bf16* h_top, float* dX, float* dW_o, const wm_grads& G, void* ws,
                         hipStream_t s) {
  const PassBwdLayout Ly = passes_bwd_layout(d, n_grad);
  const Layout Lf = layout(d, WM_OP_PASSES);
  void* fw = at(ws, Ly.fw);
  const int g = group_stride(d), Tg = d.T_new / g, L = d.L, D = d.D, HQ = d.Hq * d.d;
  const int Ng = d.B * Tg;
  const long gsz = (long)Ng * L * D;                        // one group's states
  const long cslice = (long)d.B * d.Hkv * d.S_cap * d.d;  // one channel of a cache
  const long cache_elems = (long)d.k * cslice;
  const long crows = (long)d.k * d.B * d.Hkv;              // cache rows of S_cap slots
  const int first = passes - n_grad;                       // passes before the window
  bf16* K = (bf16*)at(ws, Ly.kv);
  bf16* V = (bf16*)at(ws, Ly.kv + al256(Ly.cache));
  bf16* Hg = (bf16*)at(fw, Lf.hg);
  bf16* topg = (bf16*)at(fw, Lf.topg);
  float* tab = (float*)at(fw, Lf.tab);
  // window step j = (t - first - 1) g + q
  auto Hs = [&](int j) { return (bf16*)at(ws, Ly.hs + Ly.state * j); };
  auto Uk = [&](int j) { return (bf16*)at(ws, Ly.undo + Ly.slots * (2 * j)); };
  auto Uv = [&](int j) { return (bf16*)at(ws, Ly.undo + Ly.slots * (2 * j + 1)); };
  auto Os = [&](int j) { return (bf16*)at(ws, Ly.op + Ly.outs * j); };
  const wm::Shape sh0 = make_shape(group_dims(d, 0));
  wm::launch_router_fold<bf16>(sh0, router_layers(d), (const bf16*)P.g_pre,
                               (const bf16*)P.W_alpha, (bf16*)at(fw, Lf.wa), s);
  wm::launch_kv_fold<bf16>(sh0, (const bf16*)P.g_mid, (const bf16*)P.Wk, (const bf16*)P.Wv,
                           (bf16*)at(fw, Lf.wkv), s);
  wm::launch_q_fold<bf16>(sh0, (const bf16*)P.g_in, (const bf16*)P.Wq, (bf16*)at(fw, Lf.wq), 0,
                          L, s);
  // H^(0) = X in every layer, group by group; the initial pool
  wm::launch_group_gather<bf16>(X, Hg, d.B, d.T_new, g, L, D, s);
  for (int q = 0; q < g; ++q)
    run_pool<bf16>(group_dims(d, q), P, Hg + q * gsz, nullptr, K, V, Lf, fw, s, false, false,
                   true);
  // one step: group q's states in Hq (layer 0 holds X) from the cache, its layers' outputs
  // into O (layer l at l Ng HQ) or scratch, the slots it overwrites into (uk, uv) if given,
  // then its pool unless it is the last step (whose pool nothing reads)
  auto step = [&](int q, bf16* Hq, bf16* O, bf16* uk, bf16* uv, bool pool) {
    const wm_dims dq = group_dims(d, q);
    wm::launch_rope_table(make_shape(dq), nullptr, tab, s);
    for (int l = 0; l < L; ++l) {
      bf16* Ol = O ? O + (long)l * Ng * HQ : (bf16*)at(fw, Lf.ol);
      run_layer_attend<bf16>(dq, P, l, Hq, chan_map, nullptr, K, V, Ol, Lf, fw, s, true, true);
      const bool last = l + 1 == L;
      wm::launch_block_residual<bf16>(Ng, D, HQ, Ol, W_o + (long)l * D * HQ, Hq + (long)l * D,
                                      (long)L * D,
                                      last ? topg + (long)q * Ng * D : Hq + (long)(l + 1) * D,
                                      last ? D : (long)L * D, s);
    }
    if (!pool) return;
    if (uk) wm::launch_grad_slots(K, V, uk, uv, nullptr, nullptr, crows, Tg, g, q, d.S_cap, d.d,
                                  false, s);
    run_pool<bf16>(dq, P, Hq, nullptr, K, V, Lf, fw, s, true, true, true);
  };
  const int nsteps = n_grad * g;
  for (int t = 1; t <= first; ++t)
    for (int q = 0; q < g; ++q) step(q, Hg + q * gsz, nullptr, nullptr, nullptr, true);
  for (int j = 0; j < nsteps; ++j) {
    const int q = j % g;
    (void)hipMemcpyAsync(Hs(j), Hg + q * gsz, (size_t)gsz * sizeof(bf16), hipMemcpyDeviceToDevice,
                         s);
    step(q, Hs(j), Os(j), Uk(j), Uv(j), j + 1 < nsteps);
  }
  if (h_top) wm::launch_group_scatter<bf16>(topg, h_top, d.B, d.T_new, g, D, s);

  // backward
  float* gcur = (float*)at(ws, Ly.gcur);
  bf16* gb = (bf16*)at(ws, Ly.gb);
  float* dof = (float*)at(ws, Ly.dof);
  bf16* dob = (bf16*)at(ws, Ly.dob);
  float* dql = (float*)at(ws, Ly.dql);
  bf16* h1 = (bf16*)at(ws, Ly.h1);
  float* dpk = (float*)at(ws, Ly.dpk);
  float* dpv = (float*)at(ws, Ly.dpv);
  float* dhn = (float*)at(ws, Ly.dhn);
  float* gkd = (float*)at(ws, Ly.gkd);
  void* sub = at(ws, Ly.sub);
  wm::LayerTable m0{};
  wm::ChannelGroups cg0{};
  cg0.offsets[1] = 1;
  const Layout Lp = layout(group_dims(d, 0), WM_OP_POOL_BACKWARD);
  wm_dims dq1 = group_dims(d, 0);
  dq1.L = 1;
  const Layout Lq = layout(dq1, WM_OP_Q_BACKWARD);
  const bool paper = d.mask_mode == WM_MASK_PAPER;
  bf16* Ql = (bf16*)at(fw, Lf.q);
  float* rinv = (float*)at(fw, Lf.rinv);
  wm::launch_grad_fill(dpk, cache_elems, 0.f, s);
  wm::launch_grad_fill(dpv, cache_elems, 0.f, s);
  for (int j = nsteps - 1; j >= 0; --j) {
    const int q = j % g;
    const bool last_pass = j >= (n_grad - 1) * g, pooled = j + 1 < nsteps;
    const wm_dims dq = group_dims(d, q);
    const wm::Shape shq = make_shape(dq), sh1 = make_shape(one_consumer(dq));
    const bf16* H = Hs(j);
    const bf16* O = Os(j);
    // the step's pool: the gradient at its slots goes to its states (dhn); the slots then
    // hold what the step read, their gradient cleared
    if (pooled) {
      wm::launch_grad_fill(dhn, gsz, 0.f, s);
      run_pool_backward(dq, P, H, nullptr, dpk, dpv, dhn, G, Lp, sub, s);
      wm::launch_grad_slots(K, V, Uk(j), Uv(j), dpk, dpv, crows, Tg, g, q, d.S_cap, d.d, true, s);
    }
    // gcur: the gradient in h_{l+1}, from the loss at the top of the last pass
    wm::launch_grad_fill(gcur, (long)Ng * D, 0.f, s);
    if (last_pass) wm::launch_grad_add_rows(gcur, D, dh_top + (long)q * D, Ng, D, (long)g * D, 1, s);
    wm::launch_rope_table(shq, nullptr, tab, s);
    for (int l = L - 1; l >= 0; --l) {
      const int c = chan_map[l];
      const bf16* Ol = O + (long)l * Ng * HQ;
      // do_l = W_o[l]^T gcur, dW_o[l] += gcur^T o_l
      wm::launch_grad_cast(gcur, gb, (long)Ng * D, s);
      gemm(opnd(gb, D, 1, 0, false), opnd(W_o + (long)l * D * HQ, 1, HQ, 0, false), dof, HQ, 1, 0,
           Ng, HQ, D, 1, false, s);
      wm::launch_grad_cast(dof, dob, (long)Ng * HQ, s);
      gemm(opnd(gb, 1, D, 0, false), opnd(Ol, 1, HQ, 0, false), dW_o + (long)l * D * HQ, HQ, 1, 0,
           D, HQ, Ng, 1, true, s, 0, 0, 0, 0, (float*)at(ws, Ly.split));
      // layer l's queries again, then its attention gradients on channel c alone
      wm::launch_row_rms_strided<bf16>(H + (long)l * D, Ng, D, (long)L * D, L, d.eps, rinv + l,
                                       s);
      wm::launch_q_layers<bf16>(shq, H, rinv, (const bf16*)P.g_qnorm, tab, Ql,
                                (const bf16*)at(fw, Lf.wq), l, 1, s);
      const long dofs = ((long)c * d.Hkv) * d.d;
      wm::launch_attend_backward(sh1, m0, cg0, Ql, K + c * cslice, V + c * cslice,
                                 (const bf16*)P.Kd + dofs, (const bf16*)P.Vd + dofs, Ol, dob,
                                 nullptr, dql, dpk + c * cslice, dpv + c * cslice,
                                 paper ? G.Kd + dofs : gkd,
                                 paper ? G.Vd + dofs : gkd + (long)d.Hkv * d.d,
                                 (float*)at(ws, Ly.rows), s, true);
      // the queries' backward adds its h_l gradient into gcur, then the pool's
      wm::launch_grad_copy_rows(H + (long)l * D, (long)L * D, h1, Ng, D, s);
      wm_params P1 = P;
      P1.g_in = (const bf16*)P.g_in + (long)l * D;
      P1.Wq = (const bf16*)P.Wq + (long)l * HQ * D;
      P1.g_qnorm = (const bf16*)P.g_qnorm + (long)l * d.d;
      wm_grads G1 = G;
      G1.g_in = G.g_in + (long)l * D;
      G1.Wq = G.Wq + (long)l * HQ * D;
      G1.g_qnorm = G.g_qnorm + (long)l * d.d;
      wm_dims dl = dq;
      dl.L = 1;
      run_q_backward(dl, P1, h1, nullptr, dql, gcur, G1, Lq, sub, s);
      if (pooled) wm::launch_grad_add_rows(gcur, D, dhn + (long)l * D, Ng, D, (long)L * D, 1, s);
    }
    wm::launch_grad_add_rows(dX + (long)q * D, (long)g * D, gcur, Ng, D, D, 1, s);  // h_0 = X
  }
  if (n_grad == passes) {  // the initial pool read X in every layer
    wm::launch_group_gather<bf16>(X, Hg, d.B, d.T_new, g, L, D, s);
    for (int q = 0; q < g; ++q) {
      wm::launch_grad_fill(dhn, gsz, 0.f, s);
      run_pool_backward(group_dims(d, q), P, Hg + q * gsz, nullptr, dpk, dpv, dhn, G, Lp, sub, s);
      wm::launch_grad_add_rows(dX + (long)q * D, (long)g * D, dhn, Ng, D, (long)L * D, L, s);
    }
  }
}

}  // namespace

extern "C" {

const char* wm_last_error(void) { return g_err; }
const char* wm_version(void) { return "whitematter-gfx950 0.1.0"; }

int wm_calibrate_mfma(int32_t blocks, int32_t iters, int32_t operands, float* sink,
                      wm_stream_t stream) {
  if (blocks <= 0 || iters <= 0) return fail(WM_ERR_ARG, "blocks and iters must be positive");
  if (blocks > (1 << 20) || iters > (1 << 24)) return fail(WM_ERR_ARG, "blocks or iters too large");
  if (operands != 0 && operands != 1) return fail(WM_ERR_ARG, "operands must be 0 or 1");
  if (!sink) return fail(WM_ERR_ARG, "sink is NULL");
  wm::launch_mfma_loop(blocks, iters, operands == 1, sink, (hipStream_t)stream);
  return launched();
}

int wm_calibrate_read(const void* buf, size_t bytes, float* sink, wm_stream_t stream) {
  if (!buf || !sink) return fail(WM_ERR_ARG, "buf or sink is NULL");
  if ((uintptr_t)buf % 16 != 0 || bytes % 16 != 0 || bytes == 0)
    return fail(WM_ERR_ARG, "buf must be 16-byte aligned and bytes a positive multiple of 16");
  wm::launch_read_loop(buf, (long)(bytes / 16), sink, (hipStream_t)stream);
  return launched();
}

int wm_validate(const wm_dims* dims, int op, const int32_t* chan_map) {
  return validate_dims(dims, op, chan_map);
}

size_t wm_workspace_size(const wm_dims* dims, int op) {
  if (validate_dims(dims, op, nullptr) != WM_OK) return 0;
  return layout(*dims, op).total;
}

int wm_channel_groups(int32_t L, int32_t k, const int32_t* chan_map, int32_t* offsets,
                      int32_t* members) {
  if (!chan_map || !offsets || !members) return fail(WM_ERR_ARG, "NULL argument");
  if (L < 1 || k < 1) return fail(WM_ERR_SHAPE, "L and k must be >= 1");
  for (int l = 0; l < L; ++l)
    if (chan_map[l] < 0 || chan_map[l] >= k)
      return fail(WM_ERR_MAP, "chan_map[%d] = %d is outside [0, %d)", l, chan_map[l], k);
  int pos = 0;
  for (int c = 0; c < k; ++c) {
    offsets[c] = pos;
    for (int l = 0; l < L; ++l)
      if (chan_map[l] == c) members[pos++] = l;
  }
  offsets[k] = pos;
  return WM_OK;
}

int wm_default_map(int32_t L, int32_t k, int32_t* chan_map) {
  if (!chan_map) return fail(WM_ERR_ARG, "NULL argument");
  if (L < 1 || k < 1 || k > L) return fail(WM_ERR_SHAPE, "need 1 <= k <= L");
  for (int l = 0; l < L; ++l) chan_map[l] = l % k;
  return WM_OK;
}

int wm_init_bias(int32_t L, int32_t k, float* b) {
  if (!b) return fail(WM_ERR_ARG, "NULL argument");
  if (L < 1 || k < 1 || k > L) return fail(WM_ERR_SHAPE, "need 1 <= k <= L");
  std::memset(b, 0, sizeof(float) * (size_t)k * L);
  if (k == 1) {
    b[L - 1] = 1.f;  // the single channel starts on the top layer
  } else if (k < L) {
    for (int l = 0; l < L; ++l) b[(l % k) * L + l] = 1.f;  // cyclic
  } else {
    for (int j = 0; j < k; ++j) b[j * L + (j + 1 < L - 1 ? j + 1 : L - 1)] = 1.f;  // shifted identity
  }
  return WM_OK;
}

int wm_router_mix(const wm_dims* dims, const wm_params* params, const void* H, float* alpha_out,
                  void* mixed_out, void* ws, size_t ws_bytes, wm_stream_t stream) {
  WM_TRY(validate_dims(dims, WM_OP_ROUTER_MIX, nullptr));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  if (d.router_mode == WM_ROUTER_STATIC) WM_TRY(check_params(params, {P_GPRE, P_BA}));
  else WM_TRY(check_params(params, {P_GPRE, P_WA, P_BA}));
  WM_TRY(need_ptr(H, "H"));
  WM_TRY(need_ptr(mixed_out, "mixed_out"));
  if (alpha_out && (uintptr_t)alpha_out % 16) return fail(WM_ERR_ARG, "alpha_out is not 16-byte aligned");
  WM_TRY(check_ws(d, WM_OP_ROUTER_MIX, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  if (d.dtype == WM_BF16)
    run_router_mix<bf16>(d, *params, (const bf16*)H, alpha_out, (bf16*)mixed_out, ws, s);
  else
    run_router_mix<float>(d, *params, (const float*)H, alpha_out, (float*)mixed_out, ws, s);
  return launched();
}

int wm_kv_project(const wm_dims* dims, const wm_params* params, const void* mixed,
                  const int32_t* ctx_len, void* Kc, void* Vc, void* ws, size_t ws_bytes,
                  wm_stream_t stream) {
  WM_TRY(validate_dims(dims, WM_OP_KV_PROJECT, nullptr));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  WM_TRY(check_params(params, {P_GMID, P_WK, P_WV, P_GKN}));
  WM_TRY(need_ptr(mixed, "mixed"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(check_ws(d, WM_OP_KV_PROJECT, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  if (d.dtype == WM_BF16)
    run_kv_project<bf16>(d, *params, (const bf16*)mixed, ctx_len, (bf16*)Kc, (bf16*)Vc, ws, s);
  else
    run_kv_project<float>(d, *params, (const float*)mixed, ctx_len, (float*)Kc, (float*)Vc, ws, s);
  return launched();
}

int wm_q_project(const wm_dims* dims, const wm_params* params, const void* H,
                 const int32_t* ctx_len, void* Q, void* ws, size_t ws_bytes, wm_stream_t stream) {
  WM_TRY(validate_dims(dims, WM_OP_Q_PROJECT, nullptr));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  WM_TRY(check_params(params, {P_GIN, P_WQ, P_GQN}));
  WM_TRY(need_ptr(H, "H"));
  WM_TRY(need_ptr(Q, "Q"));
  WM_TRY(check_ws(d, WM_OP_Q_PROJECT, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  if (d.dtype == WM_BF16)
    run_q_project<bf16>(d, *params, (const bf16*)H, ctx_len, (bf16*)Q, ws, s);
  else
    run_q_project<float>(d, *params, (const float*)H, ctx_len, (float*)Q, ws, s);
  return launched();
}

static int channel_attend_impl(const wm_dims* dims, const wm_params* params, const void* Q,
                               const int32_t* chan_map, const int32_t* ctx_len,
                               const int32_t* doc, const void* Kc, const void* Vc, void* O,
                               void* ws, size_t ws_bytes, wm_stream_t stream) {
  if (!chan_map) return fail(WM_ERR_ARG, "chan_map is NULL");
  WM_TRY(validate_dims(dims, WM_OP_CHANNEL_ATTEND, chan_map));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  if (d.mask_mode == WM_MASK_PAPER) WM_TRY(check_params(params, {P_KD, P_VD}));
  else if (!params) return fail(WM_ERR_ARG, "params is NULL");
  WM_TRY(need_ptr(Q, "Q"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(need_ptr(O, "O"));
  WM_TRY(check_ws(d, WM_OP_CHANNEL_ATTEND, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  float* part = (float*)at(ws, layout(d, WM_OP_CHANNEL_ATTEND).part);
  if (d.dtype == WM_BF16)
    run_attend<bf16>(d, *params, (const bf16*)Q, chan_map, ctx_len, doc, (const bf16*)Kc,
                     (const bf16*)Vc, (bf16*)O, part, s);
  else
    run_attend<float>(d, *params, (const float*)Q, chan_map, ctx_len, doc, (const float*)Kc,
                      (const float*)Vc, (float*)O, part, s);
  return launched();
}

int wm_channel_attend(const wm_dims* dims, const wm_params* params, const void* Q,
                      const int32_t* chan_map, const int32_t* ctx_len, const void* Kc,
                      const void* Vc, void* O, void* ws, size_t ws_bytes, wm_stream_t stream) {
  return channel_attend_impl(dims, params, Q, chan_map, ctx_len, nullptr, Kc, Vc, O, ws,
                             ws_bytes, stream);
}

int wm_channel_attend_static(const wm_dims* dims, const wm_params* params, const void* Q,
                             const int32_t* chan_map, const int32_t* ctx_len, const void* Kc,
                             const void* Vc, void* O, wm_stream_t stream) {
  if (!chan_map) return fail(WM_ERR_ARG, "chan_map is NULL");
  WM_TRY(validate_dims(dims, WM_OP_CHANNEL_ATTEND, chan_map));
  const size_t need = layout(*dims, WM_OP_CHANNEL_ATTEND).total;
  if (need > kStaticScratchBytes)
    return fail(WM_ERR_WORKSPACE, "the call needs %zu bytes of scratch, more than the %zu the "
                "library holds for wm_channel_attend_static", need, kStaticScratchBytes);
  void* ws = nullptr;
  if (need > 0) WM_TRY(static_scratch(&ws));
  return channel_attend_impl(dims, params, Q, chan_map, ctx_len, nullptr, Kc, Vc, O, ws, need,
                             stream);
}

int wm_channel_attend_doc(const wm_dims* dims, const wm_params* params, const void* Q,
                          const int32_t* chan_map, const int32_t* ctx_len,
                          const int32_t* doc_start, const void* Kc, const void* Vc, void* O,
                          void* ws, size_t ws_bytes, wm_stream_t stream) {
  if (!doc_start) return fail(WM_ERR_ARG, "doc_start is NULL");
  if ((uintptr_t)doc_start % 4 != 0) return fail(WM_ERR_ARG, "doc_start is not 4-byte aligned");
  return channel_attend_impl(dims, params, Q, chan_map, ctx_len, doc_start, Kc, Vc, O, ws,
                             ws_bytes, stream);
}

static int layer_step_impl(const wm_dims* dims, const wm_params* params, const void* H,
                           const int32_t* chan_map, const int32_t* ctx_len, const int32_t* doc,
                           void* Kc, void* Vc, void* O, void* ws, size_t ws_bytes,
                           wm_stream_t stream, void* const* events) {
  if (!chan_map) return fail(WM_ERR_ARG, "chan_map is NULL");
  WM_TRY(validate_dims(dims, WM_OP_LAYER_STEP, chan_map));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  if (d.router_mode == WM_ROUTER_STATIC)  // W_alpha is not read
    WM_TRY(check_params(params, {P_GPRE, P_BA, P_GMID, P_WK, P_WV, P_GKN, P_KD, P_VD, P_GIN,
                                 P_WQ, P_GQN}));
  else
    WM_TRY(check_params(params, {P_GPRE, P_WA, P_BA, P_GMID, P_WK, P_WV, P_GKN, P_KD, P_VD,
                                 P_GIN, P_WQ, P_GQN}));
  WM_TRY(need_ptr(H, "H"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(need_ptr(O, "O"));
  WM_TRY(check_ws(d, WM_OP_LAYER_STEP, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  if (d.dtype == WM_BF16)
    WM_TRY(run_layer_step<bf16>(d, *params, (const bf16*)H, chan_map, ctx_len, doc, (bf16*)Kc,
                                (bf16*)Vc, (bf16*)O, ws, s, events));
  else
    WM_TRY(run_layer_step<float>(d, *params, (const float*)H, chan_map, ctx_len, doc,
                                 (float*)Kc, (float*)Vc, (float*)O, ws, s, events));
  return launched();
}

int wm_layer_step(const wm_dims* dims, const wm_params* params, const void* H,
                  const int32_t* chan_map, const int32_t* ctx_len, void* Kc, void* Vc, void* O,
                  void* ws, size_t ws_bytes, wm_stream_t stream) {
  return layer_step_impl(dims, params, H, chan_map, ctx_len, nullptr, Kc, Vc, O, ws, ws_bytes,
                         stream, nullptr);
}

int wm_layer_step_doc(const wm_dims* dims, const wm_params* params, const void* H,
                      const int32_t* chan_map, const int32_t* ctx_len, const int32_t* doc_start,
                      void* Kc, void* Vc, void* O, void* ws, size_t ws_bytes,
                      wm_stream_t stream) {
  if (!doc_start) return fail(WM_ERR_ARG, "doc_start is NULL");
  if ((uintptr_t)doc_start % 4 != 0) return fail(WM_ERR_ARG, "doc_start is not 4-byte aligned");
  return layer_step_impl(dims, params, H, chan_map, ctx_len, doc_start, Kc, Vc, O, ws, ws_bytes,
                         stream, nullptr);
}

int wm_layer_step_profiled(const wm_dims* dims, const wm_params* params, const void* H,
                           const int32_t* chan_map, const int32_t* ctx_len,
                           const int32_t* doc_start, void* Kc, void* Vc, void* O, void* ws,
                           size_t ws_bytes, wm_stream_t stream, void* const* events) {
  if (!events) return fail(WM_ERR_ARG, "events is NULL");
  for (int i = 0; i < WM_PROFILE_EVENTS; ++i)
    if (!events[i]) return fail(WM_ERR_ARG, "events[%d] is NULL", i);
  if ((uintptr_t)doc_start % 4 != 0) return fail(WM_ERR_ARG, "doc_start is not 4-byte aligned");
  return layer_step_impl(dims, params, H, chan_map, ctx_len, doc_start, Kc, Vc, O, ws, ws_bytes,
                         stream, events);
}

int wm_channel_attend_dense(const wm_dims* dims, const wm_params* params, const float* read_w,
                            const void* Q, const int32_t* ctx_len, const void* Kc,
                            const void* Vc, void* O, void* ws, size_t ws_bytes,
                            wm_stream_t stream) {
  WM_TRY(validate_dims(dims, WM_OP_DENSE_ATTEND, nullptr));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  if (d.mask_mode == WM_MASK_PAPER) WM_TRY(check_params(params, {P_KD, P_VD}));
  else if (!params) return fail(WM_ERR_ARG, "params is NULL");
  WM_TRY(need_ptr(read_w, "read_w"));
  WM_TRY(need_ptr(Q, "Q"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(need_ptr(O, "O"));
  WM_TRY(check_ws(d, WM_OP_DENSE_ATTEND, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  if (d.dtype == WM_BF16)
    run_attend_dense<bf16>(d, *params, read_w, (const bf16*)Q, ctx_len, (const bf16*)Kc,
                           (const bf16*)Vc, (bf16*)O, ws, s);
  else
    run_attend_dense<float>(d, *params, read_w, (const float*)Q, ctx_len, (const float*)Kc,
                            (const float*)Vc, (float*)O, ws, s);
  return launched();
}

int wm_channel_attend_backward(const wm_dims* dims, const wm_params* params, const void* Q,
                               const int32_t* chan_map, const int32_t* ctx_len, const void* Kc,
                               const void* Vc, const void* O, const void* dO, float* dQ,
                               float* dKc, float* dVc, float* dKd, float* dVd, void* ws,
                               size_t ws_bytes, wm_stream_t stream) {
  if (!chan_map) return fail(WM_ERR_ARG, "chan_map is NULL");
  WM_TRY(validate_dims(dims, WM_OP_ATTEND_BACKWARD, chan_map));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  if (d.dtype != WM_BF16) return fail(WM_ERR_DTYPE, "the attention gradients are built for bf16");
  if (d.d != 64 && d.d != 96)
    return fail(WM_ERR_SHAPE, "the attention gradients support head dims 64 and 96");
  if (decode_path(d))
    return fail(WM_ERR_SHAPE, "the attention gradients need a full-sequence call (T_new > 4)");
  if (d.mask_mode == WM_MASK_PAPER) WM_TRY(check_params(params, {P_KD, P_VD}));
  else if (!params) return fail(WM_ERR_ARG, "params is NULL");
  WM_TRY(need_ptr(Q, "Q"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(need_ptr(O, "O"));
  WM_TRY(need_ptr(dO, "dO"));
  WM_TRY(need_ptr(dQ, "dQ"));
  WM_TRY(need_ptr(dKc, "dKc"));
  WM_TRY(need_ptr(dVc, "dVc"));
  WM_TRY(need_ptr(dKd, "dKd"));
  WM_TRY(need_ptr(dVd, "dVd"));
  WM_TRY(check_ws(d, WM_OP_ATTEND_BACKWARD, ws, ws_bytes));
  (void)hipGetLastError();
  const Layout Ly = layout(d, WM_OP_ATTEND_BACKWARD);
  wm::launch_attend_backward(make_shape(d), map_table(d, chan_map), groups(d, chan_map),
                             (const bf16*)Q, (const bf16*)Kc, (const bf16*)Vc,
                             (const bf16*)params->Kd, (const bf16*)params->Vd, (const bf16*)O,
                             (const bf16*)dO, ctx_len, dQ, dKc, dVc, dKd, dVd,
                             (float*)at(ws, Ly.part), (hipStream_t)stream);
  return launched();
}

int wm_pool(const wm_dims* dims, const wm_params* params, const void* H, const int32_t* ctx_len,
            void* Kc, void* Vc, void* ws, size_t ws_bytes, wm_stream_t stream) {
  WM_TRY(validate_dims(dims, WM_OP_POOL, nullptr));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  if (d.router_mode == WM_ROUTER_STATIC)
    WM_TRY(check_params(params, {P_GPRE, P_BA, P_GMID, P_WK, P_WV, P_GKN}));
  else
    WM_TRY(check_params(params, {P_GPRE, P_WA, P_BA, P_GMID, P_WK, P_WV, P_GKN}));
  WM_TRY(need_ptr(H, "H"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(check_ws(d, WM_OP_POOL, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  const Layout Ly = layout(d, WM_OP_POOL);
  if (d.dtype == WM_BF16)
    run_pool<bf16>(d, *params, (const bf16*)H, ctx_len, (bf16*)Kc, (bf16*)Vc, Ly, ws, s, false,
                   false, false);
  else
    run_pool<float>(d, *params, (const float*)H, ctx_len, (float*)Kc, (float*)Vc, Ly, ws, s,
                    false, false, false);
  return launched();
}

int wm_layer_attend(const wm_dims* dims, const wm_params* params, int32_t layer, const void* H,
                    const int32_t* chan_map, const int32_t* ctx_len, const void* Kc,
                    const void* Vc, void* O_l, void* ws, size_t ws_bytes, wm_stream_t stream) {
  if (!chan_map) return fail(WM_ERR_ARG, "chan_map is NULL");
  WM_TRY(validate_dims(dims, WM_OP_LAYER_ATTEND, chan_map));
  const wm_dims& d = *dims;
  if (layer < 0 || layer >= d.L) return fail(WM_ERR_ARG, "layer %d is outside [0, L)", layer);
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  if (d.mask_mode == WM_MASK_PAPER) WM_TRY(check_params(params, {P_GIN, P_WQ, P_GQN, P_KD, P_VD}));
  else WM_TRY(check_params(params, {P_GIN, P_WQ, P_GQN}));
  WM_TRY(need_ptr(H, "H"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(need_ptr(O_l, "O_l"));
  WM_TRY(check_ws(d, WM_OP_LAYER_ATTEND, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  const Layout Ly = layout(d, WM_OP_LAYER_ATTEND);
  if (d.dtype == WM_BF16)
    run_layer_attend<bf16>(d, *params, layer, (const bf16*)H, chan_map, ctx_len, (const bf16*)Kc,
                           (const bf16*)Vc, (bf16*)O_l, Ly, ws, s, false, false);
  else
    run_layer_attend<float>(d, *params, layer, (const float*)H, chan_map, ctx_len,
                            (const float*)Kc, (const float*)Vc, (float*)O_l, Ly, ws, s, false,
                            false);
  return launched();
}

int wm_prefill_passes(const wm_dims* dims, const wm_params* params, const void* W_o,
                      const void* X, const int32_t* chan_map, int32_t passes, void* Kc, void* Vc,
                      void* H, void* h_top, void* ws, size_t ws_bytes, wm_stream_t stream) {
  if (!chan_map) return fail(WM_ERR_ARG, "chan_map is NULL");
  WM_TRY(validate_dims(dims, WM_OP_PASSES, chan_map));
  const wm_dims& d = *dims;
  if (passes < 1) return fail(WM_ERR_ARG, "passes must be >= 1");
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  if (d.router_mode == WM_ROUTER_STATIC)
    WM_TRY(check_params(params, {P_GPRE, P_BA, P_GMID, P_WK, P_WV, P_GKN, P_KD, P_VD, P_GIN,
                                 P_WQ, P_GQN}));
  else
    WM_TRY(check_params(params, {P_GPRE, P_WA, P_BA, P_GMID, P_WK, P_WV, P_GKN, P_KD, P_VD,
                                 P_GIN, P_WQ, P_GQN}));
  WM_TRY(need_ptr(W_o, "W_o"));
  WM_TRY(need_ptr(X, "X"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(need_ptr(H, "H"));
  if (h_top && (uintptr_t)h_top % 16 != 0) return fail(WM_ERR_ARG, "h_top is not 16-byte aligned");
  WM_TRY(check_ws(d, WM_OP_PASSES, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  if (d.dtype == WM_BF16)
    run_passes<bf16>(d, *params, (const bf16*)W_o, (const bf16*)X, chan_map, passes, (bf16*)Kc,
                     (bf16*)Vc, (bf16*)H, (bf16*)h_top, ws, s);
  else
    run_passes<float>(d, *params, (const float*)W_o, (const float*)X, chan_map, passes,
                      (float*)Kc, (float*)Vc, (float*)H, (float*)h_top, ws, s);
  return launched();
}

int wm_q_project_backward(const wm_dims* dims, const wm_params* params, const void* H,
                          const int32_t* ctx_len, const float* dQ, float* dH,
                          const wm_grads* grads, void* ws, size_t ws_bytes, wm_stream_t stream) {
  WM_TRY(validate_dims(dims, WM_OP_Q_BACKWARD, nullptr));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  WM_TRY(check_backward(d));
  WM_TRY(check_params(params, {P_GIN, P_WQ, P_GQN}));
  if (!grads) return fail(WM_ERR_ARG, "grads is NULL");
  WM_TRY(grad_ptr(grads->g_in, "g_in"));
  WM_TRY(grad_ptr(grads->Wq, "Wq"));
  WM_TRY(grad_ptr(grads->g_qnorm, "g_qnorm"));
  WM_TRY(need_ptr(H, "H"));
  WM_TRY(grad_ptr(dQ, "(dQ)"));
  WM_TRY(grad_ptr(dH, "(dH)"));
  WM_TRY(check_ws(d, WM_OP_Q_BACKWARD, ws, ws_bytes));
  (void)hipGetLastError();
  run_q_backward(d, *params, (const bf16*)H, ctx_len, dQ, dH, *grads,
                 layout(d, WM_OP_Q_BACKWARD), ws, (hipStream_t)stream);
  return launched();
}

static int check_pool_grads(const wm_dims& d, const wm_params* params, const wm_grads* grads) {
  if (d.router_mode == WM_ROUTER_STATIC)
    WM_TRY(check_params(params, {P_GPRE, P_BA, P_GMID, P_WK, P_WV, P_GKN}));
  else
    WM_TRY(check_params(params, {P_GPRE, P_WA, P_BA, P_GMID, P_WK, P_WV, P_GKN}));
  if (!grads) return fail(WM_ERR_ARG, "grads is NULL");
  WM_TRY(grad_ptr(grads->g_pre, "g_pre"));
  if (d.router_mode != WM_ROUTER_STATIC) WM_TRY(grad_ptr(grads->W_alpha, "W_alpha"));
  WM_TRY(grad_ptr(grads->b_alpha, "b_alpha"));
  WM_TRY(grad_ptr(grads->g_mid, "g_mid"));
  WM_TRY(grad_ptr(grads->Wk, "Wk"));
  WM_TRY(grad_ptr(grads->Wv, "Wv"));
  WM_TRY(grad_ptr(grads->g_knorm, "g_knorm"));
  return WM_OK;
}

int wm_pool_backward(const wm_dims* dims, const wm_params* params, const void* H,
                     const int32_t* ctx_len, const float* dKc, const float* dVc, float* dH,
                     const wm_grads* grads, void* ws, size_t ws_bytes, wm_stream_t stream) {
  WM_TRY(validate_dims(dims, WM_OP_POOL_BACKWARD, nullptr));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  WM_TRY(check_backward(d));
  WM_TRY(check_pool_grads(d, params, grads));
  WM_TRY(need_ptr(H, "H"));
  WM_TRY(need_ptr(dKc, "dKc"));
  WM_TRY(need_ptr(dVc, "dVc"));
  WM_TRY(grad_ptr(dH, "(dH)"));
  WM_TRY(check_ws(d, WM_OP_POOL_BACKWARD, ws, ws_bytes));
  (void)hipGetLastError();
  run_pool_backward(d, *params, (const bf16*)H, ctx_len, dKc, dVc, dH, *grads,
                    layout(d, WM_OP_POOL_BACKWARD), ws, (hipStream_t)stream);
  return launched();
}

int wm_layer_step_backward(const wm_dims* dims, const wm_params* params, const void* H,
                           const int32_t* chan_map, const int32_t* ctx_len, const void* Kc,
                           const void* Vc, const void* O, const void* dO, float* dKc,
                           float* dVc, float* dH, const wm_grads* grads, void* ws,
                           size_t ws_bytes, wm_stream_t stream) {
  if (!chan_map) return fail(WM_ERR_ARG, "chan_map is NULL");
  WM_TRY(validate_dims(dims, WM_OP_STEP_BACKWARD, chan_map));
  const wm_dims& d = *dims;
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  WM_TRY(check_backward(d));
  if (decode_path(d))
    return fail(WM_ERR_SHAPE, "the step's gradients need a full-sequence call (T_new > 4)");
  WM_TRY(check_pool_grads(d, params, grads));
  WM_TRY(check_params(params, {P_GIN, P_WQ, P_GQN}));
  if (d.mask_mode == WM_MASK_PAPER) WM_TRY(check_params(params, {P_KD, P_VD}));
  WM_TRY(grad_ptr(grads->g_in, "g_in"));
  WM_TRY(grad_ptr(grads->Wq, "Wq"));
  WM_TRY(grad_ptr(grads->g_qnorm, "g_qnorm"));
  if (d.mask_mode == WM_MASK_PAPER) {
    WM_TRY(grad_ptr(grads->Kd, "Kd"));
    WM_TRY(grad_ptr(grads->Vd, "Vd"));
  }
  WM_TRY(need_ptr(H, "H"));
  WM_TRY(need_ptr(Kc, "Kc"));
  WM_TRY(need_ptr(Vc, "Vc"));
  WM_TRY(need_ptr(O, "O"));
  WM_TRY(need_ptr(dO, "dO"));
  WM_TRY(need_ptr(dKc, "dKc"));
  WM_TRY(need_ptr(dVc, "dVc"));
  WM_TRY(grad_ptr(dH, "(dH)"));
  WM_TRY(check_ws(d, WM_OP_STEP_BACKWARD, ws, ws_bytes));
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  const wm::Shape sh = make_shape(d);
  const Layout Ly = layout(d, WM_OP_STEP_BACKWARD);
  const wm_params& P = *params;
  // the forward's queries, with the forward's kernels
  bf16* Q = (bf16*)at(ws, Ly.q);
  float* rinv = (float*)at(ws, Ly.rinv);
  float* tab = (float*)at(ws, Ly.tab);
  wm::launch_row_rms<bf16>((const bf16*)H, (long)sh.N() * sh.L, sh.D, sh.eps, rinv, s);
  wm::launch_rope_table(sh, ctx_len, tab, s);
  wm::launch_q_project<bf16>(sh, (const bf16*)H, rinv, (const bf16*)P.g_in, (const bf16*)P.Wq,
                             (const bf16*)P.g_qnorm, tab, Q, (bf16*)at(ws, Ly.wq), s);
  // attention gradients: dQ, and the slots' and dummy's gradients added to the caller's
  float* dQ = (float*)at(ws, Ly.dq);
  float* gkd = (float*)at(ws, Ly.gkd);
  const bool paper = d.mask_mode == WM_MASK_PAPER;
  const long nd = (long)d.k * d.Hkv * d.d;
  wm::launch_attend_backward(sh, map_table(d, chan_map), groups(d, chan_map), Q,
                             (const bf16*)Kc, (const bf16*)Vc, (const bf16*)P.Kd,
                             (const bf16*)P.Vd, (const bf16*)O, (const bf16*)dO, ctx_len, dQ,
                             dKc, dVc, paper ? grads->Kd : gkd, paper ? grads->Vd : gkd + nd,
                             (float*)at(ws, Ly.part), s, true);
  run_q_backward(d, P, (const bf16*)H, ctx_len, dQ, dH, *grads, Ly, ws, s);
  run_pool_backward(d, P, (const bf16*)H, ctx_len, dKc, dVc, dH, *grads, Ly, ws, s);
  return launched();
}

size_t wm_passes_backward_workspace(const wm_dims* dims, int32_t n_grad) {
  if (validate_dims(dims, WM_OP_PASSES_BACKWARD, nullptr) != WM_OK || n_grad < 1) return 0;
  return passes_bwd_layout(*dims, n_grad).total;
}

int wm_prefill_passes_backward(const wm_dims* dims, const wm_params* params, const void* W_o,
                               const void* X, const int32_t* chan_map, int32_t passes,
                               int32_t n_grad, const float* dh_top, void* h_top, float* dX,
                               float* dW_o, const wm_grads* grads, void* ws, size_t ws_bytes,
                               wm_stream_t stream) {
  if (!chan_map) return fail(WM_ERR_ARG, "chan_map is NULL");
  WM_TRY(validate_dims(dims, WM_OP_PASSES_BACKWARD, chan_map));
  const wm_dims& d = *dims;
  if (passes < 1) return fail(WM_ERR_ARG, "passes must be >= 1");
  if (n_grad < 1 || n_grad > passes) return fail(WM_ERR_ARG, "n_grad must be in [1, passes]");
  if ((size_t)d.B * d.T_new == 0) return WM_OK;
  WM_TRY(check_backward(d));
  if (decode_path(group_dims(d, 0)))
    return fail(WM_ERR_SHAPE, "the pass gradients need T_new / groups > 4");
  WM_TRY(check_pool_grads(d, params, grads));
  WM_TRY(check_params(params, {P_GIN, P_WQ, P_GQN}));
  if (d.mask_mode == WM_MASK_PAPER) WM_TRY(check_params(params, {P_KD, P_VD}));
  WM_TRY(grad_ptr(grads->g_in, "g_in"));
  WM_TRY(grad_ptr(grads->Wq, "Wq"));
  WM_TRY(grad_ptr(grads->g_qnorm, "g_qnorm"));
  if (d.mask_mode == WM_MASK_PAPER) {
    WM_TRY(grad_ptr(grads->Kd, "Kd"));
    WM_TRY(grad_ptr(grads->Vd, "Vd"));
  }
  WM_TRY(need_ptr(W_o, "W_o"));
  WM_TRY(need_ptr(X, "X"));
  if (h_top) WM_TRY(need_ptr(h_top, "h_top"));
  WM_TRY(grad_ptr(dh_top, "(dh_top)"));
  WM_TRY(grad_ptr(dX, "(dX)"));
  WM_TRY(grad_ptr(dW_o, "(dW_o)"));
  const size_t need = passes_bwd_layout(d, n_grad).total;
  if (!ws) return fail(WM_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if ((uintptr_t)ws % 256 != 0) return fail(WM_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (ws_bytes < need)
    return fail(WM_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  (void)hipGetLastError();
  run_passes_backward(d, *params, (const bf16*)W_o, (const bf16*)X, chan_map, passes, n_grad,
                      dh_top, (bf16*)h_top, dX, dW_o, *grads, ws, (hipStream_t)stream);
  return launched();
}

}  // extern "C"
