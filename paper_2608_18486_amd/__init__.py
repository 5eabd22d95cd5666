"""Python binding of libwhitematter.so -- the MI355X (gfx950) WhiteMatter hot path.

Argument marshalling only: every step of the computation runs in the HIP
kernels of the library (see include/whitematter.h for the C ABI). PyTorch
supplies device memory and streams. There is no fallback: if the library is
missing, importing the compute entry points raises.

The library shares the HIP runtime that torch has loaded, so torch is
imported before the library is opened.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (loads the HIP runtime the library binds to)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwhitematter.so")

OK, ERR_ARG, ERR_SHAPE, ERR_DTYPE, ERR_MAP, ERR_CAPACITY, ERR_WORKSPACE, ERR_LAUNCH = range(8)
F32, BF16 = 0, 1
MIX_LINEAR, MIX_SOFTMAX = 0, 1
MASK_PAPER, MASK_INCLUSIVE = 0, 1
ROUTER_DYNAMIC, ROUTER_STATIC, ROUTER_NOFEEDBACK = 0, 1, 2
(OP_ROUTER_MIX, OP_KV_PROJECT, OP_Q_PROJECT, OP_CHANNEL_ATTEND, OP_LAYER_STEP, OP_POOL,
 OP_LAYER_ATTEND, OP_PASSES, OP_DENSE_ATTEND, OP_ATTEND_BACKWARD, OP_Q_BACKWARD,
 OP_POOL_BACKWARD, OP_STEP_BACKWARD, OP_PASSES_BACKWARD) = range(14)

PARAM_NAMES = ("g_pre", "W_alpha", "b_alpha", "g_mid", "Wk", "Wv", "g_knorm",
               "Kd", "Vd", "g_in", "Wq", "g_qnorm")


class WMError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("whitematter error %d: %s" % (code, msg))
        self.code = code


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("B", "T_new", "L", "k", "D", "Hq", "Hkv", "d", "p", "S_cap", "ctx_max",
                 "dtype", "mix_mode", "mask_mode", "router_mode")] + [
        ("eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("groups", ctypes.c_int32),
        ("group", ctypes.c_int32)]

    @property
    def N(self) -> int:
        return self.B * self.T_new


class Params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_NAMES]


class Grads(ctypes.Structure):
    """wm_grads: fp32 device pointers named like the parameters (NULL where unused)."""
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_NAMES]


_lib = None
_vp, _i32p, _sz = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32), ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """Open libwhitematter.so (built by paper_2608_18486_amd.build); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libwhitematter.so is not built (%s); run "
                          "`python -m paper_2608_18486_amd.build`" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    D, P, G = ctypes.POINTER(Dims), ctypes.POINTER(Params), ctypes.POINTER(Grads)
    sig = {
        "wm_router_mix": [D, P, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_kv_project": [D, P, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_q_project": [D, P, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_channel_attend": [D, P, _vp, _i32p, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_layer_step": [D, P, _vp, _i32p, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_channel_attend_doc": [D, P, _vp, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_layer_step_doc": [D, P, _vp, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_layer_step_profiled": [D, P, _vp, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp,
                                   _vp],
        "wm_pool": [D, P, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_channel_attend_static": [D, P, _vp, _i32p, _vp, _vp, _vp, _vp, _vp],
        "wm_channel_attend_dense": [D, P, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_channel_attend_backward": [D, P, _vp, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_q_project_backward": [D, P, _vp, _vp, _vp, _vp, G, _vp, _sz, _vp],
        "wm_pool_backward": [D, P, _vp, _vp, _vp, _vp, _vp, G, _vp, _sz, _vp],
        "wm_layer_step_backward": [D, P, _vp, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, G,
                                   _vp, _sz, _vp],
        "wm_prefill_passes_backward": [D, P, _vp, _vp, _i32p, ctypes.c_int32, ctypes.c_int32,
                                       _vp, _vp, _vp, _vp, G, _vp, _sz, _vp],
        "wm_layer_attend": [D, P, ctypes.c_int32, _vp, _i32p, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
        "wm_prefill_passes": [D, P, _vp, _vp, _i32p, ctypes.c_int32, _vp, _vp, _vp, _vp, _vp,
                              _sz, _vp],
        "wm_validate": [D, ctypes.c_int, _i32p],
        "wm_channel_groups": [ctypes.c_int32, ctypes.c_int32, _i32p, _i32p, _i32p],
        "wm_default_map": [ctypes.c_int32, ctypes.c_int32, _i32p],
        "wm_init_bias": [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_float)],
        "wm_calibrate_mfma": [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp],
        "wm_calibrate_read": [_vp, _sz, _vp, _vp],
    }
    for name, argtypes in sig.items():
        fn = getattr(L, name)
        fn.argtypes = argtypes
        fn.restype = ctypes.c_int
    L.wm_workspace_size.argtypes = [D, ctypes.c_int]
    L.wm_workspace_size.restype = ctypes.c_size_t
    L.wm_passes_backward_workspace.argtypes = [D, ctypes.c_int32]
    L.wm_passes_backward_workspace.restype = ctypes.c_size_t
    L.wm_last_error.restype = ctypes.c_char_p
    L.wm_version.restype = ctypes.c_char_p
    _lib = L
    return L


def last_error() -> str:
    return lib().wm_last_error().decode()


def version() -> str:
    return lib().wm_version().decode()


def _check(rc: int):
    if rc != OK:
        raise WMError(rc, last_error())


def make_dims(B, T_new, L, k, D, Hq, Hkv, d, p=1, S_cap=0, ctx_max=0, dtype=BF16,
              mix_mode=MIX_LINEAR, mask_mode=MASK_PAPER, eps=1e-6, rope_theta=1e6,
              router_mode=ROUTER_DYNAMIC, groups=1, group=0) -> Dims:
    """groups/group: the call's tokens are the strided group q = group of a pass split into
    g = groups groups (token i of sequence b at position ctx_len[b] + q + g i)."""
    return Dims(B, T_new, L, k, D, Hq, Hkv, d, p, S_cap, ctx_max, dtype, mix_mode, mask_mode,
                router_mode, eps, rope_theta, groups, group)


def dtype_code(t: torch.dtype) -> int:
    if t == torch.bfloat16:
        return BF16
    if t == torch.float32:
        return F32
    raise ValueError("unsupported dtype %s" % t)


def _ptr(t) -> int | None:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _map(chan_map):
    arr = (ctypes.c_int32 * len(chan_map))(*[int(c) for c in chan_map])
    return arr


def _stream(stream) -> int | None:
    if stream is None:
        if not torch.cuda.is_available():
            return None  # the null stream: only calls that validation rejects get here
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


class ParamSet:
    """Device parameters (a dict of tensors keyed by PARAM_NAMES) as a wm_params."""

    def __init__(self, params: dict):
        self.tensors = {n: params[n].contiguous() for n in PARAM_NAMES}
        self.c = Params(*[self.tensors[n].data_ptr() for n in PARAM_NAMES])


def _params(params) -> ParamSet:
    return params if isinstance(params, ParamSet) else ParamSet(params)


def _pref(params):
    """ctypes reference to the parameters (None passes a NULL wm_params*)."""
    return None if params is None else ctypes.byref(_params(params).c)


def workspace_size(dims: Dims, op: int) -> int:
    return int(lib().wm_workspace_size(ctypes.byref(dims), op))


def workspace(dims: Dims, op: int, device="cuda") -> torch.Tensor:
    """Allocate the op's workspace with torch (the caching allocator aligns to >= 512 B)."""
    n = workspace_size(dims, op)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def _ws(dims, op, ws, device):
    if device is None and ws is None and not torch.cuda.is_available():
        return None, None, 0  # a call that validation rejects before any launch
    if device is None:
        device = "cuda"
    if ws is None:
        ws = workspace(dims, op, device)
    return ws, ws.data_ptr(), ws.numel()


def validate(dims: Dims, op: int, chan_map=None) -> int:
    m = _map(chan_map) if chan_map is not None else None
    return int(lib().wm_validate(ctypes.byref(dims), op, m))


def channel_groups(L: int, k: int, chan_map):
    off = (ctypes.c_int32 * (k + 1))()
    mem = (ctypes.c_int32 * L)()
    _check(lib().wm_channel_groups(L, k, _map(chan_map), off, mem))
    return list(off), list(mem)


def default_map(L: int, k: int):
    m = (ctypes.c_int32 * L)()
    _check(lib().wm_default_map(L, k, m))
    return list(m)


def init_bias(L: int, k: int):
    b = (ctypes.c_float * (k * L))()
    _check(lib().wm_init_bias(L, k, b))
    return list(b)


# ------------------------------------------------------------ compute calls

def router_mix(dims: Dims, params, H, mixed_out, alpha_out=None, ws=None, stream=None):
    P = _params(params)
    ws, wp, wn = _ws(dims, OP_ROUTER_MIX, ws, getattr(H, "device", None))
    _check(lib().wm_router_mix(ctypes.byref(dims), ctypes.byref(P.c), _ptr(H), _ptr(alpha_out),
                               _ptr(mixed_out), wp, wn, _stream(stream)))


def kv_project(dims: Dims, params, mixed, ctx_len, Kc, Vc, ws=None, stream=None):
    P = _params(params)
    ws, wp, wn = _ws(dims, OP_KV_PROJECT, ws, getattr(mixed, "device", None))
    _check(lib().wm_kv_project(ctypes.byref(dims), ctypes.byref(P.c), _ptr(mixed), _ptr(ctx_len),
                               _ptr(Kc), _ptr(Vc), wp, wn, _stream(stream)))


def q_project(dims: Dims, params, H, ctx_len, Q, ws=None, stream=None):
    P = _params(params)
    ws, wp, wn = _ws(dims, OP_Q_PROJECT, ws, getattr(H, "device", None))
    _check(lib().wm_q_project(ctypes.byref(dims), ctypes.byref(P.c), _ptr(H), _ptr(ctx_len),
                              _ptr(Q), wp, wn, _stream(stream)))


def channel_attend(dims: Dims, params, Q, chan_map, ctx_len, Kc, Vc, O, ws=None, stream=None,
                   doc_start=None):
    """doc_start (device int32 [B, T_new]) selects the document-masked entry point."""
    P = _params(params)
    ws, wp, wn = _ws(dims, OP_CHANNEL_ATTEND, ws, getattr(Q, "device", None))
    if doc_start is None:
        _check(lib().wm_channel_attend(ctypes.byref(dims), ctypes.byref(P.c), _ptr(Q),
                                       _map(chan_map), _ptr(ctx_len), _ptr(Kc), _ptr(Vc), _ptr(O),
                                       wp, wn, _stream(stream)))
    else:
        _check(lib().wm_channel_attend_doc(ctypes.byref(dims), ctypes.byref(P.c), _ptr(Q),
                                           _map(chan_map), _ptr(ctx_len), _ptr(doc_start),
                                           _ptr(Kc), _ptr(Vc), _ptr(O), wp, wn, _stream(stream)))


def layer_step(dims: Dims, params, H, chan_map, ctx_len, Kc, Vc, O, ws=None, stream=None,
               doc_start=None):
    """doc_start (device int32 [B, T_new]) selects the document-masked entry point."""
    P = _params(params)
    ws, wp, wn = _ws(dims, OP_LAYER_STEP, ws, getattr(H, "device", None))
    if doc_start is None:
        _check(lib().wm_layer_step(ctypes.byref(dims), ctypes.byref(P.c), _ptr(H), _map(chan_map),
                                   _ptr(ctx_len), _ptr(Kc), _ptr(Vc), _ptr(O), wp, wn,
                                   _stream(stream)))
    else:
        _check(lib().wm_layer_step_doc(ctypes.byref(dims), ctypes.byref(P.c), _ptr(H),
                                       _map(chan_map), _ptr(ctx_len), _ptr(doc_start), _ptr(Kc),
                                       _ptr(Vc), _ptr(O), wp, wn, _stream(stream)))


def channel_attend_dense(dims: Dims, params, read_w, Q, ctx_len, Kc, Vc, O, ws=None,
                         stream=None):
    """The dense soft read: consumer l attends all channels mixed with read_w[l] (device
    float32 [L, k])."""
    ws, wp, wn = _ws(dims, OP_DENSE_ATTEND, ws, getattr(Q, "device", None))
    _check(lib().wm_channel_attend_dense(ctypes.byref(dims), _pref(params), _ptr(read_w),
                                         _ptr(Q), _ptr(ctx_len), _ptr(Kc), _ptr(Vc), _ptr(O),
                                         wp, wn, _stream(stream)))


def channel_attend_backward(dims: Dims, params, Q, chan_map, ctx_len, Kc, Vc, O, dO, dQ, dKc,
                            dVc, dKd, dVd, ws=None, stream=None):
    """Gradients of channel_attend for the output gradient dO: dQ, dKc, dVc, dKd, dVd
    (device float32 tensors, written)."""
    ws, wp, wn = _ws(dims, OP_ATTEND_BACKWARD, ws, getattr(Q, "device", None))
    _check(lib().wm_channel_attend_backward(ctypes.byref(dims), _pref(params), _ptr(Q),
                                            _map(chan_map), _ptr(ctx_len), _ptr(Kc), _ptr(Vc),
                                            _ptr(O), _ptr(dO), _ptr(dQ), _ptr(dKc), _ptr(dVc),
                                            _ptr(dKd), _ptr(dVd), wp, wn, _stream(stream)))


def _grads(grads):
    """ctypes reference to a wm_grads from a dict of float32 tensors (missing names: NULL)."""
    if grads is None:
        return None
    return ctypes.byref(Grads(*[_ptr(grads.get(n)) for n in PARAM_NAMES]))


def q_project_backward(dims: Dims, params, H, ctx_len, dQ, dH, grads, ws=None, stream=None):
    """Gradients of q_project for dQ: added into dH and grads (dict of float32 tensors)."""
    ws, wp, wn = _ws(dims, OP_Q_BACKWARD, ws, getattr(H, "device", None))
    _check(lib().wm_q_project_backward(ctypes.byref(dims), _pref(params), _ptr(H), _ptr(ctx_len),
                                       _ptr(dQ), _ptr(dH), _grads(grads), wp, wn,
                                       _stream(stream)))


def pool_backward(dims: Dims, params, H, ctx_len, dKc, dVc, dH, grads, ws=None, stream=None):
    """Gradients of pool for the new cache rows' gradients dKc, dVc: added into dH and
    grads."""
    ws, wp, wn = _ws(dims, OP_POOL_BACKWARD, ws, getattr(H, "device", None))
    _check(lib().wm_pool_backward(ctypes.byref(dims), _pref(params), _ptr(H), _ptr(ctx_len),
                                  _ptr(dKc), _ptr(dVc), _ptr(dH), _grads(grads), wp, wn,
                                  _stream(stream)))


def layer_step_backward(dims: Dims, params, H, chan_map, ctx_len, Kc, Vc, O, dO, dKc, dVc, dH,
                        grads, ws=None, stream=None):
    """Gradients of layer_step for dO (and the gradients already in dKc, dVc): the cache
    gradients added in dKc, dVc; the state and parameter gradients added into dH, grads."""
    ws, wp, wn = _ws(dims, OP_STEP_BACKWARD, ws, getattr(H, "device", None))
    _check(lib().wm_layer_step_backward(ctypes.byref(dims), _pref(params), _ptr(H),
                                        _map(chan_map), _ptr(ctx_len), _ptr(Kc), _ptr(Vc),
                                        _ptr(O), _ptr(dO), _ptr(dKc), _ptr(dVc), _ptr(dH),
                                        _grads(grads), wp, wn, _stream(stream)))


def passes_backward_workspace(dims: Dims, n_grad: int) -> int:
    return int(lib().wm_passes_backward_workspace(ctypes.byref(dims), n_grad))


def prefill_passes_backward(dims: Dims, params, W_o, X, chan_map, passes: int, n_grad: int,
                            dh_top, dX, dW_o, grads, h_top=None, ws=None, stream=None):
    """The passes over dims.groups strided groups (1: Jacobi), then the gradients of
    <dh_top, h_top> through the last n_grad passes:
    added into dX, dW_o and grads (float32 tensors); h_top (bf16, optional) receives the
    forward's top state."""
    if ws is None and getattr(X, "device", None) is not None:
        ws = torch.empty(max(passes_backward_workspace(dims, n_grad), 256), dtype=torch.uint8,
                         device=X.device)
    wp, wn = (ws.data_ptr(), ws.numel()) if ws is not None else (None, 0)
    _check(lib().wm_prefill_passes_backward(ctypes.byref(dims), _pref(params), _ptr(W_o), _ptr(X),
                                            _map(chan_map), passes, n_grad, _ptr(dh_top),
                                            _ptr(h_top), _ptr(dX), _ptr(dW_o), _grads(grads), wp,
                                            wn, _stream(stream)))


def channel_attend_static(dims: Dims, params, Q, chan_map, ctx_len, Kc, Vc, O, stream=None):
    """wm_channel_attend without a workspace: the decode partials live in the library's
    fixed scratch array (calls on one device must not overlap)."""
    _check(lib().wm_channel_attend_static(ctypes.byref(dims), _pref(params), _ptr(Q),
                                          _map(chan_map), _ptr(ctx_len), _ptr(Kc), _ptr(Vc),
                                          _ptr(O), _stream(stream)))


def pool(dims: Dims, params, H, ctx_len, Kc, Vc, ws=None, stream=None):
    """Steps 1-2 fused: the call's tokens pooled into their cache slots."""
    ws, wp, wn = _ws(dims, OP_POOL, ws, getattr(H, "device", None))
    _check(lib().wm_pool(ctypes.byref(dims), _pref(params), _ptr(H), _ptr(ctx_len), _ptr(Kc),
                         _ptr(Vc), wp, wn, _stream(stream)))


def layer_attend(dims: Dims, params, layer: int, H, chan_map, ctx_len, Kc, Vc, O_l, ws=None,
                 stream=None):
    """One consumer layer: its query from H[:, :, layer] and its channel attention into
    O_l [B, T_new, Hq*d]."""
    ws, wp, wn = _ws(dims, OP_LAYER_ATTEND, ws, getattr(H, "device", None))
    _check(lib().wm_layer_attend(ctypes.byref(dims), _pref(params), int(layer), _ptr(H),
                                 _map(chan_map), _ptr(ctx_len), _ptr(Kc), _ptr(Vc), _ptr(O_l),
                                 wp, wn, _stream(stream)))


def prefill_passes(dims: Dims, params, W_o, X, chan_map, passes: int, Kc, Vc, H, h_top=None,
                   ws=None, stream=None):
    """Cyclic Gauss-Seidel passes (dims.groups groups; 1 = Jacobi) over sequences that start
    empty, with the stand-in decoder block h_{l+1} = h_l + W_o[l] o_l."""
    ws, wp, wn = _ws(dims, OP_PASSES, ws, getattr(X, "device", None))
    _check(lib().wm_prefill_passes(ctypes.byref(dims), _pref(params), _ptr(W_o), _ptr(X),
                                   _map(chan_map), int(passes), _ptr(Kc), _ptr(Vc), _ptr(H),
                                   _ptr(h_top), wp, wn, _stream(stream)))


PROFILE_EVENTS = 7
PHASES = ("norms", "router", "mix", "kv_project", "q_project", "attend")


def layer_step_profiled(dims: Dims, params, H, chan_map, ctx_len, Kc, Vc, O, events, ws=None,
                        stream=None, doc_start=None):
    """layer_step that records PROFILE_EVENTS caller-created hipEvent_t handles (ints) at
    its phase boundaries on the stream."""
    P = _params(params)
    ws, wp, wn = _ws(dims, OP_LAYER_STEP, ws, getattr(H, "device", None))
    ev = (ctypes.c_void_p * PROFILE_EVENTS)(*events)
    _check(lib().wm_layer_step_profiled(ctypes.byref(dims), ctypes.byref(P.c), _ptr(H),
                                        _map(chan_map), _ptr(ctx_len), _ptr(doc_start),
                                        _ptr(Kc), _ptr(Vc),
                                        _ptr(O), wp, wn, _stream(stream), ev))


def calibrate_mfma(blocks: int, iters: int, sink, stream=None, random_operands=False):
    """Launch the matrix-core ceiling loop (blocks * iters * 2**20 flop) on the stream, on
    small constant operands or (random_operands) on changing pseudo-random ones; sink is a
    device float tensor the kernel keeps but does not write."""
    _check(lib().wm_calibrate_mfma(blocks, iters, 1 if random_operands else 0, _ptr(sink),
                                   _stream(stream)))


def calibrate_read(buf, sink, stream=None):
    """Launch the HBM read-ceiling loop over all bytes of the device tensor buf."""
    _check(lib().wm_calibrate_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink),
                                   _stream(stream)))
