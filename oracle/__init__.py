"""WhiteMatter CPU oracle (test infrastructure only).

A thin ctypes binding over ``wm_oracle.c``: a plain fp64 statement of the
WhiteMatter cross-layer KV pool (Section 3.1, Steps 1-3, router
initialization) and of decode-time channel attention with the learned dummy
slot (Section 3.2). Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the GPU library never does, and the
two share no code.

Arrays are numpy float64, C-contiguous, in the layouts below (N = B*T_new):

    H       [B, T_new, L, D]        per-layer states entering each layer
    alpha   [2, N, k, L]            mixing weights, key branch then value
    mixed   [2, k, N, D]            mixed channels (before the mid RMSNorm)
    Kc, Vc  [k, B, Hkv, S_cap, d]   channel-major cache; token i of sequence b
                                    is stored at slot ctx_len[b] + i
    Q       [L, B, Hq, T_new, d]    consumer queries after q-norm and RoPE
    O       [L, B, T_new, Hq*d]     attention output per consumer layer

The fixed-point passes of Section 3.3 (jacobi, gauss_seidel, autoregressive) run
on sequences that start empty (T = T_new positions) with a stand-in for the
rest of each decoder block, h_{l+1} = h_l + W_o[l] o_l:

    X       [B, T, D]               the state entering layer 0 (embedding)
    W_o     [L, D, Hq*d]            the stand-in block's output projection
    H       [B, T, L, D]            states entering every layer after the passes
    h_top   [B, T, D]               the state leaving the top layer
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

MIX_LINEAR, MIX_SOFTMAX = 0, 1
MASK_PAPER, MASK_INCLUSIVE = 0, 1
ROUTER_DYNAMIC, ROUTER_STATIC, ROUTER_NOFEEDBACK = 0, 1, 2

PARAM_NAMES = ("g_pre", "W_alpha", "b_alpha", "g_mid", "Wk", "Wv", "g_knorm",
               "Kd", "Vd", "g_in", "Wq", "g_qnorm")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, IEEE semantics, OpenMP over rows)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in
                ("B", "T_new", "L", "k", "D", "Hq", "Hkv", "d", "p", "S_cap",
                 "mix_mode", "mask_mode", "router_mode")] + [("eps", ctypes.c_double),
                                              ("rope_theta", ctypes.c_double)]


class _Params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_NAMES]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = ctypes.CDLL(_LIB)
    return _lib


@dataclass
class Dims:
    B: int
    T_new: int
    L: int
    k: int
    D: int
    Hq: int
    Hkv: int
    d: int
    p: int = 1
    S_cap: int = 0
    mix_mode: int = MIX_LINEAR
    mask_mode: int = MASK_PAPER
    router_mode: int = ROUTER_DYNAMIC
    eps: float = 1e-6
    rope_theta: float = 1e6

    @property
    def N(self) -> int:
        return self.B * self.T_new

    @property
    def Lp(self) -> int:
        return (self.L + self.p - 1) // self.p

    def c(self) -> _Dims:
        return _Dims(self.B, self.T_new, self.L, self.k, self.D, self.Hq, self.Hkv, self.d,
                     self.p, self.S_cap, self.mix_mode, self.mask_mode, self.router_mode,
                     self.eps, self.rope_theta)


def _f64(a) -> np.ndarray:
    if hasattr(a, "detach"):  # a torch tensor: exact widening to float64 on the CPU
        a = a.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _ilist(lst):
    if lst is None:
        return None, 0, None
    arr = np.ascontiguousarray(np.asarray(lst, dtype=np.int32))
    return arr, len(arr), arr.ctypes.data_as(ctypes.c_void_p)


class Params:
    """Holds float64 copies of the parameters, keeping them alive for the C calls."""

    def __init__(self, params: dict):
        self.arrays = {n: _f64(params[n]) for n in PARAM_NAMES}
        self.c = _Params(*[_ptr(self.arrays[n]) for n in PARAM_NAMES])


def _as_params(params) -> Params:
    return params if isinstance(params, Params) else Params(params)


def _ctx(dims: Dims, ctx_len):
    if ctx_len is None:
        ctx_len = np.zeros(dims.B, dtype=np.int32)
    arr = np.ascontiguousarray(np.asarray(ctx_len, dtype=np.int32))
    assert arr.shape == (dims.B,)
    return arr


# ------------------------------------------------------------- primitives

def rmsnorm(x, g, eps: float = 1e-6) -> np.ndarray:
    x, g = _f64(x), _f64(g)
    y = np.empty_like(x)
    lib().wmo_rmsnorm(_ptr(x), _ptr(g), ctypes.c_int(x.size), ctypes.c_double(eps), _ptr(y))
    return y


def rope(x, pos: float, theta: float = 1e6) -> np.ndarray:
    y = _f64(x).copy()
    lib().wmo_rope(_ptr(y), ctypes.c_int(y.size), ctypes.c_double(pos), ctypes.c_double(theta))
    return y


def router_layers(L: int, p: int) -> list:
    n = lib().wmo_router_inputs(ctypes.c_int(L), ctypes.c_int(p))
    sel = np.zeros(n, dtype=np.int32)
    lib().wmo_router_layers(ctypes.c_int(L), ctypes.c_int(p), _ptr(sel))
    return sel.tolist()


def init_bias(L: int, k: int) -> np.ndarray:
    b = np.zeros(k * L, dtype=np.float64)
    rc = lib().wmo_init_bias(ctypes.c_int(L), ctypes.c_int(k), _ptr(b))
    if rc != 0:
        raise ValueError("k must lie in [1, L]")
    return b


def channel_groups(L: int, k: int, chan_map):
    m = np.ascontiguousarray(np.asarray(chan_map, dtype=np.int32))
    off = np.zeros(k + 1, dtype=np.int32)
    mem = np.zeros(L, dtype=np.int32)
    rc = lib().wmo_channel_groups(ctypes.c_int(L), ctypes.c_int(k), _ptr(m), _ptr(off), _ptr(mem))
    if rc != 0:
        raise ValueError("channel map entry outside [0, k)")
    return off, mem


def attend_row(q, K, V, kd=None, vd=None) -> np.ndarray:
    q, K, V = _f64(q), _f64(K), _f64(V)
    d = q.size
    o = np.zeros(d, dtype=np.float64)
    kd_p = vd_p = None
    if kd is not None:
        kd, vd = _f64(kd), _f64(vd)
        kd_p, vd_p = _ptr(kd), _ptr(vd)
    lib().wmo_attend_row(ctypes.c_int(d), _ptr(q), _ptr(K), ctypes.c_long(d), _ptr(V),
                         ctypes.c_long(d), ctypes.c_long(K.shape[0]), kd_p, vd_p, _ptr(o))
    return o


# ------------------------------------------------------------ whole tensors

def router_mix(dims: Dims, params, H, toks=None):
    P = _as_params(params)
    H = _f64(H)
    alpha = np.zeros((2, dims.N, dims.k, dims.L))
    mixed = np.zeros((2, dims.k, dims.N, dims.D))
    arr, n, p = _ilist(toks)
    lib().wmo_router_mix(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(H), p, ctypes.c_int(n),
                         _ptr(alpha), _ptr(mixed))
    return alpha, mixed


def empty_cache(dims: Dims, fill: float = np.nan):
    shape = (dims.k, dims.B, dims.Hkv, dims.S_cap, dims.d)
    return np.full(shape, fill), np.full(shape, fill)


def kv_project(dims: Dims, params, mixed, ctx_len, Kc, Vc, toks=None):
    """Writes the listed tokens' cache rows into Kc, Vc (float64, in place)."""
    P = _as_params(params)
    mixed = _f64(mixed)
    ctx = _ctx(dims, ctx_len)
    arr, n, p = _ilist(toks)
    assert Kc.dtype == np.float64 and Kc.flags.c_contiguous and Vc.flags.c_contiguous
    lib().wmo_kv_project(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(mixed), _ptr(ctx), p,
                         ctypes.c_int(n), _ptr(Kc), _ptr(Vc))


def pool(dims: Dims, params, H, ctx_len, Kc, Vc, toks=None):
    P = _as_params(params)
    H = _f64(H)
    ctx = _ctx(dims, ctx_len)
    arr, n, p = _ilist(toks)
    assert Kc.dtype == np.float64 and Kc.flags.c_contiguous and Vc.flags.c_contiguous
    lib().wmo_pool(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(H), _ptr(ctx), p,
                   ctypes.c_int(n), _ptr(Kc), _ptr(Vc))


def pool_rows(dims: Dims, params, H, ctx_len=None, toks=None):
    """Each token's cache rows (K, V), shape [N, k, Hkv, d], at position ctx_len[b] + i."""
    P = _as_params(params)
    H = _f64(H)
    ctx = _ctx(dims, ctx_len)
    Kr = np.zeros((dims.N, dims.k, dims.Hkv, dims.d))
    Vr = np.zeros_like(Kr)
    arr, n, p = _ilist(toks)
    lib().wmo_pool_rows(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(H), _ptr(ctx), p,
                        ctypes.c_int(n), _ptr(Kr), _ptr(Vr))
    return Kr, Vr


def q_project(dims: Dims, params, H, ctx_len=None, toks=None) -> np.ndarray:
    P = _as_params(params)
    H = _f64(H)
    ctx = _ctx(dims, ctx_len)
    Q = np.zeros((dims.L, dims.B, dims.Hq, dims.T_new, dims.d))
    arr, n, p = _ilist(toks)
    lib().wmo_q_project(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(H), _ptr(ctx), p,
                        ctypes.c_int(n), _ptr(Q))
    return Q


def _docs(dims: Dims, doc_start):
    """doc_start [B, T_new] int32 (position of each token's document start), or None."""
    if doc_start is None:
        return None
    a = np.ascontiguousarray(np.asarray(doc_start, dtype=np.int32).reshape(dims.B, dims.T_new))
    return a


def channel_attend(dims: Dims, params, Q, chan_map, ctx_len, Kc, Vc, rows=None,
                   doc_start=None) -> np.ndarray:
    """Consumer attention; doc_start (optional, [B, T_new]) applies the document mask."""
    P = _as_params(params)
    Q, Kc, Vc = _f64(Q), _f64(Kc), _f64(Vc)
    ctx = _ctx(dims, ctx_len)
    m = np.ascontiguousarray(np.asarray(chan_map, dtype=np.int32))
    O = np.zeros((dims.L, dims.B, dims.T_new, dims.Hq * dims.d))
    arr, n, p = _ilist(rows)
    ds = _docs(dims, doc_start)
    lib().wmo_channel_attend_doc(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(Q), _ptr(m),
                                 _ptr(ctx), _ptr(ds) if ds is not None else None, _ptr(Kc),
                                 _ptr(Vc), p, ctypes.c_int(n), _ptr(O))
    return O


def layer_step(dims: Dims, params, H, chan_map, ctx_len, Kc, Vc, doc_start=None) -> np.ndarray:
    """Fused step; Kc/Vc (float64, in place) gain the new tokens' slots."""
    P = _as_params(params)
    H = _f64(H)
    ctx = _ctx(dims, ctx_len)
    m = np.ascontiguousarray(np.asarray(chan_map, dtype=np.int32))
    O = np.zeros((dims.L, dims.B, dims.T_new, dims.Hq * dims.d))
    ds = _docs(dims, doc_start)
    lib().wmo_layer_step_doc(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(H), _ptr(m),
                             _ptr(ctx), _ptr(ds) if ds is not None else None, _ptr(Kc),
                             _ptr(Vc), _ptr(O))
    return O


def num_threads() -> int:
    return int(lib().wmo_num_threads())


# ----------------------------------------------- Section 3.3: fixed-point passes

def _pass_outputs(dims: Dims):
    H = np.zeros((dims.B, dims.T_new, dims.L, dims.D))
    top = np.zeros((dims.B, dims.T_new, dims.D))
    Kc, Vc = empty_cache(dims)
    return H, top, Kc, Vc


def _pass_args(dims, params, W_o, chan_map, X):
    assert dims.S_cap >= dims.T_new
    P = _as_params(params)
    W = _f64(W_o)
    assert W.shape == (dims.L, dims.D, dims.Hq * dims.d)
    X = _f64(X)
    assert X.shape == (dims.B, dims.T_new, dims.D)
    m = np.ascontiguousarray(np.asarray(chan_map, dtype=np.int32))
    return P, W, m, X


def jacobi(dims: Dims, params, W_o, chan_map, X, passes: int):
    """Jacobi iteration (Section 3.3) with the stand-in decoder block
    h_{l+1} = h_l + W_o[l] o_l: returns (H [B, T, L, D], h_top [B, T, D], Kc, Vc)."""
    P, W, m, X = _pass_args(dims, params, W_o, chan_map, X)
    H, top, Kc, Vc = _pass_outputs(dims)
    lib().wmo_jacobi(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(W), _ptr(m), _ptr(X),
                     ctypes.c_int(passes), _ptr(H), _ptr(top), _ptr(Kc), _ptr(Vc))
    return H, top, Kc, Vc


def gauss_seidel(dims: Dims, params, W_o, chan_map, X, g: int, passes: int):
    """Cyclic Gauss-Seidel iteration over g strided groups (Section 3.3)."""
    P, W, m, X = _pass_args(dims, params, W_o, chan_map, X)
    H, top, Kc, Vc = _pass_outputs(dims)
    lib().wmo_gauss_seidel(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(W), _ptr(m), _ptr(X),
                           ctypes.c_int(g), ctypes.c_int(passes), _ptr(H), _ptr(top), _ptr(Kc),
                           _ptr(Vc))
    return H, top, Kc, Vc


def gauss_seidel_from(dims: Dims, params, W_o, chan_map, X, g: int, Kc0, Vc0, passes: int):
    """Gauss-Seidel passes from a given cache (Kc0, Vc0 [k, B, Hkv, S_cap, d]) in place of
    Pool(H^(0))."""
    P, W, m, X = _pass_args(dims, params, W_o, chan_map, X)
    K0, V0 = np.ascontiguousarray(_f64(Kc0)), np.ascontiguousarray(_f64(Vc0))
    H, top, Kc, Vc = _pass_outputs(dims)
    assert K0.shape == Kc.shape and V0.shape == Vc.shape
    lib().wmo_gauss_seidel_from(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(W), _ptr(m),
                                _ptr(X), ctypes.c_int(g), _ptr(K0), _ptr(V0),
                                ctypes.c_int(passes), _ptr(H), _ptr(top), _ptr(Kc), _ptr(Vc))
    return H, top, Kc, Vc


def autoregressive(dims: Dims, params, W_o, chan_map, X):
    """Exact left-to-right evaluation (Section 3.2 order), the fixed point's solution."""
    P, W, m, X = _pass_args(dims, params, W_o, chan_map, X)
    H, top, Kc, Vc = _pass_outputs(dims)
    lib().wmo_autoregressive(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(W), _ptr(m),
                             _ptr(X), _ptr(H), _ptr(top), _ptr(Kc), _ptr(Vc))
    return H, top, Kc, Vc


def block_residual(dims: Dims, W_o, l: int, h, o) -> np.ndarray:
    """The stand-in decoder block: h + W_o[l] o."""
    W, h, o = _f64(W_o), _f64(h), _f64(o)
    out = np.zeros(dims.D)
    lib().wmo_block_residual(ctypes.byref(dims.c()), _ptr(W), ctypes.c_int(l), _ptr(h), _ptr(o),
                             _ptr(out))
    return out


def channel_attend_dense(dims: Dims, params, read_w, Q, ctx_len, Kc, Vc, rows=None) -> np.ndarray:
    """The dense soft read (Section 3.1 Step 3 variant): layer l attends the channels mixed
    with its weights read_w[l] ([L, k])."""
    P = _as_params(params)
    W = _f64(read_w)
    assert W.shape == (dims.L, dims.k)
    Q, Kc, Vc = _f64(Q), _f64(Kc), _f64(Vc)
    ctx = _ctx(dims, ctx_len)
    O = np.zeros((dims.L, dims.B, dims.T_new, dims.Hq * dims.d))
    arr, n, p = _ilist(rows)
    lib().wmo_channel_attend_dense(ctypes.byref(dims.c()), ctypes.byref(P.c), _ptr(W), _ptr(Q),
                                   _ptr(ctx), _ptr(Kc), _ptr(Vc), p, ctypes.c_int(n), _ptr(O))
    return O
