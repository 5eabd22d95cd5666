"""Gradients of the WhiteMatter step (test infrastructure only).

The forward of the fused step (Section 3.1 Steps 1-3 with the dummy slot of Section 3.2)
is restated here with plain PyTorch float64 CPU operations, in the paper's order and with
the same readings as ``wm_oracle.c`` (RMSNorm g x / sqrt(mean x^2 + eps), router over the
normed states of layers {L-1-p m} stacked in ascending order, row-major k x L reshape,
rotate-half RoPE at position ctx_len[b] + i, dummy K/V used verbatim, both masks). The
gradients are torch.autograd's derivatives of that forward. This module is pinned in the
tests against the C oracle's forward (the two forwards agree to rounding) and against
central finite differences of the C oracle's forward, which shares nothing with autograd,
and against closed forms of attention gradients.

Only the tests (and the benchmark's CPU baseline) may import it; the GPU library never
does. Arrays in and out are numpy float64 in the layouts of ``oracle/__init__.py``;
gradients have the shapes of what they differentiate.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

from . import PARAM_NAMES, Dims, MASK_PAPER, MIX_SOFTMAX, ROUTER_NOFEEDBACK, ROUTER_STATIC

F64 = torch.float64


def _t(a, grad=False):
    if hasattr(a, "detach"):  # a torch tensor (any dtype): exact widening to float64
        a = a.detach().to("cpu").double().numpy()
    t = torch.as_tensor(np.ascontiguousarray(np.asarray(a, dtype=np.float64)), dtype=F64)
    return t.clone().requires_grad_(grad)


def _same(t):
    return t


def bf16_store(t):
    """The value rounded to bfloat16 (round to nearest even), the gradient passed through
    unchanged: a tensor stored in bf16 between two steps of the computation."""
    return t + (t.detach().to(torch.bfloat16).to(F64) - t.detach())


def _rms(x, g, eps):
    """RMSNorm over the last axis (Section 3.1 Step 1 and Step 2)."""
    return g * x / torch.sqrt((x * x).mean(-1, keepdim=True) + eps)


def _rope(x, pos, theta):
    """Rotate-half RoPE over the last axis; pos broadcasts against x[..., 0]."""
    d = x.shape[-1]
    half = d // 2
    freq = torch.tensor([theta ** (-2.0 * m / d) for m in range(half)], dtype=F64)
    ang = pos.unsqueeze(-1) * freq
    c, s = torch.cos(ang), torch.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return torch.cat([a * c - b * s, b * c + a * s], dim=-1)


def _router_layers(L, p):
    Lp = (L + p - 1) // p
    return [L - 1 - p * m for m in range(Lp)][::-1]


def _positions(B, T, ctx, grp):
    """[B, T] float64 positions ctx[b] + q + g i of the call's tokens (grp = (g, q): the
    strided token group of Section 3.3; (1, 0): contiguous tokens)."""
    g, q = grp
    return ctx.to(F64).reshape(B, 1) + q + g * torch.arange(T, dtype=F64)


def pool(dims: Dims, P: dict, H, ctx, store=_same, grp=(1, 0)):
    """Steps 1-2 for every new token: H [B, T, L, D] -> the new cache rows
    K, V [k, B, Hkv, T, d] (key norm and RoPE applied to K, at the tokens' positions). store:
    applied to the mixed channels and to the rows (bf16_store: as a path that keeps them in
    bf16)."""
    B, T, L, k, D = dims.B, dims.T_new, dims.L, dims.k, dims.D
    Hkv, d = dims.Hkv, dims.d
    N = B * T
    h = H.reshape(N, L, D)
    sel = _router_layers(L, dims.p)
    Lp = len(sel)
    pos = _positions(B, T, ctx, grp).reshape(N)
    out = []
    for br in range(2):
        hn = _rms(h, P["g_pre"][br], dims.eps)                            # [N, L, D]
        bias = P["b_alpha"][br]                                          # [kL]
        if dims.router_mode == ROUTER_STATIC:
            a = bias.expand(N, k * L)
        else:
            W = P["W_alpha"][br].reshape(k * L, Lp, D)
            if dims.router_mode == ROUTER_NOFEEDBACK:
                # channel j's router reads source layers <= j only
                keep = torch.tensor([[1.0 if sel[m] <= o // L else 0.0 for m in range(Lp)]
                                     for o in range(k * L)], dtype=F64)
                W = W * keep.unsqueeze(-1)
            xi = hn[:, sel, :].reshape(N, Lp * D)
            a = xi @ W.reshape(k * L, Lp * D).T + bias
        alpha = a.reshape(N, k, L)
        if dims.router_mode == ROUTER_NOFEEDBACK:
            allowed = torch.tensor([[l <= j for l in range(L)] for j in range(k)])
        else:
            allowed = torch.ones(k, L, dtype=torch.bool)
        if dims.mix_mode == MIX_SOFTMAX:
            alpha = torch.softmax(alpha.masked_fill(~allowed, float("-inf")), dim=-1)
        else:
            alpha = alpha.masked_fill(~allowed, 0.0)
        mixed = store(torch.einsum("nkl,nld->nkd", alpha, hn))            # [N, k, D]
        u = _rms(mixed, P["g_mid"][br], dims.eps)
        W = (P["Wk"] if br == 0 else P["Wv"]).reshape(k, Hkv * d, D)
        y = torch.einsum("nkd,kod->nko", u, W).reshape(N, k, Hkv, d)
        if br == 0:
            y = _rms(y, P["g_knorm"].reshape(1, k, 1, d), dims.eps)
            y = _rope(y, pos.reshape(N, 1, 1).expand(N, k, Hkv), dims.rope_theta)
        out.append(store(y.reshape(B, T, k, Hkv, d).permute(2, 0, 3, 1, 4)))
    return out[0], out[1]


def queries(dims: Dims, P: dict, H, ctx, grp=(1, 0)):
    """Step 7 for every consumer: Q [L, B, Hq, T, d] (input norm, W^Q, q-norm, RoPE)."""
    B, T, L, D, Hq, d = dims.B, dims.T_new, dims.L, dims.D, dims.Hq, dims.d
    x = _rms(H, P["g_in"], dims.eps)                                       # [B, T, L, D]
    y = torch.einsum("btld,lod->btlo", x, P["Wq"].reshape(L, Hq * d, D))
    y = y.reshape(B, T, L, Hq, d)
    y = _rms(y, P["g_qnorm"].reshape(1, 1, L, 1, d), dims.eps)
    pos = _positions(B, T, ctx, grp)                                      # [B, T]
    y = _rope(y, pos.reshape(B, T, 1, 1).expand(B, T, L, Hq), dims.rope_theta)
    return y.permute(2, 0, 3, 1, 4)


def attend(dims: Dims, Kd, Vd, Q, chan_map, ctx, K, V, grp=(1, 0)):
    """Step 3 (and Section 3.2's dummy): consumer l reads channel chan_map[l]. K, V are
    the caches [k, B, Hkv, S, d]; query i of sequence b sits at position t = ctx[b] + q +
    g i (grp = (g, q)) and sees the dummy and slots < t (paper mask) or slots <= t
    (inclusive). Returns O [L, B, T, Hq*d]."""
    B, T, L, Hq, Hkv, d = dims.B, dims.T_new, dims.L, dims.Hq, dims.Hkv, dims.d
    G = Hq // Hkv
    cm = torch.as_tensor(list(chan_map), dtype=torch.long)
    paper = dims.mask_mode == MASK_PAPER
    outs = []
    for b in range(B):
        c0 = int(ctx[b])
        S = c0 + grp[1] + grp[0] * (T - 1) + 1
        Kb = K[cm, b, :, :S, :].repeat_interleave(G, dim=1)                 # [L, Hq, S, d]
        Vb = V[cm, b, :, :S, :].repeat_interleave(G, dim=1)
        q = Q[:, b]                                                        # [L, Hq, T, d]
        s = q @ Kb.transpose(-1, -2) / np.sqrt(d)                          # [L, Hq, T, S]
        t = (c0 + grp[1] + grp[0] * torch.arange(T)).reshape(T, 1)
        slot = torch.arange(S).reshape(1, S)
        vis = slot < t if paper else slot <= t
        s = s.masked_fill(~vis, float("-inf"))
        if paper:
            kd = Kd[cm].repeat_interleave(G, dim=1)                         # [L, Hq, d]
            vd = Vd[cm].repeat_interleave(G, dim=1)
            sd = (q * kd.unsqueeze(2)).sum(-1, keepdim=True) / np.sqrt(d)  # [L, Hq, T, 1]
            s = torch.cat([sd, s], dim=-1)
            Vb = torch.cat([vd.unsqueeze(2), Vb], dim=2)
        pr = torch.softmax(s, dim=-1)
        o = pr @ Vb                                                        # [L, Hq, T, d]
        outs.append(o.permute(0, 2, 1, 3).reshape(L, T, Hq * d))
    return torch.stack(outs, dim=1)


def _params(params, grad):
    arrays = params.arrays if hasattr(params, "arrays") else params
    return {n: _t(arrays[n], grad) for n in PARAM_NAMES}


def _ctx(dims, ctx_len):
    if ctx_len is None:
        return torch.zeros(dims.B, dtype=torch.long)
    return torch.as_tensor(np.asarray(ctx_len), dtype=torch.long).reshape(dims.B)


def layer_step(dims: Dims, params, H, chan_map, ctx_len=None, Kc=None, Vc=None):
    """The fused step's forward: (O [L, B, T, Hq*d], K, V caches with the new slots)."""
    P = _params(params, False)
    ctx = _ctx(dims, ctx_len)
    Ht = _t(H)
    Kn, Vn = pool(dims, P, Ht, ctx)
    Kall, Vall = _splice(dims, ctx, None if Kc is None else _t(Kc),
                         None if Vc is None else _t(Vc), Kn, Vn)
    O = attend(dims, P["Kd"], P["Vd"], queries(dims, P, Ht, ctx), chan_map, ctx, Kall, Vall)
    return O.detach().numpy(), Kall.detach().numpy(), Vall.detach().numpy()


def _splice(dims, ctx, Kc, Vc, Kn, Vn):
    """Caches [k, B, Hkv, S_cap, d]: the given context slots (< ctx[b]) and the new rows at
    slots ctx[b] + i; other slots zero."""
    k, B, Hkv, d, T = dims.k, dims.B, dims.Hkv, dims.d, dims.T_new
    S = max(dims.S_cap, int(ctx.max()) + T)
    Kcs, Vcs = [], []
    for b in range(B):
        c0 = int(ctx[b])
        parts_k, parts_v = [], []
        if c0 > 0:
            parts_k.append(Kc[:, b, :, :c0, :])
            parts_v.append(Vc[:, b, :, :c0, :])
        parts_k.append(Kn[:, b])
        parts_v.append(Vn[:, b])
        pad = torch.zeros(k, Hkv, S - c0 - T, d, dtype=F64)
        Kcs.append(torch.cat(parts_k + [pad], dim=2))
        Vcs.append(torch.cat(parts_v + [pad], dim=2))
    return torch.stack(Kcs, dim=1), torch.stack(Vcs, dim=1)


def channel_attend_grads(dims: Dims, params, Q, chan_map, ctx_len, Kc, Vc, dO,
                         grp=(1, 0)) -> dict:
    """Gradients of <dO, O> for O = channel attention over the given cache (queries at
    positions ctx[b] + q + g i, grp = (g, q)): dQ, dKc, dVc (every cache slot; zero where no
    query reads it) and the dummy's dKd, dVd."""
    P = _params(params, False)
    ctx = _ctx(dims, ctx_len)
    Qt, Kt, Vt = _t(Q, True), _t(Kc, True), _t(Vc, True)
    Kd, Vd = P["Kd"].requires_grad_(True), P["Vd"].requires_grad_(True)
    O = attend(dims, Kd, Vd, Qt, chan_map, ctx, Kt, Vt, grp)
    g = torch.autograd.grad(O, [Qt, Kt, Vt, Kd, Vd], grad_outputs=_t(dO), allow_unused=True)
    names = ("dQ", "dKc", "dVc", "dKd", "dVd")
    return {n: (x if x is not None else torch.zeros_like(v)).numpy()
            for n, x, v in zip(names, g, [Qt, Kt, Vt, Kd, Vd])}


def _splice_group(dims, ctx, Kc, Vc, Kn, Vn, grp):
    """The given caches (every slot the call's queries may read) with the call's rows
    written at slots ctx[b] + q + g i."""
    g, q = grp
    Ks, Vs = [], []
    for b in range(dims.B):
        idx = int(ctx[b]) + q + g * torch.arange(dims.T_new)
        Ks.append(Kc[:, b].index_copy(2, idx, Kn[:, b]))
        Vs.append(Vc[:, b].index_copy(2, idx, Vn[:, b]))
    return torch.stack(Ks, dim=1), torch.stack(Vs, dim=1)


def layer_step_grads(dims: Dims, params, H, chan_map, dO, ctx_len=None, Kc=None, Vc=None,
                     dKc=None, dVc=None, grp=(1, 0)) -> dict:
    """Gradients of <dO, O> (+ <dKc, K> + <dVc, V> over the new cache slots, when given:
    the gradient a later reader of this step's cache sends back) through the whole fused
    step: dH [B, T, L, D], one entry per parameter (d + name), and the gradients of the
    cache slots read that the step does not write (dKc_ctx, dVc_ctx, shaped like Kc). With
    a strided token group (grp = (g, q), tokens at ctx[b] + q + g i) Kc, Vc hold every slot
    the queries may read (the other groups' and the context's)."""
    P = _params(params, True)
    ctx = _ctx(dims, ctx_len)
    Ht = _t(H, True)
    strided = tuple(grp) != (1, 0)
    have_ctx = Kc is not None and (strided or int(ctx.max()) > 0)
    Kci = _t(Kc, True) if have_ctx else None
    Vci = _t(Vc, True) if have_ctx else None
    Kn, Vn = pool(dims, P, Ht, ctx, grp=grp)
    if strided:
        Kall, Vall = _splice_group(dims, ctx, Kci, Vci, Kn, Vn, grp)
    else:
        Kall, Vall = _splice(dims, ctx, Kci, Vci, Kn, Vn)
    O = attend(dims, P["Kd"], P["Vd"], queries(dims, P, Ht, ctx, grp), chan_map, ctx, Kall,
               Vall, grp)
    loss = (O * _t(dO)).sum()
    if dKc is not None:
        loss = loss + (Kn * _t(dKc)).sum() + (Vn * _t(dVc)).sum()
    leaves = [Ht] + [P[n] for n in PARAM_NAMES] + ([Kci, Vci] if have_ctx else [])
    g = torch.autograd.grad(loss, leaves, allow_unused=True)
    out = {"dH": g[0].numpy()}
    for n, x in zip(PARAM_NAMES, g[1:1 + len(PARAM_NAMES)]):
        out["d" + n] = (x if x is not None else torch.zeros_like(P[n])).numpy()
    if have_ctx:
        out["dKc_ctx"], out["dVc_ctx"] = g[-2].numpy(), g[-1].numpy()
    return out


POOL_PARAMS = ("g_pre", "W_alpha", "b_alpha", "g_mid", "Wk", "Wv", "g_knorm")
QUERY_PARAMS = ("g_in", "Wq", "g_qnorm")


def pool_grads(dims: Dims, params, H, dK, dV, ctx_len=None) -> dict:
    """Gradients of <dK, K_new> + <dV, V_new> through the pool of the call's tokens (Steps
    1-2): dK, dV in the new rows' layout [k, B, Hkv, T, d]. Returns dH [B, T, L, D] and
    d + name for the pool's parameters."""
    P = _params(params, True)
    ctx = _ctx(dims, ctx_len)
    Ht = _t(H, True)
    Kn, Vn = pool(dims, P, Ht, ctx)
    loss = (Kn * _t(dK)).sum() + (Vn * _t(dV)).sum()
    leaves = [Ht] + [P[n] for n in POOL_PARAMS]
    g = torch.autograd.grad(loss, leaves, allow_unused=True)
    out = {"dH": g[0].numpy()}
    for n, x in zip(POOL_PARAMS, g[1:]):
        out["d" + n] = (x if x is not None else torch.zeros_like(P[n])).numpy()
    return out


def q_project_grads(dims: Dims, params, H, dQ, ctx_len=None) -> dict:
    """Gradients of <dQ, Q> through the consumer queries (input norm, W^Q, q norm, RoPE):
    dQ [L, B, Hq, T, d]. Returns dH and d + name for g_in, Wq, g_qnorm."""
    P = _params(params, True)
    ctx = _ctx(dims, ctx_len)
    Ht = _t(H, True)
    loss = (queries(dims, P, Ht, ctx) * _t(dQ)).sum()
    leaves = [Ht] + [P[n] for n in QUERY_PARAMS]
    g = torch.autograd.grad(loss, leaves)
    out = {"dH": g[0].numpy()}
    for n, x in zip(QUERY_PARAMS, g[1:]):
        out["d" + n] = x.numpy()
    return out


def new_rows(dims: Dims, cache, ctx_len=None):
    """The call's new rows [k, B, Hkv, T, d] of a cache-layout array (slots ctx_len[b] + i)."""
    ctx = np.zeros(dims.B, dtype=np.int64) if ctx_len is None else np.asarray(ctx_len)
    c = np.asarray(cache)
    return np.stack([c[:, b, :, int(ctx[b]):int(ctx[b]) + dims.T_new] for b in range(dims.B)],
                    axis=1)


# ------------------------------------------- Section 3.3: passes, truncated backprop

def _states(dims: Dims, P: dict, W_o, X, chan_map, K, V, store=_same, grp=(1, 0)):
    """States(X; P) with the stand-in block h_{l+1} = h_l + W_o[l] o_l for the call's tokens
    (X [B, n, D] at positions q + g i, grp = (g, q)): layer l's query from h_l, its attention
    over channel chan_map[l] of the caches K, V [k, B, Hkv, S, d]. Returns (H [B, n, L, D],
    h_top [B, n, D]). store: applied to each query, attention output and state."""
    L = dims.L
    one = dataclasses.replace(dims, L=1, T_new=X.shape[1])
    ctx = torch.zeros(dims.B, dtype=torch.long)
    h = X
    Hs = []
    for l in range(L):
        Hs.append(h)
        sub = {**P, "g_in": P["g_in"][l:l + 1], "Wq": P["Wq"][l:l + 1],
               "g_qnorm": P["g_qnorm"][l:l + 1]}
        q = store(queries(one, sub, h.unsqueeze(2), ctx, grp))             # [1, B, Hq, n, d]
        o = store(attend(one, P["Kd"], P["Vd"], q, [chan_map[l]], ctx, K, V, grp)[0])
        h = store(h + o @ W_o[l].T)
    return torch.stack(Hs, dim=2), h


def passes_forward(dims: Dims, P: dict, W_o, X, chan_map, passes: int, n_grad: int,
                   store=_same, g: int = 1):
    """The fixed-point passes of Section 3.3 as the C oracle's Gauss-Seidel driver runs them
    (g = 1: Jacobi iteration): H^(0) = X in every layer and the cache starts as Pool(H^(0));
    each pass runs the strided groups G_q = {i : i mod g = q} in order, group q recomputing
    the states of its positions from the cache as it stands, then pooling them into its
    slots. The cache entering the last n_grad passes is detached (truncated
    backpropagation: the passes before run without gradient); with n_grad = passes nothing
    is cut and the initial pool's gradient reaches X. Returns (H, h_top) after the last
    pass."""
    B, T, L, D = dims.B, dims.T_new, dims.L, dims.D
    ctx = torch.zeros(B, dtype=torch.long)
    H = X.unsqueeze(2).expand(B, T, L, D)
    K, V = pool(dims, P, H, ctx, store)
    top = torch.zeros(B, T, D, dtype=F64)
    for t in range(1, passes + 1):
        if t == passes - n_grad + 1 and n_grad < passes:
            K, V = K.detach(), V.detach()
        for q in range(g):
            idx = torch.arange(q, T, g)
            dq = dataclasses.replace(dims, T_new=len(idx))
            Hq, tq = _states(dq, P, W_o, X[:, idx], chan_map, K, V, store, (g, q))
            Kn, Vn = pool(dq, P, Hq, ctx, store, (g, q))
            K, V = K.index_copy(3, idx, Kn), V.index_copy(3, idx, Vn)
            H, top = H.index_copy(1, idx, Hq), top.index_copy(1, idx, tq)
    return H, top


def passes_grads(dims: Dims, params, W_o, X, chan_map, passes: int, n_grad: int, dh_top,
                 bf16_storage: bool = False, g: int = 1) -> dict:
    """Gradients of <dh_top, h_top> after `passes` passes over g groups (passes_forward) with
    backpropagation truncated to the last n_grad (1 <= n_grad <= passes): dX, dW_o and
    d + name for every parameter. bf16_storage: the forward rounds what a bf16 path stores
    between its steps (mixed channels, cache rows, queries, attention outputs, states) to
    bf16, the derivatives passing through the rounding; how far that moves the gradients
    measures their sensitivity to the storage precision."""
    assert 1 <= n_grad <= passes
    P = _params(params, True)
    Xt, Wt = _t(X, True), _t(W_o, True)
    _, top = passes_forward(dims, P, Wt, Xt, chan_map, passes, n_grad,
                            bf16_store if bf16_storage else _same, g)
    loss = (top * _t(dh_top)).sum()
    leaves = [Xt, Wt] + [P[n] for n in PARAM_NAMES]
    g = torch.autograd.grad(loss, leaves, allow_unused=True)
    out = {"dX": g[0].numpy(), "dW_o": g[1].numpy()}
    for n, x in zip(PARAM_NAMES, g[2:]):
        out["d" + n] = (x if x is not None else torch.zeros_like(P[n])).numpy()
    return out
