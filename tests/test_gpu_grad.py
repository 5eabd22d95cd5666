"""GPU parity of the step's remaining gradients against the gradient oracle: the queries'
backward (wm_q_project_backward), the pool's backward (wm_pool_backward) and the whole
step's backward (wm_layer_step_backward), element by element on small shapes that span
several GEMM tiles and a ragged tail. The entry points add into their outputs: every test
starts the outputs at seeded nonzero values and compares the difference."""
import numpy as np
import pytest
import torch

from oracle import backward as ob
from tests import synth
from tests.parity import TOL_BF16_REL, _bias, _dev, _f64, _gdims, _odims, check_close, wm  # noqa: F401

pytestmark = pytest.mark.gpu

F32 = dict(dtype=torch.float32, device="cuda")


def _grads_like(P, names, seed):
    """Seeded nonzero starting values for the gradients (the calls add into them)."""
    return {n: synth._normal(tuple(P[n].shape), 0.5, seed + i, torch.float32).cuda()
            for i, n in enumerate(names)}


def _chain_slack(ref):
    """The step's gradients pass through two bf16 stages in a row (the attention gradients,
    then the projections' and norms' gradients of their result), each within the bf16
    bound on its own: the per-element floor of the bound, TOL rms(ref), is doubled."""
    return TOL_BF16_REL * float(np.sqrt(np.mean(np.square(ref))))


def _check_grads(name, g_gpu, g_start, ref, names, chain=False):
    for n in names:
        got = (g_gpu[n] - g_start[n]).cpu()
        r = ref["d" + n]
        check_close(got, r, "bf16", "%s d%s" % (name, n), slack=_chain_slack(r) if chain else None)


def _workload(name, d, Hq, Hkv, T_new, ctx, L=5, k=3, D=160, p=1):
    return synth.small(name, B=2, T_new=T_new, L=L, k=k, D=D, Hq=Hq, Hkv=Hkv, d=d,
                       ctx=ctx + T_new, dtype="bf16", p=p)


@pytest.mark.parametrize("d,Hq,Hkv", [(64, 4, 2), (96, 3, 3)])
@pytest.mark.parametrize("T_new,ctx", [(150, 0), (37, 90)])
def test_q_project_backward(wm, d, Hq, Hkv, T_new, ctx):
    w = _workload("qb_d%d" % d, d, Hq, Hkv, T_new, ctx)
    print("q backward d%d %d/%d T%d ctx%d" % (d, Hq, Hkv, T_new, ctx), flush=True)
    P = synth.make_params(w, _bias(w), gains="random")
    H = synth.make_states(w)
    ctx_len = torch.tensor([ctx, ctx // 3], dtype=torch.int32)
    dQ = synth._normal((w.L, w.B, w.Hq, w.T_new, w.d), 1.0, 501, torch.float32)
    ref = ob.q_project_grads(_odims(w), P, H, dQ.double().numpy(), ctx_len.numpy())
    dH0 = synth._normal(tuple(H.shape), 1.0, 502, torch.float32).cuda()
    dH = dH0.clone()
    g0 = _grads_like(P, ob.QUERY_PARAMS, 503)
    g = {n: t.clone() for n, t in g0.items()}
    dims = _gdims(wm, w, ctx_max=ctx)
    wm.q_project_backward(dims, _dev(P), H.cuda(), ctx_len.cuda(), dQ.cuda(), dH, g)
    torch.cuda.synchronize()
    check_close((dH - dH0).cpu(), ref["dH"], "bf16", "dH")
    _check_grads("q", g, g0, ref, ob.QUERY_PARAMS)


def test_weight_gradients_split_k(wm):
    """Many tokens, few weight tiles: the weight gradients' GEMMs cut K (the tokens) into
    slices summed in order (dWq here, 2 layers of 128 x 128 against 4096 tokens)."""
    w = synth.small("qb_split", B=2, T_new=2048, L=2, k=1, D=128, Hq=2, Hkv=1, d=64,
                    ctx=2048, dtype="bf16")
    print("q backward split K", flush=True)
    P = synth.make_params(w, _bias(w), gains="random")
    H = synth.make_states(w)
    dQ = synth._normal((w.L, w.B, w.Hq, w.T_new, w.d), 1.0, 511, torch.float32)
    ref = ob.q_project_grads(_odims(w), P, H, dQ.double().numpy())
    dH = torch.zeros(tuple(H.shape), dtype=torch.float32, device="cuda")
    g = {n: torch.zeros(tuple(P[n].shape), dtype=torch.float32, device="cuda")
         for n in ob.QUERY_PARAMS}
    wm.q_project_backward(_gdims(wm, w, ctx_max=0), _dev(P), H.cuda(), None, dQ.cuda(), dH, g)
    torch.cuda.synchronize()
    check_close(dH.cpu(), ref["dH"], "bf16", "dH")
    for n in ob.QUERY_PARAMS:
        check_close(g[n].cpu(), ref["d" + n], "bf16", "split d%s" % n)


def test_query_and_pool_gradients_at_full_size(wm):
    """The queries' and the pool's gradients of the 4096-token, 24-layer pass in the launch
    configuration a training step uses (256 x 256 and 128 x 128 GEMM tiles): dH of sampled
    token runs, whose rows depend only on their own states and incoming gradients, and the
    query weights' and gains' gradients of the first and the last layer, each of which
    depends only on its own layer, against the oracle on those sub-problems. (The pool's
    weight gradients mix every layer of every token; they are checked on the small shapes.)"""
    import dataclasses
    w = synth.WORKLOADS["c4_T4096_L24_k12"]
    print("query and pool gradients full size", flush=True)
    P = synth.make_params(w, _bias(w), gains="random")
    H = synth.make_states(w)
    dQ = synth._normal((w.L, w.B, w.Hq, w.T_new, w.d), 1.0, 521, torch.float32)
    rows = (w.k, w.B, w.Hkv, w.T_new, w.d)
    dK = synth._normal(rows, 1.0, 522, torch.float32)
    dV = synth._normal(rows, 1.0, 523, torch.float32)
    dims = _gdims(wm, w, S_cap=w.T_new, ctx_max=0)
    Pd, Hd = _dev(P), H.cuda()
    dHq = torch.zeros(tuple(H.shape), **F32)
    gq = {n: torch.zeros(tuple(P[n].shape), **F32) for n in ob.QUERY_PARAMS}
    wm.q_project_backward(dims, Pd, Hd, None, dQ.cuda(), dHq, gq)
    dHp = torch.zeros(tuple(H.shape), **F32)
    gp = {n: torch.zeros(tuple(P[n].shape), **F32) for n in ob.POOL_PARAMS}
    wm.pool_backward(dims, Pd, Hd, None, dK.cuda(), dV.cuda(), dHp, gp)
    torch.cuda.synchronize()
    dHq, dHp = dHq.cpu().numpy(), dHp.cpu().numpy()
    gq = {n: t.cpu() for n, t in gq.items()}
    del Pd, Hd, gp
    base = _odims(w, S_cap=w.T_new)
    for b, s0, n in ((0, 0, 24), (w.B - 1, w.T_new - 24, 24), (1, 1500, 16)):
        sub = dataclasses.replace(base, B=1, T_new=n)
        ctx = np.array([s0])
        rq = ob.q_project_grads(sub, P, H[b:b + 1, s0:s0 + n],
                                dQ[:, b:b + 1, :, s0:s0 + n].double().numpy(), ctx)
        check_close(dHq[b, s0:s0 + n], rq["dH"][0], "bf16", "queries dH b%d %d+%d" % (b, s0, n))
        rp = ob.pool_grads(sub, P, H[b:b + 1, s0:s0 + n],
                           dK[:, b:b + 1, :, s0:s0 + n].double().numpy(),
                           dV[:, b:b + 1, :, s0:s0 + n].double().numpy(), ctx)
        check_close(dHp[b, s0:s0 + n], rp["dH"][0], "bf16", "pool dH b%d %d+%d" % (b, s0, n))
    for l in (0, w.L - 1):
        sub = dataclasses.replace(base, L=1)
        Pl = dict(P)
        for n in ob.QUERY_PARAMS:
            Pl[n] = P[n][l:l + 1]
        r = ob.q_project_grads(sub, Pl, H[:, :, l:l + 1], dQ[l:l + 1].double().numpy())
        for n in ob.QUERY_PARAMS:
            check_close(gq[n][l], r["d" + n][0], "bf16", "layer %d d%s" % (l, n))


POOL_CASES = [
    dict(),
    dict(mix_mode=1),
    dict(p=2, L=6, k=4),
    dict(router_mode=2, L=4, k=4),
    dict(router_mode=2, L=4, k=4, mix_mode=1),
    dict(router_mode=1),
    dict(d=96, Hq=3, Hkv=3, k=2),
]


@pytest.mark.parametrize("case", range(len(POOL_CASES)))
@pytest.mark.parametrize("T_new,ctx", [(150, 0), (37, 90)])
def test_pool_backward(wm, case, T_new, ctx):
    kw = dict(POOL_CASES[case])
    modes = {m: kw.pop(m) for m in ("mix_mode", "router_mode") if m in kw}
    shape = dict(d=64, Hq=4, Hkv=2)
    shape.update(kw)
    w = _workload("pb%d" % case, T_new=T_new, ctx=ctx, **shape)
    print("pool backward case %d %s T%d ctx%d" % (case, modes, T_new, ctx), flush=True)
    bias = _bias(w)
    if modes.get("router_mode") == 2:
        # the default bias puts channel j on layer j + 1, a source the no-feedback router may
        # not mix; that leaves channel 0 with a router-only weight near zero and its mid norm
        # near its singular point, where any rounding of the mixed channel is amplified by
        # 1 / rms. Here channel j starts on layer j instead, and the router's weights are
        # scaled down so that its logits (std ~0.5 at this width) keep the single-source
        # weight of channel 0 away from zero in the linear mix.
        bias = np.eye(w.k, w.L).reshape(-1)
    P = synth.make_params(w, bias, gains="random")
    if modes.get("router_mode") == 2:
        P["W_alpha"] = (P["W_alpha"].float() * 0.1).to(torch.bfloat16)
    H = synth.make_states(w)
    ctx_len = torch.tensor([ctx, ctx // 3], dtype=torch.int32)
    dK = synth._normal((w.k, w.B, w.Hkv, w.T_new, w.d), 1.0, 601, torch.float32)
    dV = synth._normal((w.k, w.B, w.Hkv, w.T_new, w.d), 1.0, 602, torch.float32)
    od = _odims(w, **modes)
    ref = ob.pool_grads(od, P, H, dK.double().numpy(), dV.double().numpy(), ctx_len.numpy())
    # the cache-layout gradients hold the rows at the new slots, NaN elsewhere (never read)
    shape_c = (w.k, w.B, w.Hkv, w.S_cap, w.d)
    dKc = torch.full(shape_c, float("nan"), dtype=torch.float32)
    dVc = dKc.clone()
    for b, c0 in enumerate(ctx_len.tolist()):
        dKc[:, b, :, c0:c0 + w.T_new] = dK[:, b]
        dVc[:, b, :, c0:c0 + w.T_new] = dV[:, b]
    names = [n for n in ob.POOL_PARAMS if not (n == "W_alpha" and modes.get("router_mode") == 1)]
    dH0 = synth._normal(tuple(H.shape), 1.0, 603, torch.float32).cuda()
    dH = dH0.clone()
    g0 = _grads_like(P, names, 604)
    g = {n: t.clone() for n, t in g0.items()}
    dims = _gdims(wm, w, ctx_max=ctx, **modes)
    wm.pool_backward(dims, _dev(P), H.cuda(), ctx_len.cuda(), dKc.cuda(), dVc.cuda(), dH, g)
    torch.cuda.synchronize()
    check_close((dH - dH0).cpu(), ref["dH"], "bf16", "dH")
    _check_grads("pool", g, g0, ref, names)
    if modes.get("router_mode") == 2:
        # without feedback, router rows never read a source above their channel: untouched
        Wg = (g["W_alpha"] - g0["W_alpha"]).cpu().numpy().reshape(2, w.k * w.L, -1, w.D)
        sel = [w.L - 1 - w.p * m for m in range((w.L + w.p - 1) // w.p)][::-1]
        for o in range(w.k * w.L):
            for m, l in enumerate(sel):
                if l > o // w.L:
                    assert not np.any(Wg[:, o, m]), (o, m)


@pytest.mark.parametrize("mask_mode", [0, 1])
@pytest.mark.parametrize("d,Hq,Hkv", [(64, 4, 2), (96, 6, 3)])
@pytest.mark.parametrize("T_new,ctx", [(150, 0), (70, 60)])
def test_layer_step_backward(wm, mask_mode, d, Hq, Hkv, T_new, ctx):
    """The whole step: forward on the GPU (its caches and output), then the backward with a
    gradient already on the new slots; every gradient against the oracle's autograd of
    the step."""
    w = synth.small("sb_d%d" % d, B=2, T_new=T_new, L=5, k=3, D=128, Hq=Hq, Hkv=Hkv, d=d,
                    ctx=ctx + T_new, dtype="bf16", chan_map=[2, 0, 2, 1, 0])
    print("step backward d%d %d/%d T%d ctx%d mask%d" % (d, Hq, Hkv, T_new, ctx, mask_mode),
          flush=True)
    P = synth.make_params(w, _bias(w), gains="random")
    H = synth.make_states(w)
    ctx_len = torch.tensor([ctx, ctx // 2], dtype=torch.int32)
    Kc, Vc = synth.make_cache_cpu(w)
    dO = synth._normal((w.L, w.B, w.T_new, w.Hq * w.d), 1.0, 701, torch.bfloat16)
    dKe = synth._normal((w.k, w.B, w.Hkv, w.T_new, w.d), 0.3, 702, torch.float32)
    dVe = synth._normal((w.k, w.B, w.Hkv, w.T_new, w.d), 0.3, 703, torch.float32)
    od = _odims(w, mask_mode=mask_mode)
    ref = ob.layer_step_grads(od, P, H, w.chan_map, _f64(dO), ctx_len.numpy(), _f64(Kc),
                              _f64(Vc), dKe.double().numpy(), dVe.double().numpy())

    dims = _gdims(wm, w, ctx_max=ctx, mask_mode=mask_mode)
    Pd, Hd, cl = _dev(P), H.cuda(), ctx_len.cuda()
    Kd_, Vd_ = Kc.cuda(), Vc.cuda()
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=torch.bfloat16, device="cuda")
    wm.layer_step(dims, Pd, Hd, w.chan_map, cl, Kd_, Vd_, O)
    dKc = torch.zeros(tuple(Kc.shape), **F32)
    dVc = torch.zeros(tuple(Kc.shape), **F32)
    for b, c0 in enumerate(ctx_len.tolist()):
        dKc[:, b, :, c0:c0 + w.T_new] = dKe[:, b].cuda()
        dVc[:, b, :, c0:c0 + w.T_new] = dVe[:, b].cuda()
    names = list(ob.POOL_PARAMS) + list(ob.QUERY_PARAMS) + (["Kd", "Vd"] if mask_mode == 0
                                                            else [])
    dH0 = synth._normal(tuple(H.shape), 1.0, 704, torch.float32).cuda()
    dH = dH0.clone()
    g0 = _grads_like(P, names, 705)
    g = {n: t.clone() for n, t in g0.items()}
    wm.layer_step_backward(dims, Pd, Hd, w.chan_map, cl, Kd_, Vd_, O, dO.cuda(), dKc, dVc, dH, g)
    torch.cuda.synchronize()
    check_close((dH - dH0).cpu(), ref["dH"], "bf16", "dH", slack=_chain_slack(ref["dH"]))
    _check_grads("step", g, g0, ref, names, chain=True)
    dKc_h, dVc_h = dKc.cpu().numpy(), dVc.cpu().numpy()
    for b, c0 in enumerate(ctx_len.tolist()):
        if c0:  # one stage: the attention gradients alone
            check_close(dKc_h[:, b, :, :c0], ref["dKc_ctx"][:, b, :, :c0], "bf16", "dKc ctx b%d" % b)
            check_close(dVc_h[:, b, :, :c0], ref["dVc_ctx"][:, b, :, :c0], "bf16", "dVc ctx b%d" % b)
        # slots past the call's span are never written
        assert not np.any(dKc_h[:, b, :, c0 + w.T_new:]) and not np.any(dVc_h[:, b, :, c0 + w.T_new:])


@pytest.mark.parametrize("mask_mode", [0, 1])
def test_layer_step_backward_strided_group(wm, mask_mode):
    """The step over the strided token group q = 1 of g = 4 (Section 3.3): pool, queries and
    attention at positions ctx + 1 + 4 i, the other slots given."""
    g, q, T_new, ctx = 4, 1, 60, 30
    span = q + g * (T_new - 1) + 1
    w = synth.small("sbg", B=2, T_new=T_new, L=5, k=3, D=128, Hq=4, Hkv=2, d=64,
                    ctx=ctx + span, dtype="bf16", chan_map=[2, 0, 2, 1, 0])
    print("step backward strided group mask%d" % mask_mode, flush=True)
    P = synth.make_params(w, _bias(w), gains="random")
    H = synth.make_states(w)
    ctx_len = torch.tensor([ctx, ctx // 2], dtype=torch.int32)
    Kc, Vc = synth.make_cache_cpu(w)
    dO = synth._normal((w.L, w.B, w.T_new, w.Hq * w.d), 1.0, 711, torch.bfloat16)
    od = _odims(w, mask_mode=mask_mode)
    ref = ob.layer_step_grads(od, P, H, w.chan_map, _f64(dO), ctx_len.numpy(), _f64(Kc),
                              _f64(Vc), grp=(g, q))
    dims = _gdims(wm, w, ctx_max=ctx, mask_mode=mask_mode, groups=g, group=q)
    Pd, Hd, cl = _dev(P), H.cuda(), ctx_len.cuda()
    Kd_, Vd_ = Kc.cuda(), Vc.cuda()
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=torch.bfloat16, device="cuda")
    wm.layer_step(dims, Pd, Hd, w.chan_map, cl, Kd_, Vd_, O)
    dKc = torch.zeros(tuple(Kc.shape), **F32)
    dVc = torch.zeros(tuple(Kc.shape), **F32)
    names = list(ob.POOL_PARAMS) + list(ob.QUERY_PARAMS) + (["Kd", "Vd"] if mask_mode == 0
                                                            else [])
    dH = torch.zeros(tuple(H.shape), **F32)
    gz = {n: torch.zeros(tuple(P[n].shape), **F32) for n in names}
    wm.layer_step_backward(dims, Pd, Hd, w.chan_map, cl, Kd_, Vd_, O, dO.cuda(), dKc, dVc, dH, gz)
    torch.cuda.synchronize()
    check_close(dH.cpu(), ref["dH"], "bf16", "dH", slack=_chain_slack(ref["dH"]))
    for n in names:
        check_close(gz[n].cpu(), ref["d" + n], "bf16", "strided d%s" % n,
                    slack=_chain_slack(ref["d" + n]))
    # the slots the step reads but does not write carry the attention's gradient
    dKc_h = dKc.cpu().numpy()
    mine = np.zeros(w.S_cap, dtype=bool)
    for b, c0 in enumerate(ctx_len.tolist()):
        mine[:] = False
        mine[c0 + q + g * np.arange(T_new)] = True
        other = ~mine
        other[c0 + span:] = False
        check_close(dKc_h[:, b][:, :, other], ref["dKc_ctx"][:, b][:, :, other], "bf16",
                    "dKc others b%d" % b)


# ------------------------------------------------ passes with truncated backprop

PASS_CASES = [
    dict(),
    dict(mask_mode=1, mix_mode=1),
    dict(d=96, Hq=6, Hkv=3, p=2, L=5, k=3),
    dict(router_mode=1),
]


@pytest.mark.parametrize("case", range(len(PASS_CASES)))
@pytest.mark.parametrize("passes,n_grad,g", [(2, 2, 1), (3, 1, 1), (3, 2, 1), (2, 2, 2),
                                             (3, 2, 3)])
def test_prefill_passes_backward(wm, case, passes, n_grad, g):
    """The passes' forward and the truncated backward, over g strided groups (g = 1:
    Jacobi), against the oracle's autograd of the same passes with the cache entering the
    window detached."""
    kw = dict(PASS_CASES[case])
    modes = {m: kw.pop(m) for m in ("mix_mode", "router_mode", "mask_mode") if m in kw}
    shape = dict(d=64, Hq=4, Hkv=2, L=4, k=2, p=1)
    shape.update(kw)
    w = synth.small("pp%d" % case, B=2, T_new=150, D=128, ctx=0, dtype="bf16", **shape)
    print("passes backward case %d %s passes %d window %d groups %d"
          % (case, modes, passes, n_grad, g), flush=True)
    P = synth.make_params(w, _bias(w), gains="random")
    X = synth.make_embeddings(w)
    # the block's output projection at std 0.4 (20 times the forward tests' 0.02): at 0.02
    # the layers' states differ from the embedding by a few percent, every normed state is
    # then nearly parallel to every mixed channel, and the router's and pre-mix gains'
    # gradients (dalpha_jl = dh~_j . h^_l with dh~_j orthogonal to h~_j) become small
    # differences that the states' bf16 rounding swamps
    W_o = (synth.make_out_proj(w).float() * 20.0).to(torch.bfloat16)
    dh = synth._normal((w.B, w.T_new, w.D), 1.0, 801, torch.float32)
    od = _odims(w, S_cap=w.T_new, **modes)
    ref = ob.passes_grads(od, P, _f64(W_o), _f64(X), w.chan_map, passes, n_grad,
                          dh.double().numpy(), g=g)
    # how far bf16 storage of the states, caches, queries and outputs moves each gradient
    # (the oracle's own measure of the gradient's sensitivity to that rounding)
    stored = ob.passes_grads(od, P, _f64(W_o), _f64(X), w.chan_map, passes, n_grad,
                             dh.double().numpy(), bf16_storage=True, g=g)
    _, top_ref = ob.passes_forward(od, {n: ob._t(P[n]) for n in ob.PARAM_NAMES}, ob._t(W_o),
                                   ob._t(X), w.chan_map, passes, n_grad, g=g)
    names = [n for n in ob.PARAM_NAMES if not (n == "W_alpha" and modes.get("router_mode") == 1)
             and not (n in ("Kd", "Vd") and modes.get("mask_mode") == 1)]
    dims = _gdims(wm, w, S_cap=w.T_new, ctx_max=0, groups=g, **modes)
    dX0 = synth._normal(tuple(X.shape), 1.0, 802, torch.float32).cuda()
    dX = dX0.clone()
    dW0 = synth._normal(tuple(W_o.shape), 0.5, 803, torch.float32).cuda()
    dW = dW0.clone()
    g0 = _grads_like(P, names, 804)
    g = {n: t.clone() for n, t in g0.items()}
    top = torch.empty(tuple(X.shape), dtype=torch.bfloat16, device="cuda")
    wm.prefill_passes_backward(dims, _dev(P), W_o.cuda(), X.cuda(), w.chan_map, passes, n_grad,
                               dh.cuda(), dX, dW, g, h_top=top)
    torch.cuda.synchronize()
    check_close(top.cpu(), top_ref.detach().numpy(), "bf16", "h_top")
    # Every stage of the gradient chain (a layer's block, attention and query; a pass's
    # pool) works on bf16 operands and stays within the bf16 bound on its own; down a
    # chain of S stages the rounding adds up like a random walk. The bound is scaled by
    # sqrt(S / 4) (four stages: the depth of the single-step tests' chain), with
    # S = n_grad (3 L + 2) for the deepest path, from h_top back to X. Where the gradient
    # itself is sensitive to rounding (the linear router's logits when the layers' states
    # are nearly parallel, e.g. H^(0) = X in every layer), twice the oracle's own
    # storage-rounding shift is allowed on top.
    depth = n_grad * (3 * w.L + 2)
    scale = max(1.0, float(np.sqrt(depth / 4.0)))
    got = {"dX": (dX - dX0).cpu(), "dW_o": (dW - dW0).cpu()}
    got.update({"d" + n: (g[n] - g0[n]).cpu() for n in names})
    for n, v in got.items():
        r = ref[n]
        rms = float(np.sqrt(np.mean(np.square(r))))
        shift = float(np.abs(stored[n] - r).max())
        check_close(v, r, "bf16", "passes %s" % n,
                    slack=(scale - 1.0) * TOL_BF16_REL * (np.abs(r) + rms) + 2.0 * shift)
