"""Pins of the gradient oracle (oracle/backward.py), CPU only.

The gradient oracle is torch.autograd over a float64 torch restatement of the step. It is
pinned here against things outside it: its forward against the C oracle's forward (written
separately from the paper), its gradients against central finite differences of the C
oracle's forward (which shares no code with autograd), and its attention gradients against
closed forms (a single visible slot, the dummy alone, uniform attention).
"""
import numpy as np
import pytest

import oracle
from oracle import backward as ob

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def _dims(**kw):
    base = dict(B=2, T_new=5, L=4, k=2, D=16, Hq=4, Hkv=2, d=8, p=1, S_cap=0)
    base.update(kw)
    return oracle.Dims(**base)


def _params(dm, seed=0, scale=0.3):
    """Float64 parameters with weights large enough that every nonlinearity matters."""
    rng = np.random.default_rng(seed)
    L, k, D, Hq, Hkv, d = dm.L, dm.k, dm.D, dm.Hq, dm.Hkv, dm.d
    Lp = dm.Lp
    g = lambda *s: 1.0 + 0.2 * rng.standard_normal(s)  # noqa: E731
    n = lambda sd, *s: sd * rng.standard_normal(s)      # noqa: E731
    return {
        "g_pre": g(2, L, D), "W_alpha": n(scale / np.sqrt(Lp * D) * 4, 2, k * L, Lp * D),
        "b_alpha": n(0.5, 2, k * L), "g_mid": g(2, k, D),
        "Wk": n(scale, k, Hkv * d, D), "Wv": n(scale, k, Hkv * d, D), "g_knorm": g(k, d),
        "Kd": n(1.0, k, Hkv, d), "Vd": n(1.0, k, Hkv, d), "g_in": g(L, D),
        "Wq": n(scale, L, Hq * d, D), "g_qnorm": g(L, d),
    }


def _cache(dm, ctx, seed=1):
    """Caches [k, B, Hkv, S_cap, d]: finite context slots below ctx[b], NaN elsewhere (the
    step writes the new slots)."""
    rng = np.random.default_rng(seed)
    Kc = np.full((dm.k, dm.B, dm.Hkv, dm.S_cap, dm.d), np.nan)
    Vc = Kc.copy()
    for b in range(dm.B):
        Kc[:, b, :, :ctx[b]] = rng.standard_normal((dm.k, dm.Hkv, ctx[b], dm.d))
        Vc[:, b, :, :ctx[b]] = rng.standard_normal((dm.k, dm.Hkv, ctx[b], dm.d))
    return Kc, Vc


def _c_step(dm, P, H, cmap, ctx, Kc, Vc):
    """The C oracle's forward: O and the caches with the new slots."""
    K, V = Kc.copy(), Vc.copy()
    O = oracle.layer_step(dm, P, H, cmap, ctx, K, V)
    return O, K, V


CASES = [
    dict(),                                               # paper: linear mix, paper mask
    dict(mix_mode=oracle.MIX_SOFTMAX),
    dict(mask_mode=oracle.MASK_INCLUSIVE),
    dict(p=2, L=5, k=3),
    dict(router_mode=oracle.ROUTER_STATIC),
    dict(router_mode=oracle.ROUTER_NOFEEDBACK, L=3, k=3, mix_mode=oracle.MIX_SOFTMAX),
    dict(router_mode=oracle.ROUTER_NOFEEDBACK, L=3, k=3),
    dict(Hq=2, Hkv=2, k=1),
]


@pytest.mark.parametrize("kw", CASES)
@pytest.mark.parametrize("ctxs", [(0, 0), (3, 6)])
def test_forward_matches_c_oracle(kw, ctxs):
    dm = _dims(**kw)
    dm.S_cap = max(ctxs) + dm.T_new + 2
    P = _params(dm)
    H = np.random.default_rng(2).standard_normal((dm.B, dm.T_new, dm.L, dm.D))
    cmap = [l % dm.k for l in range(dm.L)]
    Kc, Vc = _cache(dm, ctxs)
    O, K, V = _c_step(dm, P, H, cmap, ctxs, Kc, Vc)
    Ot, Kt, Vt = ob.layer_step(dm, P, H, cmap, ctxs, Kc, Vc)
    assert np.abs(Ot - O).max() < 1e-12 * max(1.0, np.abs(O).max())
    for b in range(dm.B):
        hi = ctxs[b] + dm.T_new
        assert np.abs(Kt[:, b, :, :hi] - K[:, b, :, :hi]).max() < 1e-12
        assert np.abs(Vt[:, b, :, :hi] - V[:, b, :, :hi]).max() < 1e-12


def _fd(f, x, v, eps=1e-4):
    """Central difference along v, Richardson-extrapolated (error O(eps^4))."""
    def c(h):
        return (f(x + h * v) - f(x - h * v)) / (2 * h)
    return (4 * c(eps / 2) - c(eps)) / 3


@pytest.mark.parametrize("kw", CASES)
@pytest.mark.parametrize("ctxs", [(0, 0), (3, 6)])
def test_step_gradients_match_finite_differences(kw, ctxs):
    """Every gradient of <dO, O> + <dK, K_new> + <dV, V_new> (dH, each parameter, the
    context slots) against central differences of the C oracle's forward along a random
    direction."""
    dm = _dims(**kw)
    dm.S_cap = max(ctxs) + dm.T_new + 2
    P = _params(dm, seed=3)
    rng = np.random.default_rng(4)
    H = rng.standard_normal((dm.B, dm.T_new, dm.L, dm.D))
    cmap = [(3 * l + 1) % dm.k for l in range(dm.L)]
    Kc, Vc = _cache(dm, ctxs)
    dO = rng.standard_normal((dm.L, dm.B, dm.T_new, dm.Hq * dm.d))
    dK = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.T_new, dm.d))
    dV = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.T_new, dm.d))
    g = ob.layer_step_grads(dm, P, H, cmap, dO, ctxs, Kc, Vc, dK, dV)

    def loss(Hx, Px, Kx=Kc, Vx=Vc):
        O, K, V = _c_step(dm, Px, Hx, cmap, ctxs, Kx, Vx)
        s = (O * dO).sum()
        for b in range(dm.B):
            c0 = ctxs[b]
            s += (K[:, b, :, c0:c0 + dm.T_new] * dK[:, b]).sum()
            s += (V[:, b, :, c0:c0 + dm.T_new] * dV[:, b]).sum()
        return s

    checks = [("dH", lambda x: loss(x, P), H)]
    for n in oracle.PARAM_NAMES:
        checks.append(("d" + n, lambda x, n=n: loss(H, {**P, n: x}), P[n]))
    if max(ctxs) > 0:
        fin = np.isfinite(Kc)
        checks.append(("dKc_ctx", lambda x: loss(H, P, np.where(fin, x, np.nan), Vc),
                       np.where(fin, Kc, 0.0)))
        checks.append(("dVc_ctx", lambda x: loss(H, P, Kc, np.where(fin, x, np.nan)),
                       np.where(fin, Vc, 0.0)))
    for name, f, x in checks:
        v = rng.standard_normal(x.shape)
        if name in ("dKc_ctx", "dVc_ctx"):
            v = np.where(np.isfinite(Kc), v, 0.0)
        num = _fd(f, x, v)
        ana = (g[name] * v).sum()
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(num)), (name, num, ana)


def test_static_router_has_no_router_weight_gradient():
    dm = _dims(router_mode=oracle.ROUTER_STATIC, S_cap=5)
    P = _params(dm)
    H = np.random.default_rng(5).standard_normal((dm.B, dm.T_new, dm.L, dm.D))
    dO = np.random.default_rng(6).standard_normal((dm.L, dm.B, dm.T_new, dm.Hq * dm.d))
    g = ob.layer_step_grads(dm, P, H, [0, 1, 0, 1], dO)
    assert not np.any(g["dW_alpha"])
    assert np.any(g["db_alpha"])


# ------------------------------------------------------------- attention alone

def _attn_inputs(dm, ctxs, seed=7):
    rng = np.random.default_rng(seed)
    P = _params(dm, seed=seed)
    Q = rng.standard_normal((dm.L, dm.B, dm.Hq, dm.T_new, dm.d))
    Kc = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.S_cap, dm.d))
    Vc = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.S_cap, dm.d))
    dO = rng.standard_normal((dm.L, dm.B, dm.T_new, dm.Hq * dm.d))
    return P, Q, Kc, Vc, dO


@pytest.mark.parametrize("mask_mode", [0, 1])
def test_attention_gradients_match_finite_differences(mask_mode):
    dm = _dims(mask_mode=mask_mode, L=3, k=2, S_cap=12)
    ctxs = (2, 4)
    cmap = [1, 0, 1]
    P, Q, Kc, Vc, dO = _attn_inputs(dm, ctxs)
    g = ob.channel_attend_grads(dm, P, Q, cmap, ctxs, Kc, Vc, dO)

    def f(Qx=Q, Kx=Kc, Vx=Vc, Px=P):
        return (oracle.channel_attend(dm, Px, Qx, cmap, ctxs, Kx, Vx) * dO).sum()

    rng = np.random.default_rng(8)
    for name, fn, x in (("dQ", lambda x: f(Qx=x), Q), ("dKc", lambda x: f(Kx=x), Kc),
                        ("dVc", lambda x: f(Vx=x), Vc),
                        ("dKd", lambda x: f(Px={**P, "Kd": x}), P["Kd"]),
                        ("dVd", lambda x: f(Px={**P, "Vd": x}), P["Vd"])):
        v = rng.standard_normal(x.shape)
        num = _fd(fn, x, v)
        ana = (g[name] * v).sum()
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(num)), (name, num, ana)
    if mask_mode == 1:
        assert not np.any(g["dKd"]) and not np.any(g["dVd"])
    # slots no query sees get no gradient: at or past ctx[b] + T_new (paper: past the last
    # query's position minus one)
    for b in range(dm.B):
        hi = ctxs[b] + dm.T_new - (1 if mask_mode == 0 else 0)
        assert not np.any(g["dKc"][:, b, :, hi:]) and not np.any(g["dVc"][:, b, :, hi:])


def test_attention_gradients_closed_forms():
    """One query at position 0: in the inclusive mask it reads slot 0 alone (O = V0, so
    dV0 = dO and dQ = dK0 = 0); in the paper mask the dummy alone (dVd = dO, dKd = dQ = 0).
    With Q = 0 attention is uniform over the n visible slots: dV_s = dO / n."""
    dm = _dims(T_new=1, L=1, k=1, Hq=1, Hkv=1, S_cap=4)
    P, Q, Kc, Vc, dO = _attn_inputs(dm, (0, 0))
    g = ob.channel_attend_grads(dm, P, Q, [0], (0, 0), Kc, Vc, dO)
    assert np.allclose(g["dVd"][0, 0], dO[0, 0, 0] + dO[0, 1, 0], atol=1e-14)
    assert not np.any(g["dQ"]) and not np.any(g["dKd"]) and not np.any(g["dKc"])
    dm.mask_mode = oracle.MASK_INCLUSIVE
    g = ob.channel_attend_grads(dm, P, Q, [0], (0, 0), Kc, Vc, dO)
    for b in range(2):
        assert np.allclose(g["dVc"][0, b, 0, 0], dO[0, b, 0], atol=1e-14)
    assert not np.any(g["dQ"]) and not np.any(g["dKc"])
    # uniform attention: Q = 0, inclusive mask, positions 3 and 5 (ctx 3, 5)
    dm = _dims(T_new=1, L=1, k=1, Hq=1, Hkv=1, S_cap=8, mask_mode=oracle.MASK_INCLUSIVE)
    P, Q, Kc, Vc, dO = _attn_inputs(dm, (3, 5))
    Q[:] = 0.0
    g = ob.channel_attend_grads(dm, P, Q, [0], (3, 5), Kc, Vc, dO)
    for b, c0 in enumerate((3, 5)):
        n = c0 + 1
        for s in range(n):
            assert np.allclose(g["dVc"][0, b, 0, s], dO[0, b, 0] / n, atol=1e-14)
        # dQ = (1/sqrt d) sum_s (1/n)(dO.V_s - dO.O) K_s with O the mean of the V_s
        o = Vc[0, b, 0, :n].mean(0)
        w = (Vc[0, b, 0, :n] @ dO[0, b, 0] - o @ dO[0, b, 0]) / n
        want = (w[:, None] * Kc[0, b, 0, :n]).sum(0) / np.sqrt(dm.d)
        assert np.allclose(g["dQ"][0, b, 0, 0], want, atol=1e-13)


# ------------------------------------------------------- the step's parts alone

@pytest.mark.parametrize("kw", CASES)
def test_pool_gradients_match_finite_differences(kw):
    """pool_grads against central differences of the C oracle's pool rows (wmo_pool_rows)."""
    dm = _dims(**kw)
    ctxs = (2, 5)
    P = _params(dm, seed=11)
    rng = np.random.default_rng(12)
    H = rng.standard_normal((dm.B, dm.T_new, dm.L, dm.D))
    dK = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.T_new, dm.d))
    dV = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.T_new, dm.d))
    g = ob.pool_grads(dm, P, H, dK, dV, ctxs)

    def rows(x):  # [N, k, Hkv, d] -> [k, B, Hkv, T, d]
        return x.reshape(dm.B, dm.T_new, dm.k, dm.Hkv, dm.d).transpose(2, 0, 3, 1, 4)

    def loss(Hx, Px):
        K, V = oracle.pool_rows(dm, Px, Hx, ctxs)
        return (rows(K) * dK).sum() + (rows(V) * dV).sum()

    checks = [("dH", lambda x: loss(x, P), H)]
    for n in ob.POOL_PARAMS:
        checks.append(("d" + n, lambda x, n=n: loss(H, {**P, n: x}), P[n]))
    for name, f, x in checks:
        v = rng.standard_normal(x.shape)
        # a small step: without feedback, channel 0 mixes one source with a signed weight
        # that can sit near zero, where the mid norm's curvature is large
        num = _fd(f, x, v, eps=2e-5)
        ana = (g[name] * v).sum()
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(num)), (name, num, ana)


@pytest.mark.parametrize("kw", [dict(), dict(Hq=2, Hkv=1, d=16), dict(L=2, k=1)])
def test_query_gradients_match_finite_differences(kw):
    """q_project_grads against central differences of the C oracle's queries."""
    dm = _dims(**kw)
    ctxs = (0, 7)
    P = _params(dm, seed=13)
    rng = np.random.default_rng(14)
    H = rng.standard_normal((dm.B, dm.T_new, dm.L, dm.D))
    dQ = rng.standard_normal((dm.L, dm.B, dm.Hq, dm.T_new, dm.d))
    g = ob.q_project_grads(dm, P, H, dQ, ctxs)

    def loss(Hx, Px):
        return (oracle.q_project(dm, Px, Hx, ctxs) * dQ).sum()

    checks = [("dH", lambda x: loss(x, P), H)]
    for n in ob.QUERY_PARAMS:
        checks.append(("d" + n, lambda x, n=n: loss(H, {**P, n: x}), P[n]))
    for name, f, x in checks:
        v = rng.standard_normal(x.shape)
        num = _fd(f, x, v)
        ana = (g[name] * v).sum()
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(num)), (name, num, ana)


@pytest.mark.parametrize("kw", [dict(), dict(mask_mode=oracle.MASK_INCLUSIVE),
                                dict(router_mode=oracle.ROUTER_NOFEEDBACK, L=3, k=3)])
def test_step_gradient_is_the_sum_of_its_parts(kw):
    """The decomposition the GPU step's backward runs: attention gradients first, then the
    queries' backward of dQ and the pool's backward of the new slots' total gradient (the
    attention's plus what reaches them from elsewhere). The parts' sum equals the whole
    step's gradient (computed as one autograd graph)."""
    dm = _dims(**kw)
    ctxs = (3, 1)
    dm.S_cap = max(ctxs) + dm.T_new + 1
    P = _params(dm, seed=15)
    rng = np.random.default_rng(16)
    H = rng.standard_normal((dm.B, dm.T_new, dm.L, dm.D))
    cmap = [(l + 1) % dm.k for l in range(dm.L)]
    Kc, Vc = _cache(dm, ctxs)
    dO = rng.standard_normal((dm.L, dm.B, dm.T_new, dm.Hq * dm.d))
    dKe = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.T_new, dm.d))
    dVe = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.T_new, dm.d))
    whole = ob.layer_step_grads(dm, P, H, cmap, dO, ctxs, Kc, Vc, dKe, dVe)
    _, K, V = _c_step(dm, P, H, cmap, ctxs, Kc, Vc)
    K, V = np.nan_to_num(K), np.nan_to_num(V)
    Q = oracle.q_project(dm, P, H, ctxs)
    ga = ob.channel_attend_grads(dm, P, Q, cmap, ctxs, K, V, dO)
    gq = ob.q_project_grads(dm, P, H, ga["dQ"], ctxs)
    gp = ob.pool_grads(dm, P, H, dKe + ob.new_rows(dm, ga["dKc"], ctxs),
                       dVe + ob.new_rows(dm, ga["dVc"], ctxs), ctxs)
    tol = 1e-10
    assert np.abs(gq["dH"] + gp["dH"] - whole["dH"]).max() < tol
    for n in ob.QUERY_PARAMS:
        assert np.abs(gq["d" + n] - whole["d" + n]).max() < tol, n
    for n in ob.POOL_PARAMS:
        assert np.abs(gp["d" + n] - whole["d" + n]).max() < tol, n
    assert np.abs(ga["dKd"] - whole["dKd"]).max() < tol
    assert np.abs(ga["dVd"] - whole["dVd"]).max() < tol
    for b in range(dm.B):
        c0 = ctxs[b]
        assert np.abs(ga["dKc"][:, b, :, :c0] - whole["dKc_ctx"][:, b, :, :c0]).max() < tol
        assert np.abs(ga["dVc"][:, b, :, :c0] - whole["dVc_ctx"][:, b, :, :c0]).max() < tol


# ------------------------------------------------ passes and truncated backprop

def _pass_inputs(dm, seed=21):
    rng = np.random.default_rng(seed)
    P = _params(dm, seed=seed)
    W_o = 0.3 * rng.standard_normal((dm.L, dm.D, dm.Hq * dm.d)) / np.sqrt(dm.Hq * dm.d)
    X = rng.standard_normal((dm.B, dm.T_new, dm.D))
    dh = rng.standard_normal((dm.B, dm.T_new, dm.D))
    return P, W_o, X, dh, rng


PASS_CASES = [dict(), dict(mask_mode=oracle.MASK_INCLUSIVE, mix_mode=oracle.MIX_SOFTMAX),
              dict(p=2, L=5, k=3)]


@pytest.mark.parametrize("kw", PASS_CASES)
@pytest.mark.parametrize("g", [1, 2, 3])
def test_passes_forward_matches_c_oracle(kw, g):
    dm = _dims(T_new=6, **kw)
    dm.S_cap = dm.T_new
    P, W_o, X, _, _ = _pass_inputs(dm)
    cmap = [(l + 1) % dm.k for l in range(dm.L)]
    H, top, _, _ = oracle.gauss_seidel(dm, P, W_o, cmap, X, g, 3)
    Pt = {n: ob._t(P[n]) for n in oracle.PARAM_NAMES}
    Ht, topt = ob.passes_forward(dm, Pt, ob._t(W_o), ob._t(X), cmap, 3, 3, g=g)
    assert np.abs(Ht.detach().numpy() - H).max() < 1e-12
    assert np.abs(topt.detach().numpy() - top).max() < 1e-12


@pytest.mark.parametrize("kw", PASS_CASES)
@pytest.mark.parametrize("passes,n_grad,g", [(2, 2, 1), (3, 1, 1), (3, 2, 1), (2, 2, 2),
                                             (2, 1, 3)])
def test_truncated_pass_gradients_match_finite_differences(kw, passes, n_grad, g):
    """Full backpropagation (n_grad = passes) against central differences of the C oracle's
    passes; truncated backpropagation against central differences of the last n_grad passes
    run by the C oracle from the cache entering them, held fixed at its value."""
    dm = _dims(T_new=6, **kw)
    dm.S_cap = dm.T_new
    P, W_o, X, dh, rng = _pass_inputs(dm)
    cmap = [(2 * l + 1) % dm.k for l in range(dm.L)]
    gr = ob.passes_grads(dm, P, W_o, X, cmap, passes, n_grad, dh, g=g)
    if n_grad == passes:
        def top(Px, Wx, Xx):
            return (oracle.gauss_seidel(dm, Px, Wx, cmap, Xx, g, passes)[1] * dh).sum()
    else:
        _, _, K0, V0 = oracle.gauss_seidel(dm, P, W_o, cmap, X, g, passes - n_grad)

        def top(Px, Wx, Xx):
            return (oracle.gauss_seidel_from(dm, Px, Wx, cmap, Xx, g, K0, V0, n_grad)[1]
                    * dh).sum()
    checks = [("dX", lambda x: top(P, W_o, x), X), ("dW_o", lambda x: top(P, x, X), W_o)]
    for n in oracle.PARAM_NAMES:
        checks.append(("d" + n, lambda x, n=n: top({**P, n: x}, W_o, X), P[n]))
    for name, f, x in checks:
        v = rng.standard_normal(x.shape)
        num = _fd(f, x, v, eps=2e-5)
        ana = (gr[name] * v).sum()
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(num)), (name, num, ana)


def test_bf16_storage_rounds_values_and_passes_gradients():
    """bf16_store: the value is the bf16 rounding (round to nearest even, checked against
    the float32 bit pattern rounded to its upper half), the derivative the identity."""
    import torch
    x = torch.tensor([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -9, -3.14159, 1e-3],
                     dtype=torch.float64, requires_grad=True)
    y = ob.bf16_store(x)
    f = x.detach().numpy().astype(np.float32).view(np.uint32)
    rnd = ((f + 0x7FFF + ((f >> 16) & 1)) & 0xFFFF0000).view(np.float32).astype(np.float64)
    assert np.array_equal(y.detach().numpy(), rnd)
    (g,) = torch.autograd.grad(y.sum(), x)
    assert np.array_equal(g.numpy(), np.ones(5))
    # storage rounding moves the passes' gradients by rounding-sized amounts
    dm = _dims(T_new=5)
    dm.S_cap = dm.T_new
    P, W_o, X, dh, _ = _pass_inputs(dm)
    cmap = [l % dm.k for l in range(dm.L)]
    a = ob.passes_grads(dm, P, W_o, X, cmap, 2, 2, dh)
    b = ob.passes_grads(dm, P, W_o, X, cmap, 2, 2, dh, bf16_storage=True)
    for n in ("dX", "dW_o", "dWq", "dW_alpha"):
        rel = np.abs(a[n] - b[n]).max() / np.abs(a[n]).max()
        assert 1e-6 < rel < 0.1, (n, rel)


@pytest.mark.parametrize("mask_mode", [0, 1])
def test_strided_group_step_gradients_match_finite_differences(mask_mode):
    """A step over the strided token group q = 1 of g = 3 (positions 1, 4, 7, ...) with every
    other slot given: every gradient against central differences of the C oracle's pool and
    channel attention at those positions (the C oracle's pool with a token list, its
    attention over the spliced cache)."""
    dm = _dims(T_new=4, mask_mode=mask_mode, L=3, k=2)
    g, q = 3, 1
    dm.S_cap = q + g * (dm.T_new - 1) + 1
    P = _params(dm, seed=31)
    rng = np.random.default_rng(32)
    H = rng.standard_normal((dm.B, dm.T_new, dm.L, dm.D))
    cmap = [1, 0, 1]
    Kc = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.S_cap, dm.d))
    Vc = rng.standard_normal((dm.k, dm.B, dm.Hkv, dm.S_cap, dm.d))
    dO = rng.standard_normal((dm.L, dm.B, dm.T_new, dm.Hq * dm.d))
    gr = ob.layer_step_grads(dm, P, H, cmap, dO, None, Kc, Vc, grp=(g, q))
    # the C oracle at the group's positions: a full-length problem whose other tokens' H
    # are ignored (their rows come from Kc, Vc)
    full = _dims(T_new=dm.S_cap, mask_mode=mask_mode, L=3, k=2)
    full.S_cap = dm.S_cap
    pos = [q + g * i for i in range(dm.T_new)]

    def loss(Hx, Px, Kx=Kc, Vx=Vc):
        Hf = np.zeros((dm.B, full.T_new, dm.L, dm.D))
        Hf[:, pos] = Hx
        K, V = Kx.copy(), Vx.copy()
        oracle.pool(full, Px, Hf, None, K, V, toks=[b * full.T_new + p for b in range(dm.B)
                                                    for p in pos])
        Qf = oracle.q_project(full, Px, Hf)
        O = oracle.channel_attend(full, Px, Qf, cmap, None, K, V)
        return (O[:, :, pos] * dO).sum()

    gslots = np.zeros(dm.S_cap, dtype=bool)
    gslots[pos] = True
    checks = [("dH", lambda x: loss(x, P), H)]
    for n in oracle.PARAM_NAMES:
        checks.append(("d" + n, lambda x, n=n: loss(H, {**P, n: x}), P[n]))
    checks.append(("dKc_ctx", lambda x: loss(H, P, x, Vc), Kc))
    checks.append(("dVc_ctx", lambda x: loss(H, P, Kc, x), Vc))
    for name, f, x in checks:
        v = rng.standard_normal(x.shape)
        if name in ("dKc_ctx", "dVc_ctx"):
            v[..., gslots, :] = 0.0  # the group's own slots are overwritten by the step
        num = _fd(f, x, v)
        ana = (gr[name] * v).sum()
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(num)), (name, num, ana)
