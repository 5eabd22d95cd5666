"""CPU pins of the oracle's fixed-point passes (Section 3.3).

The paper fixes how the schedules relate: Jacobi iteration is the one-group case of
cyclic Gauss-Seidel, T groups make it autoregressive, and every schedule targets the
exact left-to-right solution (Section 3.2's decode order) of P = Pool(H),
H = States(X; P). These pins check the three oracle drivers against each other and
against the single-step oracle, which is pinned on its own (test_oracle_pins.py):
  - Gauss-Seidel with g = 1 equals Jacobi, bit for bit (states and top states);
  - Gauss-Seidel with g = T equals autoregressive evaluation after one pass, bit for bit
    (states, top states and cache);
  - after t passes, positions below t (Jacobi) or t g (Gauss-Seidel with g groups) are
    exact, bit for bit, and the next position is not yet;
  - the autoregressive result is a fixed point: pooling its states gives its cache, and
    each layer's channel attention over that cache, fed through the stand-in block,
    gives the next layer's state (the single-step oracle computes the attention).
"""
import numpy as np
import pytest

import oracle
from tests import synth

CASES = {
    "mha": synth.small("pass_mha", B=2, T_new=12, L=3, k=2, D=32, Hq=2, Hkv=2, d=16, dtype="f32",
                       seed=301),
    "gqa_p2": synth.small("pass_gqa", B=1, T_new=10, L=4, k=3, D=32, Hq=4, Hkv=2, d=16, p=2,
                          dtype="f32", seed=302),
}


def _setup(name, mask_mode=0):
    w = CASES[name]
    P = synth.make_params(w, oracle.init_bias(w.L, w.k) + 0.2)
    X = synth.make_embeddings(w)
    W_o = synth.make_out_proj(w)
    dm = oracle.Dims(B=w.B, T_new=w.T_new, L=w.L, k=w.k, D=w.D, Hq=w.Hq, Hkv=w.Hkv, d=w.d,
                     p=w.p, S_cap=w.T_new, mask_mode=mask_mode)
    return w, dm, oracle.Params(P), X, W_o


@pytest.fixture(scope="module", autouse=True)
def _built(oracle_lib):
    return oracle_lib


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("mask_mode", [0, 1])
def test_one_group_is_jacobi(name, mask_mode):
    w, dm, P, X, W_o = _setup(name, mask_mode)
    for passes in (1, 2, 3):
        Hj, tj, _, _ = oracle.jacobi(dm, P, W_o, w.chan_map, X, passes)
        Hg, tg, _, _ = oracle.gauss_seidel(dm, P, W_o, w.chan_map, X, 1, passes)
        assert np.array_equal(Hj, Hg) and np.array_equal(tj, tg), passes


# The exact left-to-right solution exists in the paper's mask, where a token never reads
# its own slot (Section 3.2); with the inclusive mask a token's attention would read the
# channels of its own states, so only the iterations themselves are defined there.
@pytest.mark.parametrize("name", list(CASES))
def test_T_groups_is_autoregressive(name):
    w, dm, P, X, W_o = _setup(name)
    Ha, ta, Ka, Va = oracle.autoregressive(dm, P, W_o, w.chan_map, X)
    Hg, tg, Kg, Vg = oracle.gauss_seidel(dm, P, W_o, w.chan_map, X, w.T_new, 1)
    for a, b in ((Ha, Hg), (ta, tg), (Ka, Kg), (Va, Vg)):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("name", list(CASES))
def test_exact_prefix_grows_with_passes(name):
    """Position i reads only slots below i: after t passes the first t (Jacobi) or t g
    (Gauss-Seidel) positions hold the exact solution, and the next one does not yet."""
    w, dm, P, X, W_o = _setup(name)
    Ha, ta, _, _ = oracle.autoregressive(dm, P, W_o, w.chan_map, X)
    for g, passes in ((1, 1), (1, 2), (1, 4), (2, 1), (2, 2), (3, 2), (4, 1)):
        if g == 1:
            H, top, _, _ = oracle.jacobi(dm, P, W_o, w.chan_map, X, passes)
        else:
            H, top, _, _ = oracle.gauss_seidel(dm, P, W_o, w.chan_map, X, g, passes)
        exact = min(passes * g, w.T_new)
        assert np.array_equal(H[:, :exact], Ha[:, :exact]), (g, passes)
        assert np.array_equal(top[:, :exact], ta[:, :exact]), (g, passes)
        if exact < w.T_new:
            assert not np.array_equal(top[:, exact], ta[:, exact]), (g, passes)


@pytest.mark.parametrize("name", list(CASES))
def test_autoregressive_solution_is_a_fixed_point(name):
    w, dm, P, X, W_o = _setup(name)
    Ha, ta, Ka, Va = oracle.autoregressive(dm, P, W_o, w.chan_map, X)
    Kc, Vc = oracle.empty_cache(dm)
    O = oracle.layer_step(dm, P, Ha, w.chan_map, None, Kc, Vc)  # Pool(H), then attention
    assert np.array_equal(Kc, Ka) and np.array_equal(Vc, Va)
    assert np.array_equal(Ha[:, :, 0], np.asarray(X, dtype=np.float64))
    Wn = np.asarray(W_o, dtype=np.float64)
    for l in range(w.L):
        nxt = Ha[:, :, l] + np.einsum("ec,btc->bte", Wn[l], O[l])
        want = Ha[:, :, l + 1] if l + 1 < w.L else ta
        np.testing.assert_allclose(nxt, want, rtol=0, atol=1e-12)


def test_stand_in_block_special_cases(oracle_lib):
    w, dm, P, X, W_o = _setup("mha")
    rng = np.random.default_rng(5)
    h = rng.normal(size=w.D)
    assert np.array_equal(oracle.block_residual(dm, W_o, 1, h, np.zeros(w.Hq * w.d)), h)
    sel = np.zeros((w.L, w.D, w.Hq * w.d))
    for e in range(w.D):
        sel[1, e, (3 * e) % (w.Hq * w.d)] = 1.0   # each output picks one attention channel
    o = rng.normal(size=w.Hq * w.d)
    got = oracle.block_residual(dm, sel, 1, np.zeros(w.D), o)
    assert np.array_equal(got, o[(3 * np.arange(w.D)) % (w.Hq * w.d)])
