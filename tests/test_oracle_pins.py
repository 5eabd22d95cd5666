"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every test here runs on the CPU. Each one checks the oracle against something
other than itself: values the paper states (golden fixtures), closed forms,
special cases that reduce to a textbook/library routine (torch's rms_norm,
linear, softmax, complex multiplication, scaled_dot_product_attention, all in
float64), invariants, and brute force on tiny inputs.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from tests import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _dims(o, w: synth.Workload, **kw):
    base = dict(B=w.B, T_new=w.T_new, L=w.L, k=w.k, D=w.D, Hq=w.Hq, Hkv=w.Hkv, d=w.d, p=w.p,
                S_cap=w.S_cap)
    base.update(kw)
    return o.Dims(**base)


def _t(a):
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


# ------------------------------------------------------------------ RMSNorm

def test_rmsnorm_constant_vector_closed_form(oracle_lib):
    """RMSNorm(c*1) = g * sign(c) / sqrt(1 + eps/c^2)."""
    o = oracle_lib
    rng = np.random.default_rng(0)
    for c in (3.0, -0.25, 1e-3, 7.5):
        for eps in (1e-6, 1e-2):
            g = rng.normal(size=17)
            y = o.rmsnorm(np.full(17, c), g, eps)
            ref = g * math.copysign(1.0, c) / math.sqrt(1.0 + eps / (c * c))
            np.testing.assert_allclose(y, ref, rtol=1e-14, atol=0)


def test_rmsnorm_matches_torch_rms_norm(oracle_lib):
    rng = np.random.default_rng(1)
    x, g = rng.normal(size=64) * 3, rng.normal(size=64)
    ref = F.rms_norm(_t(x), (64,), weight=_t(g), eps=1e-6).numpy()
    np.testing.assert_allclose(oracle_lib.rmsnorm(x, g, 1e-6), ref, rtol=1e-13, atol=1e-15)


# ------------------------------------------------------------------- RoPE

def _rope_complex(x, pos, theta):
    """Rotate-half RoPE as complex multiplication of pairs (m, m + d/2)."""
    d = x.shape[-1]
    half = d // 2
    z = torch.complex(_t(x[:half]), _t(x[half:]))
    freq = torch.tensor([theta ** (-2.0 * m / d) for m in range(half)], dtype=torch.float64)
    rot = torch.polar(torch.ones(half, dtype=torch.float64), pos * freq)
    w = z * rot
    return torch.cat([w.real, w.imag]).numpy()


@pytest.mark.parametrize("d", [2, 32, 64, 96])
def test_rope_is_complex_rotation(oracle_lib, d):
    rng = np.random.default_rng(d)
    for pos in (0, 1, 17, 2047, 32768):
        x = rng.normal(size=d)
        np.testing.assert_allclose(oracle_lib.rope(x, pos, 1e6), _rope_complex(x, pos, 1e6),
                                   rtol=0, atol=1e-12)


def test_rope_relative_position_and_norm(oracle_lib):
    """<RoPE(q,t), RoPE(k,s)> depends only on t - s; the rotation keeps norms."""
    o = oracle_lib
    rng = np.random.default_rng(3)
    q, k = rng.normal(size=64), rng.normal(size=64)
    base = o.rope(q, 40, 1e4) @ o.rope(k, 13, 1e4)
    for shift in (1, 100, 5000):
        assert abs(o.rope(q, 40 + shift, 1e4) @ o.rope(k, 13 + shift, 1e4) - base) < 1e-9
    assert abs(np.linalg.norm(o.rope(q, 123, 1e6)) - np.linalg.norm(q)) < 1e-12
    np.testing.assert_array_equal(o.rope(q, 0, 1e6), q)


# ----------------------------------------------------- router inputs, init

def test_router_layer_selection_golden(oracle_lib):
    for case in _load("router_layer_selection.json")["cases"]:
        assert oracle_lib.router_layers(case["L"], case["p"]) == case["layers"], case


def test_router_init_patterns_golden(oracle_lib):
    for case in _load("router_init_patterns.json")["cases"]:
        L, k = case["L"], case["k"]
        b = oracle_lib.init_bias(L, k).reshape(k, L)
        want = np.zeros((k, L))
        for j, srcs in enumerate(case["channel_sources"]):
            want[j, srcs] = 1.0
        np.testing.assert_array_equal(b, want, err_msg=str(case))


def test_channel_groups_cardinality(oracle_lib):
    """Under l mod k each channel has floor(L/k) or ceil(L/k) consumers; k=1 and k=L."""
    o = oracle_lib
    for L in range(1, 33):
        for k in range(1, L + 1):
            off, mem = o.channel_groups(L, k, [l % k for l in range(L)])
            sizes = np.diff(off)
            assert set(sizes.tolist()) <= {L // k, -(-L // k)}
            assert sorted(mem.tolist()) == list(range(L))
    off, mem = o.channel_groups(6, 1, [0] * 6)
    assert off.tolist() == [0, 6] and mem.tolist() == list(range(6))
    off, mem = o.channel_groups(6, 6, list(range(6)))
    assert off.tolist() == list(range(7)) and mem.tolist() == list(range(6))
    off, mem = o.channel_groups(12, 6, [l // 2 for l in range(12)])
    assert off.tolist() == [0, 2, 4, 6, 8, 10, 12] and mem.tolist() == list(range(12))
    with pytest.raises(ValueError):
        o.channel_groups(4, 2, [0, 1, 2, 0])


# --------------------------------------------------------- router + mix

def _normed(h, g, eps=1e-6):
    """Pre-mix RMSNorm of every layer via torch's rms_norm: [N, L, D]."""
    H = _t(h)
    return torch.stack([F.rms_norm(H[:, l], (H.shape[-1],), weight=_t(g[l]), eps=eps)
                        for l in range(H.shape[1])], dim=1)


def _small(**kw):
    w = synth.small(dtype="f32", **kw)
    return w


def test_zero_router_gives_bias_exactly(oracle_lib):
    """W^alpha = 0 => alpha = reshape(b) exactly (Section 3.1, Router initialization)."""
    o = oracle_lib
    w = _small(L=5, k=3, T_new=6, B=2)
    rng = np.random.default_rng(4)
    b = rng.normal(size=(2, w.k * w.L))
    P = synth.make_params(w, b, gains="random", zero_router=True)
    H = synth.make_states(w)
    alpha, _ = o.router_mix(_dims(o, w), P, H)
    bb = P["b_alpha"].double().numpy().reshape(2, 1, w.k, w.L)
    np.testing.assert_array_equal(alpha, np.broadcast_to(bb, alpha.shape))


def test_mix_with_arbitrary_static_weights(oracle_lib):
    """W^alpha = 0 and random b: channel j = sum_l b[j*L+l] * RMSNorm(h_l) (library einsum)."""
    o = oracle_lib
    w = _small(L=6, k=4, T_new=5, B=2)
    rng = np.random.default_rng(5)
    b = rng.normal(size=(2, w.k * w.L))
    P = synth.make_params(w, b, gains="random", zero_router=True)
    H = synth.make_states(w)
    _, mixed = o.router_mix(_dims(o, w), P, H)
    Hf = H.double().reshape(w.N, w.L, w.D)
    for br in range(2):
        hn = _normed(Hf, P["g_pre"][br].double())
        A = P["b_alpha"][br].double().reshape(w.k, w.L)
        ref = torch.einsum("jl,nld->jnd", A, hn).numpy()
        np.testing.assert_allclose(mixed[br], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("L,k", [(4, 1), (5, 3), (4, 4), (8, 8), (6, 2)])
def test_one_hot_patterns_select_exactly(oracle_lib, L, k):
    """The paper's one-hot initial biases make channel j equal its source layer's normed
    state bit-for-bit."""
    o = oracle_lib
    w = _small(L=L, k=k, T_new=4, B=1)
    b = o.init_bias(L, k)
    P = synth.make_params(w, b, gains="random", zero_router=True)
    H = synth.make_states(w)
    _, mixed = o.router_mix(_dims(o, w), P, H)
    Hf = H.double().reshape(w.N, w.L, w.D).numpy()
    for br in range(2):
        g = P["g_pre"][br].double().numpy()
        for j in range(k):
            srcs = np.nonzero(b.reshape(k, L)[j])[0]
            for n in range(w.N):
                ref = sum(o.rmsnorm(Hf[n, s], g[s]) for s in srcs)
                if len(srcs) == 1:
                    np.testing.assert_array_equal(mixed[br, j, n], ref)
                else:
                    np.testing.assert_allclose(mixed[br, j, n], ref, rtol=1e-14, atol=1e-14)


@pytest.mark.parametrize("p", [1, 2, 3])
def test_router_logits_match_linear_on_stacked_states(oracle_lib, p):
    """alpha = reshape(W xi + b) with xi the normed states of layers {L-1-p*m}, ascending."""
    o = oracle_lib
    w = _small(L=7, k=3, T_new=5, B=2, p=p)
    rng = np.random.default_rng(6)
    P = synth.make_params(w, rng.normal(size=(2, w.k * w.L)), gains="random")
    H = synth.make_states(w)
    alpha, _ = o.router_mix(_dims(o, w), P, H)
    sel = [l for l in range(w.L) if (w.L - 1 - l) % p == 0]
    Hf = H.double().reshape(w.N, w.L, w.D)
    for br in range(2):
        hn = _normed(Hf, P["g_pre"][br].double())
        xi = hn[:, sel].reshape(w.N, -1)
        ref = F.linear(xi, P["W_alpha"][br].double(), P["b_alpha"][br].double())
        np.testing.assert_allclose(alpha[br], ref.reshape(w.N, w.k, w.L).numpy(),
                                   rtol=1e-12, atol=1e-12)


def test_router_reads_selected_block_in_ascending_order(oracle_lib):
    """A router whose only nonzero column is element e of stacked block m reads layer
    sel[m] (ascending order of {L-1-p*m})."""
    o = oracle_lib
    w = _small(L=5, k=2, T_new=3, B=1, p=2, D=32)
    sel = [0, 2, 4]
    H = synth.make_states(w)
    Hf = H.double().reshape(w.N, w.L, w.D).numpy()
    for m in range(3):
        P = synth.make_params(w, np.zeros((2, w.k * w.L)), zero_router=True)
        Wa = torch.zeros_like(P["W_alpha"])
        Wa[:, 0, m * w.D + 7] = 1.0
        P["W_alpha"] = Wa
        alpha, _ = o.router_mix(_dims(o, w), P, H)
        for n in range(w.N):
            ref = o.rmsnorm(Hf[n, sel[m]], np.ones(w.D))[7]
            assert abs(alpha[0, n, 0, 0] - ref) < 1e-14


def test_softmax_mode_rows_sum_to_one(oracle_lib):
    """Softmax-over-depth mode: each channel's weights are positive and sum to 1, and
    equal torch.softmax of the linear-mode logits."""
    o = oracle_lib
    w = _small(L=6, k=3, T_new=7, B=2)
    rng = np.random.default_rng(8)
    P = synth.make_params(w, rng.normal(size=(2, w.k * w.L)))
    H = synth.make_states(w)
    lin, _ = o.router_mix(_dims(o, w), P, H)
    sm, mixed = o.router_mix(_dims(o, w, mix_mode=o.MIX_SOFTMAX), P, H)
    assert (sm > 0).all()
    np.testing.assert_allclose(sm.sum(-1), 1.0, rtol=0, atol=1e-14)
    np.testing.assert_allclose(sm, torch.softmax(_t(lin), dim=-1).numpy(), rtol=1e-13, atol=0)


# ------------------------------------------------------ projection, cache

def test_mid_norm_makes_cache_invariant_to_router_scale(oracle_lib):
    """Scaling (W^alpha, b) by lambda > 0 scales the mixed channels by lambda; the mid
    RMSNorm removes it, so the cache is unchanged up to the eps term."""
    o = oracle_lib
    w = _small(L=4, k=2, T_new=6, B=1)
    rng = np.random.default_rng(9)
    b = rng.normal(size=(2, w.k * w.L))
    P = synth.make_params(w, b, gains="random")
    H = synth.make_states(w)
    dm = _dims(o, w)
    K1, V1 = o.empty_cache(dm)
    o.pool(dm, P, H, None, K1, V1)
    P2 = dict(P)
    P2["W_alpha"] = P["W_alpha"] * 4.0
    P2["b_alpha"] = P["b_alpha"] * 4.0
    K2, V2 = o.empty_cache(dm)
    o.pool(dm, P2, H, None, K2, V2)
    sl = np.s_[:, :, :, :w.T_new]
    np.testing.assert_allclose(K2[sl], K1[sl], rtol=0, atol=1e-5)
    np.testing.assert_allclose(V2[sl], V1[sl], rtol=0, atol=1e-5)


def test_cache_write_set_is_exactly_the_new_slots(oracle_lib):
    """k * N * Hkv * d elements are written per cache, at slots ctx_len[b] + i only."""
    o = oracle_lib
    w = _small(L=4, k=3, T_new=5, B=3, ctx=7)
    P = synth.make_params(w, o.init_bias(w.L, w.k))
    H = synth.make_states(w)
    dm = _dims(o, w)
    ctx = np.array([0, 7, 3], dtype=np.int32)
    K, V = o.empty_cache(dm)
    o.pool(dm, P, H, ctx, K, V)
    for C in (K, V):
        written = ~np.isnan(C)
        assert written.sum() == w.k * w.N * w.Hkv * w.d
        for b in range(w.B):
            slots = np.nonzero(written[0, b, 0, :, 0])[0].tolist()
            assert slots == list(range(ctx[b], ctx[b] + w.T_new))


# -------------------------------------------------------------- attention

def test_attend_row_matches_sdpa_with_dummy(oracle_lib):
    rng = np.random.default_rng(10)
    d, n = 32, 9
    q, K, V = rng.normal(size=d), rng.normal(size=(n, d)), rng.normal(size=(n, d))
    kd, vd = rng.normal(size=d), rng.normal(size=d)
    out = oracle_lib.attend_row(q, K, V, kd, vd)
    ref = F.scaled_dot_product_attention(_t(q)[None, None], _t(np.vstack([kd, K]))[None],
                                         _t(np.vstack([vd, V]))[None])[0, 0].numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)
    out2 = oracle_lib.attend_row(q, K, V)
    ref2 = F.scaled_dot_product_attention(_t(q)[None, None], _t(K)[None], _t(V)[None])[0, 0]
    np.testing.assert_allclose(out2, ref2.numpy(), rtol=1e-12, atol=1e-13)


def test_first_token_reads_only_the_dummy(oracle_lib):
    """Paper mask at position 0: the softmax has one element, so O = Vd of the channel."""
    o = oracle_lib
    w = _small(L=5, k=3, T_new=4, B=2, Hq=4, Hkv=2)
    P = synth.make_params(w, o.init_bias(w.L, w.k))
    H = synth.make_states(w)
    dm = _dims(o, w)
    K, V = o.empty_cache(dm)
    O = o.layer_step(dm, P, H, w.chan_map, None, K, V)
    Vd = P["Vd"].double().numpy()
    for l in range(w.L):
        for b in range(w.B):
            for h in range(w.Hq):
                np.testing.assert_array_equal(O[l, b, 0, h * w.d:(h + 1) * w.d],
                                              Vd[w.chan_map[l], h // 2])


def test_equal_keys_give_mean_of_values(oracle_lib):
    rng = np.random.default_rng(11)
    d = 16
    key = rng.normal(size=d)
    K = np.tile(key, (6, 1))
    V = rng.normal(size=(6, d))
    vd = rng.normal(size=d)
    out = oracle_lib.attend_row(rng.normal(size=d), K, V, key, vd)
    np.testing.assert_allclose(out, (V.sum(0) + vd) / 7.0, rtol=1e-13, atol=1e-14)


def _vanilla_reference(w, P, H, paper_mask):
    """Vanilla per-layer Qwen3 attention built from torch library routines in float64:
    K_l = RoPE(knorm(W^K_l RMSNorm_mid(RMSNorm_pre(h_l)))), V_l = W^V_l (same input),
    Q_l = RoPE(qnorm(W^Q_l RMSNorm_in(h_l))), then causal SDPA (GQA) per layer; with the
    paper mask a dummy slot is prepended and the diagonal is excluded."""
    T, D, d = w.T_new, w.D, w.d
    Hf = H.double()[0]  # B = 1: [T, L, D]
    outs = []
    for l in range(w.L):
        x = Hf[:, l]
        xq = F.rms_norm(x, (D,), weight=P["g_in"][l].double(), eps=1e-6)
        q = F.linear(xq, P["Wq"][l].double()).reshape(T, w.Hq, d)
        q = F.rms_norm(q, (d,), weight=P["g_qnorm"][l].double(), eps=1e-6)
        kx = F.rms_norm(F.rms_norm(x, (D,), weight=P["g_pre"][0, l].double(), eps=1e-6), (D,),
                        weight=P["g_mid"][0, l].double(), eps=1e-6)
        vx = F.rms_norm(F.rms_norm(x, (D,), weight=P["g_pre"][1, l].double(), eps=1e-6), (D,),
                        weight=P["g_mid"][1, l].double(), eps=1e-6)
        kk = F.linear(kx, P["Wk"][l].double()).reshape(T, w.Hkv, d)
        kk = F.rms_norm(kk, (d,), weight=P["g_knorm"][l].double(), eps=1e-6)
        vv = F.linear(vx, P["Wv"][l].double()).reshape(T, w.Hkv, d)
        qr = torch.stack([torch.stack([_t(_rope_complex(q[t, h].numpy(), t, 1e6))
                                       for h in range(w.Hq)]) for t in range(T)])
        kr = torch.stack([torch.stack([_t(_rope_complex(kk[t, h].numpy(), t, 1e6))
                                       for h in range(w.Hkv)]) for t in range(T)])
        Qh, Kh, Vh = qr.transpose(0, 1), kr.transpose(0, 1), vv.transpose(0, 1)
        if paper_mask:
            Kh = torch.cat([P["Kd"][l].double()[:, None], Kh], dim=1)
            Vh = torch.cat([P["Vd"][l].double()[:, None], Vh], dim=1)
            mask = torch.zeros(T, T + 1, dtype=torch.bool)
            mask[:, 0] = True
            for t in range(T):
                mask[t, 1:t + 1] = True
            o = F.scaled_dot_product_attention(Qh, Kh, Vh, attn_mask=mask, enable_gqa=True)
        else:
            o = F.scaled_dot_product_attention(Qh, Kh, Vh, is_causal=True, enable_gqa=True)
        outs.append(o.transpose(0, 1).reshape(T, w.Hq * d))
    return torch.stack(outs).numpy()  # [L, T, Hq*d]


@pytest.mark.parametrize("paper_mask", [False, True])
def test_k_equals_L_identity_routing_is_vanilla_attention(oracle_lib, paper_mask):
    """k = L, W^alpha = 0 and one-hot bias on each consumer's own layer reduce the pool to
    vanilla per-layer KV (Section 3.1 Step 3, k = L), compared with torch SDPA."""
    o = oracle_lib
    w = _small(L=3, k=3, T_new=9, B=1, D=32, Hq=4, Hkv=2, d=16)
    b = np.eye(3).reshape(-1)  # channel j <- layer j
    P = synth.make_params(w, b, gains="random", zero_router=True)
    H = synth.make_states(w)
    dm = _dims(o, w, mask_mode=o.MASK_PAPER if paper_mask else o.MASK_INCLUSIVE)
    K, V = o.empty_cache(dm)
    O = o.layer_step(dm, P, H, list(range(3)), None, K, V)
    ref = _vanilla_reference(w, P, H, paper_mask)
    np.testing.assert_allclose(O[:, 0], ref, rtol=1e-10, atol=1e-12)


def test_decode_step_equals_full_sequence_row(oracle_lib):
    """A decode step at context t, over the cache of tokens < t, equals row t of the
    full-sequence step (the fixed-point definition and Section 3.2)."""
    o = oracle_lib
    w = _small(L=5, k=2, T_new=12, B=2, Hq=4, Hkv=2)
    rng = np.random.default_rng(12)
    P = synth.make_params(w, rng.normal(size=(2, w.k * w.L)), gains="random")
    H = synth.make_states(w)
    dm = _dims(o, w)
    K, V = o.empty_cache(dm)
    O = o.layer_step(dm, P, H, w.chan_map, None, K, V)
    for t in (0, 5, 11):
        dd = _dims(o, w, T_new=1)
        Kt, Vt = o.empty_cache(dd)
        Kt[:, :, :, :t] = K[:, :, :, :t]
        Vt[:, :, :, :t] = V[:, :, :, :t]
        Ot = o.layer_step(dd, P, H[:, t:t + 1], w.chan_map, np.full(w.B, t), Kt, Vt)
        np.testing.assert_allclose(Ot[:, :, 0], O[:, :, t], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(Kt[:, :, :, t], K[:, :, :, t], rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(Vt[:, :, :, t], V[:, :, :, t], rtol=1e-13, atol=1e-14)


def test_inclusive_mask_is_shift_invariant(oracle_lib):
    """Without the (unrotated) dummy, shifting every position by a constant leaves the
    output unchanged: RoPE scores depend on relative position only."""
    o = oracle_lib
    w = _small(L=3, k=2, T_new=8, B=1, ctx=40)
    rng = np.random.default_rng(13)
    P = synth.make_params(w, rng.normal(size=(2, w.k * w.L)))
    H = synth.make_states(w)
    dm0 = _dims(o, w, T_new=8, mask_mode=o.MASK_INCLUSIVE)
    K0, V0 = o.empty_cache(dm0)
    O0 = o.layer_step(dm0, P, H, w.chan_map, None, K0, V0)
    # same tokens placed at positions 40..47: the context slots are never read because
    # queries are compared through the explicit attention of the shifted copy below
    K1, V1 = o.empty_cache(dm0)
    o.pool(dm0, P, H, [40], K1, V1)
    Q1 = o.q_project(dm0, P, H, [40])
    for l in range(w.L):
        c = w.chan_map[l]
        for t in range(8):
            for h in range(w.Hq):
                kvh = h // (w.Hq // w.Hkv)
                out = o.attend_row(Q1[l, 0, h, t], K1[c, 0, kvh, 40:41 + t],
                                   V1[c, 0, kvh, 40:41 + t])
                np.testing.assert_allclose(out, O0[l, 0, t, h * w.d:(h + 1) * w.d],
                                           rtol=1e-9, atol=1e-11)


# ---------------------------------------------------------- document mask

def _doc_case(o, mask_mode, ctx=0, lengths=None, mean_len=4.0, seed=21):
    w = _small(L=3, k=2, T_new=13, B=2, Hq=4, Hkv=2, d=16, ctx=ctx, seed=seed)
    P = synth.make_params(w, o.init_bias(w.L, w.k))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w, fill=0.0)
    rng = np.random.default_rng(seed)
    Kc = torch.as_tensor(rng.normal(size=Kc.shape))  # every slot finite and distinct
    Vc = torch.as_tensor(rng.normal(size=Vc.shape))
    ctx_len = np.array([ctx, max(ctx - 3, 0)], dtype=np.int32)
    docs = synth.make_doc_start(w, torch.as_tensor(ctx_len), mean_len=mean_len,
                                lengths=lengths).numpy()
    dm = _dims(o, w, mask_mode=mask_mode)
    return w, P, Q, Kc, Vc, ctx_len, docs, dm


@pytest.mark.parametrize("mask_mode", [0, 1])
@pytest.mark.parametrize("ctx", [0, 9])
def test_document_mask_matches_sdpa_with_block_mask(oracle_lib, mask_mode, ctx):
    """Packed documents (Section 4.1): each row against torch SDPA (float64) over the dummy
    slot (paper mask) and the cached slots of its own document before (or at) it."""
    o = oracle_lib
    w, P, Q, Kc, Vc, ctx_len, docs, dm = _doc_case(o, mask_mode, ctx)
    O = o.channel_attend(dm, P, Q, w.chan_map, ctx_len, Kc, Vc, doc_start=docs)
    Qd, Kd, Vd = Q.double(), P["Kd"].double(), P["Vd"].double()
    paper = mask_mode == 0
    for l in range(w.L):
        c = w.chan_map[l]
        for b in range(w.B):
            for i in range(w.T_new):
                pos = int(ctx_len[b]) + i
                for h in range(w.Hq):
                    kv = h // (w.Hq // w.Hkv)
                    K = Kc[c, b, kv].double()
                    V = Vc[c, b, kv].double()
                    mask = torch.zeros(w.S_cap, dtype=torch.bool)
                    mask[docs[b, i]:pos + (0 if paper else 1)] = True
                    if paper:
                        K = torch.cat([Kd[c, kv][None], K])
                        V = torch.cat([Vd[c, kv][None], V])
                        mask = torch.cat([torch.ones(1, dtype=torch.bool), mask])
                    ref = F.scaled_dot_product_attention(Qd[l, b, h, i][None, None], K[None],
                                                         V[None], attn_mask=mask[None, None])
                    np.testing.assert_allclose(O[l, b, i, h * w.d:(h + 1) * w.d],
                                               ref[0, 0].numpy(), rtol=1e-12, atol=1e-13)


def test_document_mask_with_one_document_is_no_mask(oracle_lib):
    o = oracle_lib
    w, P, Q, Kc, Vc, ctx_len, docs, dm = _doc_case(o, 0, ctx=9)
    zero = np.zeros_like(docs)
    np.testing.assert_array_equal(o.channel_attend(dm, P, Q, w.chan_map, ctx_len, Kc, Vc,
                                                   doc_start=zero),
                                  o.channel_attend(dm, P, Q, w.chan_map, ctx_len, Kc, Vc))


@pytest.mark.parametrize("mask_mode", [0, 1])
def test_document_mask_ignores_other_documents(oracle_lib, mask_mode):
    """Changing every cached slot before a row's document leaves the row unchanged, and
    the first token of a document reads only the dummy (paper mask) or only itself."""
    o = oracle_lib
    w, P, Q, Kc, Vc, ctx_len, docs, dm = _doc_case(o, mask_mode, ctx=9, lengths=[5, 1, 7, 2])
    O = o.channel_attend(dm, P, Q, w.chan_map, ctx_len, Kc, Vc, doc_start=docs)
    rng = np.random.default_rng(5)
    for b in range(w.B):
        for i in range(w.T_new):
            K2, V2 = Kc.clone(), Vc.clone()
            lo = int(docs[b, i])
            K2[:, b, :, :lo] = torch.as_tensor(rng.normal(size=K2[:, b, :, :lo].shape))
            V2[:, b, :, :lo] = torch.as_tensor(rng.normal(size=V2[:, b, :, :lo].shape))
            O2 = o.channel_attend(dm, P, Q, w.chan_map, ctx_len, K2, V2, doc_start=docs)
            np.testing.assert_array_equal(O2[:, b, i], O[:, b, i])
            if lo == int(ctx_len[b]) + i:  # first token of its document
                for l in range(w.L):
                    for h in range(w.Hq):
                        kv = h // 2
                        want = (P["Vd"][w.chan_map[l], kv] if mask_mode == 0
                                else Vc[w.chan_map[l], b, kv, lo]).double().numpy()
                        np.testing.assert_allclose(O[l, b, i, h * w.d:(h + 1) * w.d], want,
                                                   rtol=1e-13, atol=1e-14)


# ------------------------------------------- router variants (ablations, Section 5.3)

@pytest.mark.parametrize("mix_mode", [0, 1])
def test_static_router_is_the_bias_whatever_the_weights(oracle_lib, mix_mode):
    """Static mixing weights: alpha = b for every token (before the optional softmax), the
    same as the content-dependent router with W^alpha = 0, bit for bit."""
    o = oracle_lib
    w = _small(L=5, k=3, T_new=6, B=2, p=2)
    rng = np.random.default_rng(41)
    b = rng.normal(size=(2, w.k * w.L))
    P = synth.make_params(w, b, gains="random")          # random W^alpha
    Pz = synth.make_params(w, b, gains="random", zero_router=True)
    H = synth.make_states(w)
    a_s, m_s = o.router_mix(_dims(o, w, mix_mode=mix_mode, router_mode=o.ROUTER_STATIC), P, H)
    a_z, m_z = o.router_mix(_dims(o, w, mix_mode=mix_mode), Pz, H)
    np.testing.assert_array_equal(a_s, a_z)
    np.testing.assert_array_equal(m_s, m_z)


def _nofeedback_case(o, mix_mode, p=1):
    w = _small(L=5, k=5, T_new=4, B=2, p=p)
    rng = np.random.default_rng(42)
    P = synth.make_params(w, rng.normal(size=(2, w.k * w.L)), gains="random")
    P["W_alpha"] = P["W_alpha"] * 20.0   # a router that matters
    H = synth.make_states(w)
    dm = _dims(o, w, mix_mode=mix_mode, router_mode=o.ROUTER_NOFEEDBACK)
    return w, P, H, dm


@pytest.mark.parametrize("mix_mode", [0, 1])
def test_nofeedback_channel_ignores_deeper_layers(oracle_lib, mix_mode):
    """Without deep-to-shallow feedback, channel j (built at layer j) depends on source
    layers 0..j only: changing the states of deeper layers leaves it bit-identical, its
    weights on deeper layers are 0, and in softmax mode its weights on 0..j sum to 1."""
    o = oracle_lib
    w, P, H, dm = _nofeedback_case(o, mix_mode)
    a, m = o.router_mix(dm, P, H)
    for j in range(w.k):
        assert (a[:, :, j, j + 1:] == 0).all()
        if mix_mode == 1:
            np.testing.assert_allclose(a[:, :, j, :j + 1].sum(-1), 1.0, rtol=1e-13)
        H2 = H.clone()
        H2[:, :, j + 1:] = torch.randn(H2[:, :, j + 1:].shape, dtype=H2.dtype)
        a2, m2 = o.router_mix(dm, P, H2)
        np.testing.assert_array_equal(m2[:, j], m[:, j])
        np.testing.assert_array_equal(a2[:, :, j], a[:, :, j])
    # and some channel does change with its own deepest layer
    H3 = H.clone()
    H3[:, :, w.L - 1] = torch.randn(H3[:, :, w.L - 1].shape, dtype=H3.dtype)
    assert not np.array_equal(o.router_mix(dm, P, H3)[1][:, w.k - 1], m[:, w.k - 1])


@pytest.mark.parametrize("p", [1, 2])
def test_nofeedback_equals_router_with_masked_parameters(oracle_lib, p):
    """Linear mode: the no-feedback mix equals the content-dependent one whose router
    weights on deeper source layers, and whose weights and bias for deeper mixing
    coefficients, are zero."""
    o = oracle_lib
    w, P, H, dm = _nofeedback_case(o, 0, p=p)
    sel = o.router_layers(w.L, w.p)
    Wm = P["W_alpha"].double().clone().reshape(2, w.k, w.L, len(sel), w.D)
    bm = P["b_alpha"].double().clone().reshape(2, w.k, w.L)
    for j in range(w.k):
        for m, layer in enumerate(sel):
            if layer > j:
                Wm[:, j, :, m] = 0.0
        Wm[:, j, j + 1:] = 0.0
        bm[:, j, j + 1:] = 0.0
    Pm = dict(P, W_alpha=Wm.reshape(2, w.k * w.L, -1), b_alpha=bm.reshape(2, -1))
    Pm = {k: v.double() for k, v in Pm.items()}
    Pd = {k: v.double() for k, v in P.items()}
    a, m = o.router_mix(dm, Pd, H.double())
    a0, m0 = o.router_mix(_dims(o, w), Pm, H.double())
    np.testing.assert_array_equal(a, a0)
    np.testing.assert_array_equal(m, m0)


# ------------------------------------------------ dense soft read (Section 3.1 Step 3)

def _dense_case(o, mask_mode=0, ctx=30):
    w = _small(B=2, T_new=12, L=5, k=3, Hq=4, Hkv=2, ctx=ctx + 12)
    w = synth.Workload(w.name, w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, w.ctx, "f32",
                       [2, 0, 2, 1, 0], w.p, w.seed)
    P = synth.make_params(w, o.init_bias(w.L, w.k))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w)
    ctx_len = np.array([ctx, ctx // 3], dtype=np.int32)
    return w, P, Q, Kc.double().numpy(), Vc.double().numpy(), ctx_len, _dims(o, w,
                                                                             mask_mode=mask_mode)


@pytest.mark.parametrize("mask_mode", [0, 1])
def test_dense_read_with_one_hot_weights_is_the_fixed_selection(oracle_lib, mask_mode):
    o = oracle_lib
    w, P, Q, Kc, Vc, ctx, dm = _dense_case(o, mask_mode)
    onehot = np.zeros((w.L, w.k))
    onehot[np.arange(w.L), w.chan_map] = 1.0
    Od = o.channel_attend_dense(dm, P, onehot, Q, ctx, Kc, Vc)
    Os = o.channel_attend(dm, P, Q, w.chan_map, ctx, Kc, Vc)
    assert np.array_equal(Od, Os)


def test_dense_read_matches_sdpa_over_mixed_channels(oracle_lib):
    """Soft weights: the mixed keys and values formed with einsum, the dummy slot mixed the
    same way, then torch's scaled_dot_product_attention (float64)."""
    o = oracle_lib
    w, P, Q, Kc, Vc, ctx, dm = _dense_case(o)
    rng = np.random.default_rng(21)
    sw = rng.normal(size=(w.L, w.k))
    sw = np.exp(sw) / np.exp(sw).sum(axis=1, keepdims=True)
    Od = o.channel_attend_dense(dm, P, sw, Q, ctx, Kc, Vc)
    Qn = Q.double().numpy()
    Kd, Vd = P["Kd"].double().numpy(), P["Vd"].double().numpy()
    grp = w.Hq // w.Hkv
    for l in range(w.L):
        Km = np.einsum("c,cbhsd->bhsd", sw[l], Kc)
        Vm = np.einsum("c,cbhsd->bhsd", sw[l], Vc)
        kd, vd = np.einsum("c,chd->hd", sw[l], Kd), np.einsum("c,chd->hd", sw[l], Vd)
        for b in range(w.B):
            for i in range(w.T_new):
                pos = int(ctx[b]) + i
                for h in range(w.Hq):
                    kv = h // grp
                    K = np.vstack([kd[kv], Km[b, kv, :pos]])
                    V = np.vstack([vd[kv], Vm[b, kv, :pos]])
                    ref = F.scaled_dot_product_attention(_t(Qn[l, b, h, i])[None, None],
                                                         _t(K)[None], _t(V)[None])[0, 0]
                    np.testing.assert_allclose(Od[l, b, i, h * w.d:(h + 1) * w.d], ref.numpy(),
                                               rtol=1e-11, atol=1e-12)


def test_dense_read_splitting_a_weight_over_equal_channels(oracle_lib):
    """Two channels holding the same cache and dummy: weights 0.3 / 0.7 on them read the
    same as 1.0 on one."""
    o = oracle_lib
    w, P, Q, Kc, Vc, ctx, dm = _dense_case(o)
    Kc[1], Vc[1] = Kc[0], Vc[0]
    P = dict(P)
    P["Kd"] = P["Kd"].clone()
    P["Vd"] = P["Vd"].clone()
    P["Kd"][1], P["Vd"][1] = P["Kd"][0], P["Vd"][0]
    split = np.zeros((w.L, w.k))
    split[:, 0], split[:, 1] = 0.3, 0.7
    one = np.zeros((w.L, w.k))
    one[:, 0] = 1.0
    np.testing.assert_allclose(o.channel_attend_dense(dm, P, split, Q, ctx, Kc, Vc),
                               o.channel_attend_dense(dm, P, one, Q, ctx, Kc, Vc),
                               rtol=1e-12, atol=1e-12)
