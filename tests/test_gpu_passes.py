"""GPU parity for strided token groups and the fixed-point pass driver (Section 3.3).

Group calls (dims.groups = g, dims.group = q) place the call's token i of sequence b
at position ctx_len[b] + q + g i: the pool writes those slots and the queries attend
from those positions. The oracle states the same thing at full positions: a sequence
of S_cap positions whose listed tokens are pooled and whose listed rows attend.

The pass driver runs cyclic Gauss-Seidel passes (g = 1: Jacobi) with the stand-in
decoder block h_{l+1} = h_l + W_o[l] o_l; it is compared with the oracle's driver,
whose schedules are pinned on the CPU (tests/test_oracle_passes.py).
"""
import numpy as np
import pytest
import torch

import oracle
from tests import synth
from tests.parity import _bias, _dev, _f64, _gdims, _odims, check_close, wm  # noqa: F401

pytestmark = pytest.mark.gpu


def _group_positions(w, ctx, g, q):
    return [[int(ctx[b]) + q + g * i for i in range(w.T_new)] for b in range(w.B)]


def _full_case(w, S):
    """The same problem stated at full positions 0 .. S-1 for the oracle."""
    return synth.Workload(w.name, w.B, S, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, 0, w.dtype,
                          w.chan_map, w.p, w.seed)


GROUP_CASES = [  # (name, workload, g, q)
    ("bf16_d64_prefill", synth.small("grp_bf16", B=2, T_new=40, L=4, k=2, D=128, Hq=2, Hkv=2,
                                     d=64, ctx=20), 4, 3),
    ("bf16_d96_decode", synth.small("grp_d96", B=2, T_new=3, L=4, k=3, D=192, Hq=6, Hkv=3, d=96,
                                    p=2, ctx=300), 8, 5),
    ("f32_d32_prefill", synth.small("grp_f32", B=2, T_new=33, L=3, k=2, D=64, Hq=2, Hkv=1, d=32,
                                    ctx=10, dtype="f32"), 3, 1),
    ("bf16_d64_one_per_seq", synth.small("grp_one", B=3, T_new=1, L=3, k=2, D=64, Hq=2, Hkv=2,
                                         d=64, ctx=70), 64, 63),
]


@pytest.mark.parametrize("name,w,g,q", GROUP_CASES)
@pytest.mark.parametrize("mask_mode", [0, 1])
def test_layer_step_on_a_token_group(wm, name, w, g, q, mask_mode):
    """wm_layer_step on the strided group q of g: cache slots, untouched slots and every
    consumer's output against the oracle at full positions."""
    print("group case", name, g, q, mask_mode, flush=True)
    ctx = np.array([w.ctx, w.ctx // 2, 0][:w.B], dtype=np.int32)
    S = w.ctx + q + g * (w.T_new - 1) + 1
    S_cap = (S + 63) // 64 * 64
    P = synth.make_params(w, _bias(w) + 0.1)
    Hg = synth.make_states(w)
    wf = _full_case(w, S_cap)
    K0, V0 = synth.make_cache_cpu(synth.Workload(w.name, w.B, 1, w.L, w.k, w.D, w.Hq, w.Hkv, w.d,
                                                 S_cap - 1, w.dtype, w.chan_map, w.p, w.seed))
    pos = _group_positions(w, ctx, g, q)
    # the oracle: states placed at their positions, listed tokens pooled, listed rows attend
    Hf = np.zeros((w.B, S_cap, w.L, w.D))
    for b in range(w.B):
        Hf[b, pos[b]] = _f64(Hg[b])
    dm = _odims(wf, S_cap=S_cap, mask_mode=mask_mode)
    toks = [b * S_cap + p for b in range(w.B) for p in pos[b]]
    Ko, Vo = _f64(K0).copy(), _f64(V0).copy()
    PP = oracle.Params(P)
    oracle.pool(dm, PP, Hf, None, Ko, Vo, toks)
    Qf = oracle.q_project(dm, PP, Hf, None, toks)
    rows = [(l * w.B + b) * S_cap + p for l in range(w.L) for b in range(w.B) for p in pos[b]]
    Of = oracle.channel_attend(dm, PP, Qf, w.chan_map, None, Ko, Vo, rows)
    Oo = np.stack([Of[:, b, pos[b]] for b in range(w.B)], axis=1)
    # the library: one call on the group
    dims = _gdims(wm, w, S_cap=S_cap, ctx_max=w.ctx, mask_mode=mask_mode, groups=g, group=q)
    Kg, Vg = K0.cuda(), V0.cuda()
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.layer_step(dims, _dev(P), Hg.cuda(), w.chan_map, torch.from_numpy(ctx).cuda(), Kg, Vg, O)
    torch.cuda.synchronize()
    written = np.zeros((w.B, S_cap), dtype=bool)
    for b in range(w.B):
        written[b, pos[b]] = True
    for G, Oref, G0, tag in ((Kg, Ko, K0, "K"), (Vg, Vo, V0, "V")):
        got = _f64(G)
        m = np.broadcast_to(written[None, :, None, :, None], got.shape)
        check_close(got[m], Oref[m], w.dtype, "%s %s written slots" % (name, tag))
        g0 = _f64(G0)
        same = ~m & ~np.isnan(g0)
        assert (got[same] == g0[same]).all(), "%s: a slot outside the group changed" % tag
        assert (np.isnan(got) == (np.isnan(g0) & ~m)).all(), "%s: write set differs" % tag
    check_close(O, Oo, w.dtype, "%s O" % name)


@pytest.mark.parametrize("name,w,g,q", GROUP_CASES[:3])
def test_pool_and_layer_attend_on_a_token_group(wm, name, w, g, q):
    """wm_pool (Steps 1-2 fused) and wm_layer_attend (one consumer) on a token group: the
    pool's cache rows and each consumer's output, against the oracle."""
    ctx = np.array([w.ctx, w.ctx // 2][:w.B], dtype=np.int32)
    S = w.ctx + q + g * (w.T_new - 1) + 1
    S_cap = (S + 63) // 64 * 64
    P = synth.make_params(w, _bias(w) + 0.1, gains="random")
    Hg = synth.make_states(w)
    wf = _full_case(w, S_cap)
    K0, V0 = synth.make_cache_cpu(synth.Workload(w.name, w.B, 1, w.L, w.k, w.D, w.Hq, w.Hkv, w.d,
                                                 S_cap - 1, w.dtype, w.chan_map, w.p, w.seed))
    pos = _group_positions(w, ctx, g, q)
    Hf = np.zeros((w.B, S_cap, w.L, w.D))
    for b in range(w.B):
        Hf[b, pos[b]] = _f64(Hg[b])
    dm = _odims(wf, S_cap=S_cap)
    toks = [b * S_cap + p for b in range(w.B) for p in pos[b]]
    Ko, Vo = _f64(K0).copy(), _f64(V0).copy()
    PP = oracle.Params(P)
    oracle.pool(dm, PP, Hf, None, Ko, Vo, toks)
    dims = _gdims(wm, w, S_cap=S_cap, ctx_max=w.ctx, groups=g, group=q)
    Pd = wm.ParamSet(_dev(P))
    Kg, Vg = K0.cuda(), V0.cuda()
    ctx_d = torch.from_numpy(ctx).cuda()
    wm.pool(dims, Pd, Hg.cuda(), ctx_d, Kg, Vg)
    torch.cuda.synchronize()
    m = np.zeros((w.B, S_cap), dtype=bool)
    for b in range(w.B):
        m[b, pos[b]] = True
    mm = np.broadcast_to(m[None, :, None, :, None], Ko.shape)
    check_close(_f64(Kg)[mm], Ko[mm], w.dtype, "%s pool K" % name)
    check_close(_f64(Vg)[mm], Vo[mm], w.dtype, "%s pool V" % name)
    Qf = oracle.q_project(dm, PP, Hf, None, toks)
    Hd = Hg.cuda()
    for l in range(w.L):
        rows = [(l * w.B + b) * S_cap + p for b in range(w.B) for p in pos[b]]
        Of = oracle.channel_attend(dm, PP, Qf, w.chan_map, None, Ko, Vo, rows)
        Oo = np.stack([Of[l, b, pos[b]] for b in range(w.B)], axis=0)
        Ol = torch.empty((w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
        wm.layer_attend(dims, Pd, l, Hd, w.chan_map, ctx_d, Kg, Vg, Ol)
        torch.cuda.synchronize()
        check_close(Ol, Oo, w.dtype, "%s layer %d O" % (name, l))


PASS_CASES = {
    "bf16_d64": synth.small("pass_bf16", B=2, T_new=32, L=4, k=2, D=128, Hq=2, Hkv=2, d=64,
                            seed=311),
    "bf16_d96_gqa_p2": synth.small("pass_d96", B=1, T_new=24, L=4, k=3, D=192, Hq=6, Hkv=3,
                                   d=96, p=2, seed=312),
    "f32_d32": synth.small("pass_f32", B=2, T_new=24, L=3, k=2, D=64, Hq=2, Hkv=1, d=32,
                           dtype="f32", seed=313),
}


def _run_passes(wm, w, g, passes, mask_mode=0, seqs=None, mix_mode=0):
    """The library's driver and the oracle's on the same inputs; the oracle runs the listed
    sequences only (all by default)."""
    P = synth.make_params(w, _bias(w) + 0.2)
    X = synth.make_embeddings(w)
    W_o = synth.make_out_proj(w)
    S_cap = (w.T_new + 63) // 64 * 64
    dims = _gdims(wm, w, S_cap=S_cap, ctx_max=0, groups=g, mask_mode=mask_mode,
                  mix_mode=mix_mode)
    Kg = torch.full((w.k, w.B, w.Hkv, S_cap, w.d), float("nan"), dtype=w.torch_dtype,
                    device="cuda")
    Vg = torch.full_like(Kg, float("nan"))
    H = torch.empty((w.B, w.T_new, w.L, w.D), dtype=w.torch_dtype, device="cuda")
    top = torch.empty((w.B, w.T_new, w.D), dtype=w.torch_dtype, device="cuda")
    wm.prefill_passes(dims, _dev(P), W_o.cuda(), X.cuda(), w.chan_map, passes, Kg, Vg, H, top)
    torch.cuda.synchronize()
    seqs = list(range(w.B)) if seqs is None else seqs
    res = []
    PP = oracle.Params(P)
    for b in seqs:
        dm = oracle.Dims(B=1, T_new=w.T_new, L=w.L, k=w.k, D=w.D, Hq=w.Hq, Hkv=w.Hkv, d=w.d,
                         p=w.p, S_cap=S_cap, mask_mode=mask_mode, mix_mode=mix_mode)
        Ho, to, Ko, Vo = oracle.gauss_seidel(dm, PP, W_o, w.chan_map, X[b:b + 1], g, passes)
        res.append((b, (Ho, to, Ko, Vo, _cache_slack(w, dm, PP, Ho, Ko, Vo))))
    return (H, top, Kg, Vg), res


def _cache_slack(w, dm, PP, Ho, Ko, Vo):
    """Per cache row, twice how far the oracle's own pool moves when the states it pools are
    rounded to the workload dtype (the library stores them so). The signed mix of nearly
    equal residual-stream states can cancel to a small channel, which the mid RMSNorm then
    scales up together with any rounding of those states."""
    if w.dtype != "bf16":
        return None, None
    Hr = torch.from_numpy(Ho).to(torch.bfloat16).double().numpy()
    K2, V2 = oracle.empty_cache(dm)
    oracle.pool(dm, PP, Hr, None, K2, V2)
    out = []
    for A, B in ((K2, Ko), (V2, Vo)):
        dev = np.abs(A - B)[:, :, :, :w.T_new]
        out.append(2.0 * np.broadcast_to(dev.max(axis=-1, keepdims=True), dev.shape))
    return tuple(out)


@pytest.mark.parametrize("name", list(PASS_CASES))
@pytest.mark.parametrize("g_kind,passes", [("1", 2), ("4", 2), ("T", 1), ("8", 3)])
def test_prefill_passes_small(wm, name, g_kind, passes):
    """Jacobi (g = 1), cyclic Gauss-Seidel (g = 4, 8) and g = T (one pass: exact
    left-to-right evaluation) against the oracle's driver: every state, top state and
    cache slot."""
    w = PASS_CASES[name]
    g = w.T_new if g_kind == "T" else int(g_kind)
    print("passes", name, "g", g, "passes", passes, flush=True)
    (H, top, Kg, Vg), res = _run_passes(wm, w, g, passes)
    for b, (Ho, to, Ko, Vo, (ks, vs)) in res:
        check_close(H[b:b + 1], Ho, w.dtype, "%s g%d H b=%d" % (name, g, b))
        check_close(top[b:b + 1], to, w.dtype, "%s g%d top b=%d" % (name, g, b))
        check_close(Kg[:, b:b + 1, :, :w.T_new], Ko[:, :, :, :w.T_new], w.dtype,
                    "%s g%d K b=%d" % (name, g, b), slack=ks)
        check_close(Vg[:, b:b + 1, :, :w.T_new], Vo[:, :, :, :w.T_new], w.dtype,
                    "%s g%d V b=%d" % (name, g, b), slack=vs)
    assert torch.isnan(Kg[:, :, :, w.T_new:]).all()


def test_prefill_passes_inclusive_mask(wm):
    """The iterations are also defined with the inclusive mask (a position then reads its
    own slot from the cache as it stands)."""
    w = PASS_CASES["bf16_d64"]
    (H, top, Kg, Vg), res = _run_passes(wm, w, 4, 2, mask_mode=1)
    for b, (Ho, to, Ko, Vo, _) in res:
        check_close(H[b:b + 1], Ho, w.dtype, "inclusive H b=%d" % b)
        check_close(top[b:b + 1], to, w.dtype, "inclusive top b=%d" % b)


def _mix_condition(w, dm, PP, Ho):
    """Per (branch, channel, token): how much the signed mix cancels, kappa =
    sum_l |alpha_jl| |h^_l| / |h~_j| (the factor by which it magnifies relative errors of
    the states it mixes), from the oracle's mixing weights and mixed channels."""
    alpha, mixed = oracle.router_mix(dm, PP, Ho)       # [2, N, k, L], [2, k, N, D]
    Hn = Ho.reshape(-1, w.L, w.D)
    g = PP.arrays["g_pre"]                               # [2, L, D]
    kap = np.zeros((2, w.k, Hn.shape[0]))
    for br in range(2):
        hn = Hn / np.sqrt(np.mean(Hn * Hn, axis=-1, keepdims=True) + 1e-6) * g[br][None]
        norms = np.linalg.norm(hn, axis=-1)              # [N, L]
        num = np.einsum("nkl,nl->kn", np.abs(alpha[br]), norms)
        kap[br] = num / np.maximum(np.linalg.norm(mixed[br], axis=-1), 1e-300)
    return kap


@pytest.mark.parametrize("mix_mode,passes", [(1, 3), (0, 2)])
def test_prefill_passes_paper_shape(wm, mix_mode, passes):
    """The paper's model shape (L 16, D 512, 6 query / 3 KV heads of 96, p = 2, k = 8,
    T = 2048, 16 sequences) with its training schedule of g = 8 groups; two sequences
    re-computed by the oracle's driver. The paper's signed linear mix of the nearly equal
    states of a residual stream can cancel: a channel whose mix magnifies relative errors
    of the states by kappa (sum_l |alpha_jl| |h^_l| / |h~_j|, from the oracle) carries the
    bf16 rounding of those states (2^-8 relative) times kappa into its cache rows, and
    twice that is allowed per row. With the softmax mix every channel is a convex
    combination (kappa = 1)."""
    w0 = synth.WORKLOADS["paper_T2048_L16_k8"]
    w = synth.Workload("paper_passes", w0.B, w0.T_new, w0.L, w0.k, w0.D, w0.Hq, w0.Hkv, w0.d,
                       0, w0.dtype, list(w0.chan_map), w0.p, w0.seed)
    print("passes paper shape, mix mode", mix_mode, flush=True)
    (H, top, Kg, Vg), res = _run_passes(wm, w, 8, passes, seqs=[0, w.B - 1], mix_mode=mix_mode)
    P = oracle.Params(synth.make_params(w, _bias(w) + 0.2))
    for b, (Ho, to, Ko, Vo, _) in res:
        check_close(H[b:b + 1], Ho, w.dtype, "paper g8 mix%d H b=%d" % (mix_mode, b))
        check_close(top[b:b + 1], to, w.dtype, "paper g8 mix%d top b=%d" % (mix_mode, b))
        dm = oracle.Dims(B=1, T_new=w.T_new, L=w.L, k=w.k, D=w.D, Hq=w.Hq, Hkv=w.Hkv, d=w.d,
                         p=w.p, S_cap=w.T_new, mix_mode=mix_mode)
        kap = _mix_condition(w, dm, P, Ho)               # [2, k, T]
        for br, (G, Ref) in enumerate(((Kg, Ko), (Vg, Vo))):
            rowmax = np.abs(Ref).max(axis=(1, 2, 4))     # [k, T]
            slack = (2.0 * kap[br] * 2.0 ** -8 * rowmax)[:, None, None, :, None]
            print("paper g8 mix%d %s b=%d: kappa median %.2f, 99th pct %.1f, max %.1f"
                  % (mix_mode, "KV"[br], b, np.median(kap[br]), np.percentile(kap[br], 99),
                     kap[br].max()))
            check_close(G[:, b:b + 1], Ref, w.dtype, "paper g8 mix%d %s b=%d"
                        % (mix_mode, "KV"[br], b), slack=np.broadcast_to(slack, Ref.shape))
