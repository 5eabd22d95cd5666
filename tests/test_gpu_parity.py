"""GPU parity: the HIP library (through its C ABI) against the fp64 CPU oracle.

Tolerances (stated in the workloads' terms): fp32 max |gpu - ref| <= 1e-5;
bf16 max |gpu - ref| / max |ref| <= 2e-2 per output tensor and, per element,
|gpu - ref| <= 2e-2 |ref| + 2e-2 rms(ref) for all but at most 0.1% of the elements
(tests/parity.py). Integer work (which slots are written,
the channel each consumer reads) must match exactly: caches start as NaN
sentinels and the set of slots the kernels wrote must equal the oracle's.
"""
import numpy as np
import pytest
import torch

import oracle
from tests import synth
from tests.parity import (TOL_BF16_REL, TOL_F32_ABS, _bias, _check_cache, _dev, _f64,  # noqa: F401
                          _gdims, _odims, _written_mask, check_close, wm)

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------- small cases

SMALL = {
    "c1_tiny_f32": synth.WORKLOADS["c1_tiny_f32"],
    "bf16_ragged_gqa": synth.small("bf16_ragged_gqa"),
    "bf16_d64_k1": synth.small("bf16_d64_k1", B=1, T_new=97, L=3, k=1, D=128, Hq=2, Hkv=1, d=64),
    "f32_d64_kL": synth.small("f32_d64_kL", B=2, T_new=70, L=4, k=4, D=64, Hq=2, Hkv=2, d=64,
                              dtype="f32"),
    "bf16_long_T300": synth.small("bf16_long_T300", B=1, T_new=300, L=2, k=2, D=64, Hq=2, Hkv=1,
                                  d=64),
    # head dim 96 with grouped queries and router subsampling (the paper's head layout)
    "bf16_d96_gqa_p2": synth.small("bf16_d96_gqa_p2", B=2, T_new=150, L=6, k=4, D=192, Hq=6,
                                   Hkv=3, d=96, p=2),
    "bf16_paper_shape": synth.small("bf16_paper_shape", B=1, T_new=70, L=16, k=8, D=512, Hq=6,
                                    Hkv=3, d=96, p=2),
}


def _layer_step_case(wm, w, mix_mode=0, mask_mode=0, gains="unit", ragged=False, p=None,
                     f32_scale=1.0):
    if p is not None:
        w = synth.Workload(w.name, w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, w.ctx, w.dtype,
                           w.chan_map, p, w.seed)
    print("case", w.name, "mix", mix_mode, "mask", mask_mode, "gains", gains, "ragged", ragged,
          "p", w.p, flush=True)
    rng = np.random.default_rng(w.seed)
    bias = _bias(w) + rng.normal(0, 0.3, size=w.k * w.L)
    P = synth.make_params(w, bias, gains=gains)
    H = synth.make_states(w)
    ctx = synth.make_ctx_len(w, ragged=ragged)
    K0, V0 = synth.make_cache_cpu(w)

    Ko, Vo = _f64(K0).copy(), _f64(V0).copy()
    Oo = oracle.layer_step(_odims(w, mix_mode=mix_mode, mask_mode=mask_mode), P, H, w.chan_map,
                           ctx.numpy(), Ko, Vo)

    dims = _gdims(wm, w, mix_mode=mix_mode, mask_mode=mask_mode)
    Kg, Vg = K0.cuda(), V0.cuda()
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.layer_step(dims, _dev(P), H.cuda(), w.chan_map, ctx.cuda(), Kg, Vg, O)
    torch.cuda.synchronize()
    _check_cache(Kg, Ko, K0, w, ctx.numpy(), w.dtype, w.name + " K", f32_scale)
    _check_cache(Vg, Vo, V0, w, ctx.numpy(), w.dtype, w.name + " V", f32_scale)
    check_close(O, Oo, w.dtype, w.name + " O", f32_scale=f32_scale)
    return O


@pytest.mark.parametrize("name", list(SMALL))
def test_layer_step_small(wm, name):
    _layer_step_case(wm, SMALL[name])


@pytest.mark.parametrize("mix_mode,mask_mode,gains", [(1, 0, "unit"), (0, 1, "random"),
                                                      (1, 1, "random"), (0, 0, "random")])
def test_layer_step_modes(wm, mix_mode, mask_mode, gains):
    _layer_step_case(wm, SMALL["bf16_ragged_gqa"], mix_mode, mask_mode, gains)
    _layer_step_case(wm, SMALL["c1_tiny_f32"], mix_mode, mask_mode, gains)


LIMITS = {
    # the most layers (L = k = 64: 4096 router rows over 4096 stacked columns)
    "L64_k64": synth.small("L64_k64", B=1, T_new=40, L=64, k=64, D=64, Hq=2, Hkv=1, d=32),
    # the most layers sharing one channel, router reading the top layer only (p = L)
    "L64_k1_p64": synth.small("L64_k1_p64", B=1, T_new=40, L=64, k=1, D=64, Hq=2, Hkv=1, d=32,
                              p=64),
    # the mix's LDS limit (a token's L states and its coefficients in 64 KiB): the most
    # layers at D = 1024, bf16 and fp32
    "L31_D1024_bf16": synth.small("L31_D1024_bf16", B=1, T_new=20, L=31, k=4, D=1024, Hq=4,
                                  Hkv=4, d=64),
    "L15_D1024_f32": synth.small("L15_D1024_f32", B=1, T_new=20, L=15, k=2, D=1024, Hq=4,
                                 Hkv=2, d=32, dtype="f32"),
    # wide states: the row norms' 8-chunk-per-lane variant (D = 2560) and their loop over
    # any width (D = 4608)
    "D2560_bf16": synth.small("D2560_bf16", B=1, T_new=20, L=3, k=2, D=2560, Hq=2, Hkv=1,
                              d=64),
    "D4608_bf16": synth.small("D4608_bf16", B=1, T_new=12, L=2, k=2, D=4608, Hq=2, Hkv=1,
                              d=32),
    "D4608_f32": synth.small("D4608_f32", B=1, T_new=12, L=2, k=2, D=4608, Hq=2, Hkv=1,
                             d=32, dtype="f32"),
    # a single new token with nothing cached: it reads only the dummy (or only itself)
    "first_token": synth.small("first_token", B=3, T_new=1, L=3, k=2, D=64, Hq=2, Hkv=2,
                               d=64),
}


@pytest.mark.parametrize("name", list(LIMITS))
@pytest.mark.parametrize("mask_mode", [0, 1])
def test_layer_step_limits(wm, name, mask_mode):
    """The largest supported layer counts and widths and the smallest step. fp32 rounding in
    a D-long projection sum grows like sqrt(D): the fp32 bound, stated for D <= 1024, is
    scaled by sqrt(D / 1024) past that width."""
    w = LIMITS[name]
    f32_scale = max(1.0, float(np.sqrt(w.D / 1024.0))) if w.dtype == "f32" else 1.0
    _layer_step_case(wm, w, mask_mode=mask_mode, f32_scale=f32_scale)


@pytest.mark.parametrize("p", [2, 3])
def test_layer_step_router_subsampling(wm, p):
    _layer_step_case(wm, SMALL["bf16_ragged_gqa"], p=p)
    _layer_step_case(wm, SMALL["c1_tiny_f32"], p=p)


@pytest.mark.parametrize("T_new", [1, 2, 4, 5, 33])
@pytest.mark.parametrize("mask_mode", [0, 1])
def test_layer_step_with_context(wm, T_new, mask_mode):
    """Decode (T_new <= 4, split-S kernels) and chunked prefill (T_new > 4) over a cached
    context of ragged length per sequence."""
    for dtype in ("bf16", "f32"):
        w = synth.small("ctx_%s_T%d" % (dtype, T_new), B=3, T_new=T_new, L=5, k=2, D=64, Hq=4,
                        Hkv=2, d=32 if dtype == "f32" else 64, ctx=700, dtype=dtype)
        _layer_step_case(wm, w, mask_mode=mask_mode, ragged=True)


@pytest.mark.parametrize("T_new", [1, 3, 33])
@pytest.mark.parametrize("mask_mode", [0, 1])
def test_layer_step_with_context_d96(wm, T_new, mask_mode):
    """Head dim 96: decode (12 of 16 lanes per slot group) and chunked prefill over a
    ragged cached context."""
    w = synth.small("ctx_d96_T%d" % T_new, B=3, T_new=T_new, L=6, k=3, D=192, Hq=6, Hkv=3,
                    d=96, ctx=700, p=2)
    _layer_step_case(wm, w, mask_mode=mask_mode, ragged=True)


def test_layer_step_is_deterministic(wm):
    w = SMALL["bf16_ragged_gqa"]
    a = _layer_step_case(wm, w)
    b = _layer_step_case(wm, w)
    assert torch.equal(a, b)


def test_empty_call_is_a_no_op(wm):
    w = synth.small("empty", B=0)
    dims = _gdims(wm, w)
    P = _dev(synth.make_params(synth.small(), _bias(synth.small())))
    wm.layer_step(dims, P, None, w.chan_map, None, None, None, None)


# --------------------------------------------------------------- single ops

@pytest.mark.parametrize("name", ["c1_tiny_f32", "bf16_ragged_gqa"])
@pytest.mark.parametrize("mix_mode", [0, 1])
def test_router_mix(wm, name, mix_mode):
    w = SMALL[name]
    rng = np.random.default_rng(3)
    P = synth.make_params(w, rng.normal(0, 1, size=(2, w.k * w.L)), gains="random")
    H = synth.make_states(w)
    ao, mo = oracle.router_mix(_odims(w, mix_mode=mix_mode), P, H)
    dims = _gdims(wm, w, mix_mode=mix_mode)
    alpha = torch.empty((2, w.N, w.k, w.L), dtype=torch.float32, device="cuda")
    mixed = torch.empty((2, w.k, w.N, w.D), dtype=w.torch_dtype, device="cuda")
    wm.router_mix(dims, _dev(P), H.cuda(), mixed, alpha)
    torch.cuda.synchronize()
    check_close(alpha, ao, w.dtype, name + " alpha")
    check_close(mixed, mo, w.dtype, name + " mixed")
    if mix_mode == 1:
        s = alpha.sum(-1)
        assert torch.allclose(s, torch.ones_like(s), atol=1e-5) and (alpha > 0).all()


@pytest.mark.parametrize("L,k,p,T_new", [(16, 4, 1, 200), (24, 3, 1, 70), (20, 8, 1, 300)])
def test_router_mix_long_k(wm, L, k, p, T_new):
    """The router's long-K path (stacked states of at least 16384 elements: the 12-wave block
    with K split at layer boundaries and the partial sums reduced), every weight and mixed
    channel against the oracle, ragged token tiles."""
    w = synth.small("router_long_L%d" % L, B=2, T_new=T_new, L=L, k=k, D=1024, Hq=4, Hkv=2,
                    d=64, dtype="bf16", p=p)
    assert (L + p - 1) // p * w.D >= 16384 and w.N > 64
    print("router long K: L%d k%d p%d N%d" % (L, k, p, w.N), flush=True)
    rng = np.random.default_rng(5)
    P = synth.make_params(w, rng.normal(0, 1, size=(2, w.k * w.L)), gains="random")
    H = synth.make_states(w)
    ao, mo = oracle.router_mix(_odims(w), P, H)
    dims = _gdims(wm, w)
    alpha = torch.empty((2, w.N, w.k, w.L), dtype=torch.float32, device="cuda")
    mixed = torch.empty((2, w.k, w.N, w.D), dtype=w.torch_dtype, device="cuda")
    wm.router_mix(dims, _dev(P), H.cuda(), mixed, alpha)
    torch.cuda.synchronize()
    check_close(alpha, ao, "bf16", "long-K alpha")
    check_close(mixed, mo, "bf16", "long-K mixed")


def test_router_zero_weights_give_bias_exactly(wm):
    """W_alpha = 0: the mixing weights are the bias, exactly (fp32 and bf16)."""
    for name in ("c1_tiny_f32", "bf16_ragged_gqa"):
        w = SMALL[name]
        P = synth.make_params(w, _bias(w), zero_router=True)
        dims = _gdims(wm, w)
        alpha = torch.empty((2, w.N, w.k, w.L), dtype=torch.float32, device="cuda")
        mixed = torch.empty((2, w.k, w.N, w.D), dtype=w.torch_dtype, device="cuda")
        wm.router_mix(dims, _dev(P), synth.make_states(w).cuda(), mixed, alpha)
        torch.cuda.synchronize()
        want = P["b_alpha"].float().reshape(2, 1, w.k, w.L).expand(2, w.N, w.k, w.L)
        assert torch.equal(alpha.cpu(), want)


@pytest.mark.parametrize("name", ["c1_tiny_f32", "bf16_ragged_gqa", "f32_d64_kL",
                                  "bf16_d96_gqa_p2"])
def test_kv_project(wm, name):
    w = SMALL[name]
    w = synth.Workload(w.name, w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, 50, w.dtype,
                       w.chan_map, w.p, w.seed)
    P = synth.make_params(w, _bias(w), gains="random")
    mixed = synth.make_mixed(w)
    ctx = synth.make_ctx_len(w, ragged=True)
    K0, V0 = synth.make_cache_cpu(w)
    Ko, Vo = _f64(K0).copy(), _f64(V0).copy()
    oracle.kv_project(_odims(w), P, mixed, ctx.numpy(), Ko, Vo)
    Kg, Vg = K0.cuda(), V0.cuda()
    wm.kv_project(_gdims(wm, w), _dev(P), mixed.cuda(), ctx.cuda(), Kg, Vg)
    torch.cuda.synchronize()
    _check_cache(Kg, Ko, K0, w, ctx.numpy(), w.dtype, name + " K")
    _check_cache(Vg, Vo, V0, w, ctx.numpy(), w.dtype, name + " V")


@pytest.mark.parametrize("name", ["c1_tiny_f32", "bf16_ragged_gqa", "bf16_d64_k1",
                                  "bf16_d96_gqa_p2"])
def test_q_project(wm, name):
    w = SMALL[name]
    P = synth.make_params(w, _bias(w), gains="random")
    H = synth.make_states(w)
    ctx = torch.arange(w.B, dtype=torch.int32) * 37
    Qo = oracle.q_project(_odims(w), P, H, ctx.numpy())
    Q = torch.empty((w.L, w.B, w.Hq, w.T_new, w.d), dtype=w.torch_dtype, device="cuda")
    wm.q_project(_gdims(wm, w, S_cap=0, ctx_max=0), _dev(P), H.cuda(), ctx.cuda(), Q)
    torch.cuda.synchronize()
    check_close(Q, Qo, w.dtype, name + " Q")


@pytest.mark.parametrize("T_new,ctx", [(64, 0), (300, 0), (40, 200), (1, 1000), (3, 513)])
@pytest.mark.parametrize("mask_mode", [0, 1])
def test_channel_attend(wm, T_new, ctx, mask_mode):
    """Attention alone on seeded queries and a seeded cache, with a channel map where
    several consumers share a channel (and one channel has none)."""
    for dtype, d in (("bf16", 64), ("f32", 32), ("bf16", 96)):
        w = synth.small("attn_%s" % dtype, B=2, T_new=T_new, L=5, k=3, D=64, Hq=4, Hkv=2, d=d,
                        ctx=ctx + T_new, dtype=dtype, chan_map=[2, 0, 2, 2, 0])
        P = synth.make_params(w, _bias(w))
        Q = synth.make_queries(w)
        Kc, Vc = synth.make_cache_cpu(w)
        ctx_len = torch.tensor([ctx, ctx // 2], dtype=torch.int32)
        Oo = oracle.channel_attend(_odims(w, mask_mode=mask_mode), P, Q, w.chan_map,
                                   ctx_len.numpy(), _f64(Kc), _f64(Vc))
        O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
        dims = _gdims(wm, w, mask_mode=mask_mode, ctx_max=ctx)
        wm.channel_attend(dims, _dev(P), Q.cuda(), w.chan_map, ctx_len.cuda(), Kc.cuda(),
                          Vc.cuda(), O)
        torch.cuda.synchronize()
        check_close(O, Oo, dtype, "attend %s d%d T%d ctx%d" % (dtype, d, T_new, ctx))


@pytest.mark.parametrize("d,L,Hq,Hkv,mask_mode,docs", [(64, 12, 16, 4, 0, False),
                                                       (64, 12, 16, 4, 1, True),
                                                       (96, 16, 6, 3, 0, False),
                                                       (96, 16, 6, 3, 0, True)])
def test_channel_attend_work_queue(wm, d, L, Hq, Hkv, mask_mode, docs):
    """More query tiles (128 queries of one consumer, sequence and head) than the CUs hold at
    once, so the bf16 kernels run persistent workgroups that take tiles from the work queue;
    every output element against the oracle, with a ragged last tile and cached context."""
    T_new, ctx = 300, 40
    w = synth.small("queue_d%d" % d, B=2, T_new=T_new, L=L, k=4, D=64, Hq=Hq, Hkv=Hkv, d=d,
                    ctx=ctx + T_new, dtype="bf16", chan_map=[l % 4 for l in range(L)])
    tiles = (T_new + 127) // 128 * Hq * w.B * L
    resident = torch.cuda.get_device_properties(0).multi_processor_count * (3 if d == 64 else 2)
    assert tiles > resident, (tiles, resident)
    print("queue case d%d tiles %d resident %d mask %d docs %s" % (d, tiles, resident, mask_mode,
                                                                   docs), flush=True)
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w)
    ctx_len = torch.tensor([ctx, ctx // 2], dtype=torch.int32)
    doc = synth.make_doc_start(w, ctx_len, mean_len=37.0) if docs else None
    Oo = oracle.channel_attend(_odims(w, mask_mode=mask_mode), P, Q, w.chan_map, ctx_len.numpy(),
                               _f64(Kc), _f64(Vc),
                               doc_start=doc.numpy() if docs else None)
    O = torch.full((w.L, w.B, w.T_new, w.Hq * w.d), float("nan"), dtype=w.torch_dtype,
                   device="cuda")
    dims = _gdims(wm, w, mask_mode=mask_mode, ctx_max=ctx)
    wm.channel_attend(dims, _dev(P), Q.cuda(), w.chan_map, ctx_len.cuda(), Kc.cuda(), Vc.cuda(),
                      O, doc_start=doc.cuda() if docs else None)
    torch.cuda.synchronize()
    assert not torch.isnan(O.float()).any(), "a query tile was never computed"
    check_close(O, Oo, "bf16", "queue d%d mask%d docs%d" % (d, mask_mode, docs))


@pytest.mark.parametrize("d,Hq,Hkv", [(64, 16, 4), (96, 6, 3)])
def test_channel_attend_work_queue_short_walks(wm, d, Hq, Hkv):
    """Persistent workgroups over one-token tiles whose walks are empty (no cached slot: the
    row reads only the dummy) or one block long, interleaved within each workgroup's run of
    tiles; every output element against the oracle."""
    T_new, ctx = 1, 9
    # 4096 (d = 64) or 1536 (d = 96) tiles: an XCD's share of the tile order
    # (sequence-major) spans two sequences, one with an empty walk and one with a one-block
    # walk, several tiles a workgroup
    w = synth.small("queue_short_d%d" % d, B=16, T_new=T_new, L=16, k=4, D=64, Hq=Hq, Hkv=Hkv,
                    d=d, ctx=ctx + T_new, dtype="bf16", chan_map=[l % 4 for l in range(16)])
    tiles = w.Hq * w.B * w.L
    resident = torch.cuda.get_device_properties(0).multi_processor_count * (3 if d == 64 else 2)
    assert tiles > resident, (tiles, resident)
    print("short-walk queue case d%d tiles %d resident %d" % (d, tiles, resident), flush=True)
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w)
    ctx_len = torch.tensor([0, 5, 0, 9] * 4, dtype=torch.int32)
    Oo = oracle.channel_attend(_odims(w, mask_mode=0), P, Q, w.chan_map, ctx_len.numpy(),
                               _f64(Kc), _f64(Vc))
    O = torch.full((w.L, w.B, w.T_new, w.Hq * w.d), float("nan"), dtype=w.torch_dtype,
                   device="cuda")
    dims = _gdims(wm, w, mask_mode=0, ctx_max=ctx)
    wm.channel_attend(dims, _dev(P), Q.cuda(), w.chan_map, ctx_len.cuda(), Kc.cuda(), Vc.cuda(),
                      O)
    torch.cuda.synchronize()
    assert not torch.isnan(O.float()).any(), "a query tile was never computed"
    check_close(O, Oo, "bf16", "short-walk queue d%d" % d)


# ------------------------------------------------------------ full workloads

FULL = ["c2_T2048_L12_k12", "c3_T2048_L12_k6", "c4_T4096_L24_k12", "paper_T2048_L16_k8",
        "paper_T2048_L16_k16", "paper_T2048_L16_k1", "paper_T2048_L16_k2", "paper_T2048_L16_k4",
        "paper_T2048_L16_k12"]


def _sample_rows(w, b):
    ls = sorted({0, 1, w.L // 2, w.L - 2, w.L - 1})
    ts = sorted({0, 1, 31, 63, 64, 255, 256, 1023, 1024, w.T_new // 2 + 7, w.T_new - 2,
                 w.T_new - 1})
    return [(l * w.B + b) * w.T_new + t for l in ls for t in ts]


# (workload, mix mode, mask mode): every full-size pass in the paper's modes, and the
# softmax-over-depth mix with the inclusive causal mask on the three bf16 passes
FULL_CASES = [(n, 0, 0) for n in FULL] + [(n, 1, 1) for n in FULL[:3]]


@pytest.mark.parametrize("name,mix_mode,mask_mode", FULL_CASES)
def test_full_sequence_step_at_full_size(wm, name, mix_mode, mask_mode):
    """The full-size pass as the benchmark runs it; sampled sequences are re-computed by the
    oracle (every cache slot of the sequence, sampled attention rows). The paper-mode pass
    of the 24-layer 4096-token workload checks every one of its 4 sequences."""
    w = synth.WORKLOADS[name]
    print("full", name, "mix", mix_mode, "mask", mask_mode, flush=True)
    P = synth.make_params(w, _bias(w))
    H = synth.make_states(w)
    dims = _gdims(wm, w, mix_mode=mix_mode, mask_mode=mask_mode)
    Kg = torch.full((w.k, w.B, w.Hkv, w.S_cap, w.d), float("nan"), dtype=w.torch_dtype,
                    device="cuda")
    Vg = torch.full_like(Kg, float("nan"))
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.layer_step(dims, _dev(P), H.cuda(), w.chan_map, None, Kg, Vg, O)
    torch.cuda.synchronize()
    assert not torch.isnan(Kg[:, :, :, :w.T_new]).any()
    assert torch.isnan(Kg[:, :, :, w.T_new:]).all()
    PP = oracle.Params(P)
    if name == "c4_T4096_L24_k12" and (mix_mode, mask_mode) == (0, 0):
        samples = tuple(range(w.B))
    elif w.T_new * w.L <= 2048 * 12 and (mix_mode, mask_mode) == (0, 0):
        samples = (0, w.B - 1)
    else:
        samples = (w.B - 1,)
    for b in samples:
        w1 = synth.Workload(w.name, 1, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, 0, w.dtype,
                            w.chan_map, w.p, w.seed)
        dm = _odims(w1, mix_mode=mix_mode, mask_mode=mask_mode)
        Ko, Vo = oracle.empty_cache(dm)
        oracle.pool(dm, PP, H[b:b + 1], None, Ko, Vo)
        check_close(Kg[:, b:b + 1, :, :w.T_new], Ko[:, :, :, :w.T_new], w.dtype,
                    "%s K b=%d" % (name, b))
        check_close(Vg[:, b:b + 1, :, :w.T_new], Vo[:, :, :, :w.T_new], w.dtype,
                    "%s V b=%d" % (name, b))
        rows = _sample_rows(w1, 0)
        toks = sorted({r % w.T_new for r in rows})
        Qo = oracle.q_project(dm, PP, H[b:b + 1], None, toks)
        Oo = oracle.channel_attend(dm, PP, Qo, w.chan_map, None, Ko, Vo, rows)
        g = O[:, b].float().cpu().numpy()
        ls = sorted({r // w.T_new for r in rows})
        check_close(g[ls][:, toks], Oo[ls, 0][:, toks], w.dtype,
                    "%s O b=%d (%d layers x %d positions)" % (name, b, len(ls), len(toks)))


def test_decode_step_at_full_size(wm):
    """The 32768-context decode step: 64 new tokens appended to 12 channels, 24 consumers
    attend; every new slot is checked, and sampled sequences' outputs are re-computed by the
    oracle over the same cached context."""
    w = synth.WORKLOADS["c5_decode_S32768"]
    print("full decode", flush=True)
    P = synth.make_params(w, _bias(w))
    H = synth.make_states(w)
    Kg, Vg = synth.make_cache_device(w)
    ctx = torch.full((w.B,), w.ctx, dtype=torch.int32)
    samples = (0, w.B - 1)
    host = {b: (Kg[:, b:b + 1, :, :w.ctx].cpu(), Vg[:, b:b + 1, :, :w.ctx].cpu())
            for b in samples}
    O = torch.empty((w.L, w.B, 1, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.layer_step(_gdims(wm, w), _dev(P), H.cuda(), w.chan_map, ctx.cuda(), Kg, Vg, O)
    torch.cuda.synchronize()
    PP = oracle.Params(P)
    Kn, Vn = oracle.pool_rows(_odims(w), PP, H, ctx.numpy())   # [B, k, Hkv, d]
    check_close(Kg[:, :, :, w.ctx], Kn.transpose(1, 0, 2, 3), w.dtype, "decode K new slot")
    check_close(Vg[:, :, :, w.ctx], Vn.transpose(1, 0, 2, 3), w.dtype, "decode V new slot")
    assert torch.isnan(Kg[:, :, :, w.ctx + 1:]).all()
    del Kg, Vg
    torch.cuda.empty_cache()
    for b in samples:
        w1 = synth.Workload(w.name, 1, 1, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, w.ctx, w.dtype,
                            w.chan_map, w.p, w.seed)
        dm = _odims(w1, S_cap=w.ctx + 1)
        Kh, Vh = host.pop(b)
        Ko = np.empty((w.k, 1, w.Hkv, w.ctx + 1, w.d))
        Ko[:, :, :, :w.ctx] = _f64(Kh)
        Ko[:, 0, :, w.ctx] = Kn[b]
        del Kh
        Vo = np.empty_like(Ko)
        Vo[:, :, :, :w.ctx] = _f64(Vh)
        Vo[:, 0, :, w.ctx] = Vn[b]
        del Vh
        Qo = oracle.q_project(dm, PP, H[b:b + 1], [w.ctx])
        Oo = oracle.channel_attend(dm, PP, Qo, w.chan_map, [w.ctx], Ko, Vo)
        check_close(O[:, b:b + 1], Oo, w.dtype, "decode O b=%d" % b)
        del Ko, Vo


@pytest.mark.gpu
def test_calibration_loop_runs(wm):
    """The matrix-core ceiling loop launches, finishes and leaves its sink untouched."""
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    for random_operands in (False, True):
        wm.calibrate_mfma(256, 16, sink, torch.cuda.current_stream(), random_operands)
        torch.cuda.synchronize()
        assert float(sink.item()) == 0.0


@pytest.mark.gpu
def test_read_calibration_runs(wm):
    """The HBM read loop (ragged tail included) finishes and leaves its sink untouched."""
    buf = torch.arange((1 << 20) + 12, dtype=torch.int32, device="cuda")
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    wm.calibrate_read(buf, sink, torch.cuda.current_stream())
    torch.cuda.synchronize()
    assert float(sink.item()) == 0.0


# ------------------------------------------------------------ document mask

DOC_CASES = [  # (T_new, ctx, doc lengths or None for seeded lengths of mean 37)
    (300, 0, None), (200, 0, [1]), (256, 0, [64]), (300, 0, [63, 65, 1, 128, 2]),
    (129, 0, [300]), (40, 200, None), (3, 513, [100, 7]), (1, 1000, None), (1, 700, [1]),
]


@pytest.mark.parametrize("T_new,ctx,lengths", DOC_CASES)
@pytest.mark.parametrize("mask_mode", [0, 1])
def test_channel_attend_doc(wm, T_new, ctx, lengths, mask_mode):
    """Attention under the document mask (packed documents), every kernel path: bf16 head
    dims 64 and 96 (the LDS-DMA prefill kernel), fp32 (the generic prefill kernel) and
    decode (T_new <= 4), against the oracle row by row."""
    for dtype, d in (("bf16", 64), ("f32", 32), ("bf16", 96)):
        w = synth.small("doc_%s_d%d" % (dtype, d), B=2, T_new=T_new, L=5, k=3, D=64, Hq=4,
                        Hkv=2, d=d, ctx=ctx + T_new, dtype=dtype, chan_map=[2, 0, 2, 2, 0])
        print("doc case", dtype, d, T_new, ctx, lengths, mask_mode, flush=True)
        P = synth.make_params(w, _bias(w))
        Q = synth.make_queries(w)
        Kc, Vc = synth.make_cache_cpu(w)
        ctx_len = torch.tensor([ctx, ctx // 2], dtype=torch.int32)
        docs = synth.make_doc_start(w, ctx_len, mean_len=37.0, lengths=lengths)
        Oo = oracle.channel_attend(_odims(w, mask_mode=mask_mode), P, Q, w.chan_map,
                                   ctx_len.numpy(), _f64(Kc), _f64(Vc), doc_start=docs.numpy())
        O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
        dims = _gdims(wm, w, mask_mode=mask_mode, ctx_max=ctx)
        wm.channel_attend(dims, _dev(P), Q.cuda(), w.chan_map, ctx_len.cuda(), Kc.cuda(),
                          Vc.cuda(), O, doc_start=docs.cuda())
        torch.cuda.synchronize()
        check_close(O, Oo, dtype, "doc %s d%d T%d ctx%d" % (dtype, d, T_new, ctx))


@pytest.mark.parametrize("name", ["bf16_paper_shape", "c1_tiny_f32", "bf16_ragged_gqa"])
def test_layer_step_doc(wm, name):
    """The fused step with packed documents: the cache writes are the plain step's, the
    outputs follow the document mask."""
    w = SMALL[name]
    rng = np.random.default_rng(w.seed)
    P = synth.make_params(w, _bias(w) + rng.normal(0, 0.3, size=w.k * w.L))
    H = synth.make_states(w)
    docs = synth.make_doc_start(w, mean_len=9.0)
    K0, V0 = synth.make_cache_cpu(w)
    Ko, Vo = _f64(K0).copy(), _f64(V0).copy()
    Oo = oracle.layer_step(_odims(w), P, H, w.chan_map, None, Ko, Vo, doc_start=docs.numpy())
    Kg, Vg = K0.cuda(), V0.cuda()
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.layer_step(_gdims(wm, w), _dev(P), H.cuda(), w.chan_map, None, Kg, Vg, O,
                  doc_start=docs.cuda())
    torch.cuda.synchronize()
    ctx = np.zeros(w.B, dtype=np.int64)
    _check_cache(Kg, Ko, K0, w, ctx, w.dtype, name + " doc K")
    _check_cache(Vg, Vo, V0, w, ctx, w.dtype, name + " doc V")
    check_close(O, Oo, w.dtype, name + " doc O")


def test_doc_entry_points_reject_bad_doc_arrays(wm):
    w = SMALL["bf16_ragged_gqa"]
    dims = _gdims(wm, w)
    P = _dev(synth.make_params(w, _bias(w)))
    Q = torch.zeros((w.L, w.B, w.Hq, w.T_new, w.d), dtype=w.torch_dtype, device="cuda")
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    Kc = torch.zeros((w.k, w.B, w.Hkv, w.S_cap, w.d), dtype=w.torch_dtype, device="cuda")
    raw = torch.zeros((4 * w.B * w.T_new + 4,), dtype=torch.uint8, device="cuda")
    with pytest.raises(wm.WMError) as e:  # misaligned: no launch
        wm.channel_attend(dims, P, Q, w.chan_map, None, Kc, Kc, O, doc_start=raw[1:])
    assert e.value.code == wm.ERR_ARG


@pytest.mark.parametrize("name", ["paper_T2048_L16_k8"])
def test_full_sequence_doc_step_at_full_size(wm, name):
    """The paper-shape pass with packed documents (mean length 512) as the benchmark runs
    it; one sequence re-computed by the oracle (all its cache slots, sampled rows)."""
    w = synth.WORKLOADS[name]
    print("full doc", name, flush=True)
    P = synth.make_params(w, _bias(w))
    H = synth.make_states(w)
    docs = synth.make_doc_start(w, mean_len=512.0)
    Kg = torch.full((w.k, w.B, w.Hkv, w.S_cap, w.d), float("nan"), dtype=w.torch_dtype,
                    device="cuda")
    Vg = torch.full_like(Kg, float("nan"))
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.layer_step(_gdims(wm, w), _dev(P), H.cuda(), w.chan_map, None, Kg, Vg, O,
                  doc_start=docs.cuda())
    torch.cuda.synchronize()
    PP = oracle.Params(P)
    b = w.B - 1
    w1 = synth.Workload(w.name, 1, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, 0, w.dtype,
                        w.chan_map, w.p, w.seed)
    dm = _odims(w1)
    Ko, Vo = oracle.empty_cache(dm)
    oracle.pool(dm, PP, H[b:b + 1], None, Ko, Vo)
    check_close(Kg[:, b:b + 1, :, :w.T_new], Ko[:, :, :, :w.T_new], w.dtype, name + " K")
    rows = _sample_rows(w1, 0)
    # rows at and just after each document start of the sequence, too
    starts = sorted(set(docs[b].tolist()))
    extra = sorted({t for s0 in starts for t in (s0, s0 + 1) if t < w.T_new})[:24]
    rows = sorted(set(rows) | {(l * 1 + 0) * w.T_new + t for l in (0, w.L - 1) for t in extra})
    toks = sorted({r % w.T_new for r in rows})
    Qo = oracle.q_project(dm, PP, H[b:b + 1], None, toks)
    Oo = oracle.channel_attend(dm, PP, Qo, w.chan_map, None, Ko, Vo, rows,
                               doc_start=docs[b:b + 1].numpy())
    g = O[:, b].float().cpu().numpy()
    for l in sorted({r // w.T_new for r in rows}):
        for t in toks:
            if (l * w.T_new + t) in rows:
                check_close(g[l, t], Oo[l, 0, t], w.dtype, "%s doc O l=%d t=%d" % (name, l, t))


# -------------------------------------------- router variants (ablations, Section 5.3)

VARIANT_CASES = {
    "f32_kL": synth.small("f32_kL", B=2, T_new=37, L=4, k=4, D=64, Hq=2, Hkv=2, d=32,
                          dtype="f32"),
    "bf16_kL_p2": synth.small("bf16_kL_p2", B=2, T_new=70, L=6, k=6, D=128, Hq=4, Hkv=2, d=64,
                              p=2),
    "bf16_ragged_gqa": SMALL["bf16_ragged_gqa"],
}


@pytest.mark.parametrize("name,router_mode", [("f32_kL", 2), ("bf16_kL_p2", 2), ("f32_kL", 1),
                                              ("bf16_ragged_gqa", 1)])
@pytest.mark.parametrize("mix_mode", [0, 1])
def test_router_mix_variants(wm, name, router_mode, mix_mode):
    """Static weights (no router) and no deep-to-shallow feedback: mixing weights and mixed
    channels against the oracle."""
    w = VARIANT_CASES[name]
    rng = np.random.default_rng(17)
    P = synth.make_params(w, rng.normal(0, 1, size=(2, w.k * w.L)), gains="random")
    P["W_alpha"] = (P["W_alpha"].float() * 10).to(P["W_alpha"].dtype)  # a router that matters
    H = synth.make_states(w)
    ao, mo = oracle.router_mix(_odims(w, mix_mode=mix_mode, router_mode=router_mode), P, H)
    dims = _gdims(wm, w, mix_mode=mix_mode, router_mode=router_mode)
    alpha = torch.empty((2, w.N, w.k, w.L), dtype=torch.float32, device="cuda")
    mixed = torch.empty((2, w.k, w.N, w.D), dtype=w.torch_dtype, device="cuda")
    ps = wm.ParamSet(_dev(P))
    if router_mode == 1:
        ps.c.W_alpha = None  # static weights do not read the router weights
    wm.router_mix(dims, ps, H.cuda(), mixed, alpha)
    torch.cuda.synchronize()
    check_close(alpha, ao, w.dtype, "%s alpha" % name)
    check_close(mixed, mo, w.dtype, "%s mixed" % name)
    if router_mode == 2:
        for j in range(w.k):
            assert (alpha[:, :, j, j + 1:] == 0).all()



@pytest.mark.parametrize("name,router_mode", [("bf16_kL_p2", 2), ("f32_kL", 2),
                                              ("bf16_ragged_gqa", 1)])
def test_layer_step_variants(wm, name, router_mode):
    w = VARIANT_CASES[name]
    rng = np.random.default_rng(19)
    P = synth.make_params(w, rng.normal(0, 1, size=(2, w.k * w.L)), gains="random")
    H = synth.make_states(w)
    K0, V0 = synth.make_cache_cpu(w)
    Ko, Vo = _f64(K0).copy(), _f64(V0).copy()
    Oo = oracle.layer_step(_odims(w, router_mode=router_mode), P, H, w.chan_map, None, Ko, Vo)
    Kg, Vg = K0.cuda(), V0.cuda()
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.layer_step(_gdims(wm, w, router_mode=router_mode), _dev(P), H.cuda(), w.chan_map, None,
                  Kg, Vg, O)
    torch.cuda.synchronize()
    ctx = np.zeros(w.B, dtype=np.int64)
    _check_cache(Kg, Ko, K0, w, ctx, w.dtype, name + " K")
    _check_cache(Vg, Vo, V0, w, ctx, w.dtype, name + " V")
    check_close(O, Oo, w.dtype, name + " O")
