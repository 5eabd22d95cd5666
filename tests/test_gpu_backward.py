"""GPU parity of the attention gradients (wm_channel_attend_backward) against the gradient
oracle: every element of dQ, of the written cache slots of dKc and dVc, and of the dummy's
dKd and dVd; the slots the call must not write keep their NaN sentinel."""
import numpy as np
import pytest
import torch

import oracle
from oracle import backward as ob
from tests import synth
from tests.parity import _bias, _dev, _f64, _gdims, _odims, check_close, wm  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("T_new,ctx", [(40, 0), (300, 0), (70, 130)])
@pytest.mark.parametrize("mask_mode", [0, 1])
@pytest.mark.parametrize("d,Hq,Hkv,B", [(64, 4, 2, 2), (96, 6, 3, 2), (64, 2, 2, 2),
                                        (64, 4, 2, 4), (96, 6, 3, 4)])
def test_channel_attend_backward(wm, T_new, ctx, mask_mode, d, Hq, Hkv, B):
    """B = 4 with Hkv = 2 gives 24 slices (channel, sequence, KV head): with their few slot
    tiles, the slot-major grid takes each XCD's heavy tiles first (slices a multiple of 8);
    Hkv = 3 at B = 4 does not divide and keeps the slice-major order."""
    w = synth.small("bwd_d%d" % d, B=B, T_new=T_new, L=5, k=3, D=64, Hq=Hq, Hkv=Hkv, d=d,
                    ctx=ctx + T_new, dtype="bf16", chan_map=[2, 0, 2, 2, 0])
    print("attention backward d%d %d/%d T%d ctx%d mask%d" % (d, Hq, Hkv, T_new, ctx, mask_mode),
          flush=True)
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w)
    ctx_len = torch.tensor([ctx, ctx // 2, ctx // 3, ctx][:B], dtype=torch.int32)
    od = _odims(w, mask_mode=mask_mode)
    O = oracle.channel_attend(od, P, Q, w.chan_map, ctx_len.numpy(), _f64(Kc), _f64(Vc))
    O_bf = torch.from_numpy(O).to(torch.bfloat16)
    dO = synth._normal(O.shape, 1.0, 4242, torch.bfloat16)
    g = ob.channel_attend_grads(od, P, Q, w.chan_map, ctx_len.numpy(), _f64(Kc), _f64(Vc),
                                _f64(dO))

    dev = "cuda"
    nan = float("nan")
    dQ = torch.full(tuple(Q.shape), nan, dtype=torch.float32, device=dev)
    dKc = torch.full(tuple(Kc.shape), nan, dtype=torch.float32, device=dev)
    dVc = torch.full(tuple(Vc.shape), nan, dtype=torch.float32, device=dev)
    dKd = torch.full(tuple(P["Kd"].shape), nan, dtype=torch.float32, device=dev)
    dVd = torch.full(tuple(P["Vd"].shape), nan, dtype=torch.float32, device=dev)
    dims = _gdims(wm, w, mask_mode=mask_mode, ctx_max=ctx)
    wm.channel_attend_backward(dims, _dev(P), Q.cuda(), w.chan_map, ctx_len.cuda(), Kc.cuda(),
                               Vc.cuda(), O_bf.cuda(), dO.cuda(), dQ, dKc, dVc, dKd, dVd)
    torch.cuda.synchronize()
    check_close(dQ, g["dQ"], "bf16", "dQ")
    check_close(dKd, g["dKd"], "bf16", "dKd")
    check_close(dVd, g["dVd"], "bf16", "dVd")
    dKc_h, dVc_h = dKc.cpu().numpy(), dVc.cpu().numpy()
    for b, c0 in enumerate(ctx_len.tolist()):
        hi = c0 + T_new
        check_close(dKc_h[:, b, :, :hi], g["dKc"][:, b, :, :hi], "bf16", "dKc b%d" % b)
        check_close(dVc_h[:, b, :, :hi], g["dVc"][:, b, :, :hi], "bf16", "dVc b%d" % b)
        # the call writes slots below ctx_len[b] + T_new only
        assert np.isnan(dKc_h[:, b, :, hi:]).all() and np.isnan(dVc_h[:, b, :, hi:]).all()
    # channel 1 has no consumer: no gradient reaches it
    for b, c0 in enumerate(ctx_len.tolist()):
        assert not np.any(dKc_h[1, b, :, :c0 + T_new]) and not np.any(dVc_h[1, b, :, :c0 + T_new])


def test_channel_attend_backward_is_deterministic(wm):
    """Every gradient is a fixed-order sum (no atomics): two calls agree bit for bit."""
    w = synth.small("bwd_det", B=2, T_new=200, L=4, k=2, D=64, Hq=4, Hkv=2, d=64, ctx=200,
                    dtype="bf16")
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w).cuda()
    Kc, Vc = synth.make_cache_cpu(w)
    Kc, Vc = Kc.cuda(), Vc.cuda()
    O = synth._normal((w.L, w.B, w.T_new, w.Hq * w.d), 0.5, 11, torch.bfloat16).cuda()
    dO = synth._normal((w.L, w.B, w.T_new, w.Hq * w.d), 1.0, 12, torch.bfloat16).cuda()
    dims = _gdims(wm, w, ctx_max=0)
    outs = []
    for _ in range(2):
        r = [torch.zeros(tuple(Q.shape), dtype=torch.float32, device="cuda"),
             torch.zeros(tuple(Kc.shape), dtype=torch.float32, device="cuda"),
             torch.zeros(tuple(Vc.shape), dtype=torch.float32, device="cuda"),
             torch.zeros(tuple(P["Kd"].shape), dtype=torch.float32, device="cuda"),
             torch.zeros(tuple(P["Vd"].shape), dtype=torch.float32, device="cuda")]
        wm.channel_attend_backward(dims, _dev(P), Q, w.chan_map, None, Kc, Vc, O, dO, *r)
        torch.cuda.synchronize()
        outs.append(r)
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def _sub_dims(w, L, Hq, mask_mode):
    return oracle.Dims(B=1, T_new=w.T_new, L=L, k=1, D=w.D, Hq=Hq, Hkv=1, d=w.d, p=1,
                       S_cap=w.T_new, mask_mode=mask_mode)


@pytest.mark.parametrize("name", ["c4_T4096_L24_k12", "paper_T2048_L16_k8"])
def test_channel_attend_backward_at_full_size(wm, name):
    """The full-size pass's attention gradients in the launch configuration a training step
    uses (the forward's output O from the GPU forward, persistent grids): sampled query rows'
    dQ, sampled channel slices' dK and dV (every reader of the slice), and one dummy's dK,
    dV, each against the oracle on the sub-problem that determines it."""
    w = synth.WORKLOADS[name]
    print("attention backward full size %s" % name, flush=True)
    G, c_of = w.Hq // w.Hkv, w.chan_map
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    shape = (w.k, w.B, w.Hkv, w.T_new, w.d)
    Kc = synth._normal(shape, 1.0, 9001, torch.bfloat16)
    Vc = synth._normal(shape, 1.0, 9002, torch.bfloat16)
    dO = synth._normal((w.L, w.B, w.T_new, w.Hq * w.d), 1.0, 9003, torch.bfloat16)
    dims = _gdims(wm, w, S_cap=w.T_new, ctx_max=0)
    Pd, Qd, Kd_, Vd_ = _dev(P), Q.cuda(), Kc.cuda(), Vc.cuda()
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=torch.bfloat16, device="cuda")
    wm.channel_attend(dims, Pd, Qd, w.chan_map, None, Kd_, Vd_, O)
    f32 = dict(dtype=torch.float32, device="cuda")
    dQ, dKc, dVc = torch.empty(tuple(Q.shape), **f32), torch.empty(shape, **f32), \
        torch.empty(shape, **f32)
    dKd, dVd = torch.empty(tuple(P["Kd"].shape), **f32), torch.empty(tuple(P["Vd"].shape), **f32)
    wm.channel_attend_backward(dims, Pd, Qd, w.chan_map, None, Kd_, Vd_, O, dO.cuda(), dQ, dKc,
                               dVc, dKd, dVd)
    torch.cuda.synchronize()
    del O, Pd, Qd, Kd_, Vd_
    dQ, dKc, dVc, dKd, dVd = (t.cpu() for t in (dQ, dKc, dVc, dKd, dVd))

    def sub_params(c, kvh):
        return {**{n: P[n] for n in oracle.PARAM_NAMES},
                "Kd": P["Kd"][c, kvh].reshape(1, 1, w.d), "Vd": P["Vd"][c, kvh].reshape(1, 1, w.d)}

    # dQ of sampled (consumer, sequence, query head) rows: the sub-problem of that row set
    for l, b, hq in ((0, 0, 0), (w.L - 1, w.B - 1, w.Hq - 1), (w.L // 2, 1, w.Hq // 2)):
        c, kvh = c_of[l], hq // G
        g = ob.channel_attend_grads(_sub_dims(w, 1, 1, 0), sub_params(c, kvh),
                                    Q[l, b, hq].reshape(1, 1, 1, w.T_new, w.d), [0], None,
                                    _f64(Kc[c, b, kvh]).reshape(1, 1, 1, w.T_new, w.d),
                                    _f64(Vc[c, b, kvh]).reshape(1, 1, 1, w.T_new, w.d),
                                    _f64(dO[l, b, :, hq * w.d:(hq + 1) * w.d]).reshape(
                                        1, 1, w.T_new, w.d))
        check_close(dQ[l, b, hq], g["dQ"][0, 0, 0], "bf16", "%s dQ l%d b%d h%d" % (name, l, b, hq))

    # dK, dV of sampled channel slices: every consumer of the channel, every grouped head
    def slice_grads(c, b, kvh):
        ls = [l for l in range(w.L) if c_of[l] == c]
        hs = list(range(kvh * G, (kvh + 1) * G))
        Qs = Q[ls][:, b, hs].reshape(len(ls), 1, G, w.T_new, w.d)
        dOs = dO[ls][:, b].reshape(len(ls), w.T_new, w.Hq, w.d)[:, :, hs].reshape(
            len(ls), 1, w.T_new, G * w.d)
        return ob.channel_attend_grads(_sub_dims(w, len(ls), G, 0), sub_params(c, kvh), Qs,
                                       [0] * len(ls), None,
                                       _f64(Kc[c, b, kvh]).reshape(1, 1, 1, w.T_new, w.d),
                                       _f64(Vc[c, b, kvh]).reshape(1, 1, 1, w.T_new, w.d),
                                       _f64(dOs))

    for c, b, kvh in ((0, 0, 0), (w.k - 1, w.B - 1, w.Hkv - 1)):
        g = slice_grads(c, b, kvh)
        check_close(dKc[c, b, kvh], g["dKc"][0, 0, 0], "bf16", "%s dK c%d b%d" % (name, c, b))
        check_close(dVc[c, b, kvh], g["dVc"][0, 0, 0], "bf16", "%s dV c%d b%d" % (name, c, b))
    # the dummy of channel 1, KV head 0: its readers in every sequence
    kd = np.zeros(w.d)
    vd = np.zeros(w.d)
    for b in range(w.B):
        g = slice_grads(1, b, 0)
        kd += g["dKd"][0, 0]
        vd += g["dVd"][0, 0]
    check_close(dKd[1, 0], kd, "bf16", "%s dKd" % name)
    check_close(dVd[1, 0], vd, "bf16", "%s dVd" % name)


@pytest.mark.parametrize("mask_mode", [0, 1])
@pytest.mark.parametrize("d,Hq,Hkv", [(64, 4, 2), (96, 6, 3)])
def test_channel_attend_backward_strided_group(wm, mask_mode, d, Hq, Hkv):
    """Queries of the strided token group q = 2 of g = 3 (positions ctx + 2 + 3 i, Section
    3.3) over a cache whose every slot is given."""
    g, q, T_new, ctx = 3, 2, 90, 40
    w = synth.small("bwd_grp_d%d" % d, B=2, T_new=T_new, L=5, k=3, D=64, Hq=Hq, Hkv=Hkv, d=d,
                    ctx=ctx + q + g * (T_new - 1) + 1, dtype="bf16", chan_map=[2, 0, 2, 1, 0])
    print("attention backward strided group d%d mask%d" % (d, mask_mode), flush=True)
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w)  # every slot below the span holds values
    ctx_len = torch.tensor([ctx, ctx // 2], dtype=torch.int32)
    od = _odims(w, mask_mode=mask_mode)
    O = ob.attend(od, ob._t(P["Kd"]), ob._t(P["Vd"]), ob._t(Q), w.chan_map,
                  torch.as_tensor(ctx_len.numpy(), dtype=torch.long), ob._t(Kc), ob._t(Vc),
                  (g, q)).detach().numpy()
    dO = synth._normal(O.shape, 1.0, 4343, torch.bfloat16)
    ref = ob.channel_attend_grads(od, P, Q, w.chan_map, ctx_len.numpy(), _f64(Kc), _f64(Vc),
                                  _f64(dO), grp=(g, q))
    dev = "cuda"
    f32 = dict(dtype=torch.float32, device=dev)
    dQ = torch.empty(tuple(Q.shape), **f32)
    dKc = torch.full(tuple(Kc.shape), float("nan"), **f32)
    dVc = torch.full(tuple(Kc.shape), float("nan"), **f32)
    dKd, dVd = torch.empty(tuple(P["Kd"].shape), **f32), torch.empty(tuple(P["Kd"].shape), **f32)
    dims = _gdims(wm, w, mask_mode=mask_mode, ctx_max=ctx, groups=g, group=q)
    wm.channel_attend_backward(dims, _dev(P), Q.cuda(), w.chan_map, ctx_len.cuda(), Kc.cuda(),
                               Vc.cuda(), torch.from_numpy(O).to(torch.bfloat16).cuda(),
                               dO.cuda(), dQ, dKc, dVc, dKd, dVd)
    torch.cuda.synchronize()
    check_close(dQ, ref["dQ"], "bf16", "dQ")
    check_close(dKd, ref["dKd"], "bf16", "dKd")
    check_close(dVd, ref["dVd"], "bf16", "dVd")
    dKc_h, dVc_h = dKc.cpu().numpy(), dVc.cpu().numpy()
    for b, c0 in enumerate(ctx_len.tolist()):
        hi = c0 + q + g * (T_new - 1) + 1
        check_close(dKc_h[:, b, :, :hi], ref["dKc"][:, b, :, :hi], "bf16", "dKc b%d" % b)
        check_close(dVc_h[:, b, :, :hi], ref["dVc"][:, b, :, :hi], "bf16", "dVc b%d" % b)
        assert np.isnan(dKc_h[:, b, :, hi:]).all() and np.isnan(dVc_h[:, b, :, hi:]).all()

