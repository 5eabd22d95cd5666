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
@pytest.mark.parametrize("d,Hq,Hkv", [(64, 4, 2), (96, 6, 3), (64, 2, 2)])
def test_channel_attend_backward(wm, T_new, ctx, mask_mode, d, Hq, Hkv):
    w = synth.small("bwd_d%d" % d, B=2, T_new=T_new, L=5, k=3, D=64, Hq=Hq, Hkv=Hkv, d=d,
                    ctx=ctx + T_new, dtype="bf16", chan_map=[2, 0, 2, 2, 0])
    print("attention backward d%d %d/%d T%d ctx%d mask%d" % (d, Hq, Hkv, T_new, ctx, mask_mode),
          flush=True)
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w)
    ctx_len = torch.tensor([ctx, ctx // 2], dtype=torch.int32)
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
