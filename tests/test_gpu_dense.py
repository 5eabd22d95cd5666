"""GPU parity of the dense soft read (Section 3.1 Step 3 variant): every consumer attends
all channels mixed with its own weights. Against the oracle on softmax weights, and bit
for bit against the fixed selection when the weights are one-hot."""
import numpy as np
import pytest
import torch

import oracle
from tests import synth
from tests.parity import _bias, _dev, _f64, _gdims, _odims, check_close, wm  # noqa: F401

pytestmark = pytest.mark.gpu

CASES = [  # (dtype, d, T_new, ctx): prefill over a cached context, decode, a fresh prefill
    ("bf16", 64, 70, 100), ("bf16", 96, 2, 1000), ("f32", 32, 40, 0), ("bf16", 64, 1, 5000),
]


def _case(w, ctx):
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w)
    ctx_len = torch.tensor([ctx, ctx // 2], dtype=torch.int32)
    return P, Q, Kc, Vc, ctx_len


@pytest.mark.parametrize("dtype,d,T_new,ctx", CASES)
@pytest.mark.parametrize("mask_mode", [0, 1])
def test_dense_read_matches_oracle(wm, dtype, d, T_new, ctx, mask_mode):
    w = synth.small("dense_%s_d%d" % (dtype, d), B=2, T_new=T_new, L=5, k=3, D=64, Hq=4, Hkv=2,
                    d=d, ctx=ctx + T_new, dtype=dtype, chan_map=[2, 0, 2, 1, 0])
    print("dense", dtype, d, T_new, ctx, mask_mode, flush=True)
    P, Q, Kc, Vc, ctx_len = _case(w, ctx)
    rng = np.random.default_rng(31)
    logits = rng.normal(size=(w.L, w.k))
    rw = np.exp(logits) / np.exp(logits).sum(axis=1, keepdims=True)
    Oo = oracle.channel_attend_dense(_odims(w, mask_mode=mask_mode), P, rw, Q, ctx_len.numpy(),
                                     _f64(Kc), _f64(Vc))
    dims = _gdims(wm, w, mask_mode=mask_mode, ctx_max=ctx)
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.channel_attend_dense(dims, _dev(P), torch.tensor(rw, dtype=torch.float32).cuda(),
                            Q.cuda(), ctx_len.cuda(), Kc.cuda(), Vc.cuda(), O)
    torch.cuda.synchronize()
    check_close(O, Oo, dtype, "dense %s d%d T%d ctx%d mask%d" % (dtype, d, T_new, ctx, mask_mode))


@pytest.mark.parametrize("dtype,d,T_new,ctx", CASES)
def test_dense_read_with_one_hot_weights_is_the_fixed_selection(wm, dtype, d, T_new, ctx):
    w = synth.small("dense1_%s_d%d" % (dtype, d), B=2, T_new=T_new, L=5, k=3, D=64, Hq=4, Hkv=2,
                    d=d, ctx=ctx + T_new, dtype=dtype, chan_map=[2, 0, 2, 1, 0])
    P, Q, Kc, Vc, ctx_len = _case(w, ctx)
    onehot = torch.zeros((w.L, w.k), dtype=torch.float32)
    onehot[torch.arange(w.L), torch.tensor(w.chan_map)] = 1.0
    dims = _gdims(wm, w, ctx_max=ctx)
    Pd = wm.ParamSet(_dev(P))
    args = (Q.cuda(), ctx_len.cuda(), Kc.cuda(), Vc.cuda())
    Od = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.channel_attend_dense(dims, Pd, onehot.cuda(), *args, Od)
    Os = torch.empty_like(Od)
    wm.channel_attend(dims, Pd, args[0], w.chan_map, *args[1:], Os)
    torch.cuda.synchronize()
    assert torch.equal(Od, Os)
