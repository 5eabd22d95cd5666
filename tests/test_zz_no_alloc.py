"""The entry point that allocates nothing (wm_channel_attend_static): its decode partials
(and the split ranges' partial states of a full-sequence call on a small grid) live in the
library's fixed device array instead of a caller workspace. Checked through
the C ABI against wm_channel_attend (same kernels: bit for bit) and against the oracle
(the parity bar), on two calls in a row, the second smaller; a call that needs more than
the array holds is rejected before any launch."""
import numpy as np
import pytest
import torch

import oracle
from tests import synth
from tests.parity import _bias, _dev, _f64, _gdims, _odims, check_close, wm  # noqa: F401

pytestmark = pytest.mark.gpu


def _case(wm, w, ctx):
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    Kc, Vc = synth.make_cache_cpu(w)
    ctx_len = torch.tensor([ctx - (b % 3) * 7 for b in range(w.B)], dtype=torch.int32)
    dims = _gdims(wm, w, ctx_max=ctx)
    Pd = wm.ParamSet(_dev(P))
    args = (Q.cuda(), w.chan_map, ctx_len.cuda(), Kc.cuda(), Vc.cuda())
    O_ws = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
    wm.channel_attend(dims, Pd, *args, O_ws)
    O_st = torch.full_like(O_ws, float("nan"))
    wm.channel_attend_static(dims, Pd, *args, O_st)
    torch.cuda.synchronize()
    Oo = oracle.channel_attend(_odims(w), P, Q, w.chan_map, ctx_len.numpy(), _f64(Kc), _f64(Vc))
    return O_ws, O_st, Oo


@pytest.mark.parametrize("dtype,d", [("bf16", 64), ("bf16", 96), ("f32", 32)])
def test_static_scratch_matches_workspace_entry_point(wm, dtype, d):
    cases = [  # (workload, ctx): decode over many splits, then a smaller call, then prefill
        (synth.small("static_big", B=8, T_new=2, L=6, k=3, D=64, Hq=4, Hkv=2, d=d, ctx=9002,
                     dtype=dtype), 9000),
        (synth.small("static_small", B=2, T_new=1, L=3, k=2, D=64, Hq=2, Hkv=1, d=d, ctx=3001,
                     dtype=dtype), 3000),
        (synth.small("static_prefill", B=2, T_new=40, L=3, k=2, D=64, Hq=2, Hkv=1, d=d, ctx=140,
                     dtype=dtype), 100),
        # few query tiles over a 2000-slot context: the bf16 kernel splits the slot ranges
        (synth.small("static_split", B=2, T_new=40, L=3, k=2, D=64, Hq=2, Hkv=1, d=d, ctx=2240,
                     dtype=dtype), 2200),
    ]
    for w, ctx in cases:
        print("static scratch", w.name, dtype, d, flush=True)
        O_ws, O_st, Oo = _case(wm, w, ctx)
        assert torch.equal(O_st, O_ws), w.name
        check_close(O_st, Oo, dtype, "%s %s d%d" % (w.name, dtype, d))


def test_static_scratch_rejects_calls_past_its_size(wm):
    """24 consumers x 64 sequences x 16 heads x 4 new tokens over a 32768-slot context
    need about 233 MB of decode partials: more than the 64 MiB array, so no launch."""
    w = synth.small("static_huge", B=64, T_new=4, L=24, k=12, D=1024, Hq=16, Hkv=16, d=64,
                    ctx=32772)
    dims = _gdims(wm, w, ctx_max=32768)
    need = wm.workspace_size(dims, wm.OP_CHANNEL_ATTEND)
    assert need > 64 << 20, need
    t = torch.zeros(64, dtype=torch.bfloat16, device="cuda")
    Pd = wm.ParamSet({n: t for n in wm.PARAM_NAMES})
    with pytest.raises(wm.WMError) as e:
        wm.channel_attend_static(dims, Pd, t, w.chan_map, None, t, t, t)
    assert e.value.code == wm.ERR_WORKSPACE
