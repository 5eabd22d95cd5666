"""GPU parity of the full-sequence attention on small grids, where the bf16 kernel cuts
each query tile's slot range into split ranges walked by workgroups of their own and merges
their partial softmax states (Section 3.1 Step 3: one softmax over the visible slots;
Section 3.2: the dummy slot starts the row, so it belongs to the first range only).

Each case first checks on the host that the kernel's planner splits it (query tiles at
most a quarter of the workgroups the CUs hold, walks of at least 32 64-slot blocks), then compares
every output element with the oracle: contiguous tokens and one strided token group, both
masks, head dims 64 and 96 with grouped heads, a sequence whose shorter context leaves
some of its tiles' ranges empty, and peaked scores (the sawtooth keys of the rescale
tests, climbing 60 log2 units per 256 slots) whose references differ widely between the
ranges of one row."""
import numpy as np
import pytest
import torch

import oracle
from oracle import backward as ob
from tests import synth
from tests.parity import _bias, _dev, _f64, _gdims, _odims, check_close, wm  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("d,Hq,Hkv", [(64, 4, 2), (96, 6, 3)])
@pytest.mark.parametrize("mask_mode", [0, 1])
@pytest.mark.parametrize("g,q,peak", [(1, 0, False), (3, 2, False), (1, 0, True)])
def test_channel_attend_split_ranges(wm, d, Hq, Hkv, mask_mode, g, q, peak):
    T_new, ctx = 96, 2200
    span = q + g * (T_new - 1) + 1
    w = synth.small("split_d%d" % d, B=2, T_new=T_new, L=2, k=1, D=64, Hq=Hq, Hkv=Hkv, d=d,
                    ctx=ctx + span, dtype="bf16", chan_map=[0, 0])
    tiles = (T_new + 127) // 128 * Hq * w.B * w.L
    resident = torch.cuda.get_device_properties(0).multi_processor_count * (3 if d == 64 else 2)
    blocks = (ctx + span + 63) // 64
    assert 4 * tiles <= resident and blocks >= 32, (tiles, resident, blocks)
    print("split ranges d%d mask%d g%d q%d peaked %s: %d tiles, %d blocks"
          % (d, mask_mode, g, q, peak, tiles, blocks), flush=True)
    P = synth.make_params(w, _bias(w))
    if peak:
        Q, Kc, Vc = synth.make_peaked_attention(w, rise=60.0, period=256)
    else:
        Q = synth.make_queries(w)
        Kc, Vc = synth.make_cache_cpu(w)
    ctx_len = torch.tensor([ctx, ctx // 3], dtype=torch.int32)
    od = _odims(w, mask_mode=mask_mode)
    if g == 1:
        ref = oracle.channel_attend(od, P, Q, w.chan_map, ctx_len.numpy(), _f64(Kc), _f64(Vc))
    else:
        ref = ob.attend(od, ob._t(P["Kd"]), ob._t(P["Vd"]), ob._t(Q), w.chan_map,
                        torch.as_tensor(ctx_len.numpy(), dtype=torch.long), ob._t(Kc),
                        ob._t(Vc), (g, q)).detach().numpy()
    O = torch.full((w.L, w.B, w.T_new, w.Hq * w.d), float("nan"), dtype=torch.bfloat16,
                   device="cuda")
    dims = _gdims(wm, w, mask_mode=mask_mode, ctx_max=ctx, groups=g, group=q)
    wm.channel_attend(dims, _dev(P), Q.cuda(), w.chan_map, ctx_len.cuda(), Kc.cuda(), Vc.cuda(),
                      O)
    torch.cuda.synchronize()
    check_close(O, ref, "bf16", "split d%d mask%d g%d peaked %s" % (d, mask_mode, g, peak))


def test_split_ranges_at_the_pass_driver_shape(wm):
    """One consumer's attention over a token group at the pass driver's shape (the call it
    makes per layer and group at the paper's model shape: 16 sequences of 2048 tokens, group
    13 of 16, 6 query / 3 KV heads of 96): sampled sequences' rows against the oracle (rows
    of different sequences are independent)."""
    B, T, g, q, d, Hq, Hkv = 16, 2048, 16, 13, 96, 6, 3
    Tg = T // g
    w = synth.small("split_pass", B=B, T_new=Tg, L=1, k=1, D=512, Hq=Hq, Hkv=Hkv, d=d, ctx=T,
                    dtype="bf16", chan_map=[0])
    print("pass-driver group attention with split ranges", flush=True)
    P = synth.make_params(w, _bias(w))
    Q = synth.make_queries(w)
    Kc = synth._normal((1, B, Hkv, T, d), 1.0, 9501, torch.bfloat16)  # every slot written
    Vc = synth._normal((1, B, Hkv, T, d), 1.0, 9502, torch.bfloat16)
    O = torch.empty((1, B, Tg, Hq * d), dtype=torch.bfloat16, device="cuda")
    wm.channel_attend(_gdims(wm, w, ctx_max=0, S_cap=T, groups=g, group=q), _dev(P), Q.cuda(),
                      [0], None, Kc.cuda(), Vc.cuda(), O)
    torch.cuda.synchronize()
    for b in (0, B - 1):
        sub = _odims(w, B=1, S_cap=T)
        ref = ob.attend(sub, ob._t(P["Kd"]), ob._t(P["Vd"]), ob._t(Q[:, b:b + 1]), [0],
                        torch.zeros(1, dtype=torch.long), ob._t(Kc[:, b:b + 1]),
                        ob._t(Vc[:, b:b + 1]), (g, q)).detach().numpy()
        check_close(O[:, b:b + 1], ref, "bf16", "pass-driver group, sequence %d" % b)
