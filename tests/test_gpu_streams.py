"""The boundary's call conventions on the GPU: calls keep no state between them, so two
host threads may run steps on two streams at once (one of them capturing its step into a
graph), and a ctx_len entry outside its documented range gives unspecified values for
that sequence but no access outside the caller's buffers."""
import threading

import numpy as np
import pytest
import torch

import oracle
from tests import synth
from tests.parity import _bias, _dev, _f64, _gdims, _odims, check_close, wm  # noqa: F401

pytestmark = pytest.mark.gpu


def _case(wm, w, seed_shift=0):
    P = synth.make_params(w, _bias(w))
    H = synth.make_states(w, sub=20 + seed_shift)
    return {"w": w, "P": P, "Pd": wm.ParamSet(_dev(P)), "H": H, "Hd": H.cuda(),
            "dims": _gdims(wm, w)}


def _buffers(wm, c):
    w = c["w"]
    Kc = torch.full((w.k, w.B, w.Hkv, w.S_cap, w.d), float("nan"), dtype=w.torch_dtype,
                    device="cuda")
    return {"Kc": Kc, "Vc": torch.full_like(Kc, float("nan")),
            "O": torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype,
                             device="cuda"),
            "ws": wm.workspace(c["dims"], wm.OP_LAYER_STEP)}


def _step(wm, c, buf, stream):
    w = c["w"]
    wm.layer_step(c["dims"], c["Pd"], c["Hd"], w.chan_map, None, buf["Kc"], buf["Vc"],
                  buf["O"], ws=buf["ws"], stream=stream)


def test_two_threads_two_streams_one_capturing(wm):
    """Thread A runs eager steps of one workload on its stream while thread B captures a
    step of another workload into a graph on a second stream; the graph is then replayed
    several times with eager work and synchronisations between the replays. Every result
    equals the same step run alone, bit for bit, and the lone runs match the oracle."""
    a = _case(wm, synth.small("thr_a", B=2, T_new=150, L=4, k=2, D=128, Hq=2, Hkv=2, d=64))
    b = _case(wm, synth.small("thr_b", B=1, T_new=200, L=6, k=3, D=192, Hq=6, Hkv=3, d=96,
                              p=2), seed_shift=1)
    s_ref = torch.cuda.Stream()
    ref = {}
    for name, c in (("a", a), ("b", b)):
        buf = _buffers(wm, c)
        with torch.cuda.stream(s_ref):
            _step(wm, c, buf, s_ref)
        s_ref.synchronize()
        ref[name] = buf
        w = c["w"]
        Ko, Vo = oracle.empty_cache(_odims(w))
        Oo = oracle.layer_step(_odims(w), c["P"], c["H"], w.chan_map, None, Ko, Vo)
        check_close(buf["O"], Oo, w.dtype, "lone step %s" % name)

    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    buf_a, buf_b = _buffers(wm, a), _buffers(wm, b)
    graph = torch.cuda.CUDAGraph()
    errors = []

    def run_a():
        try:
            with torch.cuda.stream(sa):
                for _ in range(6):
                    _step(wm, a, buf_a, sa)
            sa.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    def run_b():
        try:
            with torch.cuda.graph(graph, stream=sb, capture_error_mode="thread_local"):
                _step(wm, b, buf_b, sb)
        except Exception as e:
            errors.append(e)

    ta, tb = threading.Thread(target=run_a), threading.Thread(target=run_b)
    ta.start()
    tb.start()
    ta.join()
    tb.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for key in ("O", "Kc", "Vc"):
        assert torch.equal(buf_a[key].nan_to_num(7.0), ref["a"][key].nan_to_num(7.0)), key
    for rep in range(3):
        for key in ("O", "Kc", "Vc"):
            buf_b[key].fill_(-1.0)  # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for key in ("O", "Kc"):
            got = buf_b[key]
            want = ref["b"][key]
            # slots the step does not write stay as the fill left them
            if key == "Kc":
                got, want = got[:, :, :, :b["w"].T_new], want[:, :, :, :b["w"].T_new]
            assert torch.equal(got, want), "replay %d: %s differs" % (rep, key)


@pytest.mark.parametrize("T_new", [150, 1])
@pytest.mark.parametrize("d", [64, 96, 32])
def test_out_of_range_ctx_len_stays_in_bounds(wm, T_new, d):
    """ctx_len entries far below 0 and past the cache: the kernels clamp them, so every
    write lands inside each sequence's own cache slice and the outputs are finite. A
    guard slice on either side of the cache (the caller's buffer is split into three)
    must come back unchanged."""
    dtype = "f32" if d == 32 else "bf16"
    w = synth.small("ctx_oob_d%d" % d, B=3, T_new=T_new, L=3, k=2, D=96 if d == 96 else 64,
                    Hq=2, Hkv=1, d=d, ctx=200, dtype=dtype)
    c = _case(wm, w)
    shape = (w.k, w.B, w.Hkv, w.S_cap, w.d)
    n = int(np.prod(shape))
    for docs in (None, synth.make_doc_start(w, torch.tensor([0, 0, 0]), mean_len=20.0)):
        K3 = torch.zeros(3 * n, dtype=w.torch_dtype, device="cuda")  # guard | cache | guard
        V3 = torch.zeros_like(K3)
        K3[:n].fill_(5.0)
        K3[2 * n:].fill_(5.0)
        V3[:n].fill_(5.0)
        V3[2 * n:].fill_(5.0)
        Kc, Vc = K3[n:2 * n].view(shape), V3[n:2 * n].view(shape)
        ctx = torch.tensor([-1000000, 50, 1 << 30], dtype=torch.int32, device="cuda")
        O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device="cuda")
        wm.layer_step(c["dims"], c["Pd"], c["Hd"], w.chan_map, ctx, Kc, Vc, O,
                      doc_start=None if docs is None else docs.cuda())
        torch.cuda.synchronize()
        assert torch.isfinite(O).all()
        for T3 in (K3, V3):
            assert (T3[:n] == 5.0).all() and (T3[2 * n:] == 5.0).all()
