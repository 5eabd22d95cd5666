"""Host-side checks of the C ABI (no GPU needed): every declared symbol is exported,
validation returns the documented error codes before anything is launched, and the
host helpers agree bit-for-bit with the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "whitematter.h")


@pytest.fixture(scope="module")
def wm():
    import paper_2608_18486_amd as wm
    from paper_2608_18486_amd import build
    if not os.path.exists(wm.LIB_PATH):
        build.build()
    wm.lib()
    return wm


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char \*)\s*\*?(wm_\w+)\s*\(", text,
                                 flags=re.M)))


def test_library_exports_every_declared_symbol(wm):
    names = _declared()
    assert len(names) >= 12, names
    for n in names:
        assert hasattr(wm.lib(), n), n
    assert wm.version().startswith("whitematter-gfx950")


def _dims(wm, **kw):
    base = dict(B=2, T_new=16, L=4, k=2, D=64, Hq=4, Hkv=2, d=32, p=1, S_cap=64, ctx_max=8,
                dtype=wm.BF16)
    base.update(kw)
    return wm.make_dims(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(L=0), "ERR_SHAPE"), (dict(L=65, k=2), "ERR_SHAPE"), (dict(k=5), "ERR_SHAPE"),
    (dict(k=0), "ERR_SHAPE"), (dict(D=48), "ERR_SHAPE"), (dict(D=0), "ERR_SHAPE"),
    (dict(Hq=3), "ERR_SHAPE"), (dict(Hkv=0), "ERR_SHAPE"), (dict(d=48), "ERR_SHAPE"),
    (dict(d=128), "ERR_SHAPE"), (dict(d=96, dtype=0), "ERR_SHAPE"), (dict(d=80), "ERR_SHAPE"),
    (dict(p=0), "ERR_SHAPE"), (dict(p=5), "ERR_SHAPE"),
    (dict(dtype=7), "ERR_DTYPE"), (dict(mix_mode=2), "ERR_DTYPE"), (dict(mask_mode=-1), "ERR_DTYPE"),
    (dict(router_mode=3), "ERR_DTYPE"), (dict(router_mode=2), "ERR_SHAPE"),
    (dict(B=-1), "ERR_ARG"), (dict(T_new=-3), "ERR_ARG"), (dict(eps=0.0), "ERR_ARG"),
    (dict(rope_theta=-1.0), "ERR_ARG"), (dict(ctx_max=-1), "ERR_ARG"),
    (dict(ctx_max=60, T_new=5), "ERR_CAPACITY"), (dict(S_cap=0), "ERR_SHAPE"),
    (dict(L=64, k=8, D=1024), "ERR_SHAPE"),
])
def test_validation_error_codes(wm, kw, code):
    d = _dims(wm, **kw)
    chan_map = [l % 2 for l in range(max(d.L, 1))]
    assert wm.validate(d, wm.OP_LAYER_STEP, chan_map) == getattr(wm, code)
    assert wm.workspace_size(_dims(wm, **kw), wm.OP_LAYER_STEP) == 0


@pytest.mark.parametrize("d,dtype", [(32, 0), (32, 1), (64, 0), (64, 1), (96, 1)])
def test_supported_head_dims(wm, d, dtype):
    """Head dims 32 and 64 in either dtype, 96 (the paper's model) in bf16."""
    dims = _dims(wm, d=d, dtype=dtype)
    assert wm.validate(dims, wm.OP_LAYER_STEP, [l % 2 for l in range(4)]) == wm.OK
    assert wm.workspace_size(dims, wm.OP_LAYER_STEP) > 0


def test_capacity_only_matters_for_cache_ops(wm):
    d = _dims(wm, ctx_max=60, T_new=5)
    assert wm.validate(d, wm.OP_ROUTER_MIX) == wm.OK
    assert wm.validate(d, wm.OP_Q_PROJECT) == wm.OK
    assert wm.validate(d, wm.OP_KV_PROJECT) == wm.ERR_CAPACITY
    assert wm.validate(d, wm.OP_CHANNEL_ATTEND, [0, 1, 0, 1]) == wm.ERR_CAPACITY


def test_map_validation(wm):
    d = _dims(wm)
    assert wm.validate(d, wm.OP_LAYER_STEP, [0, 1, 0, 1]) == wm.OK
    assert wm.validate(d, wm.OP_LAYER_STEP, [0, 2, 0, 1]) == wm.ERR_MAP
    assert wm.validate(d, wm.OP_LAYER_STEP, [0, -1, 0, 1]) == wm.ERR_MAP
    assert "chan_map[1]" in wm.last_error()


class _FakeTensor:
    """Stands in for a device tensor in calls that must fail validation before any launch."""

    def __init__(self, addr):
        self.addr = addr

    def is_contiguous(self):
        return True

    def data_ptr(self):
        return self.addr

    def numel(self):
        return 1 << 20


def _fake_params(wm, addr=0x100000):
    return {n: _FakeTensor(addr + 0x1000 * i) for i, n in enumerate(wm.PARAM_NAMES)}


class _P:
    def __init__(self, wm, params):
        self.c = wm.Params(*[params[n].data_ptr() for n in wm.PARAM_NAMES])


def _call(wm, fn, dims, *ptrs, ws=0x400000, ws_bytes=1 << 30, params=None):
    P = _P(wm, params or _fake_params(wm))
    L = wm.lib()
    f = getattr(L, fn)
    return f(ctypes.byref(dims), ctypes.byref(P.c), *ptrs, ws, ws_bytes, None)


def test_entry_points_reject_bad_pointers_before_launch(wm):
    d = _dims(wm)
    m = (ctypes.c_int32 * 4)(0, 1, 0, 1)
    good = 0x200000
    # NULL and misaligned tensors
    assert _call(wm, "wm_router_mix", d, None, None, good) == wm.ERR_ARG
    assert _call(wm, "wm_router_mix", d, good + 8, None, good) == wm.ERR_ARG
    assert _call(wm, "wm_kv_project", d, good, None, None, good) == wm.ERR_ARG
    assert _call(wm, "wm_q_project", d, good, None, None) == wm.ERR_ARG
    assert _call(wm, "wm_channel_attend", d, good, m, None, good, good, None) == wm.ERR_ARG
    assert _call(wm, "wm_layer_step", d, good, None, None, good, good, good) == wm.ERR_ARG
    # document arrays: NULL or misaligned (the other arguments are valid)
    assert _call(wm, "wm_channel_attend_doc", d, good, m, None, None, good, good, good) == \
        wm.ERR_ARG
    assert "doc_start" in wm.last_error()
    assert _call(wm, "wm_layer_step_doc", d, good, m, None, good + 2, good, good, good) == \
        wm.ERR_ARG
    assert "doc_start" in wm.last_error()
    # NULL parameter
    bad = _fake_params(wm)
    bad["Wq"] = _FakeTensor(0)
    assert _call(wm, "wm_q_project", d, good, None, good, params=bad) == wm.ERR_ARG
    assert "Wq" in wm.last_error()
    # workspace: NULL, misaligned, too small
    assert _call(wm, "wm_layer_step", d, good, m, None, good, good, good, ws=0) == wm.ERR_WORKSPACE
    assert _call(wm, "wm_layer_step", d, good, m, None, good, good, good, ws=0x400010) == \
        wm.ERR_WORKSPACE
    need = wm.workspace_size(d, wm.OP_LAYER_STEP)
    assert _call(wm, "wm_layer_step", d, good, m, None, good, good, good, ws_bytes=need - 1) == \
        wm.ERR_WORKSPACE
    # map and capacity errors surface through the entry points too
    m_bad = (ctypes.c_int32 * 4)(0, 3, 0, 1)
    assert _call(wm, "wm_layer_step", d, good, m_bad, None, good, good, good) == wm.ERR_MAP
    d_cap = _dims(wm, ctx_max=60)
    assert _call(wm, "wm_kv_project", d_cap, good, None, good, good) == wm.ERR_CAPACITY


def test_empty_inputs_are_a_no_op(wm):
    for kw in (dict(B=0), dict(T_new=0)):
        d = _dims(wm, **kw)
        assert wm.workspace_size(d, wm.OP_LAYER_STEP) == 0
        m = (ctypes.c_int32 * 4)(0, 1, 0, 1)
        # no pointers at all: an empty call returns before touching any of them
        assert _call(wm, "wm_layer_step", d, None, m, None, None, None, None, ws=0, ws_bytes=0) == wm.OK


def test_workspace_sizes_grow_with_the_problem(wm):
    small = wm.workspace_size(_dims(wm, T_new=16), wm.OP_LAYER_STEP)
    big = wm.workspace_size(_dims(wm, T_new=32, S_cap=128), wm.OP_LAYER_STEP)
    assert 0 < small < big
    for op in range(5):
        assert wm.workspace_size(_dims(wm), op) >= 0


def test_channel_groups_match_oracle(wm, oracle_lib):
    rng = np.random.default_rng(0)
    for L in (1, 4, 5, 12, 24, 64):
        for k in sorted({1, 2, max(1, L // 2), L}):
            maps = [[l % k for l in range(L)], [l * k // L for l in range(L)],
                    rng.integers(0, k, size=L).tolist()]
            for m in maps:
                off, mem = wm.channel_groups(L, k, m)
                o_off, o_mem = oracle_lib.channel_groups(L, k, m)
                assert off == o_off.tolist() and mem == o_mem.tolist()
    with pytest.raises(wm.WMError):
        wm.channel_groups(4, 2, [0, 1, 2, 0])


def test_init_bias_and_default_map_match_oracle(wm, oracle_lib):
    for L in (1, 2, 4, 5, 12, 16, 24):
        for k in range(1, L + 1):
            assert wm.init_bias(L, k) == oracle_lib.init_bias(L, k).tolist()
            assert wm.default_map(L, k) == [l % k for l in range(L)]
    with pytest.raises(wm.WMError):
        wm.init_bias(4, 5)


def test_calibration_rejects_bad_arguments(wm):
    L = wm.lib()
    assert L.wm_calibrate_mfma(0, 10, 0, None, None) == wm.ERR_ARG
    assert L.wm_calibrate_mfma(10, 0, 0, None, None) == wm.ERR_ARG
    assert L.wm_calibrate_mfma(10, 10, 2, None, None) == wm.ERR_ARG
    assert "operands" in wm.last_error()
    assert L.wm_calibrate_mfma(10, 10, 1, None, None) == wm.ERR_ARG
    assert "sink" in wm.last_error()


def test_read_calibration_rejects_bad_arguments(wm):
    L = wm.lib()
    assert L.wm_calibrate_read(None, 16, None, None) == wm.ERR_ARG
    # misaligned buffer: rejected on the host, nothing is launched or read
    assert L.wm_calibrate_read(17, 16, 16, None) == wm.ERR_ARG
    assert L.wm_calibrate_read(32, 0, 16, None) == wm.ERR_ARG
    assert L.wm_calibrate_read(32, 24, 16, None) == wm.ERR_ARG


@pytest.mark.parametrize("kw,op,code", [
    (dict(groups=-1), "OP_LAYER_STEP", "ERR_ARG"),
    (dict(groups=4, group=4), "OP_LAYER_STEP", "ERR_ARG"),
    (dict(groups=4, group=-1), "OP_POOL", "ERR_ARG"),
    # group q of g: the last token sits at q + g (T_new - 1); ctx_max 8 + 3 + 4 * 15 + 1 > 64
    (dict(groups=4, group=3), "OP_LAYER_STEP", "ERR_CAPACITY"),
    (dict(groups=4, group=3), "OP_POOL", "ERR_CAPACITY"),
    (dict(groups=4, group=3, ctx_max=0, S_cap=63), "OP_LAYER_ATTEND", "ERR_CAPACITY"),
    (dict(groups=3, ctx_max=0), "OP_PASSES", "ERR_SHAPE"),        # T_new not a multiple of g
    (dict(groups=4, group=1, ctx_max=0), "OP_PASSES", "ERR_ARG"),  # the driver runs all groups
    (dict(groups=4, S_cap=128), "OP_PASSES", "ERR_ARG"),           # sequences start empty
])
def test_group_validation(wm, kw, op, code):
    d = _dims(wm, **kw)
    assert wm.validate(d, getattr(wm, op), [l % 2 for l in range(4)]) == getattr(wm, code)


def test_group_span_fits_exactly(wm):
    """Group q of g with T_new tokens covers positions up to q + g (T_new - 1): with no
    cached context that must be below S_cap, and the bound is exact."""
    for g, q in ((4, 0), (4, 3), (16, 7)):
        last = q + g * 15
        ok = _dims(wm, groups=g, group=q, ctx_max=0, S_cap=last + 1)
        bad = _dims(wm, groups=g, group=q, ctx_max=0, S_cap=last)
        for op in ("OP_LAYER_STEP", "OP_POOL", "OP_LAYER_ATTEND", "OP_KV_PROJECT"):
            assert wm.validate(ok, getattr(wm, op), [0, 1, 0, 1]) == wm.OK, (g, q, op)
            assert wm.validate(bad, getattr(wm, op), [0, 1, 0, 1]) == wm.ERR_CAPACITY
    # zero groups means contiguous tokens, like one group
    assert wm.validate(_dims(wm, groups=0), wm.OP_LAYER_STEP, [0, 1, 0, 1]) == wm.OK


def test_new_entry_points_reject_bad_arguments_before_launch(wm):
    d = _dims(wm, ctx_max=0, groups=4)
    assert wm.validate(d, wm.OP_PASSES, [0, 1, 0, 1]) == wm.OK
    assert wm.workspace_size(d, wm.OP_PASSES) > 0
    # the driver's workspace holds every group's states plus one group's scratch
    es = 2
    assert wm.workspace_size(d, wm.OP_PASSES) >= d.B * d.T_new * d.L * d.D * es
    with pytest.raises(wm.WMError) as e:
        wm.prefill_passes(d, None, None, None, [0, 1, 0, 1], 0, None, None, None)
    assert e.value.code == wm.ERR_ARG  # passes < 1
    with pytest.raises(wm.WMError) as e:
        wm.layer_attend(_dims(wm), None, 4, None, [0, 1, 0, 1], None, None, None, None)
    assert e.value.code == wm.ERR_ARG  # layer outside [0, L)
    with pytest.raises(wm.WMError) as e:
        wm.pool(_dims(wm), None, None, None, None, None)
    assert e.value.code == wm.ERR_ARG  # params NULL


def test_attention_backward_rejects_unsupported_calls_before_launch(wm):
    """The attention gradients cover bf16 full-sequence calls at head dims 64 and 96, over
    contiguous tokens or one strided group; everything else is refused on the host with its
    own code."""
    cmap = [0, 1, 0, 1]
    args = (None, None, cmap, None, None, None, None, None, None, None, None, None, None)

    def call(**kw):
        with pytest.raises(wm.WMError) as e:
            wm.channel_attend_backward(_dims(wm, **kw), *args)
        return e.value.code

    assert call(d=64, dtype=wm.F32) == wm.ERR_DTYPE
    assert call(d=32) == wm.ERR_SHAPE
    assert call(d=64, T_new=4) == wm.ERR_SHAPE
    assert call(d=64, groups=2, group=2) == wm.ERR_ARG  # group outside [0, g)
    assert call(d=64) == wm.ERR_ARG            # params NULL
    # four floats per query row of workspace
    d = _dims(wm, d=64)
    assert wm.workspace_size(d, wm.OP_ATTEND_BACKWARD) >= 16 * d.L * d.B * d.Hq * d.T_new


def test_step_gradients_reject_unsupported_calls_before_launch(wm):
    """The queries', pool's and step's gradients: bf16, head dims 64 and 96, contiguous
    tokens or one strided group, D <= 4608, the step's only with T_new > 4; NULL parameters or gradient pointers
    are refused on the host."""
    def code(fn, *args, **kw):
        with pytest.raises(wm.WMError) as e:
            fn(_dims(wm, **kw), *args)
        return e.value.code

    q = (None, None, None, None, None, None)
    p = (None, None, None, None, None, None, None)
    s = (None, None, [0, 1, 0, 1], None, None, None, None, None, None, None, None, None)
    for fn, args in ((wm.q_project_backward, q), (wm.pool_backward, p),
                     (wm.layer_step_backward, s)):
        assert code(fn, *args, d=64, dtype=wm.F32) == wm.ERR_DTYPE
        assert code(fn, *args, d=32) == wm.ERR_SHAPE
        assert code(fn, *args, d=64, groups=2, group=2) == wm.ERR_ARG
        assert code(fn, *args, d=64) == wm.ERR_ARG  # params NULL
    assert code(wm.layer_step_backward, *s, d=64, T_new=4) == wm.ERR_SHAPE
    # the workspace grows with the tokens and holds at least the recomputed queries
    d = _dims(wm, d=64)
    for op in (wm.OP_Q_BACKWARD, wm.OP_POOL_BACKWARD, wm.OP_STEP_BACKWARD):
        assert wm.workspace_size(d, op) > 0
    assert wm.workspace_size(d, wm.OP_STEP_BACKWARD) >= 6 * d.L * d.B * d.Hq * d.T_new * d.d


def test_passes_backward_rejects_unsupported_calls_before_launch(wm):
    """The training passes: passes >= 1, 1 <= n_grad <= passes, bf16, T a multiple of the
    groups with more than 4 tokens per group (the gradients' full-sequence kernels); each is
    refused on the host with its own code, before any pointer is needed."""
    cmap = [0, 1, 0, 1]

    def code(passes, n_grad, **kw):
        kw = dict(dict(d=64, T_new=48, S_cap=48, ctx_max=0), **kw)
        with pytest.raises(wm.WMError) as e:
            wm.prefill_passes_backward(_dims(wm, **kw), None, None, None, cmap, passes, n_grad,
                                       None, None, None, None)
        return e.value.code

    assert code(0, 1) == wm.ERR_ARG
    assert code(3, 0) == wm.ERR_ARG
    assert code(3, 4) == wm.ERR_ARG
    assert code(3, 2, dtype=wm.F32) == wm.ERR_DTYPE
    assert code(3, 2, groups=5) == wm.ERR_SHAPE    # 48 tokens are not 5 groups
    assert code(3, 2, groups=12) == wm.ERR_SHAPE   # 4 tokens per group
    assert code(3, 2, groups=8) == wm.ERR_ARG      # 6 per group: params NULL comes next
    assert code(3, 2, groups=8, group=1) == wm.ERR_ARG  # the driver runs every group
    # the workspace holds each window step's states, outputs and overwritten slots
    d = _dims(wm, d=64, T_new=48, S_cap=48, ctx_max=0, groups=8)
    w1, w2 = wm.passes_backward_workspace(d, 1), wm.passes_backward_workspace(d, 2)
    assert 0 < w1 < w2
    assert wm.passes_backward_workspace(d, 0) == 0
