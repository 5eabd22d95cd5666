"""The benchmark's FLOP model against the per-token decode FLOPs the paper prints (Table 2).

The model counts, per decoded token, the WhiteMatter terms the benchmark uses for its
roofline (router on L' = ceil(L/p) stacked states, the k x L mix, k K/V projections, the
queries, attention over T cached slots) plus the unchanged parts of a Qwen3 block (output
projection and SwiGLU MLP). A vanilla model is the same with one K/V projection per layer
and no router or mix. Table 2 is reproduced to its printed precision.
"""
import json
import os

import pytest

import bench

GOLD = os.path.join(os.path.dirname(__file__), "golden", "table2_decode_gflops.json")


def decode_gflop_per_token(L, D, I, Hq, Hkv, d, T, k=None, p=1):
    o_proj = 2 * Hq * d * D
    mlp = 3 * 2 * D * I
    attn = bench.attn_flops(1, Hq, d, T)
    per_layer = o_proj + mlp + attn
    q = bench.q_flops_per_token(L, Hq, d, D)
    if k is None:
        kv, pool = bench.kv_flops_per_token(L, Hkv, d, D), 0
    else:
        kv = bench.kv_flops_per_token(k, Hkv, d, D)
        pool = bench.router_flops_per_token(L, k, D, p) + bench.mix_flops_per_token(L, k, D)
    return (L * per_layer + q + kv + pool) / 1e9


def _gold():
    with open(GOLD) as f:
        return json.load(f)


@pytest.mark.parametrize("key,L,k", [("vanilla_L16", 16, None), ("vanilla_L24", 24, None),
                                     ("vanilla_L32", 32, None), ("whitematter_L16_k8", 16, 8),
                                     ("whitematter_L16_k16", 16, 16)])
def test_decode_flops_reproduce_table2(key, L, k):
    g = _gold()
    m = g["model"]
    got = decode_gflop_per_token(L, m["D"], m["intermediate"], m["Hq"], m["Hkv"], m["d"], m["T"],
                                 k=k, p=m["p"])
    assert abs(got - g["decode_gflop_per_token"][key]) <= g["printed_precision"], (key, got)


def test_router_subsampling_is_visible_in_table2():
    """Without the p = 2 subsampling the k = 16 router would cost enough to miss the
    printed value, so the table pins L' = ceil(L/p)."""
    g = _gold()
    m = g["model"]
    got = decode_gflop_per_token(16, m["D"], m["intermediate"], m["Hq"], m["Hkv"], m["d"], m["T"],
                                 k=16, p=1)
    assert abs(got - g["decode_gflop_per_token"]["whitematter_L16_k16"]) > g["printed_precision"]


def test_step_cost_of_the_workloads():
    """Whole-step GFLOP of the five workloads (full-sequence passes count the dummy plus the
    strictly earlier slots for every query)."""
    from tests import synth
    want = {"c2_T2048_L12_k12": 1408.8, "c3_T2048_L12_k6": 1129.7, "c4_T4096_L24_k12": 5431.8,
            "c5_decode_S32768": 214.5}
    for name, gf in want.items():
        f, _ = bench.step_cost(synth.WORKLOADS[name])
        assert abs(f / 1e9 - gf) < 0.05, (name, f / 1e9)
