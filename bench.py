"""Benchmark of the fused WhiteMatter step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step = one wm_layer_step call: pool the new tokens into the channel cache
(row norms, router, mix, per-channel K/V projection with key norm + RoPE),
project every consumer's queries, and run every consumer's attention over its
channel. The default workload is the largest full-sequence (Jacobi) pass that
fits one GPU: B = 4 sequences of T = 4096 tokens, L = 24, k = 12, D = 1024, 16
heads of 64 (bf16). Inputs are synthetic and already resident in HBM when the
timed region starts.

Prints one JSON line: tokens/s of the step (K timed steps of wm_layer_step on
one stream), the roofline of the dominant kernel (timed with HIP events that
the library records at the phase boundaries of K more steps), the step against
its fused minimum, the 32768-context decode step timed in the same run, and the
CPU oracle's tokens/s on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}

WORKLOAD_LABEL = {
    "c1_tiny_f32": "full-sequence pass, B1 T64 L4 k2 D64 2x32, fp32",
    "c2_T2048_L12_k12": "full-sequence pass, B8 T2048 L12 k12 D768 12x64, bf16, map l->l",
    "c3_T2048_L12_k6": "full-sequence pass, B8 T2048 L12 k6 D768 12x64, bf16, map l->l//2",
    "c4_T4096_L24_k12": "full-sequence pass, B4 T4096 L24 k12 D1024 16x64, bf16, map l->l%12",
    "c5_decode_S32768": "decode step, B64 ctx32768 L24 k12 D1024 16x64, bf16, map l->l%12",
}
for _k in (1, 2, 4, 8, 12, 16):
    WORKLOAD_LABEL["paper_T2048_L16_k%d" % _k] = (
        "full-sequence pass, the paper's model shape: B16 T2048 L16 k%d D512 6q/3kv x96, p2, "
        "bf16, map l->l%%%d" % (_k, _k))
for _k, _tag, _what in ((16, "static", "static mixing weights, no router"),
                        (1, "static", "static mixing weights, no router"),
                        (16, "nofeedback", "no deep-to-shallow feedback")):
    WORKLOAD_LABEL["paper_T2048_L16_k%d_%s" % (_k, _tag)] = (
        "full-sequence pass, the paper's model shape, ablation: %s: B16 T2048 L16 k%d D512 "
        "6q/3kv x96, p2, bf16, map l->l%%%d" % (_what, _k, _k))
del _tag, _what
for _k in (8, 16):
    WORKLOAD_LABEL["paper_T2048_L16_k%d_docs" % _k] = (
        "full-sequence pass, the paper's model shape with the document mask (packed documents "
        "of mean length 512): B16 T2048 L16 k%d D512 6q/3kv x96, p2, bf16, map l->l%%%d"
        % (_k, _k))
del _k


# ------------------------------------------------------------ cost model
# Algorithmic work of the step (what the method must compute / move; matrix
# multiplies count 2 flops per multiply-add).

def router_flops_per_token(L, k, D, p):
    """Both branches: W_alpha [kL x L'D] times the stacked normed states."""
    return 2 * 2 * k * L * ((L + p - 1) // p) * D


def mix_flops_per_token(L, k, D):
    """Both branches: a [k x L] by [L x D] product per token."""
    return 2 * 2 * k * L * D


def kv_flops_per_token(k, Hkv, d, D):
    """W^K_j and W^V_j for every channel j."""
    return 2 * 2 * k * Hkv * d * D


def q_flops_per_token(L, Hq, d, D):
    return 2 * L * Hq * d * D


def attn_flops(L, Hq, d, visible_pairs):
    """QK^T and PV: 4 d flops per (query head, visible slot) pair, per consumer layer."""
    return 4 * d * Hq * L * visible_pairs


def visible_pairs(w, docs=None):
    """Sum over queries of the slots each one reads: dummy + slots < t in the paper's
    mask (t + 1 in total), the same count as slots <= t without the dummy; with the
    document mask, dummy + slots of the query's document before it."""
    if docs is None:
        return w.B * sum(w.ctx + i + 1 for i in range(w.T_new))
    import numpy as np
    pos = w.ctx + np.arange(w.T_new)[None, :]
    return int((pos - np.asarray(docs) + 1).sum())


def router_mode_of(w):
    from tests import synth
    return synth.ROUTER_MODE.get(w.name, 0)


def phase_costs(w, docs=None):
    """Per-phase (flops, HBM bytes) of one step."""
    es = 4 if w.dtype == "f32" else 2
    N, L, k, D, Hq, Hkv, d, p = w.N, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, w.p
    Lp = (L + p - 1) // p
    mode = router_mode_of(w)
    if mode == 1:     # static weights: no router
        router = (0, 0)
    elif mode == 2:   # no feedback: channel j's router reads the stacked layers <= j
        sel = [L - 1 - p * m for m in range(Lp)]
        blocks = sum(sum(1 for s in sel if s <= j) for j in range(k))
        router = (N * 4 * L * blocks * D, N * Lp * D * es + 2 * L * blocks * D * es)
    else:
        router = (N * router_flops_per_token(L, k, D, p), N * Lp * D * es + 2 * k * L * Lp * D * es)
    H_bytes = N * L * D * es
    cache_write = 2 * k * N * Hkv * d * es
    used = len(set(w.chan_map))
    cache_read = 2 * used * w.B * Hkv * (w.ctx + w.T_new) * d * es
    return {
        "norms": (0, H_bytes),
        "router": router,
        "mix": (N * mix_flops_per_token(L, k, D), H_bytes + 2 * k * N * D * es),
        "kv_project": (N * kv_flops_per_token(k, Hkv, d, D),
                       2 * k * N * D * es + 2 * k * Hkv * d * D * es + cache_write),
        "q_project": (N * q_flops_per_token(L, Hq, d, D),
                      H_bytes + L * Hq * d * D * es + L * N * Hq * d * es),
        "attend": (attn_flops(L, Hq, d, visible_pairs(w, docs)),
                   L * N * Hq * d * es + cache_read + L * N * Hq * d * es),
    }


def fused_min_ms(w, docs=None):
    """The step's fused minimum: four phases, each at the slower of its flops at the bf16
    (or fp32) matrix peak and its minimum HBM bytes at 8 TB/s, with the layer states read
    once (by the pool side), the mixed channels and the queries kept on chip:
      mix side   router + mix flops; H and the router weights
      K/V        projection flops; its weights and the cache write
      Q          projection flops; its weights
      attention  flops; each channel's cache read once, O written."""
    c = phase_costs(w, docs)
    es = 4 if w.dtype == "f32" else 2
    peak = PEAK_TFLOPS[w.dtype] * 1e12
    bw = PEAK_HBM_GBS * 1e9
    used = len(set(w.chan_map))
    router_w = 0 if router_mode_of(w) == 1 else 2 * w.k * w.L * ((w.L + w.p - 1) // w.p) * w.D
    phases = [
        (c["router"][0] + c["mix"][0], (w.N * w.L * w.D + router_w) * es),
        (c["kv_project"][0], (2 * w.k * w.Hkv * w.d * w.D + 2 * w.k * w.N * w.Hkv * w.d) * es),
        (c["q_project"][0], w.L * w.Hq * w.d * w.D * es),
        (c["attend"][0], (2 * used * w.B * w.Hkv * (w.ctx + w.T_new) * w.d
                          + w.L * w.N * w.Hq * w.d) * es),
    ]
    return sum(max(f / peak, b / bw) for f, b in phases) * 1e3


def step_cost(w, docs=None):
    c = phase_costs(w, docs)
    router_w = 0 if router_mode_of(w) == 1 else 2 * w.k * w.L * ((w.L + w.p - 1) // w.p) * w.D
    min_bytes = (w.N * w.L * w.D + router_w
                 + 2 * w.k * w.Hkv * w.d * w.D + w.L * w.Hq * w.d * w.D) * (
        4 if w.dtype == "f32" else 2)
    es = 4 if w.dtype == "f32" else 2
    min_bytes += 2 * w.k * w.N * w.Hkv * w.d * es  # cache write
    used = len(set(w.chan_map))
    min_bytes += 2 * used * w.B * w.Hkv * (w.ctx + w.T_new) * w.d * es  # each channel read once
    min_bytes += w.L * w.N * w.Hq * w.d * es  # O
    return sum(f for f, _ in c.values()), min_bytes


# ------------------------------------------------------------ HIP events

class HipEvents:
    """hipEvent_t handles from the HIP runtime torch has loaded (the library uses the same)."""

    def __init__(self):
        path = None
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    path = line.split()[-1]
                    break
        if path is None:
            raise RuntimeError("the HIP runtime is not loaded")
        self.hip = ctypes.CDLL(path)
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def create(self) -> int:
        ev = ctypes.c_void_p()
        rc = self.hip.hipEventCreate(ctypes.byref(ev))
        if rc != 0:
            raise RuntimeError("hipEventCreate failed: %d" % rc)
        return ev.value

    def record(self, ev, stream) -> None:
        rc = self.hip.hipEventRecord(ev, stream)
        if rc != 0:
            raise RuntimeError("hipEventRecord failed: %d" % rc)

    def elapsed_ms(self, a, b) -> float:
        ms = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b)
        if rc != 0:
            raise RuntimeError("hipEventElapsedTime failed: %d" % rc)
        return ms.value

    def destroy(self, ev):
        self.hip.hipEventDestroy(ev)


# ------------------------------------------------------------ traffic

def _strip_comments(src: str) -> str:
    """The code of a C++/HIP source without its comments and blank lines (string literals
    in these sources hold no comment markers)."""
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return "\n".join(ln.rstrip() for ln in src.splitlines() if ln.strip())


KERNEL_SOURCES = {
    "attend": ("wm_attend.hip", "wm_device.hpp", "wm_frag.hpp"),
}
POOL_SOURCES = ("wm_pool.hip", "wm_gemm.hpp", "wm_device.hpp")


def _kernel_source_hash(phase=None):
    """Hash of the code a phase's kernels are built from (comments and blank lines
    excluded), so counters taken on one build stay attached to that kernel until its own
    code changes. phase=None hashes the whole library."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_18486_amd", "csrc")
    names = sorted(os.listdir(csrc)) if phase is None else KERNEL_SOURCES.get(phase, POOL_SOURCES)
    for name in names:
        with open(os.path.join(csrc, name), encoding="utf-8") as f:
            h.update(name.encode() + _strip_comments(f.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    """HBM bytes per launch from committed rocprofv3 FETCH_SIZE/WRITE_SIZE counters, if they
    were taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    ent = rec.get(workload, {}).get(kernel)
    if not ent or ent.get("source_hash") != _kernel_source_hash(kernel):
        return None
    return ent.get("bytes_per_launch")


# ------------------------------------------------------------ CPU baseline

def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            return next(ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name"))
    except (OSError, StopIteration):
        return "unknown"


def cpu_baseline(w, P, H_cpu, cache_dev, docs=None, budget_tokens=2 * 2048):
    """The oracle, as it stands, on a bounded sample (about 10-30 s on 16 host threads).

    Small steps (at most budget_tokens tokens in up to 8 sequences) run whole. Larger
    ones run one sequence: the pool of all its tokens (every query reads the whole cache
    before it), then the queries and attention of 128 evenly spaced positions over all
    consumers and heads; that part is scaled to all positions (a position's attention
    cost grows linearly with it, so evenly spaced positions give its mean)."""
    import numpy as np

    import oracle
    from tests import synth

    oracle.build(force=False)
    nseq = min(w.B, 8)
    whole = nseq * w.T_new <= budget_tokens or w.T_new <= 4
    if not whole:
        nseq = 1
    w1 = synth.Workload(w.name, nseq, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, w.ctx, w.dtype,
                        w.chan_map, w.p, w.seed)
    dm = oracle.Dims(B=nseq, T_new=w.T_new, L=w.L, k=w.k, D=w.D, Hq=w.Hq, Hkv=w.Hkv, d=w.d,
                     p=w.p, S_cap=w.ctx + w.T_new, router_mode=router_mode_of(w))
    PP = oracle.Params(P)
    Kc, Vc = oracle.empty_cache(dm)
    if w.ctx:
        Kc[:, :, :, :w.ctx] = cache_dev[0][:, :nseq, :, :w.ctx].double().cpu().numpy()
        Vc[:, :, :, :w.ctx] = cache_dev[1][:, :nseq, :, :w.ctx].double().cpu().numpy()
    Hs = H_cpu[:nseq]
    ctx = np.full(nseq, w.ctx, dtype=np.int32)
    dsub = None if docs is None else docs[:nseq]
    if whole:
        t0 = time.perf_counter()
        oracle.layer_step(dm, PP, Hs, w.chan_map, ctx, Kc, Vc, doc_start=dsub)
        dt = time.perf_counter() - t0
        toks = nseq * w.T_new
        sample = ("%d of %d sequences (%d tokens), whole step (pool, queries, attention over "
                  "%d cached + new slots), %.1f s" % (nseq, w.B, toks, w.ctx, dt))
        value = toks / dt
    else:
        npos = 128
        pos = sorted({int(round(x)) for x in np.linspace(0, w.T_new - 1, npos)})
        rows = [l * w.T_new + t for l in range(w.L) for t in pos]
        t0 = time.perf_counter()
        oracle.pool(dm, PP, Hs, ctx, Kc, Vc)
        t1 = time.perf_counter()
        Q = oracle.q_project(dm, PP, Hs, ctx, pos)
        oracle.channel_attend(dm, PP, Q, w.chan_map, ctx, Kc, Vc, rows, doc_start=dsub)
        t2 = time.perf_counter()
        t_seq = (t1 - t0) + (t2 - t1) * w.T_new / len(pos)
        value = w.T_new / t_seq
        sample = ("1 of %d sequences: pool of all %d tokens (%.1f s), queries and attention of "
                  "%d evenly spaced positions over all %d consumers and %d heads (%.1f s), "
                  "scaled to %d positions: %.1f s per sequence"
                  % (w.B, w.T_new, t1 - t0, len(pos), w.L, w.Hq, t2 - t1, w.T_new, t_seq))
    return {"value": value, "unit": "tokens/s", "cores": oracle.num_threads(), "kind": "oracle",
            "cpu": _cpu_model(), "sample": sample}


# ------------------------------------------------------------ main

def measure_ceilings(wm, torch, dev, stream):
    """On-box ceilings reported beside the published peaks (best of several runs): the
    library's read-only stream over 1 GiB, a plain 1 GiB device-to-device copy (bytes read
    + written per second) and the library's matrix-core loop (bf16 flop per second on
    every CU)."""
    def timed(fn, reps):
        best = float("inf")
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            b.synchronize()
            best = min(best, a.elapsed_time(b) * 1e-3)
        return best
    n = 1 << 28
    x = torch.ones(n, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    t_copy = timed(lambda: y.copy_(x), 6)
    del x, y
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    xr = torch.ones(4 * n, dtype=torch.float32, device=dev)  # 4 GiB, far past the caches
    t_read = timed(lambda: wm.calibrate_read(xr, sink, stream), 4)
    del xr
    blocks, iters = 2048, 16384
    wm.calibrate_mfma(blocks, 64, sink, stream)
    t_mfma = timed(lambda: wm.calibrate_mfma(blocks, iters, sink, stream), 4)
    wm.calibrate_mfma(blocks, 64, sink, stream, random_operands=True)
    t_mfma_r = timed(lambda: wm.calibrate_mfma(blocks, iters, sink, stream,
                                               random_operands=True), 4)
    return {"hbm_read_gbs": round(16 * n / t_read / 1e9, 1),
            "hbm_copy_gbs": round(2 * 4 * n / t_copy / 1e9, 1),
            "mfma_bf16_tflops": round(blocks * iters * 2 ** 20 / t_mfma / 1e12, 1),
            "mfma_bf16_tflops_random_operands": round(blocks * iters * 2 ** 20 / t_mfma_r / 1e12,
                                                      1),
            "method": "best of 4 runs of wm_calibrate_read over 4 GiB, of 6 copies of 1 GiB "
                      "(read + written bytes) and of 4 launches of wm_calibrate_mfma(2048 "
                      "blocks, 16384 iterations) on constant and on random operands, "
                      "event-timed"}


def blas_reference(w, log):
    """Plain batched GEMMs of the projections' shapes through torch.bmm (no norms, RoPE or
    cache layout), timed with events: what the vendor library reaches on these shapes."""
    import torch

    cases = [("K/V projection", 2 * w.k, w.B * w.T_new, w.Hkv * w.d, w.D),
             ("Q projection", w.L, w.B * w.T_new, w.Hq * w.d, w.D)]
    for name, G, M, N, K in cases:
        x = torch.randn(G, M, K, device="cuda", dtype=torch.bfloat16)
        wt = torch.randn(G, K, N, device="cuda", dtype=torch.bfloat16).contiguous()
        o = torch.empty(G, M, N, device="cuda", dtype=torch.bfloat16)
        for _ in range(3):
            torch.bmm(x, wt, out=o)
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(20):
            torch.bmm(x, wt, out=o)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / 20
        log("bench: torch.bmm reference, %s (%d x [%d x %d] x [%d x %d]): %.3f ms, %.1f TFLOP/s"
            % (name, G, M, K, K, N, ms, 2.0 * G * M * N * K / ms / 1e9))
        del x, wt, o


def decode_step(wm, torch, np, synth, hip, dev, stream, log, steps=10):
    """The 32768-context decode step (B = 64 new tokens appended to 12 channels, 24
    consumers attend; bf16), event-timed: ms per step, tokens/s and the attention's
    share of the HBM peak over its algorithmic bytes (each channel's cache read once)."""
    w = synth.WORKLOADS["c5_decode_S32768"]
    log("bench: decode step %s" % w.name)
    P = wm.ParamSet({k: v.to(dev) for k, v in
                     synth.make_params(w, np.asarray(wm.init_bias(w.L, w.k))).items()})
    H = synth.make_states(w).to(dev)
    Kc, Vc = synth.make_cache_device(w, device=dev)
    ctx = torch.full((w.B,), w.ctx, dtype=torch.int32, device=dev)
    O = torch.empty((w.L, w.B, 1, w.Hq * w.d), dtype=w.torch_dtype, device=dev)
    dims = wm.make_dims(w.B, 1, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, p=w.p, S_cap=w.S_cap,
                        ctx_max=w.ctx, dtype=wm.BF16)
    ws = wm.workspace(dims, wm.OP_LAYER_STEP, dev)
    for _ in range(3):
        wm.layer_step(dims, P, H, w.chan_map, ctx, Kc, Vc, O, ws=ws, stream=stream)
    torch.cuda.synchronize()
    ev = [hip.create() for _ in range(steps + 1)]
    hip.record(ev[0], stream.cuda_stream)
    for s in range(steps):
        wm.layer_step(dims, P, H, w.chan_map, ctx, Kc, Vc, O, ws=ws, stream=stream)
        hip.record(ev[s + 1], stream.cuda_stream)
    torch.cuda.synchronize()
    ms = [hip.elapsed_ms(ev[s], ev[s + 1]) for s in range(steps)]
    pev = [hip.create() for _ in range(wm.PROFILE_EVENTS)]
    att = []
    for _ in range(steps):
        wm.layer_step_profiled(dims, P, H, w.chan_map, ctx, Kc, Vc, O, pev, ws=ws,
                               stream=stream)
        torch.cuda.synchronize()
        att.append(hip.elapsed_ms(pev[5], pev[6]))
    for e in ev + pev:
        hip.destroy(e)
    _, attn_bytes = phase_costs(w)["attend"]
    t_step = float(np.median(ms))
    t_att = float(np.median(att))
    del Kc, Vc
    torch.cuda.empty_cache()
    out = {"workload": WORKLOAD_LABEL[w.name], "ms_per_step_median": round(t_step, 4),
           "tokens_per_s": round(w.B / (t_step * 1e-3), 1),
           "attend_ms_median": round(t_att, 4),
           "attend_hbm_gb": round(attn_bytes / 1e9, 2),
           "attend_hbm_frac": round(attn_bytes / (t_att * 1e-3) / (PEAK_HBM_GBS * 1e9), 4),
           "step_hbm_frac": round(attn_bytes / (t_step * 1e-3) / (PEAK_HBM_GBS * 1e9), 4),
           "per_consumer_hbm_gb": round(attn_bytes * w.L / len(set(w.chan_map)) / 1e9, 2),
           "steps": steps}
    log("bench: decode %.3f ms/step, attention %.3f ms (%.1f%% of HBM peak)"
        % (t_step, t_att, 100 * out["attend_hbm_frac"]))
    return out


def attend_backward_bench(wm, torch, np, synth, hip, dev, stream, log, w, reps=5):
    """The attention gradients of the headline pass (wm_channel_attend_backward), the part
    of the backward pass that runs through the attention: seeded queries, cache and output
    gradient (as in the parity test), O from the forward kernel, event-timed. TFLOP/s count
    the five gradient products of the standard tally (S = QK^T, dP = dO V^T, dQ = dS K,
    dK = dS^T Q, dV = P^T dO: 10 d flops per visible pair, 2.5 times the forward's); the
    kernels also recompute S for the row log-sum-exp and S, dP in both the query-major and
    the slot-major kernel (16 d flops per pair executed)."""
    log("bench: attention gradients %s" % w.name)
    P = wm.ParamSet({k: v.to(dev) for k, v in
                     synth.make_params(w, np.asarray(wm.init_bias(w.L, w.k))).items()})
    bf = torch.bfloat16
    Q = synth._normal((w.L, w.B, w.Hq, w.T_new, w.d), 1.0, 9100, bf).to(dev)
    shape = (w.k, w.B, w.Hkv, w.T_new, w.d)
    Kc = synth._normal(shape, 1.0, 9101, bf).to(dev)
    Vc = synth._normal(shape, 1.0, 9102, bf).to(dev)
    dO = synth._normal((w.L, w.B, w.T_new, w.Hq * w.d), 1.0, 9103, bf).to(dev)
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=bf, device=dev)
    dims = wm.make_dims(w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, p=w.p, S_cap=w.T_new,
                        ctx_max=0, dtype=wm.BF16)
    wm.channel_attend(dims, P, Q, w.chan_map, None, Kc, Vc, O, stream=stream)
    f32 = dict(dtype=torch.float32, device=dev)
    g = [torch.empty(tuple(Q.shape), **f32), torch.empty(shape, **f32),
         torch.empty(shape, **f32), torch.empty((w.k, w.Hkv, w.d), **f32),
         torch.empty((w.k, w.Hkv, w.d), **f32)]
    ws = wm.workspace(dims, wm.OP_ATTEND_BACKWARD, dev)
    for _ in range(2):
        wm.channel_attend_backward(dims, P, Q, w.chan_map, None, Kc, Vc, O, dO, *g, ws=ws,
                                   stream=stream)
    torch.cuda.synchronize()
    ev = [hip.create() for _ in range(reps + 1)]
    hip.record(ev[0], stream.cuda_stream)
    for r in range(reps):
        wm.channel_attend_backward(dims, P, Q, w.chan_map, None, Kc, Vc, O, dO, *g, ws=ws,
                                   stream=stream)
        hip.record(ev[r + 1], stream.cuda_stream)
    torch.cuda.synchronize()
    ms = float(np.median([hip.elapsed_ms(ev[r], ev[r + 1]) for r in range(reps)]))
    for e in ev:
        hip.destroy(e)
    flops = 2.5 * attn_flops(w.L, w.Hq, w.d, visible_pairs(w))
    tf = flops / (ms * 1e-3) / 1e12
    del Q, Kc, Vc, dO, O, g, ws
    torch.cuda.empty_cache()
    log("bench: attention gradients %.3f ms, %.1f TFLOP/s (%.1f%% of the bf16 peak)"
        % (ms, tf, 100 * tf / PEAK_TFLOPS["bf16"]))
    return {"workload": WORKLOAD_LABEL[w.name], "ms_median": round(ms, 4),
            "gflop": round(flops / 1e9, 1), "tflops": round(tf, 1),
            "frac_of_bf16_peak": round(tf / PEAK_TFLOPS["bf16"], 4),
            "executed_gflop": round(flops * 16 / 10 / 1e9, 1), "reps": reps}


def step_backward_bench(wm, torch, np, synth, hip, dev, stream, log, w, reps=3):
    """The whole step's gradients for the headline pass (wm_layer_step_backward: the
    queries recomputed, the attention gradients, then the queries' and the pool's
    backward), plus the queries' and the pool's backward alone, event-timed, from the
    forward step's own caches and output. GFLOP count the MFMA products the backward
    executes outside the attention: recomputed pre-norm projections, dX = dY W and
    dW = dY^T X for W^Q, W^K (three each), W^V (two), and the router's forward and its two
    gradient products per branch."""
    log("bench: step gradients %s" % w.name)
    P = wm.ParamSet({k: v.to(dev) for k, v in
                     synth.make_params(w, np.asarray(wm.init_bias(w.L, w.k)),
                                       gains="random").items()})
    bf = torch.bfloat16
    f32 = dict(dtype=torch.float32, device=dev)
    H = synth.make_states(w).to(dev)
    dims = wm.make_dims(w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, p=w.p, S_cap=w.T_new,
                        ctx_max=0, dtype=wm.BF16)
    shape = (w.k, w.B, w.Hkv, w.T_new, w.d)
    Kc = torch.empty(shape, dtype=bf, device=dev)
    Vc = torch.empty(shape, dtype=bf, device=dev)
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=bf, device=dev)
    wm.layer_step(dims, P, H, w.chan_map, None, Kc, Vc, O, stream=stream)
    dO = synth._normal(tuple(O.shape), 1.0, 9201, bf).to(dev)
    dKc, dVc = torch.zeros(shape, **f32), torch.zeros(shape, **f32)
    dH = torch.zeros(tuple(H.shape), **f32)
    grads = {n: torch.zeros(tuple(P.tensors[n].shape), **f32) for n in wm.PARAM_NAMES}
    dQ = synth._normal((w.L, w.B, w.Hq, w.T_new, w.d), 1.0, 9202, torch.float32).to(dev)
    calls = {
        "step": (wm.OP_STEP_BACKWARD, lambda ws: wm.layer_step_backward(
            dims, P, H, w.chan_map, None, Kc, Vc, O, dO, dKc, dVc, dH, grads, ws=ws,
            stream=stream)),
        "queries": (wm.OP_Q_BACKWARD, lambda ws: wm.q_project_backward(
            dims, P, H, None, dQ, dH, grads, ws=ws, stream=stream)),
        "pool": (wm.OP_POOL_BACKWARD, lambda ws: wm.pool_backward(
            dims, P, H, None, dKc, dVc, dH, grads, ws=ws, stream=stream)),
    }
    out = {"workload": WORKLOAD_LABEL[w.name], "reps": reps}
    for name, (op, fn) in calls.items():
        ws = wm.workspace(dims, op, dev)
        fn(ws)
        torch.cuda.synchronize()
        ev = [hip.create() for _ in range(reps + 1)]
        hip.record(ev[0], stream.cuda_stream)
        for r in range(reps):
            fn(ws)
            hip.record(ev[r + 1], stream.cuda_stream)
        torch.cuda.synchronize()
        out[name + "_ms_median"] = round(float(np.median(
            [hip.elapsed_ms(ev[r], ev[r + 1]) for r in range(reps)])), 4)
        for e in ev:
            hip.destroy(e)
        del ws
        torch.cuda.empty_cache()
    N, HQ, HK, kL, Lp = w.N, w.Hq * w.d, w.Hkv * w.d, w.k * w.L, (w.L + w.p - 1) // w.p
    q_gf = 3 * 2.0 * N * w.L * HQ * w.D
    kv_gf = 5 * 2.0 * N * w.k * HK * w.D
    r_gf = 3 * 2 * 2.0 * N * kL * Lp * w.D
    out["queries_gflop"] = round(q_gf / 1e9, 1)
    out["pool_gflop"] = round((kv_gf + r_gf) / 1e9, 1)
    out["queries_tflops"] = round(q_gf / (out["queries_ms_median"] * 1e-3) / 1e12, 1)
    out["pool_tflops"] = round((kv_gf + r_gf) / (out["pool_ms_median"] * 1e-3) / 1e12, 1)
    log("bench: step gradients %.3f ms (queries %.3f ms, pool %.3f ms)"
        % (out["step_ms_median"], out["queries_ms_median"], out["pool_ms_median"]))
    del H, Kc, Vc, O, dO, dKc, dVc, dH, grads, dQ, P
    torch.cuda.empty_cache()
    return out


def passes_bench(wm, torch, np, synth, hip, dev, stream, log, groups=("8", "16", "1", "T"),
                 train=True):
    """The fixed-point passes of Section 3.3 at the paper's model shape (B16 T2048 L16 k8
    D512, 6 query / 3 KV heads of 96, p = 2, bf16) with the stand-in decoder block:
    cyclic Gauss-Seidel with the paper's g = 8 groups and with g = 16, Jacobi (g = 1), 3
    passes each, and one pass of g = T (exact left-to-right evaluation), event-timed; then
    (train) a training step's passes (wm_prefill_passes_backward): the paper's 3 passes of
    g = 8 with gradients through the last 2 or 1, and 3 Jacobi passes with gradients
    through the last 2."""
    w0 = synth.WORKLOADS["paper_T2048_L16_k8"]
    w = synth.Workload("paper_passes", w0.B, w0.T_new, w0.L, w0.k, w0.D, w0.Hq, w0.Hkv, w0.d, 0,
                       w0.dtype, list(w0.chan_map), w0.p, w0.seed)
    P = wm.ParamSet({k: v.to(dev) for k, v in
                     synth.make_params(w, np.asarray(wm.init_bias(w.L, w.k)) + 0.2).items()})
    X = synth.make_embeddings(w).to(dev)
    W_o = synth.make_out_proj(w).to(dev)
    Kc = torch.zeros((w.k, w.B, w.Hkv, w.T_new, w.d), dtype=w.torch_dtype, device=dev)
    Vc = torch.zeros_like(Kc)
    H = torch.empty((w.B, w.T_new, w.L, w.D), dtype=w.torch_dtype, device=dev)
    top = torch.empty((w.B, w.T_new, w.D), dtype=w.torch_dtype, device=dev)
    out = {"workload": "fixed-point passes, the paper's model shape: B16 T2048 L16 k8 D512 "
                       "6q/3kv x96, p2, bf16, map l->l%8, stand-in block h + W_o o"}
    runs = [(w.T_new, 1, 1) if g == "T" else (int(g), 3, 5) for g in groups]
    for g, passes, reps in runs:
        dims = wm.make_dims(w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, p=w.p,
                            S_cap=w.T_new, ctx_max=0, dtype=wm.BF16, groups=g)
        ws = wm.workspace(dims, wm.OP_PASSES, dev)
        run = lambda: wm.prefill_passes(dims, P, W_o, X, w.chan_map, passes, Kc, Vc, H, top,  # noqa: E731
                                        ws=ws, stream=stream)
        run()
        torch.cuda.synchronize()
        ev = [hip.create() for _ in range(reps + 1)]
        hip.record(ev[0], stream.cuda_stream)
        for r in range(reps):
            run()
            hip.record(ev[r + 1], stream.cuda_stream)
        torch.cuda.synchronize()
        ms = float(np.median([hip.elapsed_ms(ev[r], ev[r + 1]) for r in range(reps)]))
        for e in ev:
            hip.destroy(e)
        key = "g%d" % g if g < w.T_new else "g_T"
        out[key] = {"passes": passes, "ms": round(ms, 3), "ms_per_pass": round(ms / passes, 3),
                    "tokens_per_s": round(w.B * w.T_new / (ms * 1e-3), 1),
                    "s_per_sequence": round(ms * 1e-3 / w.B, 6)}
        log("bench: passes g=%d x %d: %.3f ms (%.3f ms per pass, %.0f tokens/s)"
            % (g, passes, ms, ms / passes, w.B * w.T_new / (ms * 1e-3)))
        del ws
    # a training step's passes: 3 passes, then backpropagation truncated to the last n_g
    # of them (wm_prefill_passes_backward: the forward and the backward in one call)
    if train:
        f32 = dict(dtype=torch.float32, device=dev)
        dh = synth._normal((w.B, w.T_new, w.D), 1.0, 9301, torch.float32).to(dev)
        dX = torch.zeros((w.B, w.T_new, w.D), **f32)
        dW = torch.zeros(tuple(W_o.shape), **f32)
        grads = {n: torch.zeros(tuple(P.tensors[n].shape), **f32) for n in wm.PARAM_NAMES}
        for g, n_grad in ((8, 2), (8, 1), (1, 2)):
            dims = wm.make_dims(w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, p=w.p,
                                S_cap=w.T_new, ctx_max=0, dtype=wm.BF16, groups=g)
            ws = torch.empty(wm.passes_backward_workspace(dims, n_grad), dtype=torch.uint8,
                             device=dev)
            run = lambda: wm.prefill_passes_backward(  # noqa: E731
                dims, P, W_o, X, w.chan_map, 3, n_grad, dh, dX, dW, grads, h_top=top, ws=ws,
                stream=stream)
            run()
            torch.cuda.synchronize()
            reps = 3
            ev = [hip.create() for _ in range(reps + 1)]
            hip.record(ev[0], stream.cuda_stream)
            for r in range(reps):
                run()
                hip.record(ev[r + 1], stream.cuda_stream)
            torch.cuda.synchronize()
            ms = float(np.median([hip.elapsed_ms(ev[r], ev[r + 1]) for r in range(reps)]))
            for e in ev:
                hip.destroy(e)
            out["train_g%d_x3_ng%d" % (g, n_grad)] = {
                "passes": 3, "groups": g, "n_grad": n_grad, "ms": round(ms, 3),
                "workspace_gb": round(ws.numel() / 1e9, 2),
                "tokens_per_s": round(w.B * w.T_new / (ms * 1e-3), 1)}
            log("bench: training passes (3 of g=%d, gradients through the last %d): %.3f ms"
                % (g, n_grad, ms))
            del ws
            torch.cuda.empty_cache()
    out["schedule_s44"] = schedule_bench(wm, torch, np, synth, hip, dev, stream, log)
    return out


def schedule_bench(wm, torch, np, synth, hip, dev, stream, log):
    """The schedules of the paper's prefill timing (Section 4.4: a 4-layer model, D = 512,
    k = 4, 2048-token sequences in batches of 64, time per sequence = batch time / 64) run
    by the pass driver with the stand-in block in place of the decoder layer (heads 6 / 3
    of 96 as the paper's model family; p = 1): cyclic g = 16 with the 4 passes the paper
    needs and Jacobi with its 75. Context for the paper's figures (0.01245 and 0.1393 s per
    sequence on an RTX A6000 with full decoder layers), not the same computation."""
    w = synth.Workload("paper_s44", 64, 2048, 4, 4, 512, 6, 3, 96, 0, "bf16",
                       [l % 4 for l in range(4)], 1, 1404)
    P = wm.ParamSet({k: v.to(dev) for k, v in
                     synth.make_params(w, np.asarray(wm.init_bias(w.L, w.k)) + 0.2).items()})
    X = synth.make_embeddings(w).to(dev)
    W_o = synth.make_out_proj(w).to(dev)
    Kc = torch.zeros((w.k, w.B, w.Hkv, w.T_new, w.d), dtype=torch.bfloat16, device=dev)
    Vc = torch.zeros_like(Kc)
    H = torch.empty((w.B, w.T_new, w.L, w.D), dtype=torch.bfloat16, device=dev)
    top = torch.empty((w.B, w.T_new, w.D), dtype=torch.bfloat16, device=dev)
    out = {"workload": "Section 4.4 schedules: B64 T2048 L4 k4 D512 6q/3kv x96, p1, bf16, "
                       "stand-in block h + W_o o (the paper times full decoder layers)"}
    for g, passes, reps in ((16, 4, 5), (1, 75, 2)):
        dims = wm.make_dims(w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, p=w.p,
                            S_cap=w.T_new, ctx_max=0, dtype=wm.BF16, groups=g)
        ws = wm.workspace(dims, wm.OP_PASSES, dev)
        run = lambda: wm.prefill_passes(dims, P, W_o, X, w.chan_map, passes, Kc, Vc, H, top,  # noqa: E731
                                        ws=ws, stream=stream)
        run()
        torch.cuda.synchronize()
        ev = [hip.create() for _ in range(reps + 1)]
        hip.record(ev[0], stream.cuda_stream)
        for r in range(reps):
            run()
            hip.record(ev[r + 1], stream.cuda_stream)
        torch.cuda.synchronize()
        ms = float(np.median([hip.elapsed_ms(ev[r], ev[r + 1]) for r in range(reps)]))
        for e in ev:
            hip.destroy(e)
        out["g%d_x%d" % (g, passes)] = {"passes": passes, "ms": round(ms, 3),
                                        "s_per_sequence": round(ms * 1e-3 / w.B, 6),
                                        "tokens_per_s": round(w.B * w.T_new / (ms * 1e-3), 1)}
        log("bench: Section 4.4 schedule g=%d x %d: %.3f ms per batch of 64 (%.5f s per sequence)"
            % (g, passes, ms, ms * 1e-3 / w.B))
        del ws
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c4_T4096_L24_k12", choices=sorted(WORKLOAD_LABEL))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the 32768-context decode step timed after the main workload")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the attention gradients timed on the main workload")
    ap.add_argument("--no-passes", action="store_true",
                    help="skip the fixed-point pass driver timed at the paper's model shape")
    ap.add_argument("--pass-groups", default="8,16,1,T",
                    help="group counts g of the timed pass-driver runs (T: one exact pass)")
    ap.add_argument("--blas-reference", action="store_true",
                    help="also time torch.bmm (the vendor GEMM library) on the plain GEMMs of the "
                         "K/V and query projections of this workload, for comparison (stderr)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the WhiteMatter step here runs on a single MI355X "
              "(--gpus %d is not supported)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_18486_amd as wm
    from tests import synth

    w = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log = lambda *a: print(*a, file=sys.stderr, flush=True)  # noqa: E731
    log("bench: workload %s (%s)" % (w.name, WORKLOAD_LABEL[w.name]))
    if args.blas_reference and w.dtype == "bf16":
        blas_reference(w, log)

    bias = np.asarray(wm.init_bias(w.L, w.k))
    P_cpu = synth.make_params(w, bias)
    P = wm.ParamSet({k: v.to(dev) for k, v in P_cpu.items()})
    H_cpu = synth.make_states(w)
    H = H_cpu.to(dev)
    if w.ctx:
        Kc, Vc = synth.make_cache_device(w, device=dev)
    else:
        Kc = torch.zeros((w.k, w.B, w.Hkv, w.S_cap, w.d), dtype=w.torch_dtype, device=dev)
        Vc = torch.zeros_like(Kc)
    ctx = torch.full((w.B,), w.ctx, dtype=torch.int32, device=dev)
    docs_cpu = (synth.make_doc_start(w, mean_len=synth.DOC_MEAN[w.name])
                if w.name in synth.DOC_MEAN else None)
    docs = docs_cpu.to(dev) if docs_cpu is not None else None
    O = torch.empty((w.L, w.B, w.T_new, w.Hq * w.d), dtype=w.torch_dtype, device=dev)
    dims = wm.make_dims(w.B, w.T_new, w.L, w.k, w.D, w.Hq, w.Hkv, w.d, p=w.p, S_cap=w.S_cap,
                        ctx_max=w.ctx, dtype=wm.dtype_code(w.torch_dtype),
                        router_mode=router_mode_of(w))
    ws = wm.workspace(dims, wm.OP_LAYER_STEP, dev)
    stream = torch.cuda.current_stream(dev)

    hip = HipEvents()
    for _ in range(args.warmup):
        wm.layer_step(dims, P, H, w.chan_map, ctx, Kc, Vc, O, ws=ws, stream=stream,
                      doc_start=docs)
    torch.cuda.synchronize()
    log("bench: warmup done, timing %d steps" % args.steps)

    # the timed steps: the fused step as a caller runs it, bracketed by synchronisations
    step_ev = [hip.create() for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    hip.record(step_ev[0], stream.cuda_stream)
    for s in range(args.steps):
        wm.layer_step(dims, P, H, w.chan_map, ctx, Kc, Vc, O, ws=ws, stream=stream,
                      doc_start=docs)
        hip.record(step_ev[s + 1], stream.cuda_stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall = t1 - t0
    step_ms = [hip.elapsed_ms(step_ev[s], step_ev[s + 1]) for s in range(args.steps)]
    for e in step_ev:
        hip.destroy(e)

    # then the same number of steps with phase events, for the per-phase times and the
    # roofline of each kernel
    events = [[hip.create() for _ in range(wm.PROFILE_EVENTS)] for _ in range(args.steps)]
    for s in range(args.steps):
        wm.layer_step_profiled(dims, P, H, w.chan_map, ctx, Kc, Vc, O, events[s], ws=ws,
                               stream=stream, doc_start=docs)
    torch.cuda.synchronize()

    phase_ms = {name: [] for name in wm.PHASES}
    serial_ms = []
    for ev in events:
        for i, name in enumerate(wm.PHASES):
            phase_ms[name].append(hip.elapsed_ms(ev[i], ev[i + 1]))
        serial_ms.append(hip.elapsed_ms(ev[0], ev[-1]))
    for ev in events:
        for e in ev:
            hip.destroy(e)
    mean = {k: float(np.mean(v)) for k, v in phase_ms.items()}
    docs_np = docs_cpu.numpy() if docs_cpu is not None else None
    costs = phase_costs(w, docs_np)
    flops, min_bytes = step_cost(w, docs_np)
    for name in wm.PHASES:
        f, b = costs[name]
        t = mean[name] * 1e-3
        log("bench: phase %-10s %8.3f ms  %8.1f TFLOP/s  %8.1f GB/s" % (
            name, mean[name], f / t / 1e12 if t else 0, b / t / 1e9 if t else 0))

    dom = max(mean, key=mean.get)
    f, b = costs[dom]
    t_dom = mean[dom] * 1e-3
    ridge = PEAK_TFLOPS[w.dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)
    if f / max(b, 1) >= ridge:
        achieved = f / t_dom / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_TFLOPS[w.dtype],
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_TFLOPS[w.dtype], 4)}
    else:
        achieved = b / t_dom / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    gemm = "proj_gemm_dma_kernel" if w.dtype == "bf16" else "proj_gemm_kernel"
    mix = "mix_mfma_kernel" if (w.dtype == "bf16" and w.L <= 32 and w.k <= 32) else "mix_kernel"
    prefill = "attend_prefill_dma_kernel" if (w.dtype == "bf16" and w.d in (64, 96)) else \
        "attend_prefill_kernel"
    roof["kernel"] = {"attend": prefill if w.T_new > 4 else
                      "attend_decode_kernel + attend_combine_kernel",
                      "kv_project": gemm + " (K/V projection, after fold_gain_kernel)",
                      "q_project": gemm + " (Q projection, after fold_gain_kernel)",
                      "router": gemm + " (router, with router_fold/reduce kernels)",
                      "mix": mix, "norms": "row_rms_kernel + rope_table_kernel"}[dom]
    roof["phase"] = dom
    roof["duration_ms"] = round(mean[dom], 4)
    roof["traffic"] = measured_traffic(w.name, dom)
    ceilings = measure_ceilings(wm, torch, dev, stream)
    if roof["bound"] == "hbm":
        roof["measured_ceiling"] = ceilings["hbm_read_gbs"]
    elif w.dtype == "bf16":
        roof["measured_ceiling"] = ceilings["mfma_bf16_tflops"]
        # the same loop on changing random operands: the rate real data gets
        roof["measured_ceiling_random_operands"] = ceilings["mfma_bf16_tflops_random_operands"]
        roof["frac_of_measured_ceiling_random_operands"] = round(
            achieved / roof["measured_ceiling_random_operands"], 4)
    if "measured_ceiling" in roof:
        roof["frac_of_measured_ceiling"] = round(achieved / roof["measured_ceiling"], 4)

    ms_per_step = wall / args.steps * 1e3
    # this design's phase-wise roofline: each of its phases at the slower of its flops and
    # its bytes, with the intermediates it keeps in HBM (row norms, mixed channels, Q)
    t_roof = sum(max(f / (PEAK_TFLOPS[w.dtype] * 1e12), b / (PEAK_HBM_GBS * 1e9))
                 for f, b in costs.values())
    t_min = fused_min_ms(w, docs_np)
    tokens = w.N * args.steps
    line = {
        "metric": "tokens/s of mix+KV-proj+channel-attention step; % of HBM / MFMA roofline",
        "value": round(tokens / wall, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": WORKLOAD_LABEL[w.name], "B": w.B, "T_new": w.T_new,
                   "ctx": w.ctx, "L": w.L, "k": w.k, "D": w.D, "Hq": w.Hq, "Hkv": w.Hkv,
                   "d": w.d, "p": w.p, "tokens_per_step": w.N},
        "roofline": roof,
        "ceilings": ceilings,
        "step_roofline": {"gflop": round(flops / 1e9, 2), "min_hbm_gb": round(min_bytes / 1e9, 3),
                          "fused_min_ms": round(t_min, 4),
                          "frac": round(t_min / ms_per_step, 4),
                          "this_design_roof_ms": round(t_roof * 1e3, 4),
                          "frac_of_this_design_roof": round(t_roof / (ms_per_step * 1e-3), 4),
                          "event_ms_per_step_median": round(float(np.median(step_ms)), 4),
                          "serial_phases_ms_per_step_median": round(float(np.median(serial_ms)), 4),
                          "phases_ms": {k: round(v, 4) for k, v in mean.items()}},
    }
    if not args.no_decode and w.name != "c5_decode_S32768":
        del Kc, Vc, O, ws, H
        torch.cuda.empty_cache()
        line["decode_c5"] = decode_step(wm, torch, np, synth, hip, dev, stream, log)
    if not args.no_backward and w.dtype == "bf16" and w.d in (64, 96) and w.T_new > 4 \
            and w.ctx == 0:
        torch.cuda.empty_cache()
        line["attention_backward"] = attend_backward_bench(wm, torch, np, synth, hip, dev,
                                                           stream, log, w)
        line["step_backward"] = step_backward_bench(wm, torch, np, synth, hip, dev, stream,
                                                    log, w)
    if not args.no_passes:
        torch.cuda.empty_cache()
        line["prefill_passes"] = passes_bench(wm, torch, np, synth, hip, dev, stream, log,
                                              args.pass_groups.split(","),
                                              train=not args.no_backward)
    if not args.no_cpu_baseline:
        log("bench: CPU oracle baseline ...")
        line["cpu_baseline"] = cpu_baseline(w, P_cpu, H_cpu, (Kc, Vc) if w.ctx else None, docs_np)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
