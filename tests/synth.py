"""Seeded synthetic inputs for the WhiteMatter step (shared by tests and bench).

This module draws random tensors and states workload shapes; it holds none of
the method's arithmetic. The paper's pretraining data (FineWeb-Edu, Qwen3
tokenizer) and trained weights are not available, so every input is a seeded
stand-in with the shapes of the paper's workloads:

  * layer states H ~ N(0, 1)   (the pre-mix RMSNorm removes their scale)
  * router / K / V / Q weights ~ N(0, 0.02)
  * RMSNorm gains = 1 (or 1 + N(0, 0.1) to catch an ignored gain)
  * learned dummy K/V ~ N(0, 1); cached context K/V ~ N(0, 1)
  * router biases are passed in by the caller (the paper's initial pattern)

Float tensors are drawn in fp32 on a seeded CPU generator and rounded to bf16
(round-to-nearest-even) where the workload is bf16. The one tensor too large
for the host, the 32768-token decode cache, is drawn with torch's seeded
device generator directly in place.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

PARAM_NAMES = ("g_pre", "W_alpha", "b_alpha", "g_mid", "Wk", "Wv", "g_knorm",
               "Kd", "Vd", "g_in", "Wq", "g_qnorm")


@dataclass
class Workload:
    name: str
    B: int
    T_new: int
    L: int
    k: int
    D: int
    Hq: int
    Hkv: int
    d: int
    ctx: int          # cached tokens per sequence before the step
    dtype: str        # "f32" or "bf16"
    chan_map: list = field(default_factory=list)
    p: int = 1
    seed: int = 0

    @property
    def N(self) -> int:
        return self.B * self.T_new

    @property
    def S_cap(self) -> int:
        need = self.ctx + self.T_new
        return (need + 63) // 64 * 64

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


def _map_mod(L, k):
    return [l % k for l in range(L)]


# The five workloads (tiny fp32; two 2048-token passes with and without 2x
# KV compression; a 24-layer 4096-token pass; a 32768-context decode step).
WORKLOADS = {
    "c1_tiny_f32": Workload("c1_tiny_f32", 1, 64, 4, 2, 64, 2, 2, 32, 0, "f32",
                            _map_mod(4, 2), seed=1001),
    "c2_T2048_L12_k12": Workload("c2_T2048_L12_k12", 8, 2048, 12, 12, 768, 12, 12, 64, 0,
                                 "bf16", list(range(12)), seed=1002),
    "c3_T2048_L12_k6": Workload("c3_T2048_L12_k6", 8, 2048, 12, 6, 768, 12, 12, 64, 0, "bf16",
                                [l // 2 for l in range(12)], seed=1003),
    "c4_T4096_L24_k12": Workload("c4_T4096_L24_k12", 4, 4096, 24, 12, 1024, 16, 16, 64, 0,
                                 "bf16", _map_mod(24, 12), seed=1004),
    "c5_decode_S32768": Workload("c5_decode_S32768", 64, 1, 24, 12, 1024, 16, 16, 64, 32768,
                                 "bf16", _map_mod(24, 12), seed=1005),
}
# The paper's own model shape (Section 4.1): L = 16, D = 512, 6 query and 3 KV heads of
# dimension 96, routers reading every second source layer (p = 2), sequences packed to
# 2048 tokens, 16 sequences (a global batch of 128 over 8 GPUs), fixed selection
# l -> l mod k, for the channel counts of the compression study (Section 5.2).
for _k in (1, 2, 4, 8, 12, 16):
    WORKLOADS["paper_T2048_L16_k%d" % _k] = Workload(
        "paper_T2048_L16_k%d" % _k, 16, 2048, 16, _k, 512, 6, 3, 96, 0, "bf16",
        _map_mod(16, _k), p=2, seed=1100 + _k)
del _k
# The same passes with the document mask: each 2048-token row packs documents whose
# lengths are 1 + an exponential draw of mean 511 (mean document 512 tokens), a seeded
# stand-in for the paper's packed pretraining text (FineWeb-Edu, Section 4.1).
DOC_MEAN = {}
for _k in (8, 16):
    _w = WORKLOADS["paper_T2048_L16_k%d" % _k]
    _n = "paper_T2048_L16_k%d_docs" % _k
    WORKLOADS[_n] = Workload(_n, _w.B, _w.T_new, _w.L, _w.k, _w.D, _w.Hq, _w.Hkv, _w.d, _w.ctx,
                             _w.dtype, list(_w.chan_map), _w.p, _w.seed)
    DOC_MEAN[_n] = 512.0
# The ablations of Section 5.3 at the paper's shape: static mixing weights (k = 16 and
# k = 1) and no deep-to-shallow feedback (k = L = 16).
ROUTER_MODE = {}
for _k, _mode, _tag in ((16, 1, "static"), (1, 1, "static"), (16, 2, "nofeedback")):
    _w = WORKLOADS["paper_T2048_L16_k%d" % _k]
    _n = "paper_T2048_L16_k%d_%s" % (_k, _tag)
    WORKLOADS[_n] = Workload(_n, _w.B, _w.T_new, _w.L, _w.k, _w.D, _w.Hq, _w.Hkv, _w.d, _w.ctx,
                             _w.dtype, list(_w.chan_map), _w.p, _w.seed)
    ROUTER_MODE[_n] = _mode
del _k, _w, _n, _mode, _tag


def small(name="small", B=2, T_new=40, L=5, k=3, D=96, Hq=4, Hkv=2, d=32, ctx=0,
          dtype="bf16", chan_map=None, p=1, seed=7) -> Workload:
    """A small workload for fuzz/parity cases (defaults: ragged, k does not divide L, GQA)."""
    if chan_map is None:
        chan_map = _map_mod(L, k)
    return Workload(name, B, T_new, L, k, D, Hq, Hkv, d, ctx, dtype, list(chan_map), p, seed)


def _gen(seed: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return g


def _normal(shape, std, seed, dtype, mean=0.0):
    x = torch.randn(shape, generator=_gen(seed), dtype=torch.float32) * std + mean
    return x.to(dtype)


def make_params(w: Workload, b_alpha, gains: str = "unit", zero_router: bool = False) -> dict:
    """Random parameters on the CPU in the workload dtype.

    b_alpha: the router bias, shape [2, k*L] (or [k*L], used for both branches).
    gains: "unit" (all RMSNorm gains 1) or "random" (1 + N(0, 0.1)).
    zero_router: W_alpha = 0, so the mixing weights equal the bias.
    """
    dt = w.torch_dtype
    Lp = (w.L + w.p - 1) // w.p
    s = w.seed * 100

    def gain(shape, sub):
        if gains == "unit":
            return torch.ones(shape, dtype=torch.float32).to(dt)
        return _normal(shape, 0.1, s + sub, dt, mean=1.0)

    b = torch.as_tensor(b_alpha, dtype=torch.float32)
    if b.dim() == 1:
        b = torch.stack([b, b])
    P = {
        "g_pre": gain((2, w.L, w.D), 1),
        "W_alpha": (torch.zeros((2, w.k * w.L, Lp * w.D), dtype=dt) if zero_router
                    else _normal((2, w.k * w.L, Lp * w.D), 0.02, s + 2, dt)),
        "b_alpha": b.reshape(2, w.k * w.L).to(dt),
        "g_mid": gain((2, w.k, w.D), 3),
        "Wk": _normal((w.k, w.Hkv * w.d, w.D), 0.02, s + 4, dt),
        "Wv": _normal((w.k, w.Hkv * w.d, w.D), 0.02, s + 5, dt),
        "g_knorm": gain((w.k, w.d), 6),
        "Kd": _normal((w.k, w.Hkv, w.d), 1.0, s + 7, dt),
        "Vd": _normal((w.k, w.Hkv, w.d), 1.0, s + 8, dt),
        "g_in": gain((w.L, w.D), 9),
        "Wq": _normal((w.L, w.Hq * w.d, w.D), 0.02, s + 10, dt),
        "g_qnorm": gain((w.L, w.d), 11),
    }
    return P


def make_states(w: Workload, sub: int = 20) -> torch.Tensor:
    """Layer states H[B, T_new, L, D] ~ N(0, 1)."""
    return _normal((w.B, w.T_new, w.L, w.D), 1.0, w.seed * 100 + sub, w.torch_dtype)


def make_mixed(w: Workload, sub: int = 21) -> torch.Tensor:
    """Stand-in mixed channels [2, k, N, D] ~ N(0, 1) for testing the projection alone."""
    return _normal((2, w.k, w.N, w.D), 1.0, w.seed * 100 + sub, w.torch_dtype)


def make_queries(w: Workload, sub: int = 22) -> torch.Tensor:
    """Stand-in queries [L, B, Hq, T_new, d] ~ N(0, 1) for testing attention alone."""
    return _normal((w.L, w.B, w.Hq, w.T_new, w.d), 1.0, w.seed * 100 + sub, w.torch_dtype)


def make_ctx_len(w: Workload, ragged: bool = False, sub: int = 23) -> torch.Tensor:
    """Cached tokens per sequence: w.ctx everywhere, or uniform in [0, w.ctx]."""
    if not ragged or w.ctx == 0:
        return torch.full((w.B,), w.ctx, dtype=torch.int32)
    return torch.randint(0, w.ctx + 1, (w.B,), generator=_gen(w.seed * 100 + sub),
                         dtype=torch.int32)


def make_doc_start(w: Workload, ctx_len=None, mean_len: float = 512.0, sub: int = 31,
                   lengths=None) -> torch.Tensor:
    """Packed documents: [B, T_new] int32, the position of the first token of the document
    holding each new token (token i of sequence b sits at ctx_len[b] + i).

    Each sequence is cut into documents from position 0 on, with lengths 1 + a seeded
    exponential draw of mean `mean_len` - 1 (rounded down), or the given `lengths`
    cycled (for hand-placed boundaries)."""
    ctx = torch.zeros(w.B, dtype=torch.int32) if ctx_len is None else ctx_len.to(torch.int32)
    g = _gen(w.seed * 100 + sub)
    out = torch.empty((w.B, w.T_new), dtype=torch.int32)
    for b in range(w.B):
        end = int(ctx[b]) + w.T_new
        starts = torch.empty(end, dtype=torch.int32)
        pos, k = 0, 0
        while pos < end:
            if lengths is not None:
                n = int(lengths[k % len(lengths)])
            else:
                e = torch.empty(1).exponential_(1.0 / max(mean_len - 1.0, 1e-6), generator=g)
                n = 1 + int(e.item())
            n = max(n, 1)
            starts[pos:pos + n] = pos
            pos += n
            k += 1
        out[b] = starts[int(ctx[b]):end]
    return out


def make_cache_cpu(w: Workload, sub: int = 24, fill=float("nan")):
    """Host cache [k, B, Hkv, S_cap, d]: slots < ctx ~ N(0, 1), the rest `fill`."""
    shape = (w.k, w.B, w.Hkv, w.S_cap, w.d)
    K = torch.full(shape, fill, dtype=w.torch_dtype)
    V = torch.full(shape, fill, dtype=w.torch_dtype)
    if w.ctx:
        K[:, :, :, :w.ctx] = _normal((w.k, w.B, w.Hkv, w.ctx, w.d), 1.0, w.seed * 100 + sub,
                                     w.torch_dtype)
        V[:, :, :, :w.ctx] = _normal((w.k, w.B, w.Hkv, w.ctx, w.d), 1.0,
                                     w.seed * 100 + sub + 1, w.torch_dtype)
    return K, V


def make_cache_device(w: Workload, device="cuda", sub: int = 24, fill=float("nan")):
    """Device cache for large contexts, drawn in place with the seeded device generator
    one (channel, sequence) slice at a time; slots >= ctx hold `fill`."""
    shape = (w.k, w.B, w.Hkv, w.S_cap, w.d)
    g = torch.Generator(device=device)
    g.manual_seed(w.seed * 100 + sub)
    K = torch.empty(shape, dtype=w.torch_dtype, device=device)
    V = torch.empty(shape, dtype=w.torch_dtype, device=device)
    for T in (K, V):
        for j in range(w.k):
            for b in range(w.B):
                T[j, b, :, :w.ctx].normal_(0.0, 1.0, generator=g)
                T[j, b, :, w.ctx:].fill_(fill)
    return K, V


def _unit_dirs(n, d, seed):
    """n seeded unit vectors of length d (float64 rows)."""
    u = torch.randn((n, d), generator=_gen(seed), dtype=torch.float64)
    return u / u.norm(dim=1, keepdim=True)


def make_peaked_attention(w: Workload, rise: float = 60.0, period: int = 256, a: float = 16.0,
                          sub: int = 40):
    """Queries and a cache whose attention scores climb steeply along the slots.

    Q = a u + N(0, 1) and K[s] = beta(s) u + N(0, 1), with u a seeded unit vector per KV
    head (query heads use their KV head's) and beta(s) a sawtooth over slots, rising
    linearly through each `period` slots so that a beta(s) log2(e) / sqrt(d), the
    score's trend in log2 units, climbs by `rise` per period. V ~ N(0, 1). Returns
    Q [L, B, Hq, T_new, d] and Kc, Vc [k, B, Hkv, S_cap, d] with slots < w.ctx filled and
    the rest NaN, in the workload dtype."""
    s = w.seed * 100 + sub
    u = _unit_dirs(w.Hkv, w.d, s)
    grp = w.Hq // w.Hkv
    beta_max = rise * w.d ** 0.5 / (a * 1.4426950408889634)
    Q = torch.randn((w.L, w.B, w.Hq, w.T_new, w.d), generator=_gen(s + 1), dtype=torch.float64)
    Q += a * u.repeat_interleave(grp, dim=0)[None, None, :, None, :]
    shape = (w.k, w.B, w.Hkv, w.S_cap, w.d)
    K = torch.full(shape, float("nan"), dtype=torch.float64)
    V = torch.full(shape, float("nan"), dtype=torch.float64)
    slots = torch.arange(w.ctx, dtype=torch.float64)
    beta = beta_max * torch.remainder(slots, period) / (period - 1)
    K[:, :, :, :w.ctx] = (torch.randn((w.k, w.B, w.Hkv, w.ctx, w.d), generator=_gen(s + 2),
                                      dtype=torch.float64)
                          + beta[None, None, None, :, None] * u[None, None, :, None, :])
    V[:, :, :, :w.ctx] = torch.randn((w.k, w.B, w.Hkv, w.ctx, w.d), generator=_gen(s + 3),
                                     dtype=torch.float64)
    dt = w.torch_dtype
    return Q.to(dt), K.to(dt), V.to(dt)


def make_low_score_attention(w: Workload, level: float = -300.0, step: float = 4.0,
                             floor: float = 40.0, a: float = 16.0, sub: int = 41):
    """Queries and a cache whose scores all lie far below zero: Q = a u and K[s] =
    -beta(s) u with u a seeded unit vector per KV head, beta(s) chosen so that the score
    q.k log2(e) / sqrt(d) is `level` - min(step s, floor) log2 units (slot 0 the largest).
    V ~ N(0, 1). Shapes and fill as make_peaked_attention."""
    s = w.seed * 100 + sub
    u = _unit_dirs(w.Hkv, w.d, s)
    grp = w.Hq // w.Hkv
    Q = (a * u.repeat_interleave(grp, dim=0))[None, None, :, None, :].expand(
        w.L, w.B, w.Hq, w.T_new, w.d).clone()
    shape = (w.k, w.B, w.Hkv, w.S_cap, w.d)
    K = torch.full(shape, float("nan"), dtype=torch.float64)
    V = torch.full(shape, float("nan"), dtype=torch.float64)
    slots = torch.arange(w.ctx, dtype=torch.float64)
    score = level - torch.clamp(step * slots, max=floor)
    beta = -score * w.d ** 0.5 / (a * 1.4426950408889634)
    K[:, :, :, :w.ctx] = -beta[None, None, None, :, None] * u[None, None, :, None, :]
    V[:, :, :, :w.ctx] = torch.randn((w.k, w.B, w.Hkv, w.ctx, w.d), generator=_gen(s + 3),
                                     dtype=torch.float64)
    dt = w.torch_dtype
    return Q.to(dt), K.to(dt), V.to(dt)


def make_embeddings(w: Workload, sub: int = 50) -> torch.Tensor:
    """Token states entering layer 0 (stand-ins for embeddings) X[B, T_new, D] ~ N(0, 1)."""
    return _normal((w.B, w.T_new, w.D), 1.0, w.seed * 100 + sub, w.torch_dtype)


def make_out_proj(w: Workload, sub: int = 51) -> torch.Tensor:
    """Output projection of the stand-in decoder block, W_o[L, D, Hq*d] ~ N(0, 0.02)."""
    return _normal((w.L, w.D, w.Hq * w.d), 0.02, w.seed * 100 + sub, w.torch_dtype)
