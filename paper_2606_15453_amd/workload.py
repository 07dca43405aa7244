"""Seeded synthetic workloads for the decode-step MoE layer.

This module is the one piece of code that both the HIP path's callers and the
CPU oracle consume.  It only *draws inputs*: a planted Markov routing trace,
router rows, token hidden states and expert weights.  It computes nothing the
method computes (no gating, no prediction, no table update, no FFN).

Stand-in for the paper's workloads.  The paper routes real model traces from
summarisation, maths and code datasets (Section 5.1, Table 2).  Those traces are
not available, so a planted Markov chain stands in for them:

* temporal correlation (Section 3.2): each slot keeps the previous token's
  expert with probability ``p_stay``;
* spatial correlation (Section 3.1): otherwise the expert is drawn from a
  per-layer transition matrix whose rows are Dirichlet(alpha) draws, indexed by
  the same token's expert at the previous layer;
* the hidden state is ``3 * sum(W_g[planted]) + noise`` so that the router's
  top-k recovers the planted set up to rare near-ties.

Random streams.  Small arrays (router rows, transition matrices, the chain)
come from ``numpy.random.SeedSequence(seed, spawn_key=(stream, ...))``.  Large
arrays (expert weights, hidden-state noise) come from a counter-based hash so
that any single expert can be regenerated on its own and so that the same
values can be produced on the GPU with plain integer tensor ops:

    u   = fmix32((idx * 0x9E3779B9 + key) mod 2^32)   (MurmurHash3 finaliser)
    val = Q[u >> 16]

where ``Q`` is a 65536-entry quantile table of the target normal distribution
(``sigma * Phi^-1((j + 0.5) / 65536)``), rounded to the storage format.  Both
backends gather from the same table, so they agree bit for bit.

Streams: 0 router rows, 1 transition matrices, 2 chain, 3 hidden-state noise,
4 routed expert weights, 5 shared expert weights.
"""
from __future__ import annotations

import dataclasses
from functools import lru_cache

import numpy as np

M32 = 0xFFFFFFFF
GOLDEN = 0x9E3779B9

S_ROUTER, S_TRANS, S_CHAIN, S_NOISE, S_EXPERT, S_SHARED = range(6)

#: standard deviation of expert weights (ML initialisation convention)
W_SIGMA = 0.02
#: standard deviation of hidden-state noise: variance 1/256
NOISE_SIGMA = 1.0 / 16.0
#: scale of the planted signal in the hidden state
PLANT_SCALE = 3.0


@dataclasses.dataclass(frozen=True)
class MoEConfig:
    """Shape and routing statistics of one synthetic MoE decode workload."""
    name: str
    L: int          # MoE layers
    H: int          # hidden size
    I: int          # expert SwiGLU intermediate size
    E: int          # routed experts per layer
    K: int          # experts selected per token
    B: int          # decode batch (tokens per step)
    T: int          # decode tokens per batch row
    P: int          # profiling tokens per batch row (T/4, cf. Table 2 ratios)
    C: int          # HBM cache slots per layer for routed experts
    n_shared: int = 0
    dtype: str = "bf16"     # "bf16" or "f32": weights and activations
    p_stay: float = 0.6
    alpha: float = 0.1
    seed: int = 1234

    @property
    def wbytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    @property
    def blob_elems(self) -> int:
        return 3 * self.H * self.I

    @property
    def blob_bytes(self) -> int:
        return self.blob_elems * self.wbytes

    def scaled(self, **kw) -> "MoEConfig":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    # 4 layers, hidden 256, intermediate 512, 8 experts top-2, fp32, batch 1
    "tiny": MoEConfig("tiny-L4-H256-I512-E8-K2-f32-B1", L=4, H=256, I=512, E=8, K=2,
                      B=1, T=64, P=16, C=4, dtype="f32", p_stay=0.6, alpha=0.1, seed=1234),
    # Mixtral-8x7B shapes: 32 layers, hidden 4096, intermediate 14336, 8 experts top-2
    "mixtral": MoEConfig("mixtral8x7b-L32-H4096-I14336-E8-K2-bf16-B1", L=32, H=4096, I=14336,
                         E=8, K=2, B=1, T=256, P=64, C=3, p_stay=0.6, alpha=0.1, seed=1235),
    # Qwen3-30B-A3B shapes: 48 layers, hidden 2048, intermediate 768, 128 experts top-8
    "qwen30b": MoEConfig("qwen3-30b-a3b-L48-H2048-I768-E128-K8-bf16-B1", L=48, H=2048, I=768,
                         E=128, K=8, B=1, T=512, P=128, C=32, p_stay=0.5, alpha=0.05, seed=1236),
    "qwen30b-b8": MoEConfig("qwen3-30b-a3b-L48-H2048-I768-E128-K8-bf16-B8", L=48, H=2048, I=768,
                            E=128, K=8, B=8, T=512, P=128, C=32, p_stay=0.5, alpha=0.05, seed=1236),
    # DeepSeek-V2-Lite shapes: 26 layers, hidden 2048, intermediate 1408, 64 experts top-6 + 2 shared
    "dsv2lite": MoEConfig("deepseek-v2-lite-L26-H2048-I1408-E64+2-K6-bf16-B4", L=26, H=2048,
                          I=1408, E=64, K=6, B=4, T=512, P=128, C=24, n_shared=2,
                          p_stay=0.6, alpha=0.1, seed=1237),
    # Qwen3-235B-A22B shapes: 94 layers, hidden 4096, intermediate 1536, 128 experts top-8
    "qwen235b": MoEConfig("qwen3-235b-a22b-L94-H4096-I1536-E128-K8-bf16-B16", L=94, H=4096,
                          I=1536, E=128, K=8, B=16, T=256, P=64, C=45, p_stay=0.5, alpha=0.05,
                          seed=1238),
}


def paper_matched_stay(E: int, K: int, ratio: float = 2.0) -> float:
    """Stay probability whose expected consecutive-token overlap is `ratio`
    times the independent-routing value K^2/E (Section 3.2 reports about 2x).

    With stay probability p per slot the overlap is about p*K + (1-p)*K^2/E.
    """
    base = K * K / E
    return (ratio - 1.0) * base / (K - base)


#: Predictor-only shapes of the paper's evaluated models (Table 1: layers,
#: experts, top-K).  Hidden sizes are not needed: only routing traces feed the
#: predictor.  Routing statistics: paper-matched temporal overlap (2x random)
#: and peaked spatial transitions.
TABLE1_SHAPES = {
    "qwen1.5-moe": dict(L=24, E=60, K=4),
    "qwen2-moe": dict(L=28, E=64, K=6),
    "deepseek-v2": dict(L=60, E=160, K=8),
    "deepseek-moe": dict(L=60, E=128, K=8),
}


def table1_config(name: str, B: int = 1, T: int = 256, alpha: float = 0.05, seed: int = 2000) -> MoEConfig:
    sh = TABLE1_SHAPES[name]
    return MoEConfig(f"{name}-L{sh['L']}-E{sh['E']}-K{sh['K']}-B{B} (predictor only)", L=sh["L"], H=8, I=8,
                     E=sh["E"], K=sh["K"], B=B, T=T, P=T // 4, C=sh["E"] // 4,
                     p_stay=paper_matched_stay(sh["E"], sh["K"]), alpha=alpha,
                     seed=seed + list(TABLE1_SHAPES).index(name))


# ----------------------------------------------------------------------------
# counter-based hash (MurmurHash3 fmix32), numpy and torch backends
# ----------------------------------------------------------------------------

def fmix32(h):
    """MurmurHash3 32-bit finaliser on Python ints or uint64 numpy arrays."""
    h = h & M32
    h = h ^ (h >> 16)
    h = (h * 0x85EBCA6B) & M32
    h = h ^ (h >> 13)
    h = (h * 0xC2B2AE35) & M32
    h = h ^ (h >> 16)
    return h


def stream_key(seed: int, *path: int) -> int:
    """Fold a seed and a path of small integers into one 32-bit key."""
    k = fmix32(int(seed) & M32)
    for p in path:
        k = fmix32((k ^ (int(p) & M32)) + GOLDEN)
    return int(k)


def hash_u16_np(key: int, start: int, n: int) -> np.ndarray:
    """Top 16 bits of fmix32((idx*GOLDEN + key) mod 2^32) for idx in [start, start+n)."""
    idx = np.arange(start, start + n, dtype=np.uint64)
    u = fmix32((idx * np.uint64(GOLDEN) + np.uint64(key)) & np.uint64(M32))
    return (u >> np.uint64(16)).astype(np.int64)


def _fmix32_torch(h):
    h = h & M32
    h = h ^ (h >> 16)
    h = (h * 0x85EBCA6B) & M32
    h = h ^ (h >> 13)
    h = (h * 0xC2B2AE35) & M32
    h = h ^ (h >> 16)
    return h


def hash_u16_torch(key: int, start: int, n: int, device):
    """Same values as :func:`hash_u16_np`, computed with int64 torch ops.

    Products of two values below 2^32 may wrap in int64; masking with 2^32-1
    keeps the exact low 32 bits, so the result equals the unsigned definition.
    """
    import torch
    idx = torch.arange(start, start + n, dtype=torch.int64, device=device)
    u = _fmix32_torch((idx * GOLDEN + key) & M32)
    return u >> 16


# ----------------------------------------------------------------------------
# storage formats
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest even); returns uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounding = ((u >> np.uint64(16)) & np.uint64(1)) + np.uint64(0x7FFF)
    return ((u + rounding) >> np.uint64(16)).astype(np.uint16)


@lru_cache(maxsize=None)
def quantile_table(sigma: float, dtype: str) -> np.ndarray:
    """65536-entry table of N(0, sigma^2) quantiles in the storage format.

    bf16: uint16 bit patterns; f32: float32 values.
    """
    from scipy.special import ndtri
    j = np.arange(65536, dtype=np.float64)
    q = (sigma * ndtri((j + 0.5) / 65536.0)).astype(np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(q)
    return q


# ----------------------------------------------------------------------------
# expert weights
# ----------------------------------------------------------------------------

def expert_key(cfg: MoEConfig, layer: int, expert: int, shared: bool = False) -> int:
    return stream_key(cfg.seed, S_SHARED if shared else S_EXPERT, layer, expert)


def expert_blob(cfg: MoEConfig, layer: int, expert: int, shared: bool = False) -> np.ndarray:
    """One expert's packed weights, flat, in storage format.

    Element order: W_gate [I][H], then W_up [I][H], then W_down [H][I], each
    row-major.  bf16 configs return uint16 bit patterns, f32 configs float32.
    """
    key = expert_key(cfg, layer, expert, shared)
    q = hash_u16_np(key, 0, cfg.blob_elems)
    return quantile_table(W_SIGMA, cfg.dtype)[q]


def expert_matrices(cfg: MoEConfig, layer: int, expert: int, shared: bool = False):
    """(W_gate [I][H], W_up [I][H], W_down [H][I]) in storage format (views of one blob)."""
    b = expert_blob(cfg, layer, expert, shared)
    n = cfg.H * cfg.I
    return (b[:n].reshape(cfg.I, cfg.H), b[n:2 * n].reshape(cfg.I, cfg.H),
            b[2 * n:].reshape(cfg.H, cfg.I))


def expert_blob_torch(cfg: MoEConfig, layer: int, expert: int, out, shared: bool = False,
                      chunk: int = 1 << 26):
    """Fill ``out`` (a flat torch tensor of ``blob_elems`` elements, bfloat16 or
    float32, on any device) with the same values as :func:`expert_blob`."""
    import torch
    key = expert_key(cfg, layer, expert, shared)
    tab = quantile_table(W_SIGMA, cfg.dtype)
    if cfg.dtype == "bf16":
        ttab = torch.from_numpy(tab.view(np.int16).copy()).to(out.device).view(torch.bfloat16)
    else:
        ttab = torch.from_numpy(tab.copy()).to(out.device)
    n = cfg.blob_elems
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        out[s:s + m] = ttab[hash_u16_torch(key, s, m, out.device)]
    return out


# ----------------------------------------------------------------------------
# router rows
# ----------------------------------------------------------------------------

def _rng(cfg: MoEConfig, *key) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(cfg.seed, spawn_key=tuple(key)))


def router_rows_f64(cfg: MoEConfig, layer: int) -> np.ndarray:
    """Unit-norm router rows W_g[e] (E x H), as the exact values stored.

    Drawn as normalised standard normals, then rounded to the storage format
    (bf16: via float32 with round-to-nearest-even).
    """
    g = _rng(cfg, S_ROUTER, layer).standard_normal((cfg.E, cfg.H))
    g /= np.linalg.norm(g, axis=1, keepdims=True)
    f = g.astype(np.float32)
    if cfg.dtype == "bf16":
        bits = f32_to_bf16_bits(f).astype(np.uint32) << np.uint32(16)
        f = bits.view(np.float32)
    return f.astype(np.float64)


def router_rows(cfg: MoEConfig, layer: int) -> np.ndarray:
    """Router rows in storage format (uint16 bf16 bits or float32)."""
    f = router_rows_f64(cfg, layer).astype(np.float32)
    return f32_to_bf16_bits(f) if cfg.dtype == "bf16" else f


# ----------------------------------------------------------------------------
# planted Markov routing trace
# ----------------------------------------------------------------------------

def transition_matrices(cfg: MoEConfig) -> np.ndarray:
    """T[l][e][f]: probability that layer-l slot draws f after layer l-1 chose e.

    Rows ~ Dirichlet(alpha * 1_E), drawn once.  T[0] is unused (layer 0 draws
    uniformly when it does not stay).
    """
    rng = _rng(cfg, S_TRANS)
    T = np.zeros((cfg.L, cfg.E, cfg.E))
    T[0] = 1.0 / cfg.E
    for l in range(1, cfg.L):
        T[l] = rng.dirichlet(np.full(cfg.E, cfg.alpha), size=cfg.E)
    return T


def planted_trace(cfg: MoEConfig, n_tokens: int | None = None, trans: np.ndarray | None = None,
                  p_stay: float | None = None) -> np.ndarray:
    """Planted expert selections sel[tok][b][l][k] for P profiling + T decode tokens.

    Per batch row and slot k: with probability p_stay keep the previous token's
    slot-k expert; otherwise draw from T[l][this token's layer l-1 slot-k
    expert] (uniform at layer 0).  A draw that collides with slots 0..k-1 is
    redrawn (non-stay distribution) up to 16 times, after which the most
    probable unused expert is taken (lower index on ties).
    """
    E, K, B, L = cfg.E, cfg.K, cfg.B, cfg.L
    n = cfg.P + cfg.T if n_tokens is None else n_tokens
    ps = cfg.p_stay if p_stay is None else p_stay
    T = transition_matrices(cfg) if trans is None else trans
    cdf = np.cumsum(T, axis=2)
    cdf[:, :, -1] = 1.0 + 1e-12
    rng = _rng(cfg, S_CHAIN)
    sel = np.zeros((n, B, L, K), dtype=np.int32)
    rows = np.arange(B)

    def draw_dist(l, b, k, t):
        if l == 0:
            return np.full(E, 1.0 / E)
        return T[l][sel[t, b, l - 1, k]]

    for t in range(n):
        for l in range(L):
            for k in range(K):
                u_stay = rng.random(B)
                u_draw = rng.random(B)
                if l == 0:
                    cand = np.minimum((u_draw * E).astype(np.int64), E - 1)
                else:
                    prev = sel[t, :, l - 1, k]
                    cand = (cdf[l][prev] > u_draw[:, None]).argmax(axis=1)
                if t > 0:
                    stay = u_stay < ps
                    cand = np.where(stay, sel[t - 1, :, l, k], cand)
                for b in rows:
                    c = int(cand[b])
                    used = sel[t, b, l, :k]
                    if k > 0 and np.any(used == c):
                        p = draw_dist(l, b, k, t)
                        c_cdf = np.cumsum(p)
                        c_cdf[-1] = 1.0 + 1e-12
                        ok = False
                        for _ in range(16):
                            c = int((c_cdf > rng.random()).argmax())
                            if not np.any(used == c):
                                ok = True
                                break
                        if not ok:
                            pm = p.copy()
                            pm[used] = -1.0
                            c = int(np.argmax(pm))   # argmax takes the lowest index on ties
                    sel[t, b, l, k] = c
    return sel


# ----------------------------------------------------------------------------
# hidden states
# ----------------------------------------------------------------------------

def hidden_f64(cfg: MoEConfig, planted: np.ndarray, tok: int, layer: int,
               wg: np.ndarray | None = None) -> np.ndarray:
    """Hidden state x[b][h] (exact stored values as float64) for trace token ``tok``.

    x = 3 * sum_{e in planted} W_g[e] + noise, noise ~ N(0, 1/256) from the
    hash stream keyed by (tok, layer); then rounded to the storage format.
    """
    if wg is None:
        wg = router_rows_f64(cfg, layer)
    B, H = cfg.B, cfg.H
    sig = PLANT_SCALE * wg[planted[tok, :, layer, :]].sum(axis=1)        # [B][H]
    key = stream_key(cfg.seed, S_NOISE, tok, layer)
    nz = quantile_table(NOISE_SIGMA, "f32")[hash_u16_np(key, 0, B * H)].reshape(B, H)
    x = (sig + nz.astype(np.float64)).astype(np.float32)
    if cfg.dtype == "bf16":
        x = (f32_to_bf16_bits(x).astype(np.uint32) << np.uint32(16)).view(np.float32)
    return x.astype(np.float64)


def to_storage(cfg: MoEConfig, a_f64: np.ndarray) -> np.ndarray:
    """Exact stored values (float64) -> storage format (uint16 bf16 bits or float32)."""
    f = np.asarray(a_f64, dtype=np.float32)
    return f32_to_bf16_bits(f) if cfg.dtype == "bf16" else f


def profiling_selections(cfg: MoEConfig, planted: np.ndarray) -> np.ndarray:
    """The P profiling tokens' selections sel[p][b][l][k] (the planted sets)."""
    return np.ascontiguousarray(planted[:cfg.P])
