"""Seeded synthetic inputs for the routed mixture-of-experts layer.

This module is shared by the HIP path's tests/benchmark and by the oracle. It
holds none of the layer's arithmetic: it only draws random bytes, normal and
Gumbel variates, and converts fp32 samples to bf16 bit patterns.

Every array is a pure function of (config, stream, index), so any expert or
token range can be regenerated alone, in any order, without drawing the rest:
the fp64 oracle regenerates just the experts a token sample touches, while the
GPU side uploads the full stacks.

Workloads (the paper's regimes, stood in for by synthetic data; the paper's
own inputs are a public-source code-prompt corpus on a real checkpoint):

=========  ======  =====  ====  ==  =====  ======  =========================
name       T       H      E     k   I      shared  routing
=========  ======  =====  ====  ==  =====  ======  =========================
tiny       16      256    8     2   128    0       bf16 router weights N(0, 0.02)
decode     64      4096   256   8   2048   1       logits N(0, 1)
prefill8k  8192    4096   256   8   2048   1       logits N(0, 1)
skew32k    32768   4096   256   8   2048   0       Zipf(1.2) popularity + Gumbel
tpshard    4096    4096   256   8   256    0       logits N(0, 1)
=========  ======  =====  ====  ==  =====  ======  =========================

prefill8k_bal is prefill8k with 'balanced' routing (every routed expert gets
exactly T*k/E = 256 rows, so no row tile is ragged): a measurement companion
of prefill8k, not a separate workload.

Common to all: activations x ~ N(0, 1) rounded to bf16; expert weights are FP4
e2m1 codes uniform over the 16 codes (bytes uniform over 0..255 hold two
independent codes); one E8M0 scale per 32 weights with exponent uniform over
-4..0 (bytes 123..127).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# stream ids of SeedSequence spawn keys
S_X, S_ROUTE, S_W13, S_W13S, S_W2, S_W2S, S_SPARE = 0, 1, 2, 3, 4, 5, 7
SCALE_LO, SCALE_HI = 123, 127          # e8m0 bytes: exponents -4..0


@dataclass(frozen=True)
class LayerConfig:
    name: str
    T: int
    H: int
    E: int
    k: int
    I: int
    n_shared: int = 0
    routing: str = "normal"      # 'router' | 'normal' | 'zipf' | 'balanced'
    seed: int = 0
    zipf_s: float = 1.2
    zipf_empty: int = 8          # least-popular experts forced empty (zipf only)

    @property
    def NE(self) -> int:
        return self.E + self.n_shared

    @property
    def k_total(self) -> int:
        return self.k + self.n_shared

    @property
    def A(self) -> int:
        return self.T * self.k_total

    def with_(self, **kw) -> "LayerConfig":
        d = dict(self.__dict__)
        d.update(kw)
        return LayerConfig(**d)


CONFIGS = {
    "tiny": LayerConfig("tiny", 16, 256, 8, 2, 128, 0, "router"),
    "decode": LayerConfig("decode", 64, 4096, 256, 8, 2048, 1, "normal"),
    "prefill8k": LayerConfig("prefill8k", 8192, 4096, 256, 8, 2048, 1, "normal"),
    "skew32k": LayerConfig("skew32k", 32768, 4096, 256, 8, 2048, 0, "zipf"),
    "tpshard": LayerConfig("tpshard", 4096, 4096, 256, 8, 256, 0, "normal"),
    "prefill8k_bal": LayerConfig("prefill8k_bal", 8192, 4096, 256, 8, 2048, 1, "balanced"),
}


def _rng(cfg: LayerConfig, stream: int, index: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(cfg.seed, spawn_key=(stream, index)))


def f32_to_bf16_bits(a) -> np.ndarray:
    """Round fp32 samples to bf16 (nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def gen_x(cfg: LayerConfig, rows=None) -> np.ndarray:
    """Activations x [T, H] as bf16 bits; token t is drawn from its own stream.

    ``rows``: optional token indices to generate (default all).
    """
    rows = range(cfg.T) if rows is None else rows
    out = np.empty((len(rows), cfg.H), np.uint16)
    for i, t in enumerate(rows):
        out[i] = f32_to_bf16_bits(_rng(cfg, S_X, int(t)).standard_normal(cfg.H, dtype=np.float32))
    return out


def gen_router_weight(cfg: LayerConfig) -> np.ndarray:
    """bf16 router weights Wr [E, H] ~ N(0, 0.02) (the 'router' routing only)."""
    r = _rng(cfg, S_ROUTE, 0).standard_normal((cfg.E, cfg.H), dtype=np.float32)
    return f32_to_bf16_bits(r * np.float32(0.02))


def gen_logits(cfg: LayerConfig) -> np.ndarray:
    """fp32 router logits [T, E] for 'normal', 'zipf' and 'balanced' routing.

    normal: iid N(0, 1), near-uniform expert load.
    zipf:   expert with popularity rank r gets bias -s*ln(r) (the ``zipf_empty``
            least popular get -30, which keeps them empty); logit = bias +
            Gumbel(0, 1) in fp64, then rounded to fp32. Top-k of Gumbel-perturbed
            log-weights samples k experts without replacement with probability
            proportional to r**-s.
    """
    if cfg.routing == "normal":
        return _rng(cfg, S_ROUTE, 1).standard_normal((cfg.T, cfg.E), dtype=np.float32)
    if cfg.routing == "balanced":
        # token t picks experts (t*k + j) % E, j = 0..k-1, in that order
        # (logit 16 - j); every other logit is N(0, 1) clipped to [-8, 8].
        # Expert e then holds exactly T*k/E assignments when E divides T*k.
        lg = np.clip(_rng(cfg, S_ROUTE, 3).standard_normal((cfg.T, cfg.E), dtype=np.float32),
                     -8, 8)
        t = np.arange(cfg.T)[:, None]
        j = np.arange(cfg.k)[None, :]
        lg[np.broadcast_to(t, (cfg.T, cfg.k)), (t * cfg.k + j) % cfg.E] = 16.0 - j
        return lg
    if cfg.routing == "zipf":
        rng = _rng(cfg, S_ROUTE, 2)
        rank = rng.permutation(cfg.E) + 1
        bias = -cfg.zipf_s * np.log(rank.astype(np.float64))
        bias[rank > cfg.E - cfg.zipf_empty] = -30.0
        u = rng.random((cfg.T, cfg.E))
        gumbel = -np.log(-np.log(u))
        return (bias[None, :] + gumbel).astype(np.float32)
    raise ValueError(f"routing {cfg.routing!r} has no given logits")


@dataclass
class Expert:
    w13: np.ndarray     # uint8 [2I, H/2]
    w13s: np.ndarray    # uint8 [2I, H/32]
    w2: np.ndarray      # uint8 [H, I/2]
    w2s: np.ndarray     # uint8 [H, I/32]


def gen_expert(cfg: LayerConfig, e: int) -> Expert:
    """Weights of expert e (0 <= e < NE; e == E is the shared expert)."""
    if not 0 <= e < cfg.NE:
        raise IndexError(e)
    h, i = cfg.H, cfg.I

    def codes(stream, n, kk):
        return np.frombuffer(_rng(cfg, stream, e).bytes(n * kk // 2), np.uint8).reshape(n, kk // 2)

    def scales(stream, n, kk):
        return _rng(cfg, stream, e).integers(SCALE_LO, SCALE_HI + 1, (n, kk // 32), dtype=np.uint8)

    return Expert(codes(S_W13, 2 * i, h), scales(S_W13S, 2 * i, h),
                  codes(S_W2, h, i), scales(S_W2S, h, i))


class LazyExperts:
    """Indexable view ``[e]`` of one weight array kind, generating on demand.

    kind: 'w13' | 'w13s' | 'w2' | 'w2s'. A small cache keeps the last few
    experts so the four kinds of one expert are drawn once.
    """

    _cache: dict = {}

    def __init__(self, cfg: LayerConfig, kind: str, cache_size: int = 4):
        self.cfg, self.kind, self.cache_size = cfg, kind, cache_size

    def __getitem__(self, e):
        key = (self.cfg, int(e))
        ex = LazyExperts._cache.get(key)
        if ex is None:
            ex = gen_expert(self.cfg, int(e))
            if len(LazyExperts._cache) >= self.cache_size:
                LazyExperts._cache.pop(next(iter(LazyExperts._cache)))
            LazyExperts._cache[key] = ex
        return getattr(ex, self.kind)

    def __len__(self):
        return self.cfg.NE


def lazy_weights(cfg: LayerConfig):
    """(w13, w13s, w2, w2s) as :class:`LazyExperts` views."""
    return tuple(LazyExperts(cfg, k) for k in ("w13", "w13s", "w2", "w2s"))


def gen_all_experts(cfg: LayerConfig):
    """Stacked weights (w13 [NE,2I,H/2], w13s [NE,2I,H/32], w2 [NE,H,I/2], w2s [NE,H,I/32])."""
    h, i, ne = cfg.H, cfg.I, cfg.NE
    w13 = np.empty((ne, 2 * i, h // 2), np.uint8)
    w13s = np.empty((ne, 2 * i, h // 32), np.uint8)
    w2 = np.empty((ne, h, i // 2), np.uint8)
    w2s = np.empty((ne, h, i // 32), np.uint8)
    for e in range(ne):
        ex = gen_expert(cfg, e)
        w13[e], w13s[e], w2[e], w2s[e] = ex.w13, ex.w13s, ex.w2, ex.w2s
    return w13, w13s, w2, w2s


@dataclass
class LayerInputs:
    cfg: LayerConfig
    x: np.ndarray                       # uint16 [T, H]
    logits: np.ndarray | None           # float32 [T, E] or None
    wr: np.ndarray | None               # uint16 [E, H] or None
    weights: tuple = field(repr=False)  # (w13, w13s, w2, w2s), stacked or lazy


def make_inputs(cfg: LayerConfig, lazy: bool = False) -> LayerInputs:
    """All inputs of one workload; ``lazy`` keeps the weights as generators."""
    logits = None if cfg.routing == "router" else gen_logits(cfg)
    wr = gen_router_weight(cfg) if cfg.routing == "router" else None
    weights = lazy_weights(cfg) if lazy else gen_all_experts(cfg)
    return LayerInputs(cfg, gen_x(cfg), logits, wr, weights)
