"""Seeded synthetic inputs for the sharded expert-FFN MoE layer.

This module only draws random numbers: activations, gate and expert weights, and the
per-token routing targets that stand in for the paper's skewed router (Section 4.1,
"Router" paragraph and its probability formula).  It holds none of the layer's own
arithmetic -- no logits, softmax, top-k, grouping, GEMM or activation -- so that the
fp64 oracle and the HIP path can both consume it without sharing any method code.

Skew is injected through a per-token selection bias: every expert in a token's sampled
target set gets +BIAS_BETA added to its gate logit before top-k, every other expert gets
0.  BIAS_BETA is far above the spread of the raw logits (std about 0.6 for these
weight scales), so the selected set equals the sampled set while the order inside it and
the gate weights still come from the unbiased logits.  The paper's own evaluation runs
Switch-Base on BookCorpus; neither the trained weights nor the dataset are used here --
these Gaussian tensors of the same shapes stand in for them.

All tensors are returned as float32 arrays holding values that are exactly
representable in the configuration's dtype (bf16 configs are rounded to nearest-even
bf16 here, once); ``bf16_bits`` gives the matching uint16 bit patterns.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

BIAS_BETA = 32.0

# stream ids for np.random.SeedSequence(seed, spawn_key=(stream, shard))
_X, _WG, _W1, _W3, _W2, _ROUTE = range(6)


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    """One MoE layer workload.

    h: model hidden size (the paper's h_i); F: full FFN inner width (the paper's h_o);
    G: number of shards the inner width is split into; shard: which contiguous slice
    [shard*f, (shard+1)*f) of the inner width this device holds (Section 3.2).
    routing: ("gate",) pure gate, no bias; ("zipf", s) Zipf popularity with exponent s;
    ("paper", k_r, alpha_r) the paper's router; ("pair", frac) a fixed hot pair for a
    fraction of tokens, uniform distinct pairs otherwise; ("uniform",).
    """

    name: str
    T: int
    h: int
    E: int
    k: int
    F: int
    G: int = 1
    shard: int = 0
    act: str = "gelu"  # "gelu" (erf form) | "gelu_tanh" | "swiglu"
    dtype: str = "bf16"  # "bf16" | "f32"
    w_std: float = 0.02
    routing: tuple = ("gate",)
    renorm: int = 0

    @property
    def f(self) -> int:
        return self.F // self.G

    @property
    def A(self) -> int:
        return self.T * self.k

    def with_(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


def _alpha_for_share(k_r: int, E: int, share: float) -> float:
    """alpha_r of the paper's router that gives the k_r hot experts `share` of tokens."""
    return (share - k_r / E) / ((1.0 - share) * k_r)


CONFIGS = {
    # tiny top-1 layer, fp32, full experts
    "c1": LayerConfig("c1", T=512, h=768, E=8, k=1, F=3072, dtype="f32", routing=("gate",)),
    # Switch-base-like layer, 32 x 256 tokens, Zipf(1.0) popularity
    "c2": LayerConfig("c2", T=8192, h=768, E=64, k=1, F=3072, routing=("zipf", 1.0)),
    # one device's 1/8 shard of a 128-expert layer, 8 hot experts get 80 % of tokens
    "c3": LayerConfig("c3", T=16384, h=1024, E=128, k=1, F=4096, G=8,
                      routing=("paper", 8, _alpha_for_share(8, 128, 0.8))),
    # Mixtral-shaped top-2 SwiGLU layer, one device's 1/8 shard
    "c4": LayerConfig("c4", T=4096, h=4096, E=8, k=2, F=14336, G=8, act="swiglu",
                      w_std=0.01, routing=("zipf", 1.2), renorm=1),
    # extreme skew: 95 % of tokens send both picks to one hot pair
    "c5": LayerConfig("c5", T=32768, h=1024, E=64, k=2, F=4096, routing=("pair", 0.95), renorm=1),
    # decode-shaped run of the same layer
    "c5dec": LayerConfig("c5dec", T=64, h=1024, E=64, k=2, F=4096, routing=("pair", 0.95), renorm=1),
    # uniform-routing twins (baselines for the skew comparison)
    "c3u": LayerConfig("c3u", T=16384, h=1024, E=128, k=1, F=4096, G=8, routing=("uniform",)),
    "c5u": LayerConfig("c5u", T=32768, h=1024, E=64, k=2, F=4096, routing=("uniform",), renorm=1),
    # the paper's own evaluation shape: b=250, s=120, h=768, 4-way shard of a 3072 FFN,
    # 128 experts, k_r = 10 % of experts, alpha_r = 0.6
    "paper128": LayerConfig("paper128", T=30000, h=768, E=128, k=1, F=3072, G=4,
                            routing=("paper", 13, 0.6)),
}


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    return bf16_bits_to_f32(f32_to_bf16_bits(a))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(seed: int, stream: int, sub: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(stream, sub)))


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    v = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        v *= np.float32(std)
    return v


def _draw_distinct(rng: np.random.Generator, p: np.ndarray, T: int, k: int) -> np.ndarray:
    """k distinct ids per token, drawn one after another without replacement from p."""
    E = p.shape[0]
    out = np.empty((T, k), dtype=np.int32)
    taken = np.zeros((T, E), dtype=bool)
    for j in range(k):
        q = np.broadcast_to(p, (T, E)).copy()
        q[taken] = 0.0
        c = np.cumsum(q, axis=1)
        u = rng.random(T) * c[:, -1]
        # first slot whose cumulative mass exceeds u: it has nonzero mass, so it is free
        pick = (c <= u[:, None]).sum(axis=1)
        if (pick >= E).any() or taken[np.arange(T), pick].any():
            raise AssertionError("inverse-CDF draw landed outside the free slots")
        out[:, j] = pick
        taken[np.arange(T), pick] = True
    return out


def routing_targets(cfg: LayerConfig, seed: int) -> Optional[np.ndarray]:
    """Sampled target expert set S_t for each token (sorted ids), or None for the pure gate."""
    kind = cfg.routing[0]
    if kind == "gate":
        return None
    rng = _rng(seed, _ROUTE)
    E, T, k = cfg.E, cfg.T, cfg.k
    perm = rng.permutation(E)
    if kind == "uniform":
        tg = _draw_distinct(rng, np.full(E, 1.0 / E), T, k)
    elif kind == "zipf":
        s = float(cfg.routing[1])
        p = np.empty(E)
        p[perm] = 1.0 / np.arange(1, E + 1, dtype=np.float64) ** s
        tg = _draw_distinct(rng, p / p.sum(), T, k)
    elif kind == "paper":
        # the paper's router: p_i proportional to 1/|E| + alpha_r for the k_r skewed
        # experts, 1/|E| for the others; skewed ids are a seeded permutation's first k_r
        k_r, alpha = int(cfg.routing[1]), float(cfg.routing[2])
        p = np.full(E, 1.0 / E)
        p[perm[:k_r]] += alpha
        tg = _draw_distinct(rng, p / p.sum(), T, k)
    elif kind == "pair":
        frac = float(cfg.routing[1])
        if k != 2:
            raise ValueError("pair routing needs k = 2")
        hot = np.sort(perm[:2])
        tg = _draw_distinct(rng, np.full(E, 1.0 / E), T, k)
        use_hot = rng.random(T) < frac
        tg[use_hot] = hot
    else:
        raise ValueError(f"unknown routing {cfg.routing}")
    return np.sort(tg, axis=1).astype(np.int32)


@dataclasses.dataclass
class Layer:
    cfg: LayerConfig
    seed: int
    x: np.ndarray  # [T, h]
    wg: np.ndarray  # [E, h]  (nn.Linear layout: row e is expert e's gate vector)
    w1: Optional[np.ndarray]  # [E, h, f]  shard columns of W_i (SwiGLU: the gate projection)
    w3: Optional[np.ndarray]  # [E, h, f]  SwiGLU up projection, same columns
    w2: Optional[np.ndarray]  # [E, f, h]  shard rows of W_o
    sel_bias: Optional[np.ndarray]  # [T, E] float32
    targets: Optional[np.ndarray]  # [T, k] sorted target ids

    def bits(self, name: str) -> np.ndarray:
        return f32_to_bf16_bits(getattr(self, name))


def _expert_weights(cfg: LayerConfig, seed: int, stream: int, shard: int, rows_are_inner: bool):
    shape = (cfg.E, cfg.f, cfg.h) if rows_are_inner else (cfg.E, cfg.h, cfg.f)
    w = _normal(_rng(seed, stream, shard), shape, cfg.w_std)
    return round_to_bf16(w) if cfg.dtype == "bf16" else w


def make(cfg, seed: int = 0, weights: bool = True, **overrides) -> Layer:
    """Generate one layer's inputs.  `cfg` is a LayerConfig or a name in CONFIGS.

    Shard g of the full width-F weights is drawn from its own stream, so the full
    layer is by definition the concatenation of its G shards along the inner width.
    weights=False skips the expert weights (w1/w3/w2 are None) for routing-only use.
    """
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    if overrides:
        cfg = cfg.with_(**overrides)
    if cfg.F % cfg.G:
        raise ValueError("F must divide into G shards")
    rnd = round_to_bf16 if cfg.dtype == "bf16" else (lambda a: a)
    x = rnd(_normal(_rng(seed, _X), (cfg.T, cfg.h), 1.0))
    wg = rnd(_normal(_rng(seed, _WG), (cfg.E, cfg.h), cfg.w_std))
    w1 = w3 = w2 = None
    if weights:
        w1 = _expert_weights(cfg, seed, _W1, cfg.shard, False)
        w3 = _expert_weights(cfg, seed, _W3, cfg.shard, False) if cfg.act == "swiglu" else None
        w2 = _expert_weights(cfg, seed, _W2, cfg.shard, True)
    tg = routing_targets(cfg, seed)
    bias = None
    if tg is not None:
        bias = np.zeros((cfg.T, cfg.E), dtype=np.float32)
        np.put_along_axis(bias, tg.astype(np.int64), np.float32(BIAS_BETA), axis=1)
    return Layer(cfg, seed, x, wg, w1, w3, w2, bias, tg)


def full_width_weights(cfg, seed: int = 0):
    """All G shards concatenated along the inner width: (w1, w3, w2) of the unsharded layer."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    w1 = np.concatenate([_expert_weights(cfg, seed, _W1, g, False) for g in range(cfg.G)], axis=2)
    w3 = (np.concatenate([_expert_weights(cfg, seed, _W3, g, False) for g in range(cfg.G)], axis=2)
          if cfg.act == "swiglu" else None)
    w2 = np.concatenate([_expert_weights(cfg, seed, _W2, g, True) for g in range(cfg.G)], axis=1)
    return w1, w3, w2
