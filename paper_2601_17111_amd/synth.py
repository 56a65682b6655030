"""Seeded synthetic inputs for the imbalanced MoE expert layer.

This module only draws inputs: routing ids, gates, token activations and
expert weights. It holds none of the layer's arithmetic and is the one piece
of code that both the CPU checks and the GPU library's callers use.

Recipe (the paper's controlled experiments, Sec. 5.1, concentrate a fraction
of the routing onto a hot set of experts and spread the rest evenly over the
other experts; the layer shapes are those of Sec. 5.1 and of public MoE
models):

* ids: i.i.d. per token-expert pair (an expert may repeat inside a token),
  except where a config asks for distinct experts per token;
    - "hot":   with probability f the pair goes to a uniform expert of the hot
               set {0, .., k-1}, else to a uniform expert of {k, .., E-1};
    - "zipf":  expert perm[r] has probability proportional to (r+1)^-s, with
               perm a seeded permutation of the experts;
    - "forced_tokens": a seeded set of round(f*T) tokens each route one of
               their K distinct slots to expert 0; every other slot is a
               distinct uniform expert;
    - "balanced": exactly R/E pairs per expert, shuffled (R % E == 0);
    - "loads":  exactly the given number of pairs per expert, shuffled
               (the counts sum to T*K);
* gates: softmax over K i.i.d. N(0, 1) logits per token, float32;
* x: N(0, 1), rounded to bfloat16 (round-to-nearest-even) for bf16 layers;
* weights: N(0, 0.02^2) per expert, drawn with torch's generator on the
  device that will hold them (seeded per expert), rounded to the layer dtype.

Random streams: numpy PCG64 seeded by SeedSequence(seed), spawned in the fixed
order (ids, gates, x).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from fractions import Fraction
from typing import Optional, Sequence, Tuple

import numpy as np


@dataclass(frozen=True)
class LayerConfig:
    name: str
    T: int          # tokens in the layer
    D: int          # hidden size
    F: int          # SwiGLU intermediate size
    E: int          # experts
    K: int          # experts per token
    P: int          # devices
    alpha: Fraction  # capacity factor
    dtype: str      # "bf16" or "f32"
    routing: Tuple  # see module docstring
    distinct: bool = False
    min_chunk: int = 1
    lam: float = 0.0
    seeds: Tuple[int, ...] = (0,)

    @property
    def R(self) -> int:
        return self.T * self.K

    @property
    def M(self) -> int:
        return self.E // self.P

    @property
    def capacity(self) -> int:
        """ceil(alpha * T * K / P) pairs per device."""
        return int(math.ceil(Fraction(self.alpha) * self.R / self.P))

    def with_(self, **kw) -> "LayerConfig":
        return replace(self, **kw)


CONFIGS = {
    "tiny-fp32": LayerConfig(
        "tiny-fp32", T=256, D=64, F=128, E=8, K=2, P=4,
        alpha=Fraction(5, 4), dtype="f32",
        routing=("forced_tokens", 0.7), distinct=True),
    "gpt-oss-20b": LayerConfig(
        "gpt-oss-20b", T=16384, D=2880, F=2880, E=32, K=4, P=8,
        alpha=Fraction(11, 10), dtype="bf16", routing=("hot", 0.6, 4)),
    "gpt-oss-120b": LayerConfig(
        "gpt-oss-120b", T=32768, D=2880, F=2880, E=128, K=4, P=8,
        alpha=Fraction(11, 10), dtype="bf16", routing=("hot", 0.8, 1),
        seeds=(0, 1, 2)),
    "qwen3-30b-a3b": LayerConfig(
        "qwen3-30b-a3b", T=65536, D=2048, F=768, E=128, K=8, P=8,
        alpha=Fraction(11, 10), dtype="bf16", routing=("zipf", 1.2)),
    "deepseek-v3": LayerConfig(
        "deepseek-v3", T=8192, D=7168, F=2048, E=256, K=8, P=8,
        alpha=Fraction(1, 1), dtype="bf16", routing=("hot", 0.95, 1)),
}

# the gpt-oss-120b layer is swept over hot sets of 16, 4 and 1 experts
GPT_OSS_120B_HOT_SETS = (16, 4, 1)


def gpt_oss_120b(hot: int) -> LayerConfig:
    c = CONFIGS["gpt-oss-120b"]
    return c.with_(name=f"gpt-oss-120b-hot{hot}", routing=("hot", 0.8, hot))


# ---------------------------------------------------------------------------
# drawing
# ---------------------------------------------------------------------------

def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(3)]


def draw_ids(cfg: LayerConfig, rng: np.random.Generator) -> np.ndarray:
    """Routing ids, int32 [T, K]."""
    T, K, E = cfg.T, cfg.K, cfg.E
    kind = cfg.routing[0]
    if kind == "hot":
        f, k = cfg.routing[1], cfg.routing[2]
        R = T * K
        is_hot = rng.random(R) < f
        hot = rng.integers(0, k, size=R)
        rest = rng.integers(k, E, size=R) if k < E else hot
        ids = np.where(is_hot, hot, rest)
    elif kind == "zipf":
        s = cfg.routing[1]
        perm = rng.permutation(E)
        w = np.arange(1, E + 1, dtype=np.float64) ** (-s)
        prob = np.empty(E)
        prob[perm] = w / w.sum()
        ids = rng.choice(E, size=T * K, p=prob)
    elif kind == "forced_tokens":
        f = cfg.routing[1]
        assert cfg.distinct and K == 2
        n_forced = int(round(f * T))
        forced = np.zeros(T, dtype=bool)
        forced[rng.choice(T, size=n_forced, replace=False)] = True
        first = rng.integers(0, E, size=T)
        second = (first + rng.integers(1, E, size=T)) % E
        slot = rng.integers(0, 2, size=T)
        other = rng.integers(1, E, size=T)
        a = np.where(forced, np.where(slot == 0, 0, other), first)
        b = np.where(forced, np.where(slot == 0, other, 0), second)
        ids = np.stack([a, b], axis=1)
    elif kind == "balanced":
        R = T * K
        assert R % E == 0
        ids = rng.permutation(np.repeat(np.arange(E), R // E))
    elif kind == "loads":
        counts = np.asarray(cfg.routing[1], dtype=np.int64)
        assert len(counts) == E and counts.sum() == T * K
        ids = rng.permutation(np.repeat(np.arange(E), counts))
    else:
        raise ValueError(kind)
    return np.ascontiguousarray(ids.reshape(T, K).astype(np.int32))


def draw_gates(cfg: LayerConfig, rng: np.random.Generator) -> np.ndarray:
    """Softmax over K i.i.d. N(0, 1) logits per token, float32 [T, K]."""
    z = rng.standard_normal((cfg.T, cfg.K))
    z = z - z.max(axis=1, keepdims=True)
    w = np.exp(z)
    return np.ascontiguousarray((w / w.sum(axis=1, keepdims=True)).astype(np.float32))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); the result
    is float32 holding bf16-representable values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) >> 16 << 16
    return bits.astype(np.uint32).view(np.float32)


def draw_x(cfg: LayerConfig, rng: np.random.Generator) -> np.ndarray:
    """Token activations N(0, 1), float32 [T, D] (bf16-valued for bf16)."""
    x = rng.standard_normal((cfg.T, cfg.D), dtype=np.float32)
    return round_to_bf16(x) if cfg.dtype == "bf16" else x


@dataclass
class LayerInputs:
    cfg: LayerConfig
    seed: int
    ids: np.ndarray      # int32 [T, K]
    gates: np.ndarray    # float32 [T, K]
    x: np.ndarray        # float32 [T, D] (bf16-valued for bf16 layers)
    extra: dict = field(default_factory=dict)

    @property
    def capacity(self) -> int:
        return self.cfg.capacity


def make_inputs(cfg: LayerConfig, seed: int = 0, with_x: bool = True) -> LayerInputs:
    r_ids, r_gates, r_x = _streams(seed)
    ids = draw_ids(cfg, r_ids)
    gates = draw_gates(cfg, r_gates)
    x = draw_x(cfg, r_x) if with_x else np.zeros((0, cfg.D), np.float32)
    return LayerInputs(cfg, seed, ids, gates, x)


def expert_seed(seed: int, e: int) -> int:
    """A 63-bit seed for expert e's weights."""
    return int(np.random.SeedSequence([seed, e]).generate_state(1, np.uint64)[0]
               & np.uint64(0x7FFFFFFFFFFFFFFF))


def make_weights(cfg: LayerConfig, seed: int, device="cpu",
                 experts: Optional[Sequence[int]] = None, std: float = 0.02):
    """Expert weights as torch tensors on `device`.

    Returns (w_gate [E, D, F], w_up [E, D, F], w_down [E, F, D]) in the
    layer dtype; experts not in `experts` (default: all) are left zero.
    """
    import torch

    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    E, D, F = cfg.E, cfg.D, cfg.F
    wg = torch.zeros((E, D, F), dtype=dt, device=device)
    wu = torch.zeros((E, D, F), dtype=dt, device=device)
    wd = torch.zeros((E, F, D), dtype=dt, device=device)
    gen = torch.Generator(device=device)
    for e in (range(E) if experts is None else experts):
        gen.manual_seed(expert_seed(seed, e))
        for w, shape in ((wg, (D, F)), (wu, (D, F)), (wd, (F, D))):
            w[e].copy_((torch.randn(shape, generator=gen, device=device,
                                    dtype=torch.float32) * std).to(dt))
    return wg, wu, wd
