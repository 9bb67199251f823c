"""Workload recipes: shapes, lengths, per-fragment K scales and delivery lists.

Every recipe is a pure function of its seed (numpy PCG64). Fragments carry
per-layer K and V of shape [1, H, T, d]; the thinker-side RoPE at local
positions 0..T-1 is applied *in distribution*: for an isotropic Gaussian key
k ~ N(0, s^2 I), the rotated key R(t) k has exactly the same law, so drawing
N(0, s^2 I) directly samples post-rotation keys without any rotation code here.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    L: int                       # layers
    H: int                       # KV heads
    d: int                       # head dimension
    dtype: str                   # "float32" | "bfloat16"
    rope_base: float
    routing_layer: int           # 0-based layer index used for the K-norm score
    lengths: Tuple[int, ...]     # token count of each distinct fragment
    k_scale: Tuple[float, ...]   # standard deviation of each distinct fragment's K
    deliveries: Tuple[int, ...]  # arrival list: index of the distinct fragment delivered
    shared_k: Tuple[Tuple[int, int], ...] = ()  # (src, dst): dst reuses src's K at every layer
    seed: int = 42
    description: str = field(default="", compare=False)

    @property
    def n_distinct(self) -> int:
        return len(self.lengths)

    @property
    def n_deliveries(self) -> int:
        return len(self.deliveries)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "float32" else 2

    def fragment_bytes(self, i: int) -> int:
        """Bytes of all layers' K and V of distinct fragment i."""
        return 2 * self.L * self.H * self.lengths[i] * self.d * self.elem_bytes

    @property
    def merged_tokens(self) -> int:
        return int(sum(self.lengths))

    @property
    def render_bytes(self) -> int:
        """Read + write bytes of rendering every distinct fragment once."""
        return 2 * sum(self.fragment_bytes(i) for i in range(self.n_distinct))

    @property
    def delivery_bytes(self) -> int:
        return sum(self.fragment_bytes(i) for i in self.deliveries)


def _spread_lognormal(rng: np.random.Generator, n: int, sigma: float,
                      min_log_gap: float) -> Tuple[float, ...]:
    """Log-normal scales exp(sigma * z), pushed apart so that any two differ by
    at least min_log_gap in log space (keeps fragments' K-norm scores separable)."""
    z = rng.standard_normal(n) * sigma
    order = np.argsort(z, kind="stable")
    ls = z[order].copy()
    for k in range(1, n):
        ls[k] = max(ls[k], ls[k - 1] + min_log_gap)
    out = np.empty(n)
    out[order] = ls
    return tuple(float(np.exp(v)) for v in out)


def tiny(seed: int = 42) -> Workload:
    """2 fragments of 16 and 24 tokens; L=2, H=2, d=64, fp32; K scaled by 1+0.5j."""
    return Workload(
        name="tiny", L=2, H=2, d=64, dtype="float32", rope_base=1e4, routing_layer=1,
        lengths=(16, 24), k_scale=(1.0, 1.5), deliveries=(0, 1), seed=seed,
        description="Tiny: N=2 (16+24 tokens), L=2, H=2, d=64, fp32, base 1e4, layer 1")


def qwen3_17b_n2(seed: int = 42) -> Workload:
    rng = np.random.default_rng(seed)
    return Workload(
        name="qwen3-1.7b-n2", L=28, H=8, d=128, dtype="bfloat16", rope_base=1e6,
        routing_layer=14, lengths=(512, 768),
        k_scale=_spread_lognormal(rng, 2, 0.3, 0.01), deliveries=(0, 1), seed=seed,
        description="Qwen3-1.7B-shaped N=2 (512+768 tokens), bf16, base 1e6, layer 14")


def qwen3_17b_n5(seed: int = 42) -> Workload:
    rng = np.random.default_rng(seed)
    lengths = tuple(int(t) for t in rng.integers(256, 2049, size=5))
    scales = _spread_lognormal(rng, 5, 0.3, 0.01)
    mult = rng.integers(1, 4, size=5)
    deliveries = np.repeat(np.arange(5), mult)
    rng.shuffle(deliveries)
    return Workload(
        name="qwen3-1.7b-n5", L=28, H=8, d=128, dtype="bfloat16", rope_base=1e6,
        routing_layer=14, lengths=lengths, k_scale=scales,
        deliveries=tuple(int(x) for x in deliveries), seed=seed,
        description="Qwen3-1.7B-shaped N=5, T~U[256,2048], each delivered 1-3x, shuffled")


def qwen3_4b_n4(seed: int = 42) -> Workload:
    rng = np.random.default_rng(seed)
    return Workload(
        name="qwen3-4b-n4", L=36, H=8, d=128, dtype="bfloat16", rope_base=1e6,
        routing_layer=18, lengths=(4096,) * 4,
        k_scale=_spread_lognormal(rng, 4, 0.3, 0.01), deliveries=(0, 1, 2, 3), seed=seed,
        description="Qwen3-4B-shaped N=4 x 4096 tokens, bf16, base 1e6, layer 18")


def qwen3_4b_large(seed: int = 42) -> Workload:
    """31 distinct fragments (T~U[2048,16384], total in [250k, 270k] tokens)
    delivered 32 times: one fragment arrives twice, and one pair shares every
    layer's K (equal scores, so their order falls to the content hash)."""
    n = 31
    s = seed
    while True:
        rng = np.random.default_rng(s)
        lengths = rng.integers(2048, 16385, size=n)
        a, b = (int(x) for x in rng.choice(n, size=2, replace=False))
        lengths[b] = lengths[a]          # the equal-score pair shares K, hence T
        if 250_000 <= int(lengths.sum()) <= 270_000:
            break
        s += 1
    scales = _spread_lognormal(rng, n, 0.3, 0.01)
    dup = int(rng.integers(0, n))
    deliveries = np.concatenate([np.arange(n), [dup]])
    rng.shuffle(deliveries)
    return Workload(
        name="qwen3-4b-large", L=36, H=8, d=128, dtype="bfloat16", rope_base=1e6,
        routing_layer=18, lengths=tuple(int(t) for t in lengths), k_scale=scales,
        deliveries=tuple(int(x) for x in deliveries), shared_k=((a, b),), seed=seed,
        description="Qwen3-4B-shaped large: 32 deliveries / 31 distinct, ~260k merged tokens, "
                    "one duplicate delivery, one equal-score pair")


def custom(name: str = "custom", *, L: int = 2, H: int = 2, d: int = 128,
           dtype: str = "bfloat16", rope_base: float = 1e6, routing_layer: int = 0,
           lengths=(300, 517), deliveries=None, k_scale=None, shared_k=(),
           seed: int = 7) -> Workload:
    """Small workload for parity tests (ragged lengths, many tiles)."""
    rng = np.random.default_rng(seed)
    lengths = tuple(int(t) for t in lengths)
    if k_scale is None:
        k_scale = _spread_lognormal(rng, len(lengths), 0.3, 0.01)
    if deliveries is None:
        deliveries = tuple(range(len(lengths)))
    return Workload(name=name, L=L, H=H, d=d, dtype=dtype, rope_base=rope_base,
                    routing_layer=routing_layer, lengths=lengths,
                    k_scale=tuple(float(x) for x in k_scale),
                    deliveries=tuple(int(x) for x in deliveries),
                    shared_k=tuple(shared_k), seed=seed)


WORKLOADS: Dict[str, callable] = {
    "tiny": tiny,
    "qwen3-1.7b-n2": qwen3_17b_n2,
    "qwen3-1.7b-n5": qwen3_17b_n5,
    "qwen3-4b-n4": qwen3_4b_n4,
    "qwen3-4b-large": qwen3_4b_large,
}


def workload(name: str, seed: int = 42) -> Workload:
    return WORKLOADS[name](seed)
