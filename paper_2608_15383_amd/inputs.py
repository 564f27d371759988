"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module only draws random numbers and rounds them to bf16; it holds none
of the layer's arithmetic.  Shapes follow the OLMoE-shaped MoE layer studied
in the paper (16 sparse layers, 64 experts, top-8, hidden 2048, expert
intermediate 1024).  Draw order for one layer: W_gate, W_up [E][f][d],
W_down [E][d][f], W_router [E][d], h [T][d].
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even); returns uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to the float32 values they denote (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class LayerShape:
    d_model: int
    d_ff: int
    n_experts: int
    top_k: int


@dataclass
class LayerInputs:
    shape: LayerShape
    w_gate: np.ndarray    # uint16 bf16 bits [E, f, d]
    w_up: np.ndarray      # uint16 bf16 bits [E, f, d]
    w_down: np.ndarray    # uint16 bf16 bits [E, d, f]
    w_router: np.ndarray  # uint16 bf16 bits [E, d]
    h: np.ndarray         # uint16 bf16 bits [T, d]

    def f32(self, name: str) -> np.ndarray:
        return bf16_bits_to_f32(getattr(self, name))


def _normal_bf16(rng, shape, std):
    x = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std)
    return f32_to_bf16_bits(x)


def make_layer(shape: LayerShape, tokens: int, seed: int, weight_std: float = 0.02,
               router_std: float = 0.02, act_std: float = 1.0, n_experts_drawn=None) -> LayerInputs:
    """Draw one layer's weights ~N(0, 0.02), router ~N(0, 0.02) and h ~N(0, 1) as bf16."""
    rng = np.random.default_rng(seed)
    e, f, d = shape.n_experts, shape.d_ff, shape.d_model
    ne = e if n_experts_drawn is None else n_experts_drawn
    w_gate = _normal_bf16(rng, (ne, f, d), weight_std)
    w_up = _normal_bf16(rng, (ne, f, d), weight_std)
    w_down = _normal_bf16(rng, (ne, d, f), weight_std)
    w_router = _normal_bf16(rng, (e, d), router_std)
    h = _normal_bf16(rng, (tokens, d), act_std)
    return LayerInputs(shape, w_gate, w_up, w_down, w_router, h)


def spread_logits(tokens: int, n_experts: int, top_k: int, distinct: int, seed: int) -> np.ndarray:
    """Logits that make the batch touch exactly `distinct` experts.

    Token t prefers experts (top_k*t + j) mod distinct for j < top_k with
    logits 3 - 0.25 j; every other logit is -4 + N(0, 0.1).  Used for the
    16-token multi-wave workload.
    """
    rng = np.random.default_rng(seed)
    z = (-4.0 + 0.1 * rng.standard_normal((tokens, n_experts))).astype(np.float32)
    for t in range(tokens):
        for j in range(top_k):
            z[t, (top_k * t + j) % distinct] = np.float32(3.0 - 0.25 * j)
    return z


def zipf_gumbel_logits(tokens: int, n_experts: int, s: float, perm: np.ndarray, rng) -> np.ndarray:
    """Skewed routing logits: z[t, e] = ln p_rank(e) + Gumbel(0, 1) with p_r ~ r^-s.

    The top-k of such logits samples k experts without replacement from the
    Zipf(s) popularity law; `perm` maps popularity rank to expert id.
    """
    ranks = np.empty(n_experts, dtype=np.int64)
    ranks[perm] = np.arange(n_experts)
    logp = -s * np.log(ranks + 1.0)
    g = rng.gumbel(size=(tokens, n_experts))
    return (logp[None, :] + g).astype(np.float32)


# Workload shapes (name -> (shape, tokens, capacity, seed)).
TINY = LayerShape(256, 128, 8, 2)
OLMOE = LayerShape(2048, 1024, 64, 8)
WORKLOADS = {
    "tiny": dict(shape=TINY, tokens=16, capacity=8, seed=0),
    "decode": dict(shape=OLMOE, tokens=1, capacity=64, seed=1),
    "batch16_waves": dict(shape=OLMOE, tokens=16, capacity=16, seed=2),
    "prefill": dict(shape=OLMOE, tokens=2048, capacity=64, seed=3),
    "stack16": dict(shape=OLMOE, tokens=64, capacity=16, seed=4, layers=16, zipf_s=1.1),
}
