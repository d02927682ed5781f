"""Seeded synthetic inputs shared by the GPU path's tests/benchmark and the oracle.

This module only draws random numbers; it holds none of the stage's arithmetic.
Distributions follow the GPT-3-shaped workloads of the paper's evaluation:
hidden states x ~ N(0, 1), linear weights and biases ~ N(0, 0.02), LayerNorm
gain 1 and bias 0 (the tiny configuration draws gain 1 + N(0, 0.1) and bias
N(0, 0.1) so that LayerNorm-parameter gradients are exercised), upstream
gradient dy ~ N(0, 1), batch 1.

Every tensor has its own torch.Generator seeded from (seed, stream id), so a
tensor's values do not depend on which other tensors were drawn.  Values are
drawn in float32 and rounded (round-to-nearest-even) to the storage dtype; the
oracle consumes exactly the rounded values.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

PARAM_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w1", "b1", "w2", "b2")

SEED_X, SEED_PARAMS, SEED_DY = 0, 1, 2


def param_shapes(hidden: int, op_parts: int = 1) -> Dict[str, tuple]:
    """Parameter shapes of one layer; op_parts p > 1: one device's shard of
    p-way operation partitioning (attention width H / p, FFN width 4H / p)."""
    H, A, F = hidden, hidden // op_parts, 4 * hidden // op_parts
    return {"ln1_g": (H,), "ln1_b": (H,), "w_qkv": (3 * A, H), "b_qkv": (3 * A,),
            "w_o": (H, A), "b_o": (H,), "ln2_g": (H,), "ln2_b": (H,),
            "w1": (F, H), "b1": (F,), "w2": (H, F), "b2": (H,)}


def _gen(seed: int, stream: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1_000_003 + stream * 7_919 + 12_345) % (2 ** 63 - 1))
    return g


def normal(shape, seed: int, stream: int, std: float = 1.0, mean: float = 0.0,
           dtype=torch.float32, device="cpu") -> torch.Tensor:
    g = _gen(seed, stream, device)
    t = torch.randn(shape, generator=g, dtype=torch.float32, device=device)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(dtype)


def stage_params(n_layers: int, hidden: int, seed: int = SEED_PARAMS, dtype=torch.float32,
                 device="cpu", randomize_ln: bool = False,
                 weight_std: float = 0.02, op_parts: int = 1) -> List[Dict[str, torch.Tensor]]:
    shapes = param_shapes(hidden, op_parts)
    layers = []
    for li in range(n_layers):
        p = {}
        for pi, name in enumerate(PARAM_NAMES):
            stream = 1000 + li * 64 + pi
            shp = shapes[name]
            if name.endswith("_g"):
                p[name] = (normal(shp, seed, stream, 0.1, 1.0, dtype, device) if randomize_ln
                           else torch.ones(shp, dtype=dtype, device=device))
            elif name.startswith("ln"):
                p[name] = (normal(shp, seed, stream, 0.1, 0.0, dtype, device) if randomize_ln
                           else torch.zeros(shp, dtype=dtype, device=device))
            else:
                p[name] = normal(shp, seed, stream, weight_std, 0.0, dtype, device)
        layers.append(p)
    return layers


def hidden_states(seq: int, hidden: int, seed: int = SEED_X, dtype=torch.float32,
                  device="cpu") -> torch.Tensor:
    return normal((seq, hidden), seed, 1, 1.0, 0.0, dtype, device)


def upstream_grad(seq: int, hidden: int, seed: int = SEED_DY, dtype=torch.float32,
                  device="cpu") -> torch.Tensor:
    return normal((seq, hidden), seed, 2, 1.0, 0.0, dtype, device)


def batch_hidden_states(seq: int, batch: int, hidden: int, seed: int = SEED_X,
                        dtype=torch.float32, device="cpu") -> torch.Tensor:
    """[seq, batch, hidden]: sequence s is hidden_states(seq, hidden, seed * 1000 + s)."""
    return torch.stack([hidden_states(seq, hidden, seed * 1000 + s, dtype, device)
                        for s in range(batch)], dim=1)


def batch_upstream_grad(seq: int, batch: int, hidden: int, seed: int = SEED_DY,
                        dtype=torch.float32, device="cpu") -> torch.Tensor:
    """[seq, batch, hidden]: sequence s is upstream_grad(seq, hidden, seed * 1000 + s)."""
    return torch.stack([upstream_grad(seq, hidden, seed * 1000 + s, dtype, device)
                        for s in range(batch)], dim=1)


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy().copy()


def params_f64(layers: List[Dict[str, torch.Tensor]]) -> List[Dict[str, np.ndarray]]:
    return [{k: to_f64(v) for k, v in p.items()} for p in layers]


def random_composition(total_units: int, rng: np.random.Generator,
                       max_units: Optional[int] = None) -> List[int]:
    """A random composition of ``total_units`` (every part >= 1)."""
    parts, left = [], total_units
    while left > 0:
        hi = left if max_units is None else min(left, max_units)
        k = int(rng.integers(1, hi + 1))
        parts.append(k)
        left -= k
    return parts


def cost_table(U: int, kind: str, seed: int) -> np.ndarray:
    """Seeded int64 [U][U] slice-cost tables (cost[k-1, j] = t(k units, j units of
    context), entries with k + j > U unused) of several shapes: ``random``
    (uniform), ``ties`` (small range, many equal values), ``linear`` (a + b k +
    c j + e k j with noise, the shape of the paper's Eq. 9 model) and ``flops``
    (proportional to a block's forward+backward arithmetic plus a fixed launch
    cost)."""
    rng = np.random.default_rng(seed)
    k = np.arange(1, U + 1)[:, None].astype(np.float64)
    j = np.arange(U)[None, :].astype(np.float64)
    if kind == "random":
        t = rng.integers(1, 1000, size=(U, U)).astype(np.float64)
    elif kind == "ties":
        t = rng.integers(1, 4, size=(U, U)).astype(np.float64)
    elif kind == "linear":
        a0, a1, a2, a3 = rng.uniform(50, 200), rng.uniform(5, 20), rng.uniform(0, 2), rng.uniform(0, 1)
        t = a0 + a1 * k + a2 * j + a3 * k * j + rng.uniform(0, 3, size=(U, U))
    elif kind == "flops":
        H = 64.0
        t = 100.0 + (72 * k * H * H + 12 * H * (k * j + k * (k + 1) / 2)) / 5000.0
    else:
        raise ValueError(kind)
    t = np.rint(t).astype(np.int64)
    t[(k + j) > U] = -7  # unused entries; never read
    return np.ascontiguousarray(t)
