"""Seeded tensor generators.

Seeds follow one rule for every workload: ``1000*config + 10*layer + which``
with ``which`` = 0 for activations, 1 for weights, 2 for bias.  Values are
drawn in fp32 with ``numpy.random.default_rng``; for bf16 workloads they are
then rounded to bf16 (round to nearest, ties to even) and kept as uint16 bit
patterns, so that every consumer sees identical bits.
"""

from __future__ import annotations

import numpy as np

SEED_X, SEED_W, SEED_B = 0, 1, 2


def seed_for(config: int, layer: int, which: int) -> int:
    return 1000 * int(config) + 10 * int(layer) + int(which)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    # finite values never overflow 32 bits here (largest: 0xFF7FFFFF + 0x8000)
    r = (u >> np.uint32(16)) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _draw_f32(seed: int, shape, dist) -> np.ndarray:
    rng = np.random.default_rng(seed)
    kind = dist[0]
    if kind == "uniform":
        lo, hi = float(dist[1]), float(dist[2])
        v = rng.random(size=shape, dtype=np.float32)
        v *= np.float32(hi - lo)          # same fp32 operations, in place
        v += np.float32(lo)
        return v
    if kind == "normal":
        mean, std = float(dist[1]), float(dist[2])
        v = rng.standard_normal(size=shape, dtype=np.float32)
        v *= np.float32(std)
        v += np.float32(mean)
        return v
    raise ValueError(f"unknown distribution {dist!r}")


def draw(seed: int, shape, dist, dtype: str) -> np.ndarray:
    """Draw a tensor; dtype 'f32' returns float32, 'bf16' returns uint16 bits."""
    a = _draw_f32(seed, shape, dist)
    if dtype == "f32":
        return a
    if dtype == "bf16":
        return f32_to_bf16_bits(a)
    raise ValueError(f"unknown dtype {dtype!r}")


def draw_layer(layer, config: int, index: int, with_bias: bool = False) -> dict:
    """Activations, weights (and optionally bias, always fp32) for one layer."""
    out = {
        "x": draw(seed_for(config, index, SEED_X), layer.x_shape, layer.x_dist, layer.dtype),
        "w": draw(seed_for(config, index, SEED_W), layer.w_shape, layer.w_dist, layer.dtype),
    }
    if with_bias:
        out["bias"] = _draw_f32(seed_for(config, index, SEED_B), (layer.cout,), ("normal", 0.0, 0.1))
    return out


def draw_device(seed: int, shape, dist, dtype: str, device="cuda"):
    """Seeded draw on the GPU with torch's generator (same distributions as
    ``draw``, different stream of numbers).  Used where the host generator is
    too slow for the data volume (benchmark activations); values are fp32,
    then rounded to nearest even bf16 when dtype is 'bf16'."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    kind = dist[0]
    if kind == "normal":
        t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        t = t * float(dist[2]) + float(dist[1])
    elif kind == "uniform":
        t = torch.rand(shape, generator=g, device=device, dtype=torch.float32)
        t = t * float(dist[2] - dist[1]) + float(dist[1])
    else:
        raise ValueError(dist)
    return t if dtype == "f32" else t.to(torch.bfloat16)
