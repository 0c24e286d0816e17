"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This module holds no arithmetic of the method itself: it only draws random numbers,
rounds them to the storage dtype and lays them out.  Both the HIP path and the CPU
oracle consume what it produces; neither is imported here.

Recipe (host side, bit-reproducible):
  * a numpy ``PCG64`` stream per (workload, layer, tensor) seed,
  * standard normal draws in float64, scaled by the requested std,
  * rounded to float32, then round-to-nearest-even to bf16 when bf16 is asked for.
Large device-resident tensors for timing only are drawn with torch's own device
generator (``device_normal``); their values never feed a parity comparison.
"""
from __future__ import annotations

import hashlib

import numpy as np


def seed_for(*parts) -> int:
    """Stable 63-bit seed from any printable parts (workload, layer, tensor name...)."""
    h = hashlib.sha256(repr(parts).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def normal(seed: int, shape, std: float = 1.0) -> np.ndarray:
    """float64 N(0, std^2) draws."""
    return rng(seed).standard_normal(size=shape) * std


def to_bf16_bits(x) -> np.ndarray:
    """Round to float32, then round-to-nearest-even to bf16; returns uint16 bit patterns."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    bias = ((u >> 16) & 1) + 0x7FFF
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def scale_rows_bf16(bits: np.ndarray, frac: float, factor: float, seed: int) -> np.ndarray:
    """Multiply floor(frac * rows) distinct rows (last axis = one row) by ``factor``.

    Rows are drawn without replacement from a seeded permutation.  With a power-of-two
    factor the product is exact in bf16, so the result stays a valid bf16 tensor.
    """
    flat = bits.reshape(-1, bits.shape[-1])
    count = int(np.floor(frac * flat.shape[0]))
    pick = rng(seed).permutation(flat.shape[0])[:count]
    vals = bf16_bits_to_f32(flat[pick]) * np.float32(factor)
    out = flat.copy()
    out[pick] = to_bf16_bits(vals)
    return out.reshape(bits.shape)


def sfa_inputs(B, L, n, Hq, Hkv, D, *, seed, dtype="bf16", qkv_std=1.0, dout_std=1.0,
               k_spike=None):
    """q, k, v, dO as numpy arrays in the layouts [B][n*L][H][D].

    dtype "bf16" gives uint16 bit patterns, "f32" gives float32.  k_spike=(frac, factor)
    scales that fraction of K rows (one row = one (b, p, kv-head) vector of D values).
    """
    N = n * L
    shapes = {"q": (B, N, Hq, D), "k": (B, N, Hkv, D), "v": (B, N, Hkv, D),
              "dout": (B, N, Hq, D)}
    out = {}
    for name, shape in shapes.items():
        std = dout_std if name == "dout" else qkv_std
        x = normal(seed_for(seed, name), shape, std)
        out[name] = to_bf16_bits(x) if dtype == "bf16" else x.astype(np.float32)
    if k_spike is not None:
        frac, factor = k_spike
        if dtype == "bf16":
            out["k"] = scale_rows_bf16(out["k"], frac, factor, seed_for(seed, "k_spike"))
        else:
            flat = out["k"].reshape(-1, D)
            pick = rng(seed_for(seed, "k_spike")).permutation(flat.shape[0])[
                :int(np.floor(frac * flat.shape[0]))]
            flat[pick] *= np.float32(factor)
    return out


def token_ids(seed: int, B: int, L: int, V: int) -> np.ndarray:
    """int32 token ids uniform in [0, V)."""
    return rng(seed).integers(0, V, size=(B, L), dtype=np.int64).astype(np.int32)


def device_normal(shape, std, seed, device, dtype):
    """Timing-only device tensor: torch's device generator, N(0, std^2), cast to dtype."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed & ((1 << 62) - 1))
    t = torch.empty(shape, dtype=torch.float32, device=device)
    t.normal_(0.0, std, generator=g)
    return t.to(dtype)
