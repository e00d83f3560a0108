"""Seeded synthetic inputs shared by the oracle checks and the HIP path.

This module only draws random numbers and rounds them to the storage type;
it holds none of the denoising step's arithmetic, and neither the oracle nor
the HIP library is imported here.

Every tensor has its own stream ``numpy.random.default_rng([seed, crc32(name)])``
so that a tensor's values do not depend on which other tensors are drawn.
Weights and biases ~ N(0, 0.02^2), activations ~ N(0, 1), drawn in fp32; a
bf16 workload rounds every value once (round to nearest even) so that both
sides consume identical numbers.

Full-size workloads (tens of GB of weights) are drawn on the device with
torch's seeded generator instead (``device_normal``); a test that needs some of
those values on the host copies them back.
"""
from __future__ import annotations

import zlib
from typing import Dict, Iterable, Tuple

import numpy as np

WEIGHT_STD = 0.02


def _rng(seed: int, name: str) -> np.random.Generator:
    return np.random.default_rng([int(seed), zlib.crc32(name.encode())])


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even), returned as fp32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    nan = np.isnan(x)
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of fp32 values that are already bf16-representable."""
    return (np.ascontiguousarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def normal(seed: int, name: str, shape: Tuple[int, ...], std: float = 1.0,
           bf16: bool = False) -> np.ndarray:
    """One seeded N(0, std^2) tensor in fp32 (bf16-representable if ``bf16``)."""
    x = _rng(seed, name).standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x = x * np.float32(std)
    return bf16_round(x) if bf16 else x


def uniform(seed: int, name: str, shape: Tuple[int, ...], lo: float = 0.0, hi: float = 1.0) -> np.ndarray:
    """Seeded U[lo, hi) values in fp32 (used for per-request timesteps)."""
    return _rng(seed, name).uniform(lo, hi, size=shape).astype(np.float32)


def make_params(shapes: Iterable[Tuple[str, Tuple[int, ...]]], seed: int,
                bf16: bool, std: float = WEIGHT_STD) -> Dict[str, np.ndarray]:
    """Host-side weights for every (name, shape), N(0, std^2)."""
    return {name: normal(seed, "w:" + name, tuple(shape), std, bf16) for name, shape in shapes}


def device_normal(seed: int, name: str, shape: Tuple[int, ...], std: float, dtype, device):
    """Seeded N(0, std^2) tensor drawn directly on ``device`` by torch's
    generator (fp32 draw, then one rounding to ``dtype``)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((int(seed) << 32) ^ zlib.crc32(name.encode()))
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)
