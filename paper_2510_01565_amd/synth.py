"""Seeded synthetic inputs shared by the oracle checks and the HIP path.

This module only draws random numbers and rounds them to the storage type;
it holds none of the denoising step's arithmetic, and neither the oracle nor
the HIP library is imported here.

Every tensor has its own stream ``numpy.random.default_rng([seed, crc32(name)])``
so that a tensor's values do not depend on which other tensors are drawn.
A tensor of more than ``CHUNK`` elements is drawn in row chunks of at most
``CHUNK`` elements, chunk i from the stream ``[seed, crc32(name), i]`` (chunk 0
from the plain tensor stream), so that any row range can be drawn without the
rows before it and the chunks of a large model can be drawn in parallel.
Weights and biases ~ N(0, 0.02^2), activations ~ N(0, 1), drawn in fp32; a
bf16 workload rounds every value once (round to nearest even) so that both
sides consume identical numbers.

Full-size workloads (tens of GB of weights) are drawn on the device with
torch's seeded generator instead (``device_normal``); a test that needs some of
those values on the host copies them back.
"""
from __future__ import annotations

import zlib
from typing import Dict, Iterable, List, Tuple

import numpy as np

WEIGHT_STD = 0.02


CHUNK = 1 << 24   # elements per row chunk of a large tensor


def _rng(seed: int, name: str, chunk: int = 0) -> np.random.Generator:
    key = [int(seed), zlib.crc32(name.encode())]
    return np.random.default_rng(key if chunk == 0 else key + [int(chunk)])


def row_chunks(shape: Tuple[int, ...]) -> List[Tuple[int, int]]:
    """Row ranges [r0, r1) of the chunks a tensor of ``shape`` is drawn in."""
    shape = tuple(int(s) for s in shape)
    if not shape:
        return [(0, 1)]
    row = int(np.prod(shape[1:], dtype=np.int64)) if len(shape) > 1 else 1
    if shape[0] * row <= CHUNK:
        return [(0, shape[0])]
    per = max(1, CHUNK // max(row, 1))
    return [(r, min(r + per, shape[0])) for r in range(0, shape[0], per)]


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


def normal_chunk(seed: int, name: str, shape: Tuple[int, ...], i: int, std: float = 1.0,
                 bf16: bool = False) -> np.ndarray:
    """Chunk i (rows ``row_chunks(shape)[i]``) of the seeded N(0, std^2) tensor."""
    r0, r1 = row_chunks(shape)[i]
    sub = (r1 - r0,) + tuple(shape[1:]) if len(shape) else ()
    x = _rng(seed, name, i).standard_normal(size=sub, dtype=np.float32)
    if std != 1.0:
        x = x * np.float32(std)
    return bf16_round(x) if bf16 else x


def normal(seed: int, name: str, shape: Tuple[int, ...], std: float = 1.0,
           bf16: bool = False) -> np.ndarray:
    """One seeded N(0, std^2) tensor in fp32 (bf16-representable if ``bf16``)."""
    shape = tuple(int(s) for s in shape)
    parts = [normal_chunk(seed, name, shape, i, std, bf16) for i in range(len(row_chunks(shape)))]
    return parts[0] if len(parts) == 1 else np.concatenate(parts)


def normal_rows(seed: int, name: str, shape: Tuple[int, ...], r0: int, r1: int, std: float = 1.0,
                bf16: bool = False) -> np.ndarray:
    """Rows [r0, r1) of the seeded tensor ``normal(seed, name, shape, ...)``,
    drawing only the chunks that overlap them."""
    shape = tuple(int(s) for s in shape)
    out = []
    for i, (c0, c1) in enumerate(row_chunks(shape)):
        if c1 <= r0 or c0 >= r1:
            continue
        x = normal_chunk(seed, name, shape, i, std, bf16)
        out.append(x[max(r0, c0) - c0:min(r1, c1) - c0])
    return out[0] if len(out) == 1 else np.concatenate(out)


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
