"""Shared helpers of the GPU parity tests: seeded inputs on both sides,
device uploads, and the error measure (normwise: max|g - r| / max|r|)."""
from __future__ import annotations

import numpy as np

import oracle as O
from paper_2510_01565_amd import dit, synth, workloads

BF16_TOL = 2e-2   # bf16 outputs against the fp64 oracle
F32_TOL = 1e-4    # fp32 outputs against the fp64 oracle


def normwise_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), "non-finite GPU output"
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))


def oracle_cfg(m: workloads.ModelShape) -> O.OracleConfig:
    return O.OracleConfig(hidden=m.hidden, heads=m.heads, head_dim=m.head_dim, mlp_ratio=m.mlp_ratio,
                          n_double=m.n_double, n_single=m.n_single, in_channels=m.in_channels,
                          text_dim=m.text_dim, time_freq_dim=m.time_freq_dim, tie_streams=m.tie_streams,
                          rope_theta=m.rope_theta, ln_eps=m.ln_eps)


def torch_dtype(m: workloads.ModelShape):
    import torch
    return torch.bfloat16 if m.dtype == "bf16" else torch.float32


def to_dev(x: np.ndarray, dtype):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(device="cuda", dtype=dtype)


def host_params(m: workloads.ModelShape, seed: int):
    cfg = dit.make_config(m)
    shapes = dit.weight_manifest(cfg)
    return cfg, shapes, synth.make_params(shapes, seed, bf16=(m.dtype == "bf16"))


def upload_params(params, shapes, dtype):
    tensors = [to_dev(params[n], dtype) for n, _ in shapes]
    return dit.Weights(tensors)


def workspace(cfg, batch):
    import torch
    n = dit.workspace_size(cfg, batch)
    return torch.empty(n, dtype=torch.uint8, device="cuda"), n


def request_inputs(m: workloads.ModelShape, grids, n_txt, seed: int):
    """Per-request seeded latents [h*w, C_in] and text [L_txt, D_txt]."""
    bf = m.dtype == "bf16"
    lat = [synth.normal(seed, f"latents.{r}", (gh * gw, m.in_channels), bf16=bf) for r, (gh, gw) in enumerate(grids)]
    txt = [synth.normal(seed, f"text.{r}", (nt, m.text_dim), bf16=bf) for r, nt in enumerate(n_txt)]
    return lat, txt
