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


def upload_host_drawn_params(m: workloads.ModelShape, seed: int, workers: int = 16):
    """Every parameter of model ``m`` drawn on the host from its seeded
    streams (row chunks in parallel threads, as ``synth.make_params`` would
    draw them) and copied to the device in bf16 chunk by chunk, so the host
    never holds more than a few chunks.  Returns (dit_config, Weights)."""
    import torch
    from concurrent.futures import ThreadPoolExecutor

    assert m.dtype == "bf16"
    cfg = dit.make_config(m)
    shapes = dit.weight_manifest(cfg)
    tensors = [torch.empty(s, dtype=torch.bfloat16, device="cuda") for _, s in shapes]
    jobs = [(ti, name, s, i) for ti, (name, s) in enumerate(shapes) for i in range(len(synth.row_chunks(s)))]

    def draw(job):
        ti, name, s, i = job
        x = synth.normal_chunk(seed, "w:" + name, s, i, synth.WEIGHT_STD, bf16=True)
        return ti, synth.row_chunks(s)[i], synth.bf16_bits(x)

    with ThreadPoolExecutor(workers) as ex:
        for ti, (r0, r1), bits in ex.map(draw, jobs):
            src = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
            tensors[ti][r0:r1].copy_(src)
    torch.cuda.synchronize()
    return cfg, dit.Weights(tensors)


def error_histogram(got, ref) -> dict:
    """Fractions of elements by |g - r| / max|r| (the normwise scale), and the
    median / 99th percentile of the elementwise relative error |g - r| / |r|
    over elements with |r| above a tenth of the rms."""
    got = np.asarray(got, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    e = np.abs(got - ref) / np.abs(ref).max()
    edges = [1e-4, 1e-3, 3e-3, 1e-2, 2e-2]
    hist, lo = {}, 0.0
    for hi in edges:
        hist[f"<{hi:g}"] = float(((e >= lo) & (e < hi)).mean())
        lo = hi
    hist[f">={edges[-1]:g}"] = float((e >= edges[-1]).mean())
    big = np.abs(ref) > 0.1 * np.sqrt((ref * ref).mean())
    rel = np.abs(got - ref)[big] / np.abs(ref)[big]
    return {"normwise_bins": hist, "rel_median": float(np.median(rel)), "rel_p99": float(np.quantile(rel, 0.99))}
