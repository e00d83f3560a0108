"""Block- and step-level parity on the GPU against the oracle, plus the
properties that must hold at any size: packed = unpacked, run-to-run
bitwise determinism, dit_step = embed + blocks + final."""
import numpy as np
import pytest

import oracle as O
from paper_2510_01565_amd import dit, synth, workloads
from harness import (BF16_TOL, F32_TOL, host_params, normwise_err, oracle_cfg, request_inputs, to_dev,
                     torch_dtype, upload_params, workspace)

pytestmark = pytest.mark.gpu

# a small bf16 model with every feature of the full one (untied double blocks, single blocks)
TINY_BF16 = workloads.ModelShape(hidden=256, heads=2, head_dim=128, mlp_ratio=4, n_double=2, n_single=2,
                                 in_channels=64, text_dim=96)


# the SD3-Medium block structure (joint blocks only, untied streams, 64-wide heads) at a small width
TINY_SD3_BF16 = workloads.ModelShape(hidden=192, heads=3, head_dim=64, mlp_ratio=4, n_double=3, n_single=0,
                                     in_channels=64, text_dim=80)


def _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt):
    import torch
    dt = torch_dtype(m)
    w = upload_params(params, shapes, dt)
    b = dit.Batch([g[0] for g in grids], [g[1] for g in grids], n_txt, ts)
    ws, nws = workspace(cfg, b)
    lat_d = to_dev(np.concatenate(lat), dt)
    txt_d = to_dev(np.concatenate(txt), dt) if sum(n_txt) else None
    vel = torch.full_like(lat_d, float("nan"))
    dit.dit_step(cfg, w, b, lat_d, txt_d, vel, ws, nws)
    torch.cuda.synchronize()
    return vel, lat_d, b


def _oracle_step(m, params, grids, n_txt, ts, lat, txt):
    oc = oracle_cfg(m)
    p64 = {k: v.astype(np.float64) for k, v in params.items()}
    return [O.dit_velocity(p64, oc, lat[r], txt[r], ts[r], grids[r]) for r in range(len(grids))]


def test_small_block_step_f32():
    """One tied adaLN block, 384 wide, 6x64 heads, 256 image + 32 text tokens,
    fp32; one velocity prediction plus the Euler update with dt = 1/28."""
    wl = workloads.WORKLOADS["small_block_256px_f32"]
    m = wl.model
    cfg, shapes, params = host_params(m, 0)
    grids, n_txt, ts = [(16, 16)], [32], [0.5]
    lat, txt = request_inputs(m, grids, n_txt, 0)
    vel, lat_d, b = _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt)
    ref = _oracle_step(m, params, grids, n_txt, ts, lat, txt)[0]
    assert normwise_err(vel.cpu().numpy(), ref) < F32_TOL
    dit.euler_update(b, m.in_channels, dit.DIT_F32, lat_d, vel, [wl.dt])
    import torch
    torch.cuda.synchronize()
    ref_x = O.euler_update(lat[0].astype(np.float64), ref, wl.dt)
    assert normwise_err(lat_d.cpu().numpy(), ref_x) < F32_TOL


def test_tiny_bf16_packed_step():
    m = TINY_BF16
    cfg, shapes, params = host_params(m, 1)
    grids, n_txt, ts = [(6, 10), (16, 16), (3, 4)], [17, 40, 0], [0.9, 0.25, 0.6]
    lat, txt = request_inputs(m, grids, n_txt, 1)
    vel, _, _ = _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt)
    ref = np.concatenate(_oracle_step(m, params, grids, n_txt, ts, lat, txt))
    assert normwise_err(vel.float().cpu().numpy(), ref) < BF16_TOL


def test_text_free_batch_step():
    """A batch with no text tokens at all (no text embedder rows, text_emb NULL)."""
    m = TINY_BF16
    cfg, shapes, params = host_params(m, 6)
    grids, n_txt, ts = [(8, 8), (4, 12)], [0, 0], [0.4, 0.8]
    lat, txt = request_inputs(m, grids, n_txt, 6)
    vel, _, _ = _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt)
    ref = np.concatenate(_oracle_step(m, params, grids, n_txt, ts, lat, txt))
    assert normwise_err(vel.float().cpu().numpy(), ref) < BF16_TOL


def test_tiny_sd3_shaped_bf16_packed_step():
    """Joint blocks only with 64-wide bf16 heads; three requests packed, one of
    them without text."""
    m = TINY_SD3_BF16
    cfg, shapes, params = host_params(m, 4)
    grids, n_txt, ts = [(8, 12), (16, 16), (5, 3)], [21, 77, 0], [0.3, 0.95, 0.05]
    lat, txt = request_inputs(m, grids, n_txt, 4)
    vel, _, _ = _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt)
    ref = np.concatenate(_oracle_step(m, params, grids, n_txt, ts, lat, txt))
    assert normwise_err(vel.float().cpu().numpy(), ref) < BF16_TOL


def test_packed_equals_unpacked_and_deterministic():
    m = TINY_BF16
    cfg, shapes, params = host_params(m, 2)
    cfg = dit.make_config(m, dit.DIT_FLAG_BATCH_INVARIANT)
    grids, n_txt, ts = [(8, 8), (5, 9), (16, 12)], [33, 8, 64], [0.1, 0.5, 0.77]
    lat, txt = request_inputs(m, grids, n_txt, 2)
    packed, _, _ = _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt)
    again, _, _ = _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt)
    assert bool((packed.view(dtype=__import__("torch").int16) == again.view(dtype=__import__("torch").int16)).all())
    off = 0
    for r in range(3):
        one, _, _ = _run_step(m, params, shapes, cfg, [grids[r]], [n_txt[r]], [ts[r]], [lat[r]], [txt[r]])
        n = grids[r][0] * grids[r][1]
        assert bool((one == packed[off:off + n]).all()), r
        off += n


def test_sixteen_requests_and_extreme_grid_sides():
    """The largest batch (16 requests) with the extreme grid shapes: a 1 x 256
    and a 256 x 1 grid (RoPE positions up to the table's last row), single
    tokens, no text, one text token, and requests whose lengths are not
    multiples of 16; every request's velocity against the oracle."""
    m = TINY_BF16
    cfg, shapes, params = host_params(m, 5)
    grids = [(1, 256), (256, 1), (1, 1), (1, 1), (2, 3), (7, 5), (16, 16), (3, 1), (1, 9), (12, 4), (5, 5), (9, 2),
             (4, 4), (1, 2), (6, 6), (2, 17)]
    n_txt = [0, 3, 0, 1, 77, 5, 0, 64, 2, 0, 31, 1, 16, 0, 9, 40]
    ts = [float(t) for t in synth.uniform(5, "timesteps", (16,))]
    lat, txt = request_inputs(m, grids, n_txt, 5)
    vel, _, _ = _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt)
    refs = _oracle_step(m, params, grids, n_txt, ts, lat, txt)
    got = vel.float().cpu().numpy()
    off = 0
    for r, ref in enumerate(refs):
        n = ref.shape[0]
        assert normwise_err(got[off:off + n], ref) < BF16_TOL, r
        off += n


def test_double_block_c2():
    """One double-stream block, 3072 wide, 24x128 heads, 512 text + 1024 image
    tokens (512 px) with 2-D RoPE, bf16 weights and inputs, fp32 residual."""
    import torch
    m = workloads.FLUX_DOUBLE
    cfg, shapes, params = host_params(m, 0)
    H = m.hidden
    x_txt = synth.normal(0, "hidden.txt", (512, H), bf16=True)
    x_img = synth.normal(0, "hidden.img", (1024, H), bf16=True)
    c = synth.normal(0, "cond", (1, H), bf16=True)
    w = upload_params(params, shapes, torch.bfloat16)
    b = dit.Batch([32], [32], [512], [0.5])
    ws, nws = workspace(cfg, b)
    hidden = to_dev(np.concatenate([x_txt, x_img]), torch.float32)
    dit.dit_block_forward(cfg, w, 0, 0, b, hidden, to_dev(c, torch.float32), ws, nws)
    torch.cuda.synchronize()
    got = hidden.cpu().numpy()
    p64 = {k: v.astype(np.float64) for k, v in params.items()}
    rt, ri = O.double_block(p64, oracle_cfg(m), 0, x_txt, x_img, c[0], (32, 32))
    assert normwise_err(got[:512], rt) < BF16_TOL
    assert normwise_err(got[512:], ri) < BF16_TOL


def test_step_equals_composed_blocks():
    """dit_step's velocity equals embed -> dit_block_forward x n -> final, with
    the composition done by the oracle's embedders and final layer on the
    host and every block on the GPU (checks the block entry point and the
    modulation offsets of every block)."""
    import torch
    m = TINY_BF16
    cfg, shapes, params = host_params(m, 3)
    grids, n_txt, ts = [(7, 9)], [12], [0.4]
    lat, txt = request_inputs(m, grids, n_txt, 3)
    vel, _, _ = _run_step(m, params, shapes, cfg, grids, n_txt, ts, lat, txt)
    oc = oracle_cfg(m)
    p64 = {k: v.astype(np.float64) for k, v in params.items()}
    c = O.conditioning(p64, oc, ts[0])
    xi = O.linear(lat[0].astype(np.float64), p64["img_in.w"], p64["img_in.b"])
    xt = O.linear(txt[0].astype(np.float64), p64["txt_in.w"], p64["txt_in.b"])
    w = upload_params(params, shapes, torch.bfloat16)
    b = dit.Batch([7], [9], [12], ts)
    ws, nws = workspace(cfg, b)
    hidden = to_dev(np.concatenate([xt, xi]).astype(np.float32), torch.float32)
    cd = to_dev(c[None].astype(np.float32), torch.float32)
    for i in range(m.n_double):
        dit.dit_block_forward(cfg, w, 0, i, b, hidden, cd, ws, nws)
    for i in range(m.n_single):
        dit.dit_block_forward(cfg, w, 1, i, b, hidden, cd, ws, nws)
    torch.cuda.synchronize()
    h = hidden.cpu().numpy().astype(np.float64)
    v_comp = O.final_layer(p64, oc, h[12:], c)
    assert normwise_err(vel.float().cpu().numpy(), v_comp) < BF16_TOL
