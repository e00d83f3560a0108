"""Run-to-run determinism of the 57-block step where its GEMMs split K, and
replay of the step from a captured HIP graph.

At 256 px (512 text + 256 image tokens) the single-stream blocks' second
linear (768 x 3072 x 15360) runs as K pieces whose partial sums meet in the
workspace and are added, in piece order, by the last piece to arrive; the
result must not depend on which piece arrives last, so repeated steps are
bitwise identical.  A graph captured from dit_step + euler_update (both
enqueue kernels only, no memset nodes) replays to the eager result bit for
bit, with the program's own eager work and synchronisations between replays.
"""
import pytest

from paper_2510_01565_amd import dit, synth, workloads

pytestmark = pytest.mark.gpu


def _setup(name):
    import torch
    wl = workloads.WORKLOADS[name]
    m = wl.model
    dev = torch.device("cuda:0")
    cfg = dit.make_config(m)
    shapes = dit.weight_manifest(cfg)
    w = dit.Weights([synth.device_normal(7, "w:" + n, s, synth.WEIGHT_STD, torch.bfloat16, dev) for n, s in shapes])
    grids = wl.grids()
    b = dit.Batch(grids, grids, wl.n_txt, [0.37] * len(grids))
    nws = dit.workspace_size(cfg, b)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    lat = synth.device_normal(7, "latents", (sum(wl.n_img()), m.in_channels), 1.0, torch.bfloat16, dev)
    txt = synth.device_normal(7, "text", (sum(wl.n_txt), m.text_dim), 1.0, torch.bfloat16, dev)
    return wl, m, cfg, w, b, ws, nws, lat, txt


def test_split_k_step_is_deterministic_256px():
    import torch
    wl, m, cfg, w, b, ws, nws, lat, txt = _setup("dit57_256px_bf16")
    vels = []
    for rep in range(8):
        vel = torch.empty_like(lat)
        dit.dit_step(cfg, w, b, lat, txt, vel, ws, nws)
        vels.append(vel)
    torch.cuda.synchronize()
    assert torch.isfinite(vels[0].float()).all()
    for i, v in enumerate(vels[1:], 1):
        assert torch.equal(v, vels[0]), f"step {i} differs from step 0"


def test_graph_replay_equals_eager_256px():
    import torch
    wl, m, cfg, w, b, ws, nws, lat0, txt = _setup("dit57_256px_bf16")
    dts = [wl.dt] * len(wl.grids())
    lat = lat0.clone()
    vel = torch.empty_like(lat)

    def step():
        dit.dit_step(cfg, w, b, lat, txt, vel, ws, nws)
        dit.euler_update(b, m.in_channels, dit.DIT_BF16, lat, vel, dts)

    step()
    torch.cuda.synchronize()
    ref_v, ref_x = vel.clone(), lat.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        lat.copy_(lat0)
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        lat.copy_(lat0)
        vel.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(vel, ref_v), f"replay {rep}: velocity differs from the eager step"
        assert torch.equal(lat, ref_x), f"replay {rep}: latents differ from the eager step"
        # eager work of the program between replays
        step()
        torch.cuda.synchronize()
