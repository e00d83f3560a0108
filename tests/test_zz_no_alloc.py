"""dit_step_noalloc (the step on the library's static scratch) against
dit_step (the step on a caller workspace), through the C ABI: the 57-block
model at 512 px and then, in the next call, at 256 px (a smaller input on
the same scratch, whose split-K launches use the scratch's counters and
partial sums).  Both calls must give dit_step's output bit for bit, and so
within the bf16 tolerance of each other."""
import numpy as np
import pytest

from harness import BF16_TOL, normwise_err
from paper_2510_01565_amd import dit, synth, workloads

pytestmark = pytest.mark.gpu


def test_noalloc_step_matches_dit_step_on_two_calls():
    import torch
    dev = torch.device("cuda")
    m = workloads.FLUX_FULL
    cfg = dit.make_config(m)
    shapes = dit.weight_manifest(cfg)
    w = dit.Weights([synth.device_normal(11, "w:" + n, s, synth.WEIGHT_STD, torch.bfloat16, dev) for n, s in shapes])
    for res, t in ((512, 0.3), (256, 0.8)):
        g = res // 16
        b = dit.Batch([g], [g], [512], [t])
        assert dit.workspace_size(cfg, b) <= dit.DIT_NOALLOC_SCRATCH_BYTES
        lat = synth.device_normal(11, f"latents.{res}", (g * g, m.in_channels), 1.0, torch.bfloat16, dev)
        txt = synth.device_normal(11, f"text.{res}", (512, m.text_dim), 1.0, torch.bfloat16, dev)
        print(f"noalloc step {res} px", flush=True)
        v_na = torch.full_like(lat, float("nan"))
        dit.dit_step_noalloc(cfg, w, b, lat, txt, v_na)
        torch.cuda.synchronize()
        nws = dit.workspace_size(cfg, b)
        ws = torch.empty(nws, dtype=torch.uint8, device=dev)
        v_ref = torch.full_like(lat, float("nan"))
        dit.dit_step(cfg, w, b, lat, txt, v_ref, ws, nws)
        torch.cuda.synchronize()
        assert torch.isfinite(v_na.float()).all().item()
        assert normwise_err(v_na.float().cpu().numpy(), v_ref.float().cpu().numpy().astype(np.float64)) < BF16_TOL
        assert torch.equal(v_na.view(torch.int16), v_ref.view(torch.int16)), res
