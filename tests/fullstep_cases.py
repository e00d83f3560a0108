"""Whole-step parity cases at the workloads' full sizes: the 57-block
FLUX.1-dev-shaped model (19 double + 38 single blocks, 3072 wide, 24 x 128
heads, 512 text tokens per request) at 1024 px, at 2048 px, and on the packed
256/512/1024/2048 px batch with per-request timesteps U[0, 1).  Token counts
follow the paper's section 2.2, Table 1: (resolution / 16)^2 image tokens.

Inputs only: seeds, shapes and the seeded draws.  Both the expected-value
writer (which runs the oracle) and the GPU tests (which run the library)
take their inputs from here, so the two sides see identical numbers.  Every
value is drawn on the host and rounded to bf16 once.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

from paper_2510_01565_amd import synth, workloads

WEIGHT_SEED = 0
CASES = {
    "c3_1024px": {"workload": "dit57_1024px_bf16", "input_seed": 3},
    "c4_2048px": {"workload": "dit57_2048px_bf16", "input_seed": 4},
    "c5_packed": {"workload": "dit57_packed_mixed_bf16", "input_seed": 5},
}
# case whose hidden state is recorded after every block, and the rows kept
# (joint order [text; image] of its one request): text rows at both ends and
# the middle, image rows at the grid's corners and edges, and seeded others
TRACE_CASE = "c3_1024px"


def workload(case: str) -> workloads.Workload:
    return workloads.WORKLOADS[CASES[case]["workload"]]


def model(case: str) -> workloads.ModelShape:
    return workload(case).model


def requests(case: str) -> List[Tuple[int, int, int, float]]:
    """(grid_h, grid_w, n_txt, t) of every request of the case."""
    wl = workload(case)
    seed = CASES[case]["input_seed"]
    n = len(wl.resolutions)
    ts = wl.t if wl.t is not None else [float(x) for x in synth.uniform(seed, "timesteps", (n,))]
    return [(g, g, nt, float(t)) for g, nt, t in zip(wl.grids(), wl.n_txt, ts)]


def dt(case: str) -> float:
    return workload(case).dt


def request_inputs(case: str, r: int) -> Tuple[np.ndarray, np.ndarray]:
    """Latents [grid_h * grid_w, C_in] and text embeddings [n_txt, D_txt] of
    request r, bf16-representable fp32."""
    m = model(case)
    seed = CASES[case]["input_seed"]
    gh, gw, nt, _ = requests(case)[r]
    lat = synth.normal(seed, f"latents.{r}", (gh * gw, m.in_channels), bf16=True)
    txt = synth.normal(seed, f"text.{r}", (nt, m.text_dim), bf16=True)
    return lat, txt


def trace_rows(case: str = TRACE_CASE) -> np.ndarray:
    gh, gw, nt, _ = requests(case)[0]
    L = nt + gh * gw
    fixed = [0, nt // 2, nt - 1, nt, nt + gw - 1, nt + gw, nt + (gh - 1) * gw, L - 1]
    extra = np.random.default_rng([CASES[case]["input_seed"], 99]).choice(L, 8, replace=False)
    return np.unique(np.concatenate([np.array(fixed), extra])).astype(np.int64)


def golden_path(case: str, r: int) -> str:
    import os
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "fullstep", f"{case}_r{r}.npz")
