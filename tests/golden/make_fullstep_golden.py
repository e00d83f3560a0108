"""Writes the expected values of the whole-step parity tests with the oracle.

For every request of the 1024 px, 2048 px and packed 256/512/1024/2048 px
cases (tests/fullstep_cases.py) it runs the fp64 oracle's velocity
prediction on the seeded bf16-representable inputs and weights and stores
the velocity as fp32 in tests/golden/fullstep/<case>_r<request>.npz.  For the
1024 px case it also stores sampled rows of the hidden state after every
block (the error-growth trace).  The Euler-updated latents are not stored:
the test forms them from the stored velocity with the oracle's Euler step.

Only the oracle and the seeded input generators are used; nothing here
loads the HIP library.  Weights are drawn tensor by tensor when the oracle
asks for them and dropped afterwards, so host memory stays near one block's
weights in fp64 plus the activations (about 10 GB at 2048 px).

    python tests/golden/make_fullstep_golden.py --jobs 6      # every request
    python tests/golden/make_fullstep_golden.py --case c4_2048px --request 0

Run time on 8 host cores: about two hours for all six requests (the two
2048 px requests dominate: 418 TFLOP of fp64 each).
"""
from __future__ import annotations

import argparse
import os
import platform
import subprocess
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
TESTS = os.path.dirname(HERE)
ROOT = os.path.dirname(TESTS)
for p in (ROOT, TESTS):
    if p not in sys.path:
        sys.path.insert(0, p)

import oracle as O  # noqa: E402
import fullstep_cases as FC  # noqa: E402
from paper_2510_01565_amd import synth  # noqa: E402


class _Rows:
    """Row slices of one large seeded tensor, drawn on demand."""

    def __init__(self, name, shape):
        self.name, self.shape = name, shape

    def __getitem__(self, sl):
        assert isinstance(sl, slice) and sl.step in (None, 1)
        r0, r1, _ = sl.indices(self.shape[0])
        return synth.normal_rows(FC.WEIGHT_SEED, "w:" + self.name, self.shape, r0, r1, synth.WEIGHT_STD, bf16=True)


class LazyParams:
    """The model's parameters as the oracle reads them (params[name]), each
    drawn from its seeded stream when read and not kept.  The modulation
    weights of all blocks form one tensor of 3.2e9 values; it is read by row
    ranges only."""

    def __init__(self, cfg: O.OracleConfig, threads: int):
        self.shapes = dict(O.param_shapes(cfg))
        self.pool = ThreadPoolExecutor(max(1, threads))

    def __getitem__(self, name):
        shape = self.shapes[name]
        if name in ("mod.w", "mod.b"):
            return _Rows(name, shape)
        n = len(synth.row_chunks(shape))
        parts = list(self.pool.map(
            lambda i: synth.normal_chunk(FC.WEIGHT_SEED, "w:" + name, shape, i, synth.WEIGHT_STD, bf16=True),
            range(n)))
        return parts[0] if n == 1 else np.concatenate(parts)


def oracle_cfg(m) -> O.OracleConfig:
    return O.OracleConfig(hidden=m.hidden, heads=m.heads, head_dim=m.head_dim, mlp_ratio=m.mlp_ratio,
                          n_double=m.n_double, n_single=m.n_single, in_channels=m.in_channels,
                          text_dim=m.text_dim, time_freq_dim=m.time_freq_dim, tie_streams=m.tie_streams,
                          rope_theta=m.rope_theta, ln_eps=m.ln_eps)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def run_one(case: str, r: int, threads: int) -> str:
    m = FC.model(case)
    oc = oracle_cfg(m)
    gh, gw, nt, t = FC.requests(case)[r]
    lat, txt = FC.request_inputs(case, r)
    params = LazyParams(oc, threads)
    trace = case == FC.TRACE_CASE
    rows = FC.trace_rows(case) if trace else np.zeros(0, np.int64)
    hidden = []

    def on_block(depth, x):
        hidden.append(np.asarray(x[rows], dtype=np.float32))
        print(f"{case} r{r}: block {depth + 1}/{oc.n_double + oc.n_single} "
              f"({time.time() - t0:.0f} s)", flush=True)

    t0 = time.time()
    v = O.dit_velocity(params, oc, lat.astype(np.float64), txt.astype(np.float64), t, (gh, gw),
                       on_block=on_block)
    wall = time.time() - t0
    out = FC.golden_path(case, r)
    os.makedirs(os.path.dirname(out), exist_ok=True)
    extra = {"rows": rows, "hidden": np.stack(hidden)} if trace else {}
    np.savez(out, velocity=v.astype(np.float32), grid=np.array([gh, gw]), n_txt=np.array(nt),
             t=np.array(t, dtype=np.float64), oracle_dtype=np.array("float64"), wall_s=np.array(wall),
             host=np.array(f"{os.cpu_count()} threads, {cpu_model()}"), **extra)
    print(f"{case} r{r}: wrote {out} in {wall:.0f} s", flush=True)
    return out


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--case", choices=sorted(FC.CASES))
    ap.add_argument("--request", type=int)
    ap.add_argument("--threads", type=int, default=4, help="threads drawing weights")
    ap.add_argument("--jobs", type=int, default=0, help="run every request, this many processes at a time")
    a = ap.parse_args()
    if a.case is not None:
        reqs = range(len(FC.requests(a.case))) if a.request is None else [a.request]
        for r in reqs:
            run_one(a.case, r, a.threads)
        return
    jobs = [(c, r) for c in FC.CASES for r in range(len(FC.requests(c)))]
    # largest requests first so they start at once
    jobs.sort(key=lambda cr: -FC.requests(cr[0])[cr[1]][0])
    running = []
    n = max(1, a.jobs)
    for c, r in jobs:
        while len(running) >= n:
            running = [p for p in running if p.poll() is None]
            time.sleep(5)
        running.append(subprocess.Popen([sys.executable, os.path.abspath(__file__), "--case", c, "--request",
                                         str(r), "--threads", str(a.threads)]))
    rc = [p.wait() for p in running]
    sys.exit(max(rc) if rc else 0)


if __name__ == "__main__":
    main()
