"""The seeded input generators: row-chunked streams of large tensors, and the
expected-value writer's lazily drawn parameters equal to the plain draw.  CPU
only."""
import os
import sys

import numpy as np

import oracle as O
from paper_2510_01565_amd import synth, workloads

sys.path.insert(0, os.path.join(os.path.dirname(__file__), "golden"))
import make_fullstep_golden as G  # noqa: E402


def test_row_chunks_and_row_ranges(monkeypatch):
    monkeypatch.setattr(synth, "CHUNK", 1000)
    shape = (37, 100)
    assert synth.row_chunks(shape) == [(0, 10), (10, 20), (20, 30), (30, 37)]
    x = synth.normal(3, "a", shape, 0.02, True)
    assert x.shape == shape
    for r0, r1 in [(0, 37), (3, 29), (10, 20), (36, 37), (9, 11)]:
        np.testing.assert_array_equal(synth.normal_rows(3, "a", shape, r0, r1, 0.02, True), x[r0:r1])
    # chunk 0 is the tensor's plain stream: a small tensor is unchanged by chunking
    y = synth.normal(3, "b", (5, 7))
    np.testing.assert_array_equal(y, synth._rng(3, "b").standard_normal((5, 7), dtype=np.float32))


def test_golden_writer_params_equal_plain_draw(monkeypatch):
    monkeypatch.setattr(synth, "CHUNK", 5000)   # force several chunks per weight at this size
    m = workloads.ModelShape(hidden=128, heads=1, head_dim=128, mlp_ratio=4, n_double=2, n_single=2,
                             in_channels=64, text_dim=32)
    oc = G.oracle_cfg(m)
    lazy = G.LazyParams(oc, 3)
    full = synth.make_params(O.param_shapes(oc), G.FC.WEIGHT_SEED, bf16=True)
    for name, shape in O.param_shapes(oc):
        got = lazy[name]
        got = got[0:shape[0]] if isinstance(got, G._Rows) else got
        np.testing.assert_array_equal(got, full[name], err_msg=name)
    lat = synth.normal(1, "l", (12, 64), bf16=True).astype(np.float64)
    txt = synth.normal(1, "t", (5, 32), bf16=True).astype(np.float64)
    p64 = {k: v.astype(np.float64) for k, v in full.items()}
    seen = []
    v1 = O.dit_velocity(lazy, oc, lat, txt, 0.3, (3, 4), on_block=lambda d, x: seen.append((d, x.shape)))
    v2 = O.dit_velocity(p64, oc, lat, txt, 0.3, (3, 4))
    np.testing.assert_array_equal(v1, v2)
    assert seen == [(d, (17, 128)) for d in range(4)]
