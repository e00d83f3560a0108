"""Pins of the CPU oracle against facts that do not come from the oracle itself:
values the paper prints (Table 1 token counts), hand-derived examples, closed
forms, invariants, library routines for special cases and brute force on tiny
inputs.  CPU only."""
import math
import os

import numpy as np
import pytest
import torch

import oracle as O
from paper_2510_01565_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _read_gold(name):
    rows = {}
    with open(os.path.join(GOLD, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            rows.setdefault(key, []).append([float(v) for v in vals])
    return rows


# ---------------------------------------------------------------- Table 1
def test_image_tokens_match_table1():
    with open(os.path.join(GOLD, "table1_tokens.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    assert len(rows) == 4
    for res, tokens in rows:
        assert O.image_tokens(int(res)) == int(tokens)


# ---------------------------------------------------------------- timestep embedding
def test_timestep_embedding_special_values():
    e0 = O.timestep_embedding(np.array([0.0]))[0]
    assert e0.shape == (256,)
    np.testing.assert_array_equal(e0[:128], 1.0)   # cos(0) block comes first
    np.testing.assert_array_equal(e0[128:], 0.0)   # then sin(0)
    t = 0.37
    e = O.timestep_embedding(np.array([t]))[0]
    # frequency index 0 is 1: the angle is the scaled timestep 1000*t
    assert e[0] == pytest.approx(math.cos(370.0), abs=1e-12)
    assert e[128] == pytest.approx(math.sin(370.0), abs=1e-12)
    # index 64 = half of 128: frequency 1e4^(-1/2) = 1e-2, angle 3.7
    assert e[64] == pytest.approx(math.cos(3.7), abs=1e-12)
    assert e[192] == pytest.approx(math.sin(3.7), abs=1e-12)
    # index 96: frequency 1e4^(-3/4) = 1e-3, angle 0.37
    assert e[96] == pytest.approx(math.cos(0.37), abs=1e-12)
    # cos^2 + sin^2 = 1 for every frequency
    np.testing.assert_allclose(e[:128] ** 2 + e[128:] ** 2, 1.0, atol=1e-14)


# ---------------------------------------------------------------- activations
def test_silu_pins():
    x = np.linspace(-30, 30, 2001)
    s = O.silu(x)
    assert O.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(s - O.silu(-x), x, atol=1e-12)        # x*(sig(x)+sig(-x)) = x
    np.testing.assert_allclose(s, torch.nn.functional.silu(torch.from_numpy(x)).numpy(), rtol=1e-12, atol=1e-14)


def test_gelu_tanh_pins():
    x = np.linspace(-8, 8, 4001)
    g = O.gelu_tanh(x)
    assert O.gelu_tanh(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(g - O.gelu_tanh(-x), x, atol=1e-12)   # odd part is x/2 * 2
    ref = torch.nn.functional.gelu(torch.from_numpy(x), approximate="tanh").numpy()
    np.testing.assert_allclose(g, ref, rtol=1e-12, atol=1e-14)
    # the tanh form stays within 1e-3 of the exact erf GELU
    exact = 0.5 * x * (1 + np.vectorize(math.erf)(x / math.sqrt(2)))
    assert np.max(np.abs(g - exact)) < 1e-3


# ---------------------------------------------------------------- LayerNorm / adaLN
def test_layernorm_hand_example():
    g = _read_gold("layernorm_hand.txt")
    x = np.array(g["x"][0])
    y = O.layer_norm(x[None], 1e-6)[0]
    dev = np.array([-1.5, -0.5, 0.5, 1.5])
    np.testing.assert_allclose(y, dev / math.sqrt(g["var"][0][0] + 1e-6), rtol=1e-14)
    m = O.modulate(x[None], np.full(4, 0.5), np.ones(4), 1e-6)[0]
    np.testing.assert_allclose(m, 2 * dev / math.sqrt(1.25 + 1e-6) + 0.5, rtol=1e-14)


def test_layernorm_properties_and_library():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 96)) * 3 + 2
    y = O.layer_norm(x, 1e-6)
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-13)
    var = x.var(-1)
    np.testing.assert_allclose((y ** 2).mean(-1), var / (var + 1e-6), rtol=1e-12)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (96,), eps=1e-6).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-12)
    # zero modulation is plain LayerNorm
    np.testing.assert_array_equal(O.modulate(x, np.zeros(96), np.zeros(96), 1e-6), y)
    # a constant row normalises to zero
    np.testing.assert_array_equal(O.layer_norm(np.full((1, 8), 3.25), 1e-6), 0.0)


# ---------------------------------------------------------------- linear
def test_linear_brute_force():
    rng = np.random.default_rng(2)
    x, w, b = rng.standard_normal((3, 5)), rng.standard_normal((4, 5)), rng.standard_normal(4)
    y = O.linear(x, w, b)
    for i in range(3):
        for j in range(4):
            acc = b[j]
            for k in range(5):
                acc += x[i, k] * w[j, k]
            assert y[i, j] == pytest.approx(acc, rel=1e-13, abs=1e-13)
    np.testing.assert_array_equal(O.linear(x, np.eye(5), None), x)


# ---------------------------------------------------------------- RoPE
def test_rope_hand_example():
    g = _read_gold("rope_hand.txt")
    gw = int(g["grid_w"][0][0])
    tok = int(g["token"][0][0])
    gh = tok // gw + 1
    x = np.zeros((gh * gw, 1, 8))
    x[tok, 0] = g["x"][0]
    y = O.rope_2d(x, gh, gw, 1e4)
    np.testing.assert_allclose(y[tok, 0], g["out"][0], rtol=0, atol=1e-15)


def test_rope_properties():
    rng = np.random.default_rng(3)
    gh, gw, d = 6, 5, 16
    x = rng.standard_normal((gh * gw, 2, d))
    y = O.rope_2d(x, gh, gw, 1e4)
    np.testing.assert_array_equal(y[0], x[0])                       # position (0, 0): identity
    n_in = x[..., 0::2] ** 2 + x[..., 1::2] ** 2
    n_out = y[..., 0::2] ** 2 + y[..., 1::2] ** 2
    np.testing.assert_allclose(n_out, n_in, rtol=1e-12)             # every pair keeps its norm
    # token (0, j) leaves the row half alone, token (i, 0) the column half
    np.testing.assert_array_equal(y[3, :, : d // 2], x[3, :, : d // 2])
    np.testing.assert_array_equal(y[2 * gw, :, d // 2:], x[2 * gw, :, d // 2:])
    # complex-number form: pair k of the row axis is z * exp(i * row * 1e4^(-2k/(d/2)))
    z = x[..., 0:d // 2:2] + 1j * x[..., 1:d // 2:2]
    rows = (np.arange(gh * gw) // gw)[:, None, None]
    k = np.arange(d // 4)[None, None, :]
    zr = z * np.exp(1j * rows * (1e4 ** (-2.0 * k / (d // 2))))
    np.testing.assert_allclose(y[..., 0:d // 2:2], zr.real, atol=1e-12)
    np.testing.assert_allclose(y[..., 1:d // 2:2], zr.imag, atol=1e-12)


def test_rope_relative_position():
    """q . k after rotation depends only on the position difference."""
    rng = np.random.default_rng(4)
    d = 16
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    gh, gw = 12, 12

    def rot(vec, i, j):
        x = np.zeros((gh * gw, 1, d))
        x[i * gw + j, 0] = vec
        return O.rope_2d(x, gh, gw, 1e4)[i * gw + j, 0]

    a = rot(q, 3, 7) @ rot(k, 1, 2)
    b = rot(q, 8, 9) @ rot(k, 6, 4)     # both shifted by (5, 2)
    assert a == pytest.approx(b, rel=1e-10)


# ---------------------------------------------------------------- attention
def test_attention_hand_example():
    g = _read_gold("attention_hand.txt")
    q = np.array(g["q"])[:, None, :]
    k = np.array(g["k"])[:, None, :]
    v = np.array(g["v"])[:, None, :]
    out = O.attention(q, k, v)[0, 0]
    np.testing.assert_allclose(out, g["out"][0], rtol=1e-14)


def test_attention_brute_force_and_library():
    rng = np.random.default_rng(5)
    L, nh, d = 9, 2, 4
    q, k, v = (rng.standard_normal((L, nh, d)) for _ in range(3))
    o = O.attention(q, k, v)
    for h in range(nh):
        for i in range(L):
            s = [sum(q[i, h, c] * k[j, h, c] for c in range(d)) / math.sqrt(d) for j in range(L)]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            for c in range(d):
                assert o[i, h, c] == pytest.approx(sum(e[j] * v[j, h, c] for j in range(L)) / z, abs=1e-13)
    t = lambda a: torch.from_numpy(a).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v))[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-13)


def test_attention_invariants():
    rng = np.random.default_rng(6)
    L, nh, d = 16, 3, 8
    q, k, v = (rng.standard_normal((L, nh, d)) for _ in range(3))
    # V = identity rows: the output is P itself, whose rows sum to 1
    vi = np.broadcast_to(np.eye(L)[:, None, :], (L, nh, L)).copy()
    p = O.attention(q, k, vi)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=1e-14)
    assert (p > 0).all()
    # V = ones: output ones
    np.testing.assert_allclose(O.attention(q, k, np.ones_like(v)), 1.0, rtol=1e-14)
    # identical keys: mean of V
    ks = np.broadcast_to(k[:1], k.shape).copy()
    np.testing.assert_allclose(O.attention(q, ks, v), np.broadcast_to(v.mean(0), v.shape), rtol=1e-12)
    # one key: its value row
    np.testing.assert_allclose(O.attention(q, k[:1], v[:1]), np.broadcast_to(v[:1], v.shape), rtol=1e-14)
    # adding one vector to every key shifts each score row by a constant
    u = rng.standard_normal((1, nh, d))
    np.testing.assert_allclose(O.attention(q, k + u, v), O.attention(q, k, v), rtol=1e-11, atol=1e-13)
    # query subsets and chunking agree with the full result
    rows = np.array([0, 5, 15])
    np.testing.assert_allclose(O.attention(q, k, v, rows=rows, q_chunk=2), O.attention(q, k, v)[rows], rtol=1e-14)


# ---------------------------------------------------------------- Euler
def test_euler_closed_form():
    rng = np.random.default_rng(7)
    x, v = rng.standard_normal((5, 4)), rng.standard_normal((5, 4))
    np.testing.assert_array_equal(O.euler_update(x, v, 0.0), x)
    np.testing.assert_allclose(O.euler_update(x, v, 1 / 28), x - v / 28, rtol=1e-15)
    np.testing.assert_allclose(O.euler_update(x, 2 * v, 0.25) - x, 2 * (O.euler_update(x, v, 0.25) - x), rtol=1e-14)


# ---------------------------------------------------------------- blocks
TINY = O.OracleConfig(hidden=32, heads=2, head_dim=16, mlp_ratio=4, n_double=1, n_single=1,
                      in_channels=8, text_dim=24)


def _tiny(cfg=TINY, seed=0, zero_mod=False):
    p = synth.make_params(O.param_shapes(cfg), seed, bf16=False, std=0.2)
    if zero_mod:
        p["mod.w"][:] = 0
        p["mod.b"][:] = 0
    return {k: v.astype(np.float64) for k, v in p.items()}


def test_zero_gate_blocks_are_identity():
    p = _tiny(zero_mod=True)
    rng = np.random.default_rng(8)
    xt, xi, c = rng.standard_normal((5, 32)), rng.standard_normal((12, 32)), rng.standard_normal(32)
    yt, yi = O.double_block(p, TINY, 0, xt, xi, c, (3, 4))
    np.testing.assert_array_equal(yt, xt)
    np.testing.assert_array_equal(yi, xi)
    x = np.concatenate([xt, xi])
    np.testing.assert_array_equal(O.single_block(p, TINY, 0, x, 5, c, (3, 4)), x)


def test_text_permutation_equivariance():
    p = _tiny()
    rng = np.random.default_rng(9)
    xt, xi, c = rng.standard_normal((5, 32)), rng.standard_normal((12, 32)), rng.standard_normal(32)
    perm = np.array([3, 0, 4, 1, 2])
    yt, yi = O.double_block(p, TINY, 0, xt, xi, c, (3, 4))
    pt, pi = O.double_block(p, TINY, 0, xt[perm], xi, c, (3, 4))
    np.testing.assert_allclose(pt, yt[perm], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(pi, yi, rtol=1e-12, atol=1e-12)
    x = np.concatenate([xt, xi])
    xp = np.concatenate([xt[perm], xi])
    y = O.single_block(p, TINY, 0, x, 5, c, (3, 4))
    yp = O.single_block(p, TINY, 0, xp, 5, c, (3, 4))
    np.testing.assert_allclose(yp[:5], y[:5][perm], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(yp[5:], y[5:], rtol=1e-12, atol=1e-12)


def test_tied_double_block_equals_untied_with_equal_weights():
    tied = O.OracleConfig(hidden=32, heads=2, head_dim=16, n_double=1, in_channels=8, text_dim=24,
                          tie_streams=True)
    untied = O.OracleConfig(hidden=32, heads=2, head_dim=16, n_double=1, in_channels=8, text_dim=24)
    pt = _tiny(tied, seed=3)
    pu = {}
    lay_t, lay_u = O.modulation_layout(tied), O.modulation_layout(untied)
    for name, shape in O.param_shapes(untied):
        if name.startswith("double.0.txt."):
            pu[name] = pt["double.0.img." + name[len("double.0.txt."):]]
        elif name in ("mod.w", "mod.b"):
            src = pt[name]
            dst = np.zeros(shape)
            o_img = lay_t["double.0.img"][0]
            for key in ("double.0.img", "double.0.txt"):
                dst[lay_u[key][0]:lay_u[key][0] + 6 * 32] = src[o_img:o_img + 6 * 32]
            dst[lay_u["final"][0]:lay_u["final"][0] + 64] = src[lay_t["final"][0]:lay_t["final"][0] + 64]
            pu[name] = dst
        else:
            pu[name] = pt[name]
    rng = np.random.default_rng(10)
    xt, xi, c = rng.standard_normal((4, 32)), rng.standard_normal((9, 32)), rng.standard_normal(32)
    a = O.double_block(pt, tied, 0, xt, xi, c, (3, 3))
    b = O.double_block(pu, untied, 0, xt, xi, c, (3, 3))
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_block_attention_sees_joint_sequence():
    """A double block's text output changes when only the image input changes
    (attention couples the streams), but not when the image rows are shifted
    by a per-row constant, which the LayerNorm removes."""
    p = _tiny(zero_mod=False, seed=4)
    rng = np.random.default_rng(11)
    xt, xi, c = rng.standard_normal((5, 32)), rng.standard_normal((12, 32)), rng.standard_normal(32)
    yt, _ = O.double_block(p, TINY, 0, xt, xi, c, (3, 4))
    yt2, _ = O.double_block(p, TINY, 0, xt, xi + rng.standard_normal(xi.shape), c, (3, 4))
    assert np.abs(yt - yt2).max() > 1e-3
    yt3, _ = O.double_block(p, TINY, 0, xt, xi + rng.standard_normal((12, 1)), c, (3, 4))
    np.testing.assert_allclose(yt3, yt, atol=1e-12)


def test_fp32_oracle_agrees_with_fp64():
    cfg = O.OracleConfig(hidden=384, heads=6, head_dim=64, n_double=1, in_channels=16, text_dim=384,
                         tie_streams=True)
    p = synth.make_params(O.param_shapes(cfg), 0, bf16=False)
    lat = synth.normal(0, "latents", (256, 16))
    txt = synth.normal(0, "text", (32, 384))
    v64 = O.dit_velocity(p, cfg, lat, txt, 0.5, (16, 16), np.float64)
    v32 = O.dit_velocity(p, cfg, lat, txt, 0.5, (16, 16), np.float32)
    err = np.abs(v32 - v64).max() / np.abs(v64).max()
    assert err < 1e-5, err


def test_step_is_per_request():
    cfg = O.OracleConfig(hidden=32, heads=2, head_dim=16, n_double=1, n_single=1, in_channels=8, text_dim=24)
    p = _tiny(cfg, seed=5)
    rng = np.random.default_rng(12)
    reqs = [O.OracleRequest(2, 3, 0.2, rng.standard_normal((6, 8)), rng.standard_normal((4, 24))),
            O.OracleRequest(3, 3, 0.9, rng.standard_normal((9, 8)), rng.standard_normal((2, 24)))]
    vs, xs = O.dit_step(p, cfg, reqs, [0.1, 0.2])
    v1, x1 = O.dit_step(p, cfg, reqs[1:], [0.2])
    np.testing.assert_array_equal(vs[1], v1[0])
    np.testing.assert_array_equal(xs[1], reqs[1].latents - 0.2 * vs[1])


def test_sampled_rows_match_full_blocks():
    p = _tiny(seed=6)
    rng = np.random.default_rng(13)
    xt, xi, c = rng.standard_normal((5, 32)), rng.standard_normal((12, 32)), rng.standard_normal(32)
    yt, yi = O.double_block(p, TINY, 0, xt, xi, c, (3, 4))
    rt, ri = np.array([4, 0]), np.array([11, 3, 7])
    st, si = O.double_block(p, TINY, 0, xt, xi, c, (3, 4), rows_txt=rt, rows_img=ri)
    np.testing.assert_allclose(st, yt[rt], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(si, yi[ri], rtol=1e-13, atol=1e-13)
    x = np.concatenate([xt, xi])
    y = O.single_block(p, TINY, 0, x, 5, c, (3, 4))
    rows = np.array([16, 2, 9])
    np.testing.assert_allclose(O.single_block(p, TINY, 0, x, 5, c, (3, 4), rows=rows), y[rows], rtol=1e-13, atol=1e-13)
