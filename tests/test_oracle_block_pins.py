"""Pins of the oracle's composed functions (conditioning, modulation, final
layer, double-stream block, single-stream block) against the hand-derived
example in golden/block_hand.txt.  CPU only.

Each assertion names the plausible transcription slip it rules out; every
one of these slips, applied to a copy of the oracle, fails at least one
assertion below:
  (a) SiLU dropped before the modulation weights (modulation);
  (b) SiLU dropped inside the timestep MLP (conditioning);
  (c) shift and scale swapped in the final layer;
  (d) the double block's MLP LayerNorm fed from the input residual instead
      of the residual after the attention update;
  (e) gate1 and gate2 swapped.
"""
import os

import numpy as np

import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden", "block_hand.txt")

CFG = O.OracleConfig(hidden=4, heads=1, head_dim=4, mlp_ratio=1, n_double=1, n_single=1, in_channels=4,
                     text_dim=4, time_freq_dim=8)
I4 = np.eye(4)
X_TXT = np.array([1.0, -1.0, 1.0, -1.0])
X_IMG = np.array([3.0, 1.0, 1.0, -1.0])
TOL = dict(rtol=1e-12, atol=1e-12)


def _gold():
    rows = {}
    with open(GOLD) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                key, *vals = line.split()
                rows.setdefault(key, []).append(np.array([float(v) for v in vals]))
    return rows


G = _gold()


def _params():
    """The structured parameters of the hand example (every other entry 0)."""
    p = {name: np.zeros(shape) for name, shape in O.param_shapes(CFG)}
    p["time_in.w1"][0, :4] = 0.375
    p["time_in.w1"][1, :4] = -0.5
    p["time_in.w1"][2, :] = [0.25, 0.25, 0, 0, 7, 7, 7, 7]
    p["time_in.w1"][3, 3] = -0.5
    p["time_in.b1"][:] = [0.5, 0, 0, 0]
    p["time_in.w2"][:] = [[1, 1, 0, 0], [0, 1, 0, 0], [0, 0, 2, 0], [0, 0, 0, -1]]
    p["time_in.b2"][:] = [0.1, 0, 0, 0.2]
    lay = O.modulation_layout(CFG)
    chunks = {
        "double.0.img": [[.5, 0, 0, -.5], [0, 1, 0, 0], [.5] * 4, [0, 0, 0, .25], [0, 0, -.5, 0], [2, 1, 2, 1]],
        "double.0.txt": [[0, .25, 0, 0], [1, 0, 0, 0], [1, 0, 1, 0], [.5, 0, 0, 0], [0, 0, 0, 1], [.25] * 4],
        "single.0": [[0, 0, .5, 0], [.5, 0, 0, 0], [1, 3, 2, 4]],
    }
    for key, ch in chunks.items():
        off = lay[key][0]
        p["mod.b"][off:off + 4 * len(ch)] = np.concatenate(ch)
    off = lay["final"][0]
    p["mod.w"][off:off + 8] = [[1, 0, 0, 0], [0, 1, 0, 0], [0, 0, 0, 1], [1, 1, 0, 0],
                               [0, 0, 0, .5], [0, 0, 0, 0], [2, 0, 0, 0], [0, 0, 0, 0]]
    p["mod.b"][off:off + 8] = [0, 0, 0, 0, .1, .2, .3, .4]
    p["final.w"][:] = [[1, 0, 0, 0], [0, 0, 1, 0], [0, 1, 0, 0], [1, 0, 0, 1]]
    p["final.b"][:] = [0, 0, 0, .5]
    for s, bv in (("img", [0, 0, 0, 1]), ("txt", [0, 0, 0, 0])):
        pre = f"double.0.{s}."
        p[pre + "qkv.w"][8:12] = I4
        p[pre + "qkv.b"][8:12] = bv
        for n in ("proj.w", "mlp1.w", "mlp2.w"):
            p[pre + n][:] = I4
    p["single.0.lin1.w"][8:12] = I4
    p["single.0.lin1.w"][12:16] = I4
    p["single.0.lin2.w"][:] = np.concatenate([I4, 2 * I4], axis=1)
    return p


def test_conditioning_hand_example():
    """c at t = 0.  Kills (b): without the inner SiLU c = (.1, -2, 1, .7)."""
    c = O.conditioning(_params(), CFG, 0.0)
    np.testing.assert_allclose(c, G["cond"][0], **TOL)


def test_modulation_hand_example():
    """Final-layer chunks for c = (1, -1, 0, 2).  Kills (a): without the SiLU
    the shift chunk would read (1, -1, 2, 0)."""
    sh, sc = O.modulation(_params(), CFG, "final", np.array([1.0, -1.0, 0.0, 2.0]))
    np.testing.assert_allclose(sh, G["final_shift"][0], **TOL)
    np.testing.assert_allclose(sc, G["final_scale"][0], **TOL)


def test_final_layer_hand_example():
    """Velocity of two image tokens.  Kills (c) (scale and shift enter as
    LN(x)(1 + scale) + shift, not the other way round) and (a) again; also
    fixes the [out, in] orientation of the final weight (row 3 reads inputs 0
    and 3)."""
    x = np.stack(G["final_x"])
    v = O.final_layer(_params(), CFG, x, np.array([1.0, -1.0, 0.0, 2.0]))
    np.testing.assert_allclose(v, np.stack(G["final_v"]), **TOL)


def test_double_block_hand_example():
    """Kills (d): the MLP's LayerNorm must see x + gate1 * attention; fed
    from the input residual the image output's first entry would be 5.75...
    Kills (e): gate1 = (.5, .5, .5, .5) and gate2 = (2, 1, 2, 1) for the
    image stream differ, as do the text gates.  Also fixes the joint
    attention (the text output depends on the image token's V bias)."""
    yt, yi = O.double_block(_params(), CFG, 0, X_TXT[None], X_IMG[None], np.zeros(4), (1, 1))
    np.testing.assert_allclose(yt[0], G["double_out_txt"][0], **TOL)
    np.testing.assert_allclose(yi[0], G["double_out_img"][0], **TOL)


def test_single_block_hand_example():
    """Joint sequence [text; image]: linear2 sees [attention | GELU(MLP)] in
    that order (weights I and 2 I) and one gated residual with gate (1, 3, 2, 4)."""
    x = np.stack([X_TXT, X_IMG])
    y = O.single_block(_params(), CFG, 0, x, 1, np.zeros(4), (1, 1))
    np.testing.assert_allclose(y, np.stack(G["single_out"]), **TOL)


def test_hand_example_intermediates_are_consistent():
    """The fixture's intermediate rows follow from each other (guards the
    fixture itself): x' = x + gate1 * o and o = mean of the two V rows."""
    o = (G["double_A_txt"][0] + G["double_A_img"][0] + np.array([0, 0, 0, 1.0])) / 2
    np.testing.assert_allclose(o, G["double_attn"][0], **TOL)
    np.testing.assert_allclose(X_TXT + np.array([1, 0, 1, 0]) * o, G["double_after_attn_txt"][0], **TOL)
    np.testing.assert_allclose(X_IMG + 0.5 * o, G["double_after_attn_img"][0], **TOL)
    np.testing.assert_allclose((G["single_A"][0] + G["single_A"][1]) / 2, G["single_attn"][0], **TOL)
