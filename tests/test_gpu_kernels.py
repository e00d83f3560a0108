"""Kernel-level parity on the GPU: each entry point of the C ABI against the
oracle on the same seeded inputs, at sizes that span several tiles and end
in ragged tails."""
import numpy as np
import pytest

import oracle as O
from paper_2510_01565_amd import dit, synth
from harness import BF16_TOL, F32_TOL, normwise_err, to_dev

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


@pytest.mark.parametrize("M,N,K", [(1, 1, 8), (1, 3001, 64), (77, 64, 40), (300, 200, 136), (2500, 1100, 520),
                                   (513, 3072, 3072)])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_linear_bf16(M, N, K, out):
    torch = _torch()
    x = synth.normal(1, "x", (M, K), bf16=True)
    w = synth.normal(1, "w", (N, K), std=0.02, bf16=True)
    b = synth.normal(1, "b", (N,), std=0.02, bf16=True)
    ref = O.linear(x.astype(np.float64), w.astype(np.float64), b.astype(np.float64))
    od = torch.float32 if out == "f32" else torch.bfloat16
    y = torch.empty((M, N), dtype=od, device="cuda")
    dit.dit_linear(M, N, K, dit.DIT_BF16, to_dev(x, torch.bfloat16), to_dev(w, torch.bfloat16),
                   to_dev(b, torch.bfloat16), y, dit.DIT_F32 if out == "f32" else dit.DIT_BF16)
    torch.cuda.synchronize()
    err = normwise_err(y.float().cpu().numpy(), ref)
    assert err < (F32_TOL if out == "f32" else BF16_TOL), err
    if out == "bf16":
        # every element within 2 bf16 ulps of the exact value
        g = y.float().cpu().numpy()
        assert np.all(np.abs(g - ref) <= 2 ** -7 * np.abs(ref) + 1e-6 * np.abs(ref).max())


@pytest.mark.parametrize("M,N,K,cfg", [
    (5410, 659, 512, "256x128"), (5410, 659, 520, "256x128"),      # direct-to-LDS and register paths
    (1303, 5429, 512, "128x256"), (1303, 5429, 520, "128x256"),
    (6001, 2313, 512, "256x256"), (6001, 2313, 520, "256x256"),
    (5891, 1295, 512, "288x192"),                                  # direct-to-LDS only (96x48 wave tiles)
    (600, 500, 512, "128x128"), (600, 500, 520, "128x128"),
])
def test_linear_bf16_every_tile_config(M, N, K, cfg):
    """Shapes for which the launch model picks each tile configuration (the
    profile names the kernel that ran); 800 sampled outputs against fp64 dot
    products, including the ragged last row and column."""
    torch = _torch()
    x = synth.normal(2, "x", (M, K), bf16=True)
    w = synth.normal(2, "w", (N, K), std=0.02, bf16=True)
    b = synth.normal(2, "b", (N,), std=0.02, bf16=True)
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    dit.profile_start()
    dit.dit_linear(M, N, K, dit.DIT_BF16, to_dev(x, torch.bfloat16), to_dev(w, torch.bfloat16),
                   to_dev(b, torch.bfloat16), y, dit.DIT_F32)
    torch.cuda.synchronize()
    ran = dit.profile_stop()
    assert "gemm_bf16_" + cfg in ran, list(ran)
    rng = np.random.default_rng(M * N + K)
    ms = np.concatenate([[0, M - 1, M - 1, 127, 128], rng.integers(0, M, 795)])
    ns = np.concatenate([[0, N - 1, 0, 255, 256], rng.integers(0, N, 795)])
    ref = (x[ms].astype(np.float64) * w[ns].astype(np.float64)).sum(axis=1) + b[ns].astype(np.float64)
    got = y.cpu().numpy()[ms, ns]
    assert normwise_err(got, ref) < F32_TOL


@pytest.mark.parametrize("M,N,cfg", [(6001, 2313, "256x256"), (5891, 1295, "288x192"), (5410, 659, "256x128"),
                                     (1303, 5429, "128x256"), (600, 500, "128x128")])
@pytest.mark.parametrize("K", [192, 576])
def test_linear_bf16_odd_k_tile_count(M, N, K, cfg):
    """An odd number of 64-wide K tiles (3 and 9): the main loop runs over pairs
    of tiles and the last tile runs on its own, with the refetch of the last
    tile as its loads.  Same sampled check as above."""
    torch = _torch()
    x = synth.normal(3, "x", (M, K), bf16=True)
    w = synth.normal(3, "w", (N, K), std=0.02, bf16=True)
    b = synth.normal(3, "b", (N,), std=0.02, bf16=True)
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    dit.profile_start()
    dit.dit_linear(M, N, K, dit.DIT_BF16, to_dev(x, torch.bfloat16), to_dev(w, torch.bfloat16),
                   to_dev(b, torch.bfloat16), y, dit.DIT_F32)
    torch.cuda.synchronize()
    ran = dit.profile_stop()
    assert any(k.startswith("gemm_bf16_") for k in ran), list(ran)
    if K == 576:  # at 9 K tiles the launch model picks the named configuration for each shape
        assert "gemm_bf16_" + cfg in ran, list(ran)
    rng = np.random.default_rng(M * N + K + 7)
    ms = np.concatenate([[0, M - 1, M - 1, 127, 128], rng.integers(0, M, 795)])
    ns = np.concatenate([[0, N - 1, 0, 255, 256], rng.integers(0, N, 795)])
    ref = (x[ms].astype(np.float64) * w[ns].astype(np.float64)).sum(axis=1) + b[ns].astype(np.float64)
    got = y.cpu().numpy()[ms, ns]
    assert normwise_err(got, ref) < F32_TOL


@pytest.mark.parametrize("M,N,K", [(5, 3, 8), (130, 70, 200), (300, 1152, 384)])
def test_linear_f32(M, N, K):
    torch = _torch()
    x = synth.normal(2, "x", (M, K))
    w = synth.normal(2, "w", (N, K), std=0.02)
    b = synth.normal(2, "b", (N,), std=0.02)
    ref = O.linear(x.astype(np.float64), w.astype(np.float64), b.astype(np.float64))
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    dit.dit_linear(M, N, K, dit.DIT_F32, to_dev(x, torch.float32), to_dev(w, torch.float32),
                   to_dev(b, torch.float32), y, dit.DIT_F32)
    torch.cuda.synchronize()
    assert normwise_err(y.cpu().numpy(), ref) < F32_TOL


def _attn_case(grids, n_txt, heads, d, bf16, seed):
    torch = _torch()
    lens = [gh * gw + nt for (gh, gw), nt in zip(grids, n_txt)]
    T = sum(lens)
    q = synth.normal(seed, "q", (T, heads, d), bf16=bf16)
    k = synth.normal(seed, "k", (T, heads, d), bf16=bf16)
    v = synth.normal(seed, "v", (T, heads, d), bf16=bf16)
    ref = np.empty((T, heads, d))
    off = 0
    for L in lens:
        sl = slice(off, off + L)
        ref[sl] = O.attention(q[sl].astype(np.float64), k[sl].astype(np.float64), v[sl].astype(np.float64))
        off += L
    dt = torch.bfloat16 if bf16 else torch.float32
    b = dit.Batch([g[0] for g in grids], [g[1] for g in grids], n_txt)
    dtype = dit.DIT_BF16 if bf16 else dit.DIT_F32
    wsb = dit.attention_workspace_size(b, heads, d, dtype)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    o = torch.full((T, heads, d), float("nan"), dtype=dt, device="cuda")
    dit.dit_attention(b, heads, d, dtype, to_dev(q, dt), to_dev(k, dt), to_dev(v, dt), o, ws, wsb)
    torch.cuda.synchronize()
    return o.float().cpu().numpy(), ref


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("grids,n_txt", [
    ([(16, 16)], [32]),                       # 288 tokens: 2 full + 1 partial query tile, ragged key tile
    ([(5, 7), (16, 16), (9, 13)], [3, 32, 17]),  # packed, lengths 38 / 288 / 134
    ([(1, 1)], [0]),                          # a single token
    ([(8, 8)], [0]),                          # exactly one 64-key tile
    ([(8, 8), (11, 11)], [1, 7]),             # 65 and 128 tokens: one key past a tile, exactly two tiles
])
def test_attention_bf16(grids, n_txt, d):
    got, ref = _attn_case(grids, n_txt, 3, d, True, 3)
    assert normwise_err(got, ref) < BF16_TOL


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("gain", [4.0, 16.0])
def test_attention_bf16_large_logits(d, gain):
    """Scores far outside the unit range: q and k scaled so that the log2-domain
    logits reach tens (gain 4) or hundreds (gain 16), which takes the softmax
    off its reference-0 path and through the rescales."""
    torch = _torch()
    grids, n_txt, heads = [(12, 12), (7, 9)], [40, 5], 2
    lens = [gh * gw + nt for (gh, gw), nt in zip(grids, n_txt)]
    T = sum(lens)
    q = (synth.normal(6, "q", (T, heads, d)) * gain).astype(np.float32)
    k = (synth.normal(6, "k", (T, heads, d)) * gain).astype(np.float32)
    v = synth.normal(6, "v", (T, heads, d), bf16=True)
    qb = torch.from_numpy(q).to(torch.bfloat16)
    kb = torch.from_numpy(k).to(torch.bfloat16)
    q64 = qb.float().numpy().astype(np.float64)
    k64 = kb.float().numpy().astype(np.float64)
    ref = np.empty((T, heads, d))
    off = 0
    for L in lens:
        sl = slice(off, off + L)
        ref[sl] = O.attention(q64[sl], k64[sl], v[sl].astype(np.float64))
        off += L
    b = dit.Batch([g[0] for g in grids], [g[1] for g in grids], n_txt)
    wsb = dit.attention_workspace_size(b, heads, d, dit.DIT_BF16)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    o = torch.full((T, heads, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    dit.dit_attention(b, heads, d, dit.DIT_BF16, qb.cuda(), kb.cuda(), to_dev(v, torch.bfloat16), o, ws, wsb)
    torch.cuda.synchronize()
    assert normwise_err(o.float().cpu().numpy(), ref) < BF16_TOL


@pytest.mark.parametrize("grids,n_txt,heads", [
    ([(31, 31)], [39], 136),          # 1000 tokens, 1088 units: 64 leftover tiles x 8 key ranges, ragged tiles
    ([(31, 31)], [39], 144),          # 1152 units: 128 leftover tiles x 4 key ranges
    ([(20, 25), (25, 20)], [0, 0], 132),  # two requests of 500 tokens: 32 x 8 ranges of one key tile each
])
def test_attention_bf16_key_split(grids, n_txt, heads):
    """The launch whose last round of 128-query tiles is at most half full
    splits those tiles' keys into ranges merged afterwards; every tile,
    split or not, against the oracle, and the same bits on a second call."""
    torch = _torch()
    lens = [gh * gw + nt for (gh, gw), nt in zip(grids, n_txt)]
    T, d = sum(lens), 128
    b = dit.Batch([g[0] for g in grids], [g[1] for g in grids], n_txt)
    assert dit.attention_workspace_size(b, heads, d, dit.DIT_BF16) > 2 * T * heads * d + 4096  # the split applies
    q = synth.normal(7, "q", (T, heads, d), bf16=True)
    k = synth.normal(7, "k", (T, heads, d), bf16=True)
    v = synth.normal(7, "v", (T, heads, d), bf16=True)
    ref = np.empty((T, heads, d))
    off = 0
    for L in lens:
        sl = slice(off, off + L)
        ref[sl] = O.attention(q[sl].astype(np.float64), k[sl].astype(np.float64), v[sl].astype(np.float64))
        off += L
    wsb = dit.attention_workspace_size(b, heads, d, dit.DIT_BF16)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    qd, kd, vd = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    outs = []
    for _ in range(2):
        o = torch.full((T, heads, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        dit.dit_attention(b, heads, d, dit.DIT_BF16, qd, kd, vd, o, ws, wsb)
        torch.cuda.synchronize()
        outs.append(o)
    got = outs[0].float().cpu().numpy()
    assert normwise_err(got, ref) < BF16_TOL
    # the leftover tiles are the last heads' last query tiles: check those heads alone too
    assert normwise_err(got[:, -2:], ref[:, -2:]) < BF16_TOL
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("gain", [4.0, 16.0])
def test_attention_bf16_key_split_large_logits(gain):
    """The key-split merge with scores far outside the unit range: each key
    range has its own running max, tens to hundreds apart in the log2
    domain, and the merge rescales the ranges' sums and outputs to the
    largest (1000 tokens, 136 heads: 64 leftover query tiles x 8 key ranges)."""
    torch = _torch()
    grids, n_txt, heads, d = [(31, 31)], [39], 136, 128
    T = 31 * 31 + 39
    b = dit.Batch([31], [31], n_txt)
    q = (synth.normal(8, "q", (T, heads, d)) * gain).astype(np.float32)
    k = (synth.normal(8, "k", (T, heads, d)) * gain).astype(np.float32)
    v = synth.normal(8, "v", (T, heads, d), bf16=True)
    qb = torch.from_numpy(q).to(torch.bfloat16)
    kb = torch.from_numpy(k).to(torch.bfloat16)
    ref = O.attention(qb.float().numpy().astype(np.float64), kb.float().numpy().astype(np.float64),
                      v.astype(np.float64))
    wsb = dit.attention_workspace_size(b, heads, d, dit.DIT_BF16)
    assert wsb > 2 * T * heads * d + 4096  # the split applies
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    o = torch.full((T, heads, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    dit.dit_attention(b, heads, d, dit.DIT_BF16, qb.cuda(), kb.cuda(), to_dev(v, torch.bfloat16), o, ws, wsb)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy()
    assert normwise_err(got, ref) < BF16_TOL
    assert normwise_err(got[:, -8:], ref[:, -8:]) < BF16_TOL  # the heads whose tiles were split


@pytest.mark.parametrize("grids,n_txt", [([(16, 16)], [32]), ([(5, 7), (9, 13)], [3, 17])])
def test_attention_f32(grids, n_txt):
    got, ref = _attn_case(grids, n_txt, 2, 64, False, 4)
    assert normwise_err(got, ref) < F32_TOL


@pytest.mark.parametrize("d", [128, 64])
def test_attention_identical_keys_give_mean_of_values(d):
    torch = _torch()
    T, heads = 200, 2
    q = synth.normal(5, "q", (T, heads, d), bf16=True)
    k = np.broadcast_to(synth.normal(5, "k", (1, heads, d), bf16=True), (T, heads, d)).copy()
    v = synth.normal(5, "v", (T, heads, d), bf16=True)
    b = dit.Batch([10], [18], [20])
    wsb = dit.attention_workspace_size(b, heads, d, dit.DIT_BF16)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    o = torch.empty((T, heads, d), dtype=torch.bfloat16, device="cuda")
    dit.dit_attention(b, heads, d, dit.DIT_BF16, to_dev(q, torch.bfloat16), to_dev(k, torch.bfloat16),
                      to_dev(v, torch.bfloat16), o, ws, wsb)
    torch.cuda.synchronize()
    ref = np.broadcast_to(v.astype(np.float64).mean(0), v.shape)
    assert normwise_err(o.float().cpu().numpy(), ref) < BF16_TOL


@pytest.mark.parametrize("bf16", [False, True])
def test_euler(bf16):
    torch = _torch()
    grids = [(3, 5), (8, 8)]
    C = 16
    n = sum(g[0] * g[1] for g in grids)
    x = synth.normal(6, "x", (n, C), bf16=bf16)
    v = synth.normal(6, "v", (n, C), bf16=bf16)
    dts = [1 / 28, 0.3]
    dt = torch.bfloat16 if bf16 else torch.float32
    xd = to_dev(x, dt)
    b = dit.Batch([g[0] for g in grids], [g[1] for g in grids], [0, 0])
    dit.euler_update(b, C, dit.DIT_BF16 if bf16 else dit.DIT_F32, xd, to_dev(v, dt), dts)
    torch.cuda.synchronize()
    ref = np.concatenate([O.euler_update(x[:15].astype(np.float64), v[:15].astype(np.float64), dts[0]),
                          O.euler_update(x[15:].astype(np.float64), v[15:].astype(np.float64), dts[1])])
    got = xd.float().cpu().numpy()
    if bf16:
        assert np.all(np.abs(got - ref) <= 2 ** -8 * np.abs(ref) + 1e-30)
    else:
        assert np.all(np.abs(got - ref) <= 1e-6 * np.abs(ref) + 1e-7)
