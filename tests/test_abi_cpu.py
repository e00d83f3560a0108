"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function that include/dit.h declares, describes the same parameter set
as the oracle, sizes workspaces, and rejects invalid calls before enqueuing
anything."""
import ctypes
import os
import re

import pytest

import oracle as O
from paper_2510_01565_amd import dit, workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "dit.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:dit_status|const char\*)\s+(\w+)\s*\(", src, flags=re.M)))


def test_library_exports_every_header_function():
    names = _header_functions()
    assert len(names) >= 10
    L = dit.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(dit.EXPORTED)


def _oracle_cfg(m: workloads.ModelShape):
    return O.OracleConfig(hidden=m.hidden, heads=m.heads, head_dim=m.head_dim, mlp_ratio=m.mlp_ratio,
                          n_double=m.n_double, n_single=m.n_single, in_channels=m.in_channels,
                          text_dim=m.text_dim, time_freq_dim=m.time_freq_dim, tie_streams=m.tie_streams)


@pytest.mark.parametrize("name", ["small_block_256px_f32", "mmdit_double_512px_bf16", "dit57_1024px_bf16"])
def test_manifest_matches_oracle_parameter_set(name):
    m = workloads.WORKLOADS[name].model
    got = dit.weight_manifest(dit.make_config(m))
    assert got == [(n, tuple(s)) for n, s in O.param_shapes(_oracle_cfg(m))]


def test_full_model_parameter_count():
    m = workloads.FLUX_FULL
    n = sum(int(__import__("numpy").prod(s)) for _, s in dit.weight_manifest(dit.make_config(m)))
    # 19 double + 38 single blocks at 3072 wide: ~11.9e9 parameters, 3.25e9 of them adaLN modulation
    assert 11.8e9 < n < 12.0e9
    mod = [s for nm, s in dit.weight_manifest(dit.make_config(m)) if nm == "mod.w"][0]
    assert mod == ((19 * 12 + 38 * 3 + 2) * 3072, 3072)


def test_workspace_size_grows_with_tokens():
    cfg = dit.make_config(workloads.FLUX_FULL)
    a = dit.workspace_size(cfg, dit.Batch([64], [64], [512], [0.5]))
    b = dit.workspace_size(cfg, dit.Batch([128], [128], [512], [0.5]))
    c = dit.workspace_size(cfg, dit.Batch([16, 32, 64, 128], [16, 32, 64, 128], [512] * 4, [0.1, 0.2, 0.3, 0.4]))
    assert 0 < a < b < c
    assert c < 4 * 2 ** 30     # the 23808-token packed step needs only a few GB of scratch


def _err(fn, *args):
    with pytest.raises(dit.DitError) as e:
        fn(*args)
    return e.value.status


def test_invalid_configs_are_rejected():
    base = workloads.FLUX_FULL
    cfg = dit.make_config(base)
    cfg.heads = 23
    assert _err(dit.weight_count, cfg) == dit.DIT_ERR_INVALID_ARG
    cfg = dit.make_config(base)
    cfg.head_dim, cfg.heads = 96, 32
    assert _err(dit.weight_count, cfg) == dit.DIT_ERR_UNSUPPORTED
    cfg = dit.make_config(base)
    cfg.head_dim, cfg.heads = 64, 48   # bf16 head_dim 64 (the SD3-Medium head) is supported
    assert dit.weight_count(cfg) == dit.weight_count(dit.make_config(base))
    f32 = dit.make_config(workloads.SMALL_BLOCK)
    f32.head_dim, f32.heads = 128, 3   # fp32 attention is head_dim 64 only
    assert _err(dit.weight_count, f32) == dit.DIT_ERR_UNSUPPORTED
    cfg = dit.make_config(base)
    cfg.in_channels = 12
    assert _err(dit.weight_count, cfg) == dit.DIT_ERR_UNSUPPORTED
    cfg = dit.make_config(base)
    cfg.dtype = 7
    assert _err(dit.weight_count, cfg) == dit.DIT_ERR_INVALID_ARG
    assert "dtype" in dit.lib().dit_last_error().decode()
    cfg = dit.make_config(base, 2)   # no such flag
    assert _err(dit.weight_count, cfg) == dit.DIT_ERR_INVALID_ARG


def test_split_workspace_only_without_batch_invariance():
    """bf16 models reserve the split-K partial sums and counters unless
    DIT_FLAG_BATCH_INVARIANT is set; fp32 models never do."""
    b = dit.Batch([16], [16], [512], [0.5])
    m = workloads.FLUX_FULL
    free = dit.workspace_size(dit.make_config(m), b)
    inv = dit.workspace_size(dit.make_config(m, dit.DIT_FLAG_BATCH_INVARIANT), b)
    assert free - inv == 96 * 2 ** 20 + 4096
    f32 = workloads.SMALL_BLOCK
    assert dit.workspace_size(dit.make_config(f32), b) == \
        dit.workspace_size(dit.make_config(f32, dit.DIT_FLAG_BATCH_INVARIANT), b)


def _split_bytes(tail_units, pieces, d=128):
    return -(-(tail_units * pieces * 128 * (d + 2) * 4) // 256) * 256


def test_attention_key_split_rule():
    """The bf16 attention splits the key ranges of its last round of
    128-query tiles only when that round holds at most a quarter of the 512
    block slots and follows at least two full rounds, every request has one
    length and the head dim is 128; the extra workspace is the pieces' fp32
    partials (P = min(512 // T, key tiles) pieces per leftover tile)."""
    bf = dit.DIT_BF16

    def extra(b, heads, d=128):
        vt = dit.attention_workspace_size(b, heads, d, dit.DIT_F32) // 2  # same V^T shape, fp32 has no split
        return dit.attention_workspace_size(b, heads, d, bf) - -(-vt // 256) * 256
    one = dit.Batch([31], [31], [39])                    # 1000 tokens: 8 query tiles, 16 key tiles
    assert extra(one, 136) == _split_bytes(64, 8)        # 1088 units: 2 rounds + 64
    assert extra(one, 144) == _split_bytes(128, 4)       # 1152: 2 rounds + 128
    assert extra(one, 145) == 0                          # 1160: last round 136 > 128
    assert extra(one, 160) == 0                          # 1280: last round 256
    assert extra(one, 128) == 0                          # 1024: no leftover
    assert extra(one, 72) == 0                           # 576: one full round only
    assert extra(one, 136, 64) == 0                      # head dim 64
    two = dit.Batch([20, 20], [25, 25], [0, 0])           # two requests of 500 tokens: 8 key tiles each
    assert extra(two, 132) == _split_bytes(32, 8)        # 1056 units: P capped by the 8 key tiles
    mixed = dit.Batch([20, 25], [25, 20], [0, 1])         # 500 and 501 tokens
    assert extra(mixed, 132) == 0
    flux2048 = dit.Batch([128], [128], [512])             # 16 896 tokens, 24 heads: 3168 units
    assert extra(flux2048, 24) == _split_bytes(96, 5)


def test_invalid_batches_are_rejected():
    cfg = dit.make_config(workloads.FLUX_FULL)
    assert _err(dit.workspace_size, cfg, dit.Batch([], [], [])) == dit.DIT_ERR_INVALID_ARG
    assert _err(dit.workspace_size, cfg, dit.Batch([1] * 17, [1] * 17, [0] * 17)) == dit.DIT_ERR_INVALID_ARG
    assert _err(dit.workspace_size, cfg, dit.Batch([0], [4], [1])) == dit.DIT_ERR_INVALID_ARG
    assert _err(dit.workspace_size, cfg, dit.Batch([257], [4], [1])) == dit.DIT_ERR_INVALID_ARG
    assert _err(dit.workspace_size, cfg, dit.Batch([4], [4], [-1])) == dit.DIT_ERR_INVALID_ARG


def test_dit_step_validation_happens_before_any_launch():
    """Every one of these calls fails on the host; none reaches the GPU."""
    m = workloads.SMALL_BLOCK
    cfg = dit.make_config(m)
    n = dit.weight_count(cfg)
    fake = dit.Weights([4096 * (i + 1) for i in range(n)])
    b = dit.Batch([16], [16], [32], [0.5])
    need = dit.workspace_size(cfg, b)
    P = 1 << 20
    # missing timesteps
    assert _err(dit.dit_step, cfg, fake, dit.Batch([16], [16], [32]), P, P, P, P, need, 0) == dit.DIT_ERR_INVALID_ARG
    # timestep outside [0, 1]
    assert _err(dit.dit_step, cfg, fake, dit.Batch([16], [16], [32], [1.5]), P, P, P, P, need, 0) == \
        dit.DIT_ERR_INVALID_ARG
    # wrong number of weights
    assert _err(dit.dit_step, cfg, dit.Weights([4096] * (n - 1)), b, P, P, P, P, need, 0) == dit.DIT_ERR_INVALID_ARG
    # misaligned weight
    bad = dit.Weights([4096 * (i + 1) + (8 if i == 3 else 0) for i in range(n)])
    assert _err(dit.dit_step, cfg, bad, b, P, P, P, P, need, 0) == dit.DIT_ERR_INVALID_ARG
    # null latents
    assert _err(dit.dit_step, cfg, fake, b, 0, P, P, P, need, 0) == dit.DIT_ERR_INVALID_ARG
    # workspace too small / null / misaligned
    assert _err(dit.dit_step, cfg, fake, b, P, P, P, P, need - 1, 0) == dit.DIT_ERR_WORKSPACE
    assert _err(dit.dit_step, cfg, fake, b, P, P, P, 0, need, 0) == dit.DIT_ERR_WORKSPACE
    assert _err(dit.dit_step, cfg, fake, b, P, P, P, P + 64, need, 0) == dit.DIT_ERR_WORKSPACE
    # block index out of range, bad kind
    assert _err(dit.dit_block_forward, cfg, fake, 0, 1, b, P, P, P, need, 0) == dit.DIT_ERR_INVALID_ARG
    assert _err(dit.dit_block_forward, cfg, fake, 2, 0, b, P, P, P, need, 0) == dit.DIT_ERR_INVALID_ARG
    # attention head_dim unsupported for the dtype
    assert _err(dit.dit_attention, b, 6, 96, dit.DIT_BF16, P, P, P, P, P, need, 0) == dit.DIT_ERR_UNSUPPORTED
    assert _err(dit.dit_attention, b, 3, 128, dit.DIT_F32, P, P, P, P, P, need, 0) == dit.DIT_ERR_UNSUPPORTED
    # GEMM K not a multiple of 8
    assert _err(dit.dit_linear, 4, 4, 12, dit.DIT_BF16, P, P, 0, P, dit.DIT_F32, 0) == dit.DIT_ERR_UNSUPPORTED
    # Euler with a non-finite dt
    assert _err(dit.euler_update, b, 16, dit.DIT_F32, P, P, [float("nan")], 0) == dit.DIT_ERR_INVALID_ARG


def test_last_error_is_cleared_by_a_good_call():
    cfg = dit.make_config(workloads.FLUX_FULL)
    _err(dit.workspace_size, cfg, dit.Batch([0], [4], [1]))
    assert dit.lib().dit_last_error().decode() != ""
    dit.weight_count(cfg)
    assert dit.lib().dit_last_error().decode() == ""


def test_noalloc_step_rejects_batches_beyond_its_scratch_before_any_launch():
    """dit_step_noalloc's static scratch holds DIT_NOALLOC_SCRATCH_BYTES; a
    batch that needs more (one 1024 px request of the 57-block model) is
    refused on the host, and so is every invalid call dit_step refuses."""
    m = workloads.FLUX_FULL
    cfg = dit.make_config(m)
    n = dit.weight_count(cfg)
    fake = dit.Weights([4096 * (i + 1) for i in range(n)])
    P = 1 << 20
    big = dit.Batch([64], [64], [512], [0.5])
    assert dit.workspace_size(cfg, big) > dit.DIT_NOALLOC_SCRATCH_BYTES
    assert _err(dit.dit_step_noalloc, cfg, fake, big, P, P, P, 0) == dit.DIT_ERR_WORKSPACE
    assert "static scratch" in dit.lib().dit_last_error().decode()
    small = dit.Batch([16], [16], [512], [0.5])
    assert dit.workspace_size(cfg, small) <= dit.DIT_NOALLOC_SCRATCH_BYTES
    assert dit.workspace_size(cfg, dit.Batch([32], [32], [512], [0.5])) <= dit.DIT_NOALLOC_SCRATCH_BYTES
    assert _err(dit.dit_step_noalloc, cfg, fake, dit.Batch([16], [16], [512]), P, P, P, 0) == \
        dit.DIT_ERR_INVALID_ARG
    assert _err(dit.dit_step_noalloc, cfg, fake, small, 0, P, P, 0) == dit.DIT_ERR_INVALID_ARG
    assert _err(dit.dit_step_noalloc, cfg, dit.Weights([4096] * (n - 1)), small, P, P, P, 0) == \
        dit.DIT_ERR_INVALID_ARG
