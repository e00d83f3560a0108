"""Host logic of bench.py (no GPU): the roofline's choice of the dominant
kernel, the aggregation of the GEMM's tile configurations into one kernel, the
traffic lookup, and the --gpus guard."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _k(ms, launches, flops, nbytes):
    return {"ms": ms, "launches": launches, "flops": flops, "bytes": nbytes}


def test_gemm_families_are_one_kernel():
    assert bench.kernel_of("gemm_bf16_256x256") == "gemm_bf16"
    assert bench.kernel_of("gemm_bf16_128x256_k3") == "gemm_bf16"
    assert bench.kernel_of("attention_bf16") == "attention_bf16"
    assert bench.kernel_of("gemv") == "gemv"


def test_roofline_adds_tile_configurations_and_picks_the_dominant_kernel():
    # attention alone (40 ms) beats either GEMM family (30 + 25 ms) but not their sum
    kernels = {
        "gemm_bf16_256x256": _k(30.0, 10, 30e12, 1e9),
        "gemm_bf16_288x192": _k(25.0, 5, 20e12, 5e8),
        "attention_bf16": _k(40.0, 20, 30e12, 1e9),
        "gemv": _k(1.0, 3, 1e10, 6.5e9),
        "detail:gemm_bf16_256x256 M=1 N=1 K=1 store": _k(1e3, 1, 1e15, 1.0),  # never counted
    }
    rl = bench.roofline(kernels, "bf16", "no_such_workload")
    assert rl["kernel"] == "gemm_bf16"
    assert rl["launches"] == 15
    assert rl["families"] == {"gemm_bf16_256x256": 10, "gemm_bf16_288x192": 5}
    assert rl["bound"] == "mfma" and rl["unit"] == "TFLOP/s" and rl["peak"] == bench.BF16_PEAK_TFLOPS
    # 50 TFLOP in 55 ms
    assert rl["achieved"] == pytest.approx(50e12 / 55e-3 / 1e12)
    assert rl["frac"] == pytest.approx(rl["achieved"] / bench.BF16_PEAK_TFLOPS)
    assert rl["avg_launch_ms"] == pytest.approx(55.0 / 15)
    assert rl["traffic"] is None  # no counter summary for this workload


def test_roofline_of_a_bandwidth_kernel():
    rl = bench.roofline({"gemv": _k(2.0, 2, 0.0, 13e9)}, "bf16", "no_such_workload")
    assert rl["bound"] == "hbm" and rl["unit"] == "GB/s"
    assert rl["achieved"] == pytest.approx(6.5e9 / 1e-3 / 1e9)


def test_traffic_lookup_needs_current_sources():
    assert bench.measured_traffic("gemm_bf16_256x256", "no_such_workload") is None
    assert bench.measured_traffic("no_such_family", "dit57_1024px_bf16") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_split_family_takes_its_kernels_traffic(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    h = bench.kernel_source_hash("gemm_bf16_128x128")
    (prof / "hbm_traffic.txt").write_text(f"# header\ngemm_bf16_128x128 wl {h} 1.5e+08 1e+08 5e+07 4\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda fam: h)
    assert bench.measured_traffic("gemm_bf16_128x128_k2", "wl") == pytest.approx(1.5e8)
    assert bench.measured_traffic("gemm_bf16_128x128", "wl") == pytest.approx(1.5e8)
    assert bench.measured_traffic("gemm_bf16_128x256_k2", "wl") is None


def test_double_block_flops_match_the_c2_count():
    # one FLUX double block at 512 text + 1024 image tokens: 347.9 GFLOP of
    # GEMM (2 T H (3H + H + 2F)), 29.0 of attention (4 L^2 d heads), plus the
    # block's modulation GEMV (2 streams x 6H x H)
    from paper_2510_01565_amd import workloads
    m = workloads.FLUX_DOUBLE
    f = bench.block_flops(m, [512], [1024])
    assert f["attention"] == pytest.approx(4.0 * 1536 ** 2 * 128 * 24)
    assert f["gemm"] == pytest.approx(2.0 * 1536 * 3072 * 36864 + 2.0 * 2 * 6 * 3072 * 3072)
    assert f["total"] / 1e9 == pytest.approx(377.1, abs=0.1)
