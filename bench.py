"""Throughput of one DiT denoising step on one MI355X.

A step is the whole hot path over one batch of synthetic input: timestep
embedding and all adaLN modulation vectors, the input embedders, 19
double-stream and 38 single-stream blocks (adaLN LayerNorm, QKV + 2-D RoPE,
joint attention, gated MLP, gated residuals), the final layer and the
flow-matching Euler update -- dit_step followed by euler_update.

Default workload: the 1024 px request (4096 image + 512 text tokens) of the
FLUX.1-dev-shaped model, bf16 weights with fp32 accumulation; `value` is its
steps/s.  The 256, 512 and 2048 px requests of the same model are timed too
(per_workload).  Weights and inputs are seeded random values drawn on the GPU
(no trained checkpoint).  Prints one JSON line on stdout; progress goes to
stderr.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--extra A,B]
"""
from __future__ import annotations

import argparse
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DiT denoising steps/sec per resolution; attention+GEMM TFLOP/s and % bf16 peak"
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
F32_PEAK_TFLOPS = 157.3
HBM_PEAK_GBS = 8000.0


def log(msg: str) -> None:
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def make_model(torch, dit, synth, m, seed, dev):
    cfg = dit.make_config(m)
    shapes = dit.weight_manifest(cfg)
    dt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
    tensors = [synth.device_normal(seed, "w:" + n, s, synth.WEIGHT_STD, dt, dev) for n, s in shapes]
    return cfg, dit.Weights(tensors)


def run_workload(torch, dit, synth, workloads, wl, cfg, w, steps, warmup, seed, dev, profile=True):
    m = wl.model
    dt_t = torch.bfloat16 if m.dtype == "bf16" else torch.float32
    grids = wl.grids()
    n_img = wl.n_img()
    import numpy as np
    if wl.t is None:
        ts = [float(x) for x in synth.uniform(seed, "timesteps:" + wl.name, (len(grids),))]
    else:
        ts = list(wl.t)
    b = dit.Batch(grids, grids, wl.n_txt, ts)
    nws = dit.workspace_size(cfg, b)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    lat = synth.device_normal(seed, "latents:" + wl.name, (sum(n_img), m.in_channels), 1.0, dt_t, dev)
    txt = synth.device_normal(seed, "text:" + wl.name, (sum(wl.n_txt), m.text_dim), 1.0, dt_t, dev)
    vel = torch.empty_like(lat)
    dts = [wl.dt] * len(grids)
    stream = torch.cuda.current_stream()
    dtype = dit.DIT_BF16 if m.dtype == "bf16" else dit.DIT_F32

    def step():
        dit.dit_step(cfg, w, b, lat, txt, vel, ws, nws, stream)
        dit.euler_update(b, m.in_channels, dtype, lat, vel, dts, stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    assert torch.isfinite(vel.float()).all().item(), "non-finite velocity"
    kernels = None
    if profile:
        dit.profile_start()
        for _ in range(max(1, min(steps, 3))):
            step()
        torch.cuda.synchronize()
        kernels = dit.profile_stop()
        nprof = max(1, min(steps, 3))
        for k in kernels.values():
            k["launches"] //= 1
            k["ms_per_step"] = k["ms"] / nprof
    flops = workloads.flops_per_step(m, wl.n_txt, n_img)
    ms = wall * 1000.0 / steps
    res = {
        "steps_per_s": steps / wall, "ms_per_step": ms, "ms_median_event": statistics.median(per),
        "cv_pct": 100.0 * statistics.pstdev(per) / statistics.mean(per),
        "tflop_per_step": flops["total"] / 1e12, "tflops": flops["total"] / (ms / 1e3) / 1e12,
        "gemm_tflop": flops["gemm"] / 1e12, "attention_tflop": flops["attention"] / 1e12,
        "kernels": kernels,
    }
    peak = BF16_PEAK_TFLOPS if m.dtype == "bf16" else F32_PEAK_TFLOPS
    res["frac_peak"] = res["tflops"] / peak
    del ws, lat, txt, vel
    return res


KERNEL_SOURCES = {
    "gemm_bf16": ["gemm_bf16.hip", "device_common.h", "dit_internal.h"],
    "attention_bf16": ["attention.hip", "device_common.h", "dit_internal.h"],
    "ln_modulate": ["elementwise.hip", "device_common.h", "dit_internal.h"],
    "gemv": ["elementwise.hip", "device_common.h", "dit_internal.h"],
}


def kernel_source_hash(family: str) -> str:
    """Hash of the sources a kernel family is built from (stale-counter check)."""
    import hashlib
    key = next((k for k in KERNEL_SOURCES if family.startswith(k)), None)
    if key is None:
        return ""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[key]:
        with open(os.path.join(ROOT, "paper_2510_01565_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(family: str, workload: str):
    """HBM bytes per launch from the committed counter summary
    profiles/hbm_traffic.txt (FETCH_SIZE and WRITE_SIZE passes, each scaled by
    the same counter's reading for a plain copy of known size), or None when
    no summary exists for this kernel, workload and kernel source.  The
    counters see kernels, not K splits: a family "<tile>_k<n>" takes the
    reading of its tile configuration's kernel, which is averaged over all of
    that kernel's launches in the workload, split or not."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    want = kernel_source_hash(family)
    family = re.sub(r"_k\d+$", "", family)
    for line in open(path):
        f = line.split()
        if len(f) >= 4 and not line.startswith("#") and f[0] == family and f[1] == workload and f[2] == want:
            return float(f[3])
    return None


def run_sp_share(torch, dit, synth, workloads, wl, cfg, w, steps, seed, dev):
    """One GPU's share of a k-way (Ulysses) sequence-parallel step at real shape:
    every non-attention kernel of a step on the rank's token shard (L/k tokens:
    n_txt/k text + grid^2/k image), plus one attention per block over all L
    tokens for n_heads/k heads -- the all-to-alls between them are not part of
    a one-GPU measurement.  Both parts are HIP-event-timed loops: the shard's
    whole step (dit_step + euler_update) minus the attention it runs on its own
    tokens (taken from one profiled step), and the block count of dit_attention
    calls on the rank's heads (each with the V transpose a rank would need)."""
    k = wl.extra.get("sp", 4)
    m = wl.model
    g = wl.grids()[0]
    shard_grid = (g // k, g) if g % k == 0 else (g, g)
    n_txt_shard = wl.n_txt[0] // k
    b = dit.Batch([shard_grid[0]], [shard_grid[1]], [n_txt_shard], [0.5])
    nws = dit.workspace_size(cfg, b)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    lat = synth.device_normal(seed, "latents:share", (shard_grid[0] * shard_grid[1], m.in_channels), 1.0, torch.bfloat16, dev)
    txt = synth.device_normal(seed, "text:share", (n_txt_shard, m.text_dim), 1.0, torch.bfloat16, dev)
    vel = torch.empty_like(lat)
    stream = torch.cuda.current_stream()

    def shard_step():
        dit.dit_step(cfg, w, b, lat, txt, vel, ws, nws, stream)
        dit.euler_update(b, m.in_channels, dit.DIT_BF16, lat, vel, [wl.dt], stream)

    def timed_loop(fn, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    for _ in range(3):
        shard_step()
    shard_ms = timed_loop(shard_step, steps)
    dit.profile_start()
    shard_step()
    torch.cuda.synchronize()
    kern = dit.profile_stop()
    shard_attn_ms = sum(v["ms"] for n, v in kern.items() if n.startswith("attention"))
    non_attn_ms = shard_ms - shard_attn_ms
    # attention of the rank's heads over the whole sequence, once per block
    heads = m.heads // k
    L = wl.n_txt[0] + g * g
    ab = dit.Batch([g], [g], [wl.n_txt[0]])
    q = synth.device_normal(seed, "share.q", (L, heads, m.head_dim), 1.0, torch.bfloat16, dev)
    kk = synth.device_normal(seed, "share.k", (L, heads, m.head_dim), 1.0, torch.bfloat16, dev)
    v = synth.device_normal(seed, "share.v", (L, heads, m.head_dim), 1.0, torch.bfloat16, dev)
    o = torch.empty_like(q)
    anws = dit.attention_workspace_size(ab, heads, m.head_dim, dit.DIT_BF16)
    aws = torch.empty(anws, dtype=torch.uint8, device=dev)
    nblk = m.n_double + m.n_single

    def attn_blocks():
        for _ in range(nblk):
            dit.dit_attention(ab, heads, m.head_dim, dit.DIT_BF16, q, kk, v, o, aws, anws, stream)

    attn_blocks()
    attn_ms = timed_loop(attn_blocks, max(1, steps // 2))
    share_ms = non_attn_ms + attn_ms
    fl = workloads.flops_per_step(m, [n_txt_shard], [shard_grid[0] * shard_grid[1]])
    attn_flops = nblk * 4.0 * L * L * m.head_dim * heads
    total = fl["gemm"] + attn_flops
    return {"steps_per_s": 1e3 / share_ms, "ms_per_step": share_ms, "non_attention_ms": non_attn_ms,
            "attention_ms": attn_ms, "shard_step_ms": shard_ms, "shard_step_attention_ms": shard_attn_ms,
            "tflop_per_step": total / 1e12, "tflops": total / (share_ms / 1e3) / 1e12,
            "frac_peak": total / (share_ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS,
            "note": f"composed from HIP-event-timed loops: the {L // k}-token shard's step minus its own attention "
                    f"(profiled), plus {nblk} dit_attention calls of {heads} heads over {L} tokens (V transpose "
                    f"included); all-to-alls excluded"}


def block_flops(m, n_txt, n_img) -> dict:
    """Algorithmic FLOPs of one double-stream block: its GEMMs (QKV, output
    projection, MLP up and down on every token), its modulation GEMV from the
    conditioning vector, and attention inside each request."""
    H, F = m.hidden, m.mlp_ratio * m.hidden
    T = sum(n_txt) + sum(n_img)
    streams = 1 if m.tie_streams else 2
    g = 2.0 * T * H * (3 * H + H + F + F) + 2.0 * len(n_img) * streams * 6 * H * H
    a = sum(4.0 * (lt + li) ** 2 * m.head_dim * m.heads for lt, li in zip(n_txt, n_img))
    return {"gemm": g, "attention": a, "total": g + a}


def run_block(torch, dit, synth, wl, cfg, w, steps, seed, dev):
    """One double-stream block through dit_block_forward (fp32 residual in
    place, bf16 weights), timed with HIP events on the launch stream."""
    m = wl.model
    grids = wl.grids()
    n_img = wl.n_img()
    b = dit.Batch(grids, grids, wl.n_txt, [0.5] * len(grids))
    nws = dit.workspace_size(cfg, b)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    hidden = synth.device_normal(seed, "hidden:" + wl.name, (sum(wl.n_txt) + sum(n_img), m.hidden), 1.0,
                                 torch.float32, dev)
    cond = synth.device_normal(seed, "cond:" + wl.name, (len(grids), m.hidden), 1.0, torch.float32, dev)
    stream = torch.cuda.current_stream()
    for _ in range(2):
        dit.dit_block_forward(cfg, w, 0, 0, b, hidden, cond, ws, nws, stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        dit.dit_block_forward(cfg, w, 0, 0, b, hidden, cond, ws, nws, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    assert torch.isfinite(hidden).all().item(), "non-finite block output"
    ms = e0.elapsed_time(e1) / steps
    f = block_flops(m, wl.n_txt, n_img)
    tf = f["total"] / (ms / 1e3) / 1e12
    del ws, hidden, cond
    return {"ms_per_block": ms, "gflop_per_block": f["total"] / 1e9, "tflops": tf,
            "frac_peak": tf / (BF16_PEAK_TFLOPS if m.dtype == "bf16" else F32_PEAK_TFLOPS)}


def scheduler_latency(seed: int):
    """Decision latency of the round scheduler (host C++): one ts_round_schedule
    call over R pending requests of the paper's resolution mix on N = 8 GPUs,
    their allocations from ts_allocate with the MI355X cost model, timed
    around the C call alone (arguments marshalled once)."""
    import ctypes
    import random
    from paper_2510_01565_amd import cost_model, sched
    rng = random.Random(seed)
    out = {}
    for n_req in (16, 64, 256):
        reqs = []
        for _ in range(n_req):
            res = rng.choice([256, 512, 1024, 2048])
            row = cost_model.row(res)
            steps = rng.randint(1, 28)
            deadline = rng.randint(steps * row[0] // 4, steps * row[0] * 2)
            _, alloc, _, _ = sched.allocate(row, 8, steps, deadline)
            reqs.append(sched.Request(deadline, row, alloc))
        arr = sched._requests(reqs)
        dec = (sched.ts_decision * n_req)()
        sv, used = ctypes.c_int32(), ctypes.c_int32()
        L = sched.lib()
        tau = 5 * cost_model.step_us(1024, 1)
        reps = 200
        t0 = time.perf_counter()
        for _ in range(reps):
            L.ts_round_schedule(arr, n_req, 8, tau, 0, dec, ctypes.byref(sv), ctypes.byref(used))
        out[str(n_req)] = round((time.perf_counter() - t0) / reps * 1e6, 2)
    row = cost_model.row(2048)
    t0 = time.perf_counter()
    for _ in range(200):
        sched.allocate(row, 8, 28, 28 * row[0] // 3)
    return {"round_schedule_us_by_requests": out, "n_gpus": 8,
            "allocate_us_28_steps": round((time.perf_counter() - t0) / 200 * 1e6, 2)}


def kernel_of(family: str) -> str:
    """Kernel a profiler family belongs to: the bf16 GEMM's tile configurations
    and K splits ("gemm_bf16_256x256", "gemm_bf16_128x256_k3", ...) are launch
    parameters of one kernel, "gemm_bf16"; other families are their own kernel."""
    return "gemm_bf16" if family.startswith("gemm_bf16_") else family


def roofline(kernels, dtype: str, workload: str):
    """Dominant kernel by time: algorithmic work per launch over its average
    launch duration (HIP events on the launch stream), with the measured HBM
    bytes per launch when every family of the kernel has a current counter
    summary."""
    agg = {}
    for n, v in kernels.items():
        if n.startswith("detail:"):
            continue
        a = agg.setdefault(kernel_of(n), {"ms": 0.0, "launches": 0, "flops": 0.0, "bytes": 0.0, "families": {}})
        for f in ("ms", "launches", "flops", "bytes"):
            a[f] += v[f]
        a["families"][n] = v["launches"]
    name, k = max(agg.items(), key=lambda kv: kv[1]["ms"])
    avg_ms = k["ms"] / k["launches"]
    per_family = {f: measured_traffic(f, workload) for f in k["families"]}
    traffic = None
    if all(t is not None for t in per_family.values()):
        traffic = sum(per_family[f] * n for f, n in k["families"].items()) / k["launches"]
    common = {"kernel": name, "families": {f: n for f, n in k["families"].items()}, "traffic": traffic,
              "avg_launch_ms": avg_ms, "algorithmic_bytes_per_launch": k["bytes"] / k["launches"],
              "launches": k["launches"]}
    if k["flops"] > 0:
        peak = BF16_PEAK_TFLOPS if dtype == "bf16" else F32_PEAK_TFLOPS
        ach = k["flops"] / k["launches"] / (avg_ms / 1e3) / 1e12
        return {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s", "frac": ach / peak,
                "flop_per_launch": k["flops"] / k["launches"], **common}
    ach = k["bytes"] / k["launches"] / (avg_ms / 1e3) / 1e9
    return {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS,
            **common}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(wl, seed: int):
    """The oracle (fp64, as it stands) on a bounded sample of the workload:
    one double-stream and one single-stream block at the workload's token
    counts, extrapolated to the model's block counts."""
    import numpy as np
    import oracle as O
    from paper_2510_01565_amd import synth
    m = wl.model
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads") or 0) for i in threadpool_info()) or None
    except Exception:
        pass
    cfg1 = O.OracleConfig(hidden=m.hidden, heads=m.heads, head_dim=m.head_dim, mlp_ratio=m.mlp_ratio, n_double=1,
                          n_single=1, in_channels=m.in_channels, text_dim=m.text_dim)
    shapes = [(n, s) for n, s in O.param_shapes(cfg1) if n.startswith(("double.", "single.", "mod."))]
    params = synth.make_params(shapes, seed, bf16=True)
    H = m.hidden
    gh = wl.grids()[0]
    nt = wl.n_txt[0]
    xt = synth.normal(seed, "cpu.txt", (nt, H), bf16=True).astype(np.float64)
    xi = synth.normal(seed, "cpu.img", (gh * gh, H), bf16=True).astype(np.float64)
    c = synth.normal(seed, "cpu.c", (H,)).astype(np.float64)
    p64 = {k: v.astype(np.float64) for k, v in params.items()}
    t0 = time.perf_counter()
    yt, yi = O.double_block(p64, cfg1, 0, xt, xi, c, (gh, gh))
    t_d = time.perf_counter() - t0
    x = np.concatenate([yt, yi])
    t0 = time.perf_counter()
    O.single_block(p64, cfg1, 0, x, nt, c, (gh, gh))
    t_s = time.perf_counter() - t0
    t_step = m.n_double * t_d + m.n_single * t_s
    return {"value": 1.0 / t_step, "unit": "steps/s", "cores": threads or os.cpu_count(), "kind": "oracle",
            "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"oracle (numpy fp64) on one double-stream ({t_d:.2f} s) and one single-stream block "
                      f"({t_s:.2f} s) at {nt} text + {gh * gh} image tokens, extrapolated to "
                      f"{m.n_double} + {m.n_single} blocks ({t_step:.1f} s per step)",
            "s_per_step": t_step}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="dit57_1024px_bf16")
    ap.add_argument("--extra", default="dit57_256px_bf16,dit57_512px_bf16,dit57_2048px_bf16,"
                                       "dit57_2048px_sp4_share_bf16,dit57_packed_mixed_bf16,sd3m_1024px_bf16,"
                                       "sd3m_512px_bf16,mmdit_double_512px_bf16,small_block_256px_f32",
                    help="comma-separated further workloads reported under per_workload (default: the other "
                         "resolutions of the paper's mix, one GPU's share of the 4-way 2048 px split, the packed "
                         "mixed-resolution batch, the SD3-Medium-shaped model at 1024 and 512 px, one double "
                         "block and the small fp32 block; '' for none)")
    ap.add_argument("--extra-steps", type=int, default=20,
                    help="timed steps of each further workload (after --extra-warmup untimed ones)")
    ap.add_argument("--extra-warmup", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy-gib", type=float, default=0.0,
                    help="first copy this many GiB device-to-device once (reference dispatch for HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported by this build "
              "(the step is measured on one GPU's share, see the design notes on sharding)", file=sys.stderr)
        return 2

    import torch
    from paper_2510_01565_amd import dit, synth, workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dit.lib()
    if args.calibrate_copy_gib > 0:
        n = int(args.calibrate_copy_gib * 2 ** 30) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {n * 4} bytes read, {n * 4} bytes written")
        del src, dst
    wl = workloads.WORKLOADS[args.workload]
    log(f"workload {wl.name}: {wl.note}")
    t0 = time.perf_counter()
    cfg, w = make_model(torch, dit, synth, wl.model, args.seed, dev)
    torch.cuda.synchronize()
    log(f"weights drawn on the GPU in {time.perf_counter() - t0:.1f} s")
    main_res = run_workload(torch, dit, synth, workloads, wl, cfg, w, args.steps, args.warmup, args.seed, dev)
    log(f"{wl.name}: {main_res['ms_per_step']:.2f} ms/step, {main_res['tflops']:.1f} TFLOP/s "
        f"({100 * main_res['frac_peak']:.1f}% of peak), CV {main_res['cv_pct']:.2f}%")
    per = {wl.name: {k: v for k, v in main_res.items() if k != "kernels"}}
    per[wl.name]["steps"], per[wl.name]["warmup"] = args.steps, args.warmup
    models = {wl.model: (cfg, w)}
    for name in [x for x in args.extra.split(",") if x]:
        ow = workloads.WORKLOADS[name]
        if ow.model not in models:
            # another model shape (e.g. the SD3-Medium one): its own seeded weights
            models[ow.model] = make_model(torch, dit, synth, ow.model, args.seed, dev)
        cfg, w = models[ow.model]
        if ow.kind == "attention_share":
            r = run_sp_share(torch, dit, synth, workloads, ow, cfg, w, args.extra_steps, args.seed, dev)
            log(f"{name}: {r['ms_per_step']:.2f} ms per share step, {r['tflops']:.1f} TFLOP/s ({r['note']})")
            per[name] = r
            continue
        if ow.kind == "double_block":
            r = run_block(torch, dit, synth, ow, cfg, w, max(args.extra_steps, 10), args.seed, dev)
            log(f"{name}: {r['ms_per_block'] * 1e3:.1f} us per block, {r['tflops']:.1f} TFLOP/s "
                f"({100 * r['frac_peak']:.1f}% of peak)")
            per[name] = r
            continue
        if ow.kind != "step":
            continue
        r = run_workload(torch, dit, synth, workloads, ow, cfg, w, args.extra_steps, args.extra_warmup, args.seed,
                         dev, profile=True)
        r["steps"], r["warmup"] = args.extra_steps, args.extra_warmup
        r["roofline"] = roofline(r["kernels"], ow.model.dtype, ow.name)
        r["roofline"]["step_frac_of_peak"] = r["frac_peak"]
        log(f"{name}: {r['ms_per_step']:.2f} ms/step, {r['tflops']:.1f} TFLOP/s ({100 * r['frac_peak']:.1f}% of peak), "
            f"CV {r['cv_pct']:.2f}%; dominant kernel {r['roofline']['kernel']} at "
            f"{100 * r['roofline']['frac']:.1f}% of its roofline")
        per[name] = {k: v for k, v in r.items() if k != "kernels"}

    rl = roofline(main_res["kernels"], wl.model.dtype, wl.name)
    # the whole step's share of the peak beside the dominant kernel's
    rl["step_frac_of_peak"] = main_res["frac_peak"]
    per[wl.name]["roofline"] = rl
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(wl, args.seed)
        log(f"cpu baseline: {cpu['sample']}")
    sched_lat = None
    try:
        sched_lat = scheduler_latency(args.seed)
        log(f"scheduler decision latency (us) by pending requests: {sched_lat['round_schedule_us_by_requests']}")
    except (OSError, RuntimeError) as e:  # scheduler library not built
        log(f"scheduler latency not measured: {e}")
    g = wl.grids()
    out = {
        "metric": METRIC, "value": main_res["steps_per_s"], "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": main_res["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.model.dtype, "data": "synthetic (seeded random weights and inputs)",
        "config": {"workload": wl.name, "resolution_px": wl.resolutions, "image_tokens": wl.n_img(),
                   "text_tokens": wl.n_txt, "requests": len(g), "parallelism": "single GPU"},
        "tflops": main_res["tflops"], "frac_bf16_peak": main_res["frac_peak"],
        "tflop_per_step": main_res["tflop_per_step"], "cv_pct": main_res["cv_pct"],
        "ms_median_event": main_res["ms_median_event"],
        "roofline": rl, "cpu_baseline": cpu,
        "steps_per_s_by_resolution": {str(workloads.WORKLOADS[n].resolutions[0]): round(r["steps_per_s"], 3)
                                      for n, r in per.items()
                                      if workloads.WORKLOADS[n].model == wl.model and workloads.WORKLOADS[n].kind == "step"
                                      and len(workloads.WORKLOADS[n].resolutions) == 1},
        "per_workload": per, "scheduler": sched_lat,
        "kernels_ms_per_step": {k: round(v["ms_per_step"], 4) for k, v in main_res["kernels"].items()
                                if not k.startswith("detail:")},
        "kernels": {k: {"launches_per_step": v["launches"] // max(1, min(args.steps, 3)), "avg_launch_ms": v["ms"] / v["launches"],
                        "tflops": v["flops"] / (v["ms"] / 1e3) / 1e12, "gbs": v["bytes"] / (v["ms"] / 1e3) / 1e9}
                    for k, v in main_res["kernels"].items() if not k.startswith("detail:")},
        "gemm_shapes": {k[7:]: {"ms_per_step": round(v["ms_per_step"], 4), "tflops": round(v["flops"] / (v["ms"] / 1e3) / 1e12, 1)}
                        for k, v in main_res["kernels"].items() if k.startswith("detail:")},
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
