"""Block barriers of the tiled kernels never leave LDS accesses in flight.

The bf16 attention and GEMM kernels reuse an LDS stage right after a block
barrier (the next tile's direct-to-LDS loads overwrite it), so every wave
must have received the data of all its LDS reads before it arrives at the
barrier.  The compiler places the s_waitcnt that covers an LDS read just
before the read's first use, which it may schedule after the barrier; the
kernels therefore wait explicitly.  This test compiles the kernel sources
for gfx950 to assembly and checks, for every s_barrier, that no ds_read or
ds_write issued before it (in program order) is still outstanding, i.e. an
s_waitcnt with lgkmcnt(0) lies between them.  Program order is followed
straight through the listing, which is exact for the unrolled tile loops.
"""
import os
import re
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2510_01565_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S", "-o", "-",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def barriers_with_lds_in_flight(asm: str):
    """(kernel, line) of every s_barrier reached with LDS accesses outstanding."""
    bad = []
    kernel, outstanding = None, 0
    for n, line in enumerate(asm.splitlines(), 1):
        t = line.strip()
        m = re.match(r"^([A-Za-z_][\w.]*):", line)
        if m and not t.startswith(".L"):
            kernel, outstanding = m.group(1), 0
            continue
        if t.startswith("ds_read") or t.startswith("ds_write"):
            outstanding += 1
        w = re.match(r"s_waitcnt\s+(.*)", t)
        if w:
            c = re.search(r"lgkmcnt\((\d+)\)", w.group(1))
            if c:
                outstanding = min(outstanding, int(c.group(1)))
        if t == "s_barrier":
            if outstanding:
                bad.append((kernel, n))
            outstanding = 0
    return bad


def _compile(src):
    r = subprocess.run([HIPCC, *FLAGS, os.path.join(CSRC, src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_no_lds_access_in_flight_at_block_barriers():
    srcs = ["attention.hip", "gemm_bf16.hip"]
    with ThreadPoolExecutor(len(srcs)) as ex:
        listings = dict(zip(srcs, ex.map(_compile, srcs)))
    for src, asm in listings.items():
        assert "s_barrier" in asm and "ds_read_b128" in asm, src
        bad = barriers_with_lds_in_flight(asm)
        assert not bad, f"{src}: barriers with LDS reads in flight: {bad[:8]}"


def test_checker_flags_a_read_pending_at_a_barrier():
    ok = "k:\n ds_read_b128 v[0:3], v4\n s_waitcnt lgkmcnt(0)\n s_barrier\n"
    late = "k:\n ds_read_b128 v[0:3], v4\n s_waitcnt vmcnt(0)\n s_barrier\n s_waitcnt lgkmcnt(0)\n"
    partial = "k:\n ds_read_b128 v[0:3], v4\n ds_read_b128 v[4:7], v4\n s_waitcnt lgkmcnt(1)\n s_barrier\n"
    assert barriers_with_lds_in_flight(ok) == []
    assert barriers_with_lds_in_flight(late) == [("k", 4)]
    assert barriers_with_lds_in_flight(partial) == [("k", 5)]
