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

The GEMM's main loop issues its MFMAs and fragment reads as asm statements
with LDS waits of its own, which the compiler neither checks nor repairs.  A
second check follows each GEMM kernel through its prologue, its main loop
twice (reads issued at the end of one iteration feed the next) and the rest of
the kernel, retiring LDS reads in issue order at each lgkmcnt wait, and
requires every MFMA's A and B registers to be free of outstanding reads.  A
wait that is one short would only fail now and then on the GPU; here it fails
every time.
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


def _regs(tok):
    """VGPR numbers named by an operand such as v[4:7] or v12"""
    tok = tok.strip().rstrip(",")
    m = re.match(r"^v\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"^v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def mfmas_reading_pending_lds(seq):
    """Instructions of seq (in execution order) that are MFMAs reading, as A or B,
    a register an LDS read still in flight writes; and whether an lgkmcnt wait
    other than 0 was reached with a scalar load in flight (scalar loads return
    out of order, so such a wait counts nothing reliably)."""
    outstanding, smem, bad, mixed = [], 0, [], False
    for t in seq:
        op = t.split()[0]
        if op.startswith("ds_read"):
            outstanding.append(_regs(t.split()[1]))
        elif op.startswith("ds_"):
            outstanding.append(set())
        elif op.startswith("s_load") or op.startswith("s_buffer_load"):
            smem += 1
        elif op == "s_waitcnt":
            m = re.search(r"lgkmcnt\((\d+)\)", t)
            if m:
                k = int(m.group(1))
                if k == 0:
                    smem = 0
                elif smem:
                    mixed = True
                outstanding = outstanding[len(outstanding) - k:] if k < len(outstanding) else outstanding
        elif op.startswith("v_mfma"):
            ops = t[len(op):].split(",")
            if any((_regs(ops[1]) | _regs(ops[2])) & o for o in outstanding):
                bad.append(t)
    return bad, mixed


def main_loop_sequence(klines):
    """A kernel's instructions in execution order through its first loop that
    holds MFMAs: everything up to the loop's back edge, the loop body again,
    then the rest of the kernel."""
    ins = []
    for line in klines:
        t = line.split(";")[0].strip()
        if t and (not t.startswith(".") or re.match(r"^\.LBB\d+_\d+:$", t)):
            ins.append(t)
    labels = {t[:-1]: i for i, t in enumerate(ins) if t.endswith(":")}
    for i, t in enumerate(ins):
        m = re.search(r"s_c?branch\w*\s+(\.LBB\d+_\d+)", t)
        if m and m.group(1) in labels and labels[m.group(1)] < i:
            body = ins[labels[m.group(1)]:i + 1]
            if any(x.startswith("v_mfma") for x in body):
                return ins[:i + 1] + body + ins[i + 1:]
    return None


def _compile(src):
    r = subprocess.run([HIPCC, *FLAGS, os.path.join(CSRC, src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stdout


@pytest.fixture(scope="module")
def listings():
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    srcs = ["attention.hip", "gemm_bf16.hip"]
    with ThreadPoolExecutor(len(srcs)) as ex:
        return dict(zip(srcs, ex.map(_compile, srcs)))


def test_no_lds_access_in_flight_at_block_barriers(listings):
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


def test_gemm_mfma_operands_never_pending_lds_reads(listings):
    lines = listings["gemm_bf16.hip"].splitlines()
    starts = [i for i, line in enumerate(lines) if re.match(r"^_ZN\S*gemm_bf16_kernel\S*:", line)]
    assert len(starts) >= 10
    checked = 0
    for s in starts:
        e = next(j for j in range(s, len(lines)) if "s_endpgm" in lines[j])
        name = lines[s].split(":")[0]
        seq = main_loop_sequence(lines[s:e + 1])
        assert seq is not None, name
        bad, mixed = mfmas_reading_pending_lds(seq)
        assert not bad, f"{name}: MFMAs reading registers of LDS reads in flight: {bad[:4]}"
        assert not mixed, f"{name}: an lgkmcnt wait other than 0 with a scalar load in flight"
        checked += sum(1 for t in seq if t.startswith("v_mfma"))
    assert checked > 1000


def test_lds_wait_checker_flags_a_short_wait():
    loop = ["ds_read_b128 v[0:3], v8", "ds_read_b128 v[4:7], v8 offset:64", "s_waitcnt lgkmcnt(1)",
            "v_mfma_f32_16x16x32_bf16 v[10:13], v[0:3], v[4:7], v[10:13]"]
    assert mfmas_reading_pending_lds(loop)[0] == [loop[3]]          # B still in flight
    ok = loop[:2] + ["s_waitcnt lgkmcnt(0)", loop[3]]
    assert mfmas_reading_pending_lds(ok) == ([], False)
    # a read issued after the wait into a register the MFMA reads is in flight too
    late = ["s_waitcnt lgkmcnt(0)", "ds_read_b128 v[0:3], v8", loop[3]]
    assert mfmas_reading_pending_lds(late)[0] == [loop[3]]
    mixed = ["s_load_dword s0, s[4:5], 0x0", "ds_read_b128 v[0:3], v8", "s_waitcnt lgkmcnt(1)"]
    assert mfmas_reading_pending_lds(mixed)[1]
    seq = main_loop_sequence(["k:", "ds_read_b128 v[0:3], v8", ".LBB0_1:", "s_waitcnt lgkmcnt(0)",
                              "v_mfma_f32_16x16x32_bf16 v[10:13], v[0:3], v[0:3], v[10:13]",
                              "ds_read_b128 v[0:3], v8", "s_cbranch_scc1 .LBB0_1", "s_endpgm"])
    # the body runs twice: the read at the end of the first pass is waited for at the top of the second
    assert [t for t in seq if t.startswith("v_mfma")] and mfmas_reading_pending_lds(seq) == ([], False)
