"""Python binding of the round scheduler's C ABI (``include/tetri_sched.h``).

ctypes marshalling only: the decisions are made by ``libtetri_sched.so``
(host C++, built by ``build.py``).  The first call loads the library and
fails loudly when it has not been built.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtetri_sched.so")

TS_OK, TS_ERR_INVALID_ARG, TS_INFEASIBLE = 0, 1, 2
TS_MAX_DEGREES = 8
TS_MAX_ALLOCS = 8
TS_MAX_STEPS = 256
TS_MAX_GPUS = 4096

EXPORTED = ("ts_allocate", "ts_round_schedule", "ts_select_batch")


class ts_alloc(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int32), ("gpus", ctypes.c_int32)]


class ts_request(ctypes.Structure):
    _fields_ = [("deadline_us", ctypes.c_int64), ("step_us", ctypes.c_int64 * TS_MAX_DEGREES),
                ("n_allocs", ctypes.c_int32), ("allocs", ts_alloc * TS_MAX_ALLOCS)]


class ts_decision(ctypes.Structure):
    _fields_ = [("option", ctypes.c_int32), ("gpus", ctypes.c_int32), ("steps", ctypes.c_int32),
                ("survives", ctypes.c_int32), ("best_effort", ctypes.c_int32)]


class SchedError(RuntimeError):
    pass


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"scheduler library not built: {LIB_PATH} is missing (run paper_2510_01565_amd/build.py)")
        L = ctypes.CDLL(LIB_PATH)
        i32p, i64p = ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64)
        L.ts_allocate.argtypes = [i64p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                  ctypes.POINTER(ts_alloc), i32p, i64p, i64p]
        L.ts_allocate.restype = ctypes.c_int
        L.ts_round_schedule.argtypes = [ctypes.POINTER(ts_request), ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                        ctypes.c_int64, ctypes.POINTER(ts_decision), i32p, i32p]
        L.ts_round_schedule.restype = ctypes.c_int
        L.ts_select_batch.argtypes = [ctypes.POINTER(ts_request), ctypes.c_int32, i64p, ctypes.c_int32, ctypes.c_int64,
                                      ctypes.c_int64, i32p, i32p]
        L.ts_select_batch.restype = ctypes.c_int
        _lib = L
    return _lib


def _row(step_us: Sequence[int]):
    if len(step_us) > TS_MAX_DEGREES:
        raise SchedError(f"at most {TS_MAX_DEGREES} degrees")
    row = (ctypes.c_int64 * TS_MAX_DEGREES)()
    for j, t in enumerate(step_us):
        row[j] = int(t)
    return row


def allocate(step_us: Sequence[int], max_gpus: int, steps: int, budget_us: int):
    """ts_allocate: returns (feasible, [(steps, gpus), ...], gpu_time_us, time_us)."""
    row = _row(step_us)
    out = (ts_alloc * TS_MAX_ALLOCS)()
    n = ctypes.c_int32()
    gt, tt = ctypes.c_int64(), ctypes.c_int64()
    st = lib().ts_allocate(row, len(step_us), max_gpus, steps, int(budget_us), out, ctypes.byref(n), ctypes.byref(gt),
                           ctypes.byref(tt))
    if st == TS_ERR_INVALID_ARG:
        raise SchedError("ts_allocate: invalid argument")
    return st == TS_OK, [(out[i].steps, out[i].gpus) for i in range(n.value)], gt.value, tt.value


@dataclass
class Request:
    deadline_us: int
    step_us: List[int]
    allocs: List[Tuple[int, int]]


def _requests(reqs: Sequence[Request]):
    arr = (ts_request * max(1, len(reqs)))()
    for i, r in enumerate(reqs):
        if len(r.allocs) > TS_MAX_ALLOCS:
            raise SchedError(f"at most {TS_MAX_ALLOCS} allocations per request")
        arr[i].deadline_us = int(r.deadline_us)
        arr[i].step_us = _row(r.step_us)
        arr[i].n_allocs = len(r.allocs)
        for m, (s, g) in enumerate(r.allocs):
            arr[i].allocs[m] = ts_alloc(s, g)
    return arr


def select_batch(reqs: Sequence[Request], batch_us: Sequence[int], round_us: int, now_us: int):
    """ts_select_batch: batch_us[b] for b = 0 .. max_b (entry 0 unused); returns
    (b, members in deadline order)."""
    arr = _requests(reqs)
    bt = (ctypes.c_int64 * len(batch_us))(*[int(x) for x in batch_us])
    members = (ctypes.c_int32 * max(1, len(reqs)))()
    b = ctypes.c_int32()
    st = lib().ts_select_batch(arr, len(reqs), bt, len(batch_us) - 1, int(round_us), int(now_us), members,
                               ctypes.byref(b))
    if st != TS_OK:
        raise SchedError(f"ts_select_batch: status {st}")
    return b.value, [members[i] for i in range(len(reqs))]


def round_schedule(reqs: Sequence[Request], n_gpus: int, round_us: int, now_us: int):
    """ts_round_schedule: returns ([(option, gpus, steps, survives, best_effort)], survivors, gpus_used)."""
    arr = _requests(reqs)
    out = (ts_decision * max(1, len(reqs)))()
    sv, used = ctypes.c_int32(), ctypes.c_int32()
    st = lib().ts_round_schedule(arr, len(reqs), n_gpus, int(round_us), int(now_us), out, ctypes.byref(sv),
                                 ctypes.byref(used))
    if st != TS_OK:
        raise SchedError(f"ts_round_schedule: status {st}")
    plan = [(out[i].option, out[i].gpus, out[i].steps, out[i].survives, out[i].best_effort) for i in range(len(reqs))]
    return plan, sv.value, used.value
