"""The round scheduler library (include/tetri_sched.h, host C++) against the
exhaustive oracle (oracle/sched_oracle.py) on seeded random instances small
enough to enumerate, plus edge cases and argument validation.  CPU only: the
scheduler is host code."""
import ctypes
import os
import random
import re

import pytest

from oracle import sched_oracle as O
from paper_2510_01565_amd import sched


def _row(rng, n_deg, zero_some=True):
    """A cost-model row: T(1) in [2, 20] ms and a sub-linear speedup per doubling;
    some degrees left unprofiled (0)."""
    t = [rng.randint(2000, 20000)]
    for j in range(1, n_deg):
        t.append(max(1, int(t[-1] * rng.uniform(0.5, 0.95))))
    if zero_some:
        for j in range(1, n_deg):
            if rng.random() < 0.2:
                t[j] = 0
    return t


def test_library_exports_every_header_function():
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    src = re.sub(r"/\*.*?\*/", "", open(os.path.join(root, "include", "tetri_sched.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"^\s*ts_status\s+(\w+)\s*\(", src, flags=re.M)))
    assert len(names) == 3 and set(names) == set(sched.EXPORTED)
    L = sched.lib()
    for name in names:
        assert hasattr(L, name), name


def test_struct_layout_matches_header():
    # int64 deadline, int64[8], int32 n_allocs, (int32, int32)[8] -> 140 bytes, padded to 8
    assert ctypes.sizeof(sched.ts_request) == 144
    assert ctypes.sizeof(sched.ts_decision) == 20
    assert ctypes.sizeof(sched.ts_alloc) == 8


@pytest.mark.parametrize("seed", range(40))
def test_allocate_matches_oracle(seed):
    rng = random.Random(seed)
    for _ in range(15):
        n_deg = rng.randint(1, 4)
        t = _row(rng, n_deg)
        max_gpus = rng.choice([1, 2, 4, 8])
        if not O.degrees(t, max_gpus):
            continue
        steps = rng.randint(0, 9)
        fastest = min(tt for _, tt in O.degrees(t, max_gpus))
        slowest = max(tt for _, tt in O.degrees(t, max_gpus))
        budget = rng.randint(steps * fastest - 3000, steps * slowest + 3000)
        assert sched.allocate(t, max_gpus, steps, budget) == O.allocate(t, max_gpus, steps, budget)


def _requests(rng, n_req, n_gpus, now, tau):
    reqs = []
    for _ in range(n_req):
        t = _row(rng, 4)
        steps = rng.randint(0, 12)
        fastest = min(tt for _, tt in O.degrees(t, n_gpus))
        deadline = now + rng.randint(-3 * tau, 3 * tau + steps * fastest)
        budget = deadline - now
        _, alloc, _, _ = O.allocate(t, n_gpus, steps, budget)
        if rng.random() < 0.3:  # arbitrary extra allocations, also wider than N
            alloc = alloc + [(rng.randint(0, 5), rng.choice([1, 2, 4, 8, 16]))]
        reqs.append(O.Request(deadline, t, alloc[:8]))
    return reqs


def _check_best_effort(reqs, n_gpus, tau, now, plan):
    used = sum(p[1] for p in plan if not p[4])
    late = [i for i, r in enumerate(reqs) if all(o.survives == 0 for o in O.options(r, n_gpus, tau, now))]
    eligible = [i for i in late if reqs[i].step_us[0] > 0 and min(sum(s for s, _ in reqs[i].allocs),
                                                                  tau // reqs[i].step_us[0]) > 0]
    eligible.sort(key=lambda i: (reqs[i].deadline_us, i))
    want = eligible[:max(0, n_gpus - used)]
    assert [i for i, p in enumerate(plan) if p[4]] == sorted(want)


@pytest.mark.parametrize("seed", range(60))
def test_round_schedule_matches_oracle(seed):
    rng = random.Random(1000 + seed)
    n_gpus = rng.choice([1, 2, 3, 4, 8])
    n_req = rng.randint(0, 6)
    tau = rng.randint(10_000, 100_000)
    now = rng.randint(0, 10**6)
    reqs = _requests(rng, n_req, n_gpus, now, tau)
    plan, surv, used = sched.round_schedule([sched.Request(r.deadline_us, r.step_us, r.allocs) for r in reqs],
                                            n_gpus, tau, now)
    assert surv == O.best_survivors(reqs, n_gpus, tau, now)
    s2, u2 = O.check_plan(reqs, n_gpus, tau, now, plan)
    assert (s2, u2) == (surv, used)
    _check_best_effort(reqs, n_gpus, tau, now, plan)


def test_round_schedule_hand_example():
    # the three-request example of tests/golden/sched_hand.txt with N = 2:
    # R0 survives idle, so the two GPUs go to R1 (2 GPUs) or R2 (1 GPU)
    reqs = [sched.Request(250, [50, 30], [(4, 1)]), sched.Request(150, [50, 30], [(4, 2)]),
            sched.Request(180, [50, 30], [(3, 1)])]
    plan, surv, used = sched.round_schedule(reqs, 2, 100, 0)
    assert surv == 2
    assert plan[0][0] == -1 and plan[0][3] == 1
    # the plan is read back from the smallest capacity reaching 2 survivors:
    # one GPU, running R2; R1 stays idle and, having a surviving option, gets
    # no best-effort grant (the spare GPU is left to elastic scale-up)
    assert plan[2][:4] == (0, 1, 2, 1) and plan[1][:2] == (-1, 0)
    assert plan[1][4] == 0 and used == 1


def test_empty_and_finished():
    plan, surv, used = sched.round_schedule([], 4, 1000, 0)
    assert (plan, surv, used) == ([], 0, 0)
    plan, surv, used = sched.round_schedule([sched.Request(5000, [100], [])], 1, 1000, 0)
    assert plan == [(-1, 0, 0, 1, 0)] and surv == 1


def test_invalid_arguments():
    with pytest.raises(sched.SchedError):
        sched.allocate([0, 0], 4, 3, 100)               # no profiled degree
    with pytest.raises(sched.SchedError):
        sched.allocate([100], 4, sched.TS_MAX_STEPS + 1, 100)
    with pytest.raises(sched.SchedError):
        sched.round_schedule([sched.Request(0, [100], [(1, 1)])], 0, 100, 0)   # N = 0
    with pytest.raises(sched.SchedError):
        sched.round_schedule([sched.Request(0, [100], [(1, 1)])], 2, 0, 0)    # tau = 0
    with pytest.raises(sched.SchedError):
        sched.round_schedule([sched.Request(0, [100], [(-1, 1)])], 2, 10, 0)  # negative steps


def test_decision_latency_is_small():
    # the paper reports under 10 ms per decision; this DP is O(R N)
    import time
    rng = random.Random(7)
    reqs = [sched.Request(r.deadline_us, r.step_us, r.allocs) for r in _requests(rng, 256, 8, 0, 50_000)]
    t0 = time.perf_counter()
    for _ in range(20):
        sched.round_schedule(reqs, 8, 50_000, 0)
    assert (time.perf_counter() - t0) / 20 < 0.01


@pytest.mark.parametrize("seed", range(30))
def test_select_batch_matches_oracle(seed):
    rng = random.Random(5000 + seed)
    tau = rng.randint(50_000, 200_000)
    now = rng.randint(0, 10**6)
    row = _row(rng, 4, zero_some=False)
    t1 = row[0]
    bt = [0, t1] + [int(t1 * b * rng.uniform(0.3, 1.0)) if rng.random() < 0.7 else 0 for b in range(2, 9)]
    n = rng.randint(0, 9)
    reqs = [O.Request(now + rng.randint(0, 6 * tau), row, [(rng.randint(0, 12), 1)]) for _ in range(n)]
    got = sched.select_batch([sched.Request(r.deadline_us, r.step_us, r.allocs) for r in reqs], bt, tau, now)
    assert got == O.select_batch(reqs, bt, tau, now)
