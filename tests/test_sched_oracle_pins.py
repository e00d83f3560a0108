"""Pins of the scheduler oracle (oracle/sched_oracle.py) against facts that
do not come from the oracle: hand-worked examples from the definitions of
section 4.2 (tests/golden/sched_hand.txt), closed forms for special cases
(no deadline pressure, the fastest degree only, plain 0/1 knapsack of unit
values) and invariants.  CPU only."""
import os

import pytest

from oracle import sched_oracle as S

GOLD = os.path.join(os.path.dirname(__file__), "golden", "sched_hand.txt")


def _gold():
    alloc, pack = [], []
    with open(GOLD) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            if line.startswith("allocate"):
                v = [int(x) for x in line.split()[1:]]
                # rows here have 3 degrees (T(1), T(2), T(4))
                t, (mg, st, bud), (feas, cost, time), rest = v[:3], v[3:6], v[6:9], v[9:]
                pack_alloc = list(zip(rest[0::2], rest[1::2]))
                alloc.append((t, mg, st, bud, bool(feas), cost, time, pack_alloc))
            elif line.startswith("pack"):
                head, want = line[4:].split("->")
                parts = head.split(";")
                n, tau, now = [int(x) for x in parts[0].split("|")[0].split()[:3]]
                reqs = []
                for i, p in enumerate(parts):
                    toks = p.split("|")
                    lhs = toks[0].split()
                    if i == 0:
                        lhs = lhs[3:]
                    d, t = int(lhs[0]), [int(x) for x in lhs[1:]]
                    al = [int(x) for x in toks[1].split()]
                    reqs.append(S.Request(d, t, list(zip(al[0::2], al[1::2]))))
                pack.append((n, tau, now, reqs, int(want)))
    return alloc, pack


ALLOC, PACK = _gold()


@pytest.mark.parametrize("case", ALLOC)
def test_allocate_hand_examples(case):
    t, mg, st, bud, feas, cost, time, alloc = case
    got = S.allocate(t, mg, st, bud)
    assert got == (feas, alloc, cost, time)


@pytest.mark.parametrize("case", PACK)
def test_packing_hand_examples(case):
    n, tau, now, reqs, want = case
    assert S.best_survivors(reqs, n, tau, now) == want


def test_allocate_without_deadline_pressure_uses_one_gpu():
    # k * T(k) increasing in k (sub-linear speedup): with budget >= S * T(1)
    # every step stays on one GPU
    t = [1000, 600, 400, 300]
    for steps in range(0, 9):
        feas, alloc, cost, time = S.allocate(t, 8, steps, steps * 1000)
        assert feas and cost == steps * 1000 and time == steps * 1000
        assert alloc == ([(steps, 1)] if steps else [])


def test_allocate_at_the_fastest_time_uses_the_fastest_degree():
    t = [1000, 600, 400, 300]
    for steps in range(1, 8):
        feas, alloc, cost, time = S.allocate(t, 8, steps, steps * 300)
        assert feas and alloc == [(steps, 8)] and time == steps * 300 and cost == steps * 8 * 300


def test_allocate_cost_is_monotone_in_budget():
    t = [900, 500, 300, 220]
    for steps in (3, 6):
        prev = None
        for bud in range(steps * 220, steps * 900 + 1, 97):
            feas, _, cost, time = S.allocate(t, 8, steps, bud)
            assert feas and time <= bud
            if prev is not None:
                assert cost <= prev
            prev = cost


def test_packing_reduces_to_unit_knapsack():
    # every request dies unless it runs this round, and runs on w GPUs: the most
    # survivors is the largest number of widths that fit in N (smallest first)
    widths = [1, 2, 2, 4, 1, 8, 2]
    reqs = [S.Request(105, [10, 10, 10, 10], [(1, w)]) for w in widths]  # run: 100 + 0 <= 105; idle: 100 + 10 > 105
    for n in range(1, 12):
        greedy, used = 0, 0
        for w in sorted(widths):
            if used + w <= n:
                used += w
                greedy += 1
        assert S.best_survivors(reqs, n, 100, 0) == greedy


def test_options_follow_the_definitions():
    # q = min(s, floor(tau / T(A))); options with q = 0 or A > N are dropped
    r = S.Request(10_000, [300, 200, 0, 90], [(5, 1), (2, 2), (4, 4), (3, 8)])
    opts = {o.m: o for o in S.options(r, 4, 650, 0)}
    assert set(opts) == {S.NONE, 0, 1}       # k = 4 not profiled; k = 8 > N
    assert opts[0].steps == 2 and opts[1].steps == 2 and opts[0].width == 1 and opts[1].width == 2


def test_select_batch_hand_example():
    # tau = 100 ms, 256 px-like rows: alone 24 ms/step (q_1 = 4), batch of 4 at
    # 54 ms/step (q_4 = 1), batch of 8 at 109 ms/step (q_8 = 0: never chosen).
    # Each request has 10 steps left and T_min = 20 ms.  Survival alone: 100 +
    # (10 - 4) * 20 = 220 ms; in a batch of 4: 100 + 9 * 20 = 280 ms.
    row = [24, 23, 21, 20]
    tight = [S.Request(d, row, [(10, 1)]) for d in (300, 290, 400, 500)]
    # every deadline >= 280: the batch of 4 harms nobody
    assert S.select_batch(tight, [0, 24, 0, 0, 54, 0, 0, 0, 109], 100, 0)[0] == 4
    # a request with deadline 250 survives alone (220) but not in the batch (280)
    tight[0] = S.Request(250, row, [(10, 1)])
    assert S.select_batch(tight, [0, 24, 0, 0, 54, 0, 0, 0, 109], 100, 0)[0] == 1
    # one that cannot survive alone anyway (deadline 200) does not block batching
    tight[0] = S.Request(200, row, [(10, 1)])
    tight[1] = S.Request(300, row, [(10, 1)])
    assert S.select_batch(tight, [0, 24, 0, 0, 54, 0, 0, 0, 109], 100, 0)[0] == 4
