"""Oracle for TetriServe's round-based step scheduler -- TEST INFRASTRUCTURE ONLY.

Plain, slow, exhaustive versions of the two decisions the scheduler makes at
the start of every round (section 4.2 of the paper):

* deadline-aware GPU allocation (section 4.2.1): for one request, the split
  of its remaining steps over sequence-parallel degrees k in {1, 2, 4, ...}
  that meets the deadline with the least GPU time sum(n_k * k * T(k));
* request packing (section 4.2.2, Algorithm 1): per request at most one
  option (run one of its allocations this round, or none), total width at
  most N GPUs, maximising the number of requests that survive to the next
  round start; requests that cannot survive get at most one GPU, best effort.

Both are written as enumerations of the whole decision space (every
composition of the steps; every combination of options), so they can be
checked against the paper's definitions by eye; the C++ library implements
the dynamic programs.  Times are integers (microseconds), so every comparison
is exact.  Nothing here is imported by the product path.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

NONE = -1


def degrees(step_us: Sequence[int], max_gpus: int) -> List[Tuple[int, int]]:
    """(k, T(k)) for k = 2^j <= max_gpus with a profiled time (T > 0)."""
    out = []
    for j, t in enumerate(step_us):
        k = 1 << j
        if k <= max_gpus and t > 0:
            out.append((k, int(t)))
    return out


def compositions(n: int, parts: int):
    """Every tuple of `parts` non-negative integers summing to n."""
    if parts == 1:
        yield (n,)
        return
    for first in range(n, -1, -1):
        for rest in compositions(n - first, parts - 1):
            yield (first,) + rest


def allocate(step_us: Sequence[int], max_gpus: int, steps: int, budget_us: int):
    """Deadline-aware GPU allocation of one request (section 4.2.1).

    Minimises the GPU time sum_k n_k * k * T(k) over step counts n_k >= 0 with
    sum_k n_k = steps, subject to the time sum_k n_k * T(k) <= budget_us.
    Ties: less total time, then more steps on smaller degrees (lexicographic
    from k = 1).  Returns (feasible, [(steps, k), ...] in increasing k, gpu
    time, time); when no split meets the budget, every step goes to the
    fastest degree (ties: the smaller k) and feasible is False.
    """
    ks = degrees(step_us, max_gpus)
    if not ks:
        raise ValueError("no degree with a profiled step time")
    if steps == 0:
        return True, [], 0, 0
    best = None
    for n in compositions(steps, len(ks)):
        time = sum(c * t for c, (_, t) in zip(n, ks))
        if time > budget_us:
            continue
        cost = sum(c * k * t for c, (k, t) in zip(n, ks))
        key = (cost, time, tuple(-c for c in n))
        if best is None or key < best[0]:
            best = (key, n)
    if best is None:
        k, t = min(ks, key=lambda kt: (kt[1], kt[0]))
        return False, [(steps, k)], steps * k * t, steps * t
    n = best[1]
    alloc = [(c, k) for c, (k, _) in zip(n, ks) if c > 0]
    return True, alloc, best[0][0], best[0][1]


@dataclass
class Request:
    deadline_us: int
    step_us: List[int]                      # T(2^j)
    allocs: List[Tuple[int, int]]           # (s^m, A^m)


@dataclass
class Option:
    m: int          # NONE or allocation index
    width: int      # GPUs
    steps: int      # q^m (0 for none)
    survives: int   # sv_i(o)


def options(req: Request, n_gpus: int, round_us: int, now_us: int) -> List[Option]:
    """The option set O_i of Algorithm 1 with width and survival of each."""
    t_next = now_us + round_us
    t_min = min(t for k, t in degrees(req.step_us, n_gpus))
    def step_time(k):
        j = k.bit_length() - 1
        ok = k > 0 and k == 1 << j and j < len(req.step_us) and req.step_us[j] > 0
        return req.step_us[j] if ok else None
    q = [min(s, round_us // step_time(k)) if step_time(k) else 0 for s, k in req.allocs]
    out = []
    for m in [NONE] + list(range(len(req.allocs))):
        if m != NONE and not (q[m] > 0 and req.allocs[m][1] <= n_gpus):
            continue
        remaining = sum(max(0, s - (q[mm] if mm == m else 0)) for mm, (s, _) in enumerate(req.allocs))
        lb = remaining * t_min
        out.append(Option(m, 0 if m == NONE else req.allocs[m][1], 0 if m == NONE else q[m],
                          int(t_next + lb <= req.deadline_us)))
    return out


def best_survivors(reqs: Sequence[Request], n_gpus: int, round_us: int, now_us: int) -> int:
    """Largest number of surviving requests over every choice of one option
    per request with total width <= n_gpus (exhaustive)."""
    opts = [options(r, n_gpus, round_us, now_us) for r in reqs]
    best = 0
    for combo in itertools.product(*opts):
        if sum(o.width for o in combo) <= n_gpus:
            best = max(best, sum(o.survives for o in combo))
    return best


def check_plan(reqs: Sequence[Request], n_gpus: int, round_us: int, now_us: int,
               plan: Sequence[Tuple[int, int, int, int, int]]) -> Tuple[int, int]:
    """Validates a plan [(option m, width, steps, survives, best_effort)] from
    the library against the definitions; returns (survivors, GPUs used).

    The DP's choice among equally good packings is not unique, so the test
    compares the survivor count with best_survivors() and checks here that
    every decision is one of the request's options (or a one-GPU best-effort
    grant to a request none of whose options survives), and that the widths
    fit in n_gpus."""
    used = surv = 0
    for req, (m, width, steps, sv, be) in zip(reqs, plan):
        opts = options(req, n_gpus, round_us, now_us)
        if be:
            assert all(o.survives == 0 for o in opts), "best effort for a request that can survive"
            assert width == 1 and sv == 0
            t1 = req.step_us[0]
            s_left = sum(s for s, _ in req.allocs)
            assert steps == min(s_left, round_us // t1) and steps > 0
        else:
            match = [o for o in opts if o.m == m]
            assert match, f"option {m} not in O_i"
            o = match[0]
            assert (o.width, o.steps, o.survives) == (width, steps, sv)
        used += width
        surv += sv
    assert used <= n_gpus
    return surv, used


def select_batch(reqs: Sequence[Request], batch_us: Sequence[int], round_us: int, now_us: int):
    """Selective continuous batching (sections 3 and 5): the largest measured
    batch size b whose b earliest-deadline requests each still survive to the
    next round start when batched, whenever they would survive on their own
    (q_b = floor(tau / batch_us[b]) steps against q_1 = floor(tau / batch_us[1])).
    Written as a check of every candidate b.  Returns (b, deadline order)."""
    order = sorted(range(len(reqs)), key=lambda i: (reqs[i].deadline_us, i))
    t_next = now_us + round_us

    def survives(i, q):
        r = reqs[i]
        left = sum(s for s, _ in r.allocs)
        t_min = min(t for t in r.step_us if t > 0)
        return t_next + (left - min(left, q)) * t_min <= r.deadline_us

    q1 = round_us // batch_us[1]
    best = 1 if reqs else 0
    for b in range(2, min(len(batch_us) - 1, len(reqs)) + 1):
        if batch_us[b] <= 0 or round_us // batch_us[b] <= 0:
            continue
        qb = round_us // batch_us[b]
        if all((not survives(i, q1)) or survives(i, qb) for i in order[:b]):
            best = b
    return best, order
