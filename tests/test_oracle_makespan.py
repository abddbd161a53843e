"""The full method's schedule against the exhaustive optimum in the unit-time
model of integrated prefetching and caching (Cao, Felten, Karlin and Li,
SIGMETRICS 1995): kernels take one unit each, fetches F units each over one
link, equal-size read-only tensors in a pool of ``cap`` slots.

The bound asserted here is derived in the design notes (oracle pins): the
full method keeps the replacements of farthest-next-use paging (MIN) and
issues each fetch, in demand order, once the window's previous tensor has
had its last use.  While a kernel waits for a fetch, the first unfinished
fetch in link order can always run, so the link and the kernels are never
idle together: makespan <= K + F * fetches.  MIN's fetch count m is the least
any schedule can make, and any schedule needs at least K units of kernels and
F * m units of link, so makespan <= K + F * m <= 2 * optimum.
"""
import random

import pytest

from oracle import brute
from oracle import planner as op
from workloads.format import DT_U8, KIND_PARAM, OP_TOUCH, VAR_DEMAND_BELADY, VAR_T_A_P

SLOW_LINK = (10 ** 18, 10 ** 18, 1)      # every kernel with a missing operand is CGI-bound


def _plan(acc, n, cap, variant, **kw):
    tensors = [dict(nbytes=256, dtype=DT_U8, kind=KIND_PARAM, host_init=True) for _ in range(n)]
    kernels = [dict(op=OP_TOUCH, shape=(0,), operands=[(t, 1) for t in sorted(a)], flops=1, hbm_bytes=1)
               for a in acc]
    return op.plan(tensors, kernels, cap * 256, roofs=SLOW_LINK, variant=variant, **kw)


def _fetches(r):
    return r.counters["h2d_prefetch_n"] + r.counters["h2d_demand_n"]


@pytest.mark.parametrize("acc,cap,F,want", [
    ([{0}, {1}, {2}], 3, 1, 4),          # fetches land at 1, 2, 3; kernels 1-2, 2-3, 3-4
    ([{0}, {1}, {2}], 3, 2, 7),          # fetches land at 2, 4, 6; the last kernel runs 6-7
    ([{0}, {0}, {0}, {1}], 1, 3, 10),    # 0 lands at 3, kernels 3-6; 1 waits for the slot: 6-9, runs 9-10
    ([{0}, {1}, {0}, {1}], 2, 2, 7),     # 0 at 2, 1 at 4: kernels 2-3, 4-5, 5-6, 6-7
    ([{0}, {1}, {0}], 1, 2, 9),          # one slot: 0-2 | 2-3 | 3-5 | 5-6 | 6-8 | 8-9
    ([{0, 1}, {2}, {0}], 2, 1, 6),       # 0, 1 land at 2; k0 2-3; 2 over 1 at 3-4; k1 4-5; k2 5-6
])
def test_min_makespan_hand_cases(acc, cap, F, want):
    assert brute.min_makespan(acc, cap, F) == want


@pytest.mark.parametrize("seed", range(40))
def test_min_makespan_bounds(seed):
    r = random.Random(seed)
    n = r.randint(2, 7)
    K = r.randint(1, 9)
    cap = r.randint(1, n)
    F = r.randint(1, 4)
    acc = [{r.randrange(n)} for _ in range(K)]
    opt = brute.min_makespan(acc, cap, F)
    m = brute.min_demand_fetches(acc, cap)
    assert opt >= K + F                   # the first kernel waits for one fetch
    assert opt >= F * m + 1               # m fetches on one link, then a kernel
    assert opt <= K * (F + 1)             # fetch before every kernel
    # the demand schedule of farthest-next-use paging is a schedule of the model
    b = _plan(acc, n, cap, VAR_DEMAND_BELADY, affinity_w=0)
    assert opt <= brute.schedule_makespan(b.schedule, acc, F)


def test_schedule_makespan_hand_case():
    # one slot, accesses 0, 1, 0, F = 2: every fetch is a demand fetch after the
    # previous kernel (the slot's previous tensor was just used): 9 units
    acc = [{0}, {1}, {0}]
    r = _plan(acc, 2, 1, VAR_T_A_P, guard=0, bucket=1)
    assert brute.schedule_makespan(r.schedule, acc, 2) == 9


def _ratio_cases(seed, ops):
    r = random.Random(seed)
    n = r.randint(3, 8 if ops == 1 else 6)
    K = r.randint(4, 10 if ops == 1 else 8)
    cap = r.randint(max(1, ops), n - 1)
    F = r.randint(1, 5)
    acc = [set(r.sample(range(n), r.randint(1, ops))) for _ in range(K)]
    return acc, n, cap, F


@pytest.mark.parametrize("ops", [1, 2])
def test_full_method_within_twice_the_optimum(ops):
    ratios = []
    for seed in range(150):
        acc, n, cap, F = _ratio_cases(1000 * ops + seed, ops)
        K = len(acc)
        r = _plan(acc, n, cap, VAR_T_A_P, guard=0, bucket=1)
        mk = brute.schedule_makespan(r.schedule, acc, F)
        opt = brute.min_makespan(acc, cap, F)
        m = brute.min_demand_fetches(acc, cap)
        assert _fetches(r) == m                   # MIN's replacements, no extra fetch
        assert mk <= K + F * m                    # link and kernels never idle together
        assert opt <= mk <= 2 * opt
        d = _plan(acc, n, cap, VAR_DEMAND_BELADY, affinity_w=0)
        assert mk <= brute.schedule_makespan(d.schedule, acc, F)   # moving fetches earlier never hurts
        ratios.append(mk / opt)
    print(f"{ops} operand(s) per kernel: makespan / optimum max {max(ratios):.3f}, "
          f"mean {sum(ratios) / len(ratios):.3f}, optimal in {sum(x == 1 for x in ratios)} of {len(ratios)}")


def test_default_guard_and_bucket_keep_the_idle_bound():
    # with the victim guard and the next-use bucket the demand pass may fetch
    # more than MIN, but the link and the kernels still never idle together
    for seed in range(100):
        acc, n, cap, F = _ratio_cases(5000 + seed, 1)
        r = _plan(acc, n, cap, VAR_T_A_P)
        mk = brute.schedule_makespan(r.schedule, acc, F)
        assert mk <= len(acc) + F * _fetches(r)
        assert mk >= brute.min_makespan(acc, cap, F)


@pytest.mark.parametrize("ops", [1, 2])
def test_full_method_is_the_conservative_timeline(ops):
    """The full method's second pass keeps MIN's replacements and starts every
    fetch as early as its window allows: its makespan equals that of MIN's
    demand schedule timed with every fetch turned into a prefetch (each fetch
    then waits only for the link and for the last use of the tensor it
    replaces), Cao et al.'s conservative strategy."""
    from workloads.format import S_H2D_DEMAND, S_H2D_PREFETCH
    for seed in range(200):
        r = random.Random(7000 + 100 * ops + seed)
        n = r.randint(3, 8)
        K = r.randint(4, 12)
        cap = r.randint(ops, n - 1)
        F = r.randint(1, 5)
        acc = [set(r.sample(range(n), r.randint(1, ops))) for _ in range(K)]
        for W in (0, 1):
            a = _plan(acc, n, cap, VAR_T_A_P, guard=0, bucket=1, affinity_w=W)
            d = _plan(acc, n, cap, VAR_DEMAND_BELADY, affinity_w=0)
            early = [(S_H2D_PREFETCH if e[0] == S_H2D_DEMAND else e[0],) + tuple(e[1:]) for e in d.schedule]
            assert brute.schedule_makespan(a.schedule, acc, F) == brute.schedule_makespan(early, acc, F)
