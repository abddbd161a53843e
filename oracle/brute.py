"""Exhaustive searches on tiny instances (at most 8 tensors).

``min_demand_fetches`` is the minimum number of host-to-device fetches any
demand-paging schedule can achieve on a trace of equal-size, read-only tensors
with room for ``cap`` of them: dynamic programming over every resident set and
every eviction choice.  Belady's farthest-next-use rule (MIN) attains it, which
pins the victim rule of the planner.
"""
from itertools import combinations


def min_demand_fetches(accesses, cap):
    """accesses: list of sets of tensor ids (one per kernel); cap: slots."""
    states = {frozenset(): 0}
    for need in accesses:
        need = frozenset(need)
        if len(need) > cap:
            raise ValueError("kernel needs more slots than the capacity")
        nxt = {}
        for S, cost in states.items():
            c = cost + len(need - S)
            others = sorted(S - need)
            room = cap - len(need)
            for r in range(0, min(room, len(others)) + 1):
                for keep in combinations(others, r):
                    T = need | frozenset(keep)
                    if c < nxt.get(T, 1 << 60):
                        nxt[T] = c
        states = nxt
    return min(states.values())
