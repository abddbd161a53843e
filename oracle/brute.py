"""Exhaustive searches on tiny instances (at most 8 tensors).

``min_demand_fetches`` is the minimum number of host-to-device fetches any
demand-paging schedule can achieve on a trace of equal-size, read-only tensors
with room for ``cap`` of them: dynamic programming over every resident set and
every eviction choice.  Belady's farthest-next-use rule (MIN) attains it, which
pins the victim rule of the planner.

``schedule_makespan`` and ``min_makespan`` use the unit-time model of
integrated prefetching and caching (Cao, Felten, Karlin and Li, SIGMETRICS
1995): every kernel runs for one time unit, in trace order; every fetch
occupies the one host link for ``F`` units, one fetch at a time; a fetch into
a slot may start once the kernels that last used the slot's previous tensors
have finished; a kernel starts once the previous kernel has finished and the
fetches that brought its operands have landed.  ``schedule_makespan`` times a
given schedule by these rules, with the executor's extra rule that a demand
fetch for kernel k > 0 starts no earlier than the end of kernel k - 1.
``min_makespan`` searches every schedule: at each kernel boundary any number
of fetches (of any tensor still to be used, into a free slot or over any
resident tensor the next kernel does not read), in link order, then the
launch.
"""
from itertools import combinations

from workloads.format import S_D2H_WRITEBACK, S_DROP, S_H2D_DEMAND, S_H2D_PREFETCH, S_LAUNCH


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


def schedule_makespan(schedule, accesses, F):
    """Finish time of the last kernel of ``schedule`` (planner entries in
    emission order) in the unit-time model, with fetches of F units."""
    end = {}                  # kernel -> finish time
    last_end = {}             # tensor -> finish time of the last kernel that accessed it
    avail = {}                # resident tensor -> time its fetch lands
    hazards = []              # (lo, hi, time) of vacated windows not yet refilled
    link = 0
    for op, t, off, nbytes, issue_k, _ in schedule:
        if op in (S_DROP, S_D2H_WRITEBACK):
            if op == S_D2H_WRITEBACK:
                raise ValueError("the unit-time model has read-only traces")
            hazards.append((off, off + nbytes, last_end.get(t, 0)))
            avail.pop(t, None)
        elif op in (S_H2D_PREFETCH, S_H2D_DEMAND):
            start = link
            keep = []
            for lo, hi, tm in hazards:
                if lo < off + nbytes and off < hi:
                    start = max(start, tm)
                else:
                    keep.append((lo, hi, tm))
            hazards = keep
            if op == S_H2D_DEMAND and issue_k > 0:
                start = max(start, end[issue_k - 1])
            link = start + F
            avail[t] = link
        elif op == S_LAUNCH:
            k = issue_k
            start = max([end.get(k - 1, 0)] + [avail[u] for u in accesses[k]])
            end[k] = start + 1
            for u in accesses[k]:
                last_end[u] = end[k]
        else:
            raise ValueError("the unit-time model has no first-write allocations")
    return end[len(accesses) - 1]


def min_makespan(accesses, cap, F):
    """Least finish time over every schedule of the unit-time model
    (depth-first search with a bound; exact states are visited once)."""
    K = len(accesses)
    A = [frozenset(a) for a in accesses]
    if any(len(a) > cap for a in A):
        raise ValueError("kernel needs more slots than the capacity")
    later = [set().union(*A[b:]) if b < K else set() for b in range(K + 1)]
    best = [1 << 60]
    seen = set()

    def dfs(b, res, link, tprev, nf):
        # res: frozenset of (tensor, landing time, finish time of its last access)
        if b == K:
            best[0] = min(best[0], tprev)
            return
        have = {t: (av, le) for t, av, le in res}
        missing = [t for t in A[b] if t not in have]
        lb = max(tprev, link + F * len(missing)) + (K - b)
        if lb >= best[0]:
            return
        key = (b, res, link, tprev, nf)
        if key in seen:
            return
        seen.add(key)
        if not missing:
            start = max([tprev] + [have[t][0] for t in A[b]])
            fin = start + 1
            dfs(b + 1, frozenset((t, av, fin if t in A[b] else le) for t, (av, le) in have.items()),
                link, fin, 0)
        if nf >= cap:
            return
        for t in sorted(later[b] - set(have)):
            victims = [None] if len(have) < cap else []
            victims += [v for v in sorted(have) if v not in A[b]]
            for v in victims:
                start = max(link, have[v][1] if v is not None else 0)
                land = start + F
                nres = {u: x for u, x in have.items() if u != v}
                nres[t] = (land, 0)
                dfs(b, frozenset((u, av, le) for u, (av, le) in nres.items()), land, tprev, nf + 1)

    dfs(0, frozenset(), 0, 0, 0)
    return best[0]
