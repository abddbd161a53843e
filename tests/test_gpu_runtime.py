"""GPU tests of the transfer engine and executor: random touch traces under a
device budget must read, at every launch, exactly the version of each tensor
that the trace's order of writes implies (prefetches, write-backs, drops and
pool-window reuse all correct), and the executed log must equal the plan."""
import random

import numpy as np
import pytest

from oracle import planner as op
from workloads.format import DT_U8, KIND_ACT, KIND_PARAM, MODE_R
from workloads.trace import Workload

from gpu_util import touch_expectations
from planner_cases import random_trace

pytestmark = pytest.mark.gpu


def _session_from_trace(tensors, kernels, M, **pol):
    from paper_2609_06172_amd.session import Session
    w = Workload(None)
    for i, t in enumerate(tensors):
        w.tensor(f"t{i}", (t["nbytes"],), t["dtype"], t["kind"], host_init=t["host_init"])
    for k in kernels:
        w.kernel(k["op"], k["shape"], k["operands"])
    s = Session(w, device=0, M=M, fill=False, **pol)
    return s, w


def _init_words(s, w, tensors):
    init = {}
    for i, t in enumerate(tensors):
        if t["host_init"] or t["kind"] == KIND_PARAM:
            v = 1000 + i
            s.host_view(w.tensors[i])[:] = np.full(t["nbytes"] // 4, v, np.uint32).view(np.uint8)
            init[i] = v
    # the log starts at zero
    s.host_view(w.tensors[0])[:] = 0
    return init


def feasible_budget(tensors, kernels, variant, fracs=((1, 2), (2, 3), (3, 4), (5, 6), (1, 1))):
    """Smallest of a few budgets (fractions of the footprint) the trace can run in."""
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    for num, den in fracs:
        M = max(1024, fp * num // den // 256 * 256)
        try:
            op.plan(tensors, kernels, M, variant=variant)
            return M
        except op.PlanError:
            continue
    raise AssertionError("no feasible budget")


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("variant", [0, 1, 2, 3, 4])
def test_touch_traces_read_latest_versions(seed, variant):
    tensors, kernels = random_trace(seed, touch=True, n_kernels=random.Random(seed).randint(20, 120))
    M = feasible_budget(tensors, kernels, variant)
    print(f"touch seed={seed} variant={variant} M={M} kernels={len(kernels)}", flush=True)
    s, w = _session_from_trace(tensors, kernels, M, variant=variant, validate=1)
    init = _init_words(s, w, tensors)
    # run in a few segments
    K = len(kernels)
    cuts = sorted(set([0, K] + [K // 3, 2 * K // 3]))
    for a, b in zip(cuts, cuts[1:]):
        if b > a:
            s.run(a, b - a)
    assert s.ctx.get_executed() == s.ctx.get_schedule()
    log = s.read("t0").view(np.uint32).reshape(-1, 16)
    for slot, i, v in touch_expectations(tensors, kernels, init):
        assert log[slot, 2 * i] == v and log[slot, 2 * i + 1] == v, (slot, i, v, log[slot])
    s.close()


def test_reset_and_rerun_gives_the_same_reads():
    tensors, kernels = random_trace(3, touch=True, n_kernels=60)
    M = feasible_budget(tensors, kernels, 4)
    s, w = _session_from_trace(tensors, kernels, M)
    init = _init_words(s, w, tensors)
    s.run_all()
    first = s.read("t0").copy()
    s.ctx.reset()
    _init_words(s, w, tensors)
    s.run_all()
    assert np.array_equal(first, s.read("t0"))
    s.close()


@pytest.mark.parametrize("seed,variant", [(5, 0), (5, 4), (9, 1), (9, 4)])
def test_timeline_is_complete_ordered_and_causal(seed, variant):
    """Timing policy: one timeline entry per kernel and per executed copy, each
    stream's items in order without overlap (host-to-device copies run on two
    streams), every kernel starting after the copies that brought its
    operands, and demand fetches after the kernel before their need."""
    from paper_2609_06172_amd.capi import TL_D2H, TL_H2D, TL_H2D_B, TL_KERNEL
    from workloads.format import S_ALLOC, S_D2H_WRITEBACK, S_H2D_DEMAND, S_H2D_PREFETCH, S_LAUNCH
    tensors, kernels = random_trace(seed, touch=True, n_kernels=90)
    M = feasible_budget(tensors, kernels, variant)
    print(f"timeline seed={seed} variant={variant} M={M}", flush=True)
    s, w = _session_from_trace(tensors, kernels, M, variant=variant, timing=1)
    _init_words(s, w, tensors)
    K = len(kernels)
    cuts = [0, K // 2, K]
    for a, b in zip(cuts, cuts[1:]):
        s.run(a, b - a)
    tl = s.ctx.get_timeline()
    sched = s.ctx.get_schedule()
    s.close()
    tol = 0.02   # ms
    kern = [e for e in tl if e[0] == TL_KERNEL]
    assert [e[2] for e in kern] == list(range(K))
    assert [e[1] for e in kern] == [0 if k < K // 2 else 1 for k in range(K)]
    for kinds, ops in (((TL_H2D, TL_H2D_B), (S_H2D_PREFETCH, S_H2D_DEMAND)), ((TL_D2H,), (S_D2H_WRITEBACK,))):
        got = sorted((e[2], e[3]) for e in tl if e[0] in kinds)
        want = [(i, tensors[x[1]]["nbytes"]) for i, x in enumerate(sched) if x[0] in ops]
        assert got == want
    # copies alternate between the two host-to-device streams, the first on
    # TL_H2D, unless the plan writes back (then they share one stream)
    h2d_kinds = [e[0] for e in sorted((e for e in tl if e[0] in (TL_H2D, TL_H2D_B)), key=lambda e: e[2])]
    if any(x[0] == S_D2H_WRITEBACK for x in sched):
        assert set(h2d_kinds) <= {TL_H2D}
    else:
        assert all(k == (TL_H2D, TL_H2D_B)[i % 2] for i, k in enumerate(h2d_kinds))
    for kind in (TL_KERNEL, TL_H2D, TL_H2D_B, TL_D2H):
        items = [e for e in tl if e[0] == kind]
        for a, b in zip(items, items[1:]):
            assert b[5] <= b[6] + 1e-6 and a[5] >= -tol
            if a[1] == b[1]:
                assert b[5] >= a[6] - tol and b[4] >= a[4]
    # causality through the schedule
    start = {e[2]: e[5] for e in kern}
    end = {e[2]: e[6] for e in kern}
    seg = {e[2]: e[1] for e in kern}
    copy = {e[2]: e for e in tl if e[0] in (TL_H2D, TL_H2D_B)}
    latest = {}
    for i, x in enumerate(sched):
        if x[0] in (S_H2D_PREFETCH, S_H2D_DEMAND):
            latest[x[1]] = i
            if x[0] == S_H2D_DEMAND and x[4] > 0 and seg[x[4] - 1] == copy[i][1]:
                assert copy[i][5] >= end[x[4] - 1] - tol
        elif x[0] == S_LAUNCH:
            k = x[4]
            for t, _ in kernels[k]["operands"]:
                j = latest.get(t)
                if j is not None and copy[j][1] == seg[k]:
                    assert copy[j][6] <= start[k] + tol, (k, t)
        elif x[0] == S_ALLOC:
            latest.pop(x[1], None)


def test_kernels_overlap_an_unrelated_prefetch():
    """Kernels that do not read a tensor being prefetched run while its copy is
    on the link: the compute and copy streams must not be serialized (as they
    are when two streams share a hardware queue)."""
    from paper_2609_06172_amd.capi import TL_H2D, TL_H2D_B, TL_KERNEL
    from workloads.format import DT_U8, MODE_RW, OP_TOUCH
    tensors = [dict(nbytes=4096, dtype=DT_U8, kind=KIND_ACT, host_init=True),    # log: 64 slots
               dict(nbytes=128 << 20, dtype=DT_U8, kind=KIND_PARAM, host_init=False),
               dict(nbytes=4096, dtype=DT_U8, kind=KIND_ACT, host_init=True)]
    kernels = [dict(op=OP_TOUCH, shape=(k,), operands=[(0, MODE_RW), (2, MODE_RW)], flops=1, hbm_bytes=1)
               for k in range(31)]
    kernels.append(dict(op=OP_TOUCH, shape=(31,), operands=[(0, MODE_RW), (1, MODE_R)], flops=1, hbm_bytes=1))
    M = sum(op.aligned(t["nbytes"]) for t in tensors)
    s, w = _session_from_trace(tensors, kernels, M, variant=4, timing=1)
    _init_words(s, w, tensors)
    s.run_all()
    tl = s.ctx.get_timeline()
    sched = s.ctx.get_schedule()
    s.close()
    big = [e for e in tl if e[0] in (TL_H2D, TL_H2D_B) and sched[e[2]][1] == 1]
    assert len(big) == 1
    kern = {e[2]: e for e in tl if e[0] == TL_KERNEL}
    assert big[0][5] < kern[1][5], "the prefetch is issued before the small kernels"
    # every kernel that does not read the big tensor ends before its copy does
    assert max(kern[k][6] for k in range(1, 31)) < big[0][6] - 0.5
    assert kern[31][5] >= big[0][6] - 0.02
