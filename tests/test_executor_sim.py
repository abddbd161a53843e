"""The executor on the CPU: the transfer engine's source, built against a
queue simulator instead of the HIP runtime (tests/sim), runs random touch
traces under every policy while operations execute in random orders allowed
by the engine's event waits.  Every kernel must read exactly the version of
each operand that the trace's order of writes implies, and the executed log
must equal the plan.  Evicted windows are poisoned, so a read of a window
that is not yet (or no longer) the tensor's shows up as a wrong version.

A control run with the simulator's event waits dropped must fail: the
traces are sensitive to missing ordering."""
import ctypes as C
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "sim"))

from oracle import planner as op
from workloads.format import KIND_PARAM
from workloads.trace import Workload

from gpu_util import touch_expectations
from planner_cases import random_trace

_SIM = {}


def sim_library():
    if "L" not in _SIM:
        import build_sim
        from paper_2609_06172_amd.capi import bind_library
        L = bind_library(C.CDLL(build_sim.build()))
        L.auvm_sim_seed.restype = C.c_uint64
        L.auvm_sim_seed.argtypes = [C.c_uint64]
        L.auvm_sim_drop_waits.restype = None
        L.auvm_sim_drop_waits.argtypes = [C.c_int]
        L.auvm_sim_new_stream.restype = C.c_void_p
        L.auvm_sim_new_stream.argtypes = []
        _SIM["L"] = L
    return _SIM["L"]


def feasible_budget(tensors, kernels, variant, fracs=((1, 2), (2, 3), (3, 4), (5, 6), (1, 1)), object_bytes=0):
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    for num, den in fracs:
        M = max(1024, fp * num // den // 256 * 256)
        try:
            op.plan(tensors, kernels, M, variant=variant, object_bytes=object_bytes)
            return M
        except op.PlanError:
            continue
    raise AssertionError("no feasible budget")


def run_touch_trace(seed, variant, order_seed, cuts=3, read_only=False, bind=None, timing=0, out=None,
                    object_bytes=0, tiered=False, big=0):
    """Runs a random touch trace on the simulated executor; returns (executed log
    equals the plan, reads that saw the wrong version).

    big: that many read-only parameters of 100 MiB + 4 KiB (larger than a
    staging slot) joined to the trace, each read by every fifth kernel in turn.
    tiered: a tiered host arena whose pageable tier holds every parameter that
    no kernel writes (fetched through the staging ring)."""
    from paper_2609_06172_amd.capi import Context
    L = sim_library()
    n_kernels = (60 if read_only else 40) + (seed * 7) % 60
    tensors, kernels = random_trace(seed, touch=True, n_kernels=n_kernels, read_only=read_only)
    for b in range(big):
        tensors.append(dict(nbytes=(100 << 20) + 4096, dtype=tensors[1]["dtype"] if len(tensors) > 1 else 3,
                            kind=KIND_PARAM, host_init=True))
    for k, kd in enumerate(kernels):
        if big and k % 5 == 0 and len(kd["operands"]) < 7:
            kd["operands"].append((len(tensors) - big + (k // 5) % big, 1))
    M = feasible_budget(tensors, kernels, variant, object_bytes=object_bytes,
                        fracs=((3, 4), (5, 6), (1, 1)) if big else ((1, 2), (2, 3), (3, 4), (5, 6), (1, 1)))
    w = Workload(None)
    for i, t in enumerate(tensors):
        w.tensor(f"t{i}", (t["nbytes"],), t["dtype"], t["kind"], host_init=t["host_init"])
    ctx = Context(0, library=L)
    offs = [t.off for t in w.tensors]
    if tiered:
        written = {u for kd in kernels for u, m in kd["operands"] if m & 2}
        pin = [t for t in w.tensors if t.kind != KIND_PARAM or t.tid in written]
        page = [t for t in w.tensors if not (t.kind != KIND_PARAM or t.tid in written)]
        assert page
        off = 0
        for t in pin + page:
            offs[t.tid] = off
            off += (t.nbytes + 255) // 256 * 256
        ctx.arena_init_tiered(w.arena_bytes, offs[page[0].tid])
    else:
        ctx.arena_init(w.arena_bytes)
    for t in w.tensors:
        ctx.register_tensor(offs[t.tid], t.nbytes, t.dtype, t.kind, t.flags)
    init = {}
    for i, t in enumerate(tensors):
        view = np.ctypeslib.as_array((C.c_uint8 * t["nbytes"]).from_address(ctx.tensor_host_ptr(i)))
        if i == 0:
            view[:] = 0                                  # the log
        elif t["host_init"] or t["kind"] == KIND_PARAM:
            init[i] = 1000 + i
            view[:] = np.full(t["nbytes"] // 4, init[i], np.uint32).view(np.uint8)
    for k in kernels:
        ctx.add_kernel(k["op"], k["shape"], k["operands"])
    ctx.set_budget(M)
    ctx.set_policy(variant, validate=1, timing=timing, object_bytes=object_bytes)
    ctx.plan()
    if bind is not None:
        ctx.bind_streams(*bind)
    L.auvm_sim_seed(order_seed)
    K = len(kernels)
    bounds = sorted(set([0, K] + [K * j // cuts for j in range(1, cuts)]))
    for a, b in zip(bounds, bounds[1:]):
        if b > a:
            ctx.run(a, b - a)
    executed_ok = ctx.get_executed() == ctx.get_schedule()
    if out is not None:
        out.update(timeline=ctx.get_timeline(), schedule=ctx.get_schedule(), kernels=kernels, tensors=tensors,
                   counters=ctx.get_counters(), kernel_times=ctx.get_kernel_times())
    logbuf = np.empty(tensors[0]["nbytes"], np.uint8)
    ctx.read_tensor(0, logbuf.ctypes.data, logbuf.nbytes)
    ctx.destroy()
    log = logbuf.view(np.uint32).reshape(-1, 16)
    bad = [(slot, i, v, tuple(log[slot, 2 * i:2 * i + 2]))
           for slot, i, v in touch_expectations(tensors, kernels, init)
           if log[slot, 2 * i] != v or log[slot, 2 * i + 1] != v]
    return executed_ok, bad


@pytest.mark.parametrize("variant", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("seed", range(8))
def test_touch_traces_read_latest_versions_in_any_order(seed, variant):
    for order_seed in range(4):
        executed_ok, bad = run_touch_trace(seed, variant, order_seed, cuts=1 + order_seed % 3)
        assert executed_ok
        assert not bad, (seed, variant, order_seed, bad[:4])


@pytest.mark.parametrize("seed", range(4))
def test_pageable_tier_through_the_staging_ring(seed):
    """A tiered host arena: the parameters no kernel writes live in pageable
    memory and reach the device through the pinned staging ring, two of them
    larger than a slot (they move in pieces, reusing slots): every kernel
    still reads the latest version of each operand, in any order of
    execution the event waits allow, and the executed log equals the plan."""
    for variant in (1, 4):
        executed_ok, bad = run_touch_trace(seed, variant, seed, cuts=2, tiered=True, big=2)
        assert executed_ok
        assert not bad, (seed, variant, bad[:4])


def test_tiered_arena_refuses_what_would_need_a_write_back():
    """Only parameters may live in the pageable tier, a window may not
    straddle the tiers, and no kernel may write a pageable tensor."""
    from paper_2609_06172_amd.capi import AuvmError, Context
    from workloads.format import DT_U8, KIND_ACT, MODE_R, MODE_RW, OP_TOUCH
    ctx = Context(0, library=sim_library())
    with pytest.raises(AuvmError):
        ctx.arena_init_tiered(4096, 1000)          # not a multiple of 256
    ctx.arena_init_tiered(4096, 1024)
    log = ctx.register_tensor(0, 512, DT_U8, KIND_ACT)
    with pytest.raises(AuvmError):
        ctx.register_tensor(768, 512, DT_U8, KIND_PARAM)   # straddles 1024
    with pytest.raises(AuvmError):
        ctx.register_tensor(1024, 512, DT_U8, KIND_ACT)    # activation in the pageable tier
    p = ctx.register_tensor(1024, 512, DT_U8, KIND_PARAM)
    ctx.add_kernel(OP_TOUCH, (0,), [(log, MODE_RW), (p, MODE_R)])
    with pytest.raises(AuvmError):
        ctx.add_kernel(OP_TOUCH, (1,), [(log, MODE_RW), (p, MODE_RW)])
    ctx.destroy()


@pytest.mark.parametrize("variant", [1, 2, 3, 4])
@pytest.mark.parametrize("seed", range(12))
def test_read_only_traces_on_two_copy_streams(seed, variant):
    """Data operands only read: the plans have no write-backs, so copies
    alternate between the two host-to-device streams; a kernel that ran
    before its operand's copy, or a copy that overtook an earlier fill of the
    same window, would read poison or another tensor's words."""
    for order_seed in range(3):
        executed_ok, bad = run_touch_trace(seed, variant, order_seed, cuts=1 + order_seed, read_only=True)
        assert executed_ok
        assert not bad, (seed, variant, order_seed, bad[:4])


@pytest.mark.parametrize("read_only", [False, True])
@pytest.mark.parametrize("seed", range(6))
def test_caller_bound_streams(seed, read_only):
    """One caller stream for all copies (and callers' compute and write-back
    streams): both copy sequences share it, and reads stay exact."""
    L = sim_library()
    streams = (L.auvm_sim_new_stream(), L.auvm_sim_new_stream(), L.auvm_sim_new_stream())
    for variant in (0, 4):
        if read_only and variant == 0:
            continue
        for order_seed in range(2):
            executed_ok, bad = run_touch_trace(seed, variant, order_seed, read_only=read_only, bind=streams)
            assert executed_ok and not bad, (seed, variant, order_seed, bad[:4])


@pytest.mark.parametrize("read_only", [False, True])
@pytest.mark.parametrize("seed", range(4))
def test_timing_tracks(seed, read_only):
    """Timing policy: one timeline entry per kernel and per copy, each
    stream's items in order without overlap, kernels after the copies that
    brought their operands (simulated clocks), and reads still exact."""
    from paper_2609_06172_amd.capi import TL_D2H, TL_H2D, TL_H2D_B, TL_KERNEL
    from workloads.format import S_ALLOC, S_D2H_WRITEBACK, S_H2D_DEMAND, S_H2D_PREFETCH, S_LAUNCH
    rec = {}
    executed_ok, bad = run_touch_trace(seed, 4, seed, cuts=2, read_only=read_only, timing=1, out=rec)
    assert executed_ok and not bad
    tl, sched, kernels, tensors = rec["timeline"], rec["schedule"], rec["kernels"], rec["tensors"]
    kern = [e for e in tl if e[0] == TL_KERNEL]
    assert sorted(e[2] for e in kern) == list(range(len(kernels)))
    got = sorted((e[2], e[3]) for e in tl if e[0] in (TL_H2D, TL_H2D_B))
    want = [(i, tensors[x[1]]["nbytes"]) for i, x in enumerate(sched) if x[0] in (S_H2D_PREFETCH, S_H2D_DEMAND)]
    assert got == want
    assert sum(1 for e in tl if e[0] == TL_D2H) == sum(1 for x in sched if x[0] == S_D2H_WRITEBACK)
    for kind in (TL_KERNEL, TL_H2D, TL_H2D_B, TL_D2H):
        items = [e for e in tl if e[0] == kind]
        for a, b in zip(items, items[1:]):
            if a[1] == b[1]:
                assert b[5] >= a[6] and b[6] >= b[5]
    start = {e[2]: e[5] for e in kern}
    seg = {e[2]: e[1] for e in kern}
    copy = {e[2]: e for e in tl if e[0] in (TL_H2D, TL_H2D_B)}
    latest = {}
    for i, x in enumerate(sched):
        if x[0] in (S_H2D_PREFETCH, S_H2D_DEMAND):
            latest[x[1]] = i
        elif x[0] == S_LAUNCH:
            for t, _ in kernels[x[4]]["operands"]:
                j = latest.get(t)
                if j is not None and copy[j][1] == seg[x[4]]:
                    assert copy[j][6] <= start[x[4]], (x[4], t)
        elif x[0] == S_ALLOC:
            latest.pop(x[1], None)
    # the stall counter is the compute stream's idle time between consecutive
    # kernels of a segment, as the timeline shows it
    idle = sum(b[5] - a[6] for a, b in zip(kern, kern[1:]) if a[1] == b[1])
    _, gaps = rec["kernel_times"]
    assert abs(rec["counters"]["stall_ns"] - idle * 1e6) <= 1e-3 * max(1.0, idle * 1e6)
    assert abs(sum(gaps) * 1e6 - rec["counters"]["stall_ns"]) <= 1e-3 * max(1.0, idle * 1e6)
    assert idle > 0


def test_no_stall_counted_without_timing():
    rec = {}
    executed_ok, bad = run_touch_trace(3, 4, 1, cuts=2, out=rec)
    assert executed_ok and not bad
    assert rec["counters"]["stall_ns"] == 0


def test_dropping_the_event_waits_is_caught():
    L = sim_library()
    L.auvm_sim_drop_waits(1)
    try:
        failures = 0
        for seed in range(6):
            for order_seed in range(3):
                _, bad = run_touch_trace(seed, 4, order_seed)
                failures += bool(bad)
        assert failures > 0
    finally:
        L.auvm_sim_drop_waits(0)


@pytest.mark.parametrize("seed", range(4))
def test_a_new_budget_replans_the_same_trace(seed):
    """set_budget again on a context that has run: the plan at the new budget
    is the oracle's, and a rerun from the first kernel reads exact versions
    (read-only data, so the host contents the rerun starts from are intact)."""
    from paper_2609_06172_amd.capi import Context
    L = sim_library()
    tensors, kernels = random_trace(seed, touch=True, n_kernels=70, read_only=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    w = Workload(None)
    for i, t in enumerate(tensors):
        w.tensor(f"t{i}", (t["nbytes"],), t["dtype"], t["kind"], host_init=t["host_init"])
    ctx = Context(0, library=L)
    ctx.arena_init(w.arena_bytes)
    for t in w.tensors:
        ctx.register_tensor(t.off, t.nbytes, t.dtype, t.kind, t.flags)
    init = {}
    for i, t in enumerate(tensors):
        view = np.ctypeslib.as_array((C.c_uint8 * t["nbytes"]).from_address(ctx.tensor_host_ptr(i)))
        if i == 0:
            view[:] = 0
        else:
            init[i] = 1000 + i
            view[:] = np.full(t["nbytes"] // 4, init[i], np.uint32).view(np.uint8)
    for k in kernels:
        ctx.add_kernel(k["op"], k["shape"], k["operands"], flops=k["flops"], hbm_bytes=k["hbm_bytes"])
    budgets = [fp // 256 * 256, feasible_budget(tensors, kernels, 4)]
    for i, M in enumerate(budgets):
        ctx.set_budget(M)
        ctx.set_policy(4, validate=1)
        ctx.plan()
        assert ctx.get_schedule() == op.plan(tensors, kernels, M).schedule
        L.auvm_sim_seed(seed + i)
        ctx.run(0, len(kernels))
        logbuf = np.empty(tensors[0]["nbytes"], np.uint8)
        ctx.read_tensor(0, logbuf.ctypes.data, logbuf.nbytes)
        log = logbuf.view(np.uint32).reshape(-1, 16)
        bad = [(s, j, v) for s, j, v in touch_expectations(tensors, kernels, init)
               if log[s, 2 * j] != v or log[s, 2 * j + 1] != v]
        assert not bad, (M, bad[:4])
    ctx.destroy()


@pytest.mark.parametrize("seed", range(4))
def test_run_noalloc_reads_the_same_versions(seed):
    """auvm_run_noalloc on the simulated executor: the same transfers and
    launches as auvm_run (touch traces carry no workspace operand), exact
    versions, and the timing policy refused before anything is enqueued."""
    from paper_2609_06172_amd.capi import AuvmError, Context
    L = sim_library()
    tensors, kernels = random_trace(seed, touch=True, n_kernels=60)
    M = feasible_budget(tensors, kernels, 4)
    w = Workload(None)
    for i, t in enumerate(tensors):
        w.tensor(f"t{i}", (t["nbytes"],), t["dtype"], t["kind"], host_init=t["host_init"])
    ctx = Context(0, library=L)
    ctx.arena_init(w.arena_bytes)
    for t in w.tensors:
        ctx.register_tensor(t.off, t.nbytes, t.dtype, t.kind, t.flags)
    init = {}
    for i, t in enumerate(tensors):
        view = np.ctypeslib.as_array((C.c_uint8 * t["nbytes"]).from_address(ctx.tensor_host_ptr(i)))
        if i == 0:
            view[:] = 0
        elif t["host_init"] or t["kind"] == KIND_PARAM:
            init[i] = 1000 + i
            view[:] = np.full(t["nbytes"] // 4, init[i], np.uint32).view(np.uint8)
    for k in kernels:
        ctx.add_kernel(k["op"], k["shape"], k["operands"], flops=k["flops"], hbm_bytes=k["hbm_bytes"])
    ctx.set_budget(M)
    ctx.set_policy(4, validate=1, timing=1)
    ctx.plan()
    with pytest.raises(AuvmError) as e:
        ctx.run_noalloc(0, len(kernels))
    assert e.value.code == -2 and ctx.get_executed() == []
    ctx.set_policy(4, validate=1)
    ctx.plan()
    L.auvm_sim_seed(seed)
    half = len(kernels) // 2
    ctx.run_noalloc(0, half)
    ctx.run_noalloc(half, len(kernels) - half)
    assert ctx.get_executed() == ctx.get_schedule()
    logbuf = np.empty(tensors[0]["nbytes"], np.uint8)
    ctx.read_tensor(0, logbuf.ctypes.data, logbuf.nbytes)
    log = logbuf.view(np.uint32).reshape(-1, 16)
    bad = [(s, j, v) for s, j, v in touch_expectations(tensors, kernels, init)
           if log[s, 2 * j] != v or log[s, 2 * j + 1] != v]
    assert not bad, bad[:4]
    ctx.destroy()


@pytest.mark.parametrize("variant", [0, 1, 4])
@pytest.mark.parametrize("seed", range(6))
def test_object_plans_read_latest_versions(seed, variant):
    """Plans at object granularity (whole allocator blocks moved, members
    allocated or written back together) run on the executor unchanged and
    read exact versions in any allowed order."""
    for order_seed in range(3):
        executed_ok, bad = run_touch_trace(seed, variant, order_seed, cuts=1 + order_seed,
                                           object_bytes=(1024, 4096, 16384)[order_seed])
        assert executed_ok
        assert not bad, (seed, variant, order_seed, bad[:4])
