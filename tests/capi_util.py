"""Helpers to load traces into a plan-only C-ABI context and compare with the oracle."""
import os

from paper_2609_06172_amd.capi import Context

_LIB = {}


def plan_library():
    """None (the package's library) unless AUVM_SIM_SANITIZE=1: then the
    host-only build of the same sources with the sanitizers."""
    if os.environ.get("AUVM_SIM_SANITIZE") != "1":
        return None
    if "L" not in _LIB:
        import ctypes
        import sys
        sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "sim"))
        import build_sim
        from paper_2609_06172_amd.capi import bind_library
        _LIB["L"] = bind_library(ctypes.CDLL(build_sim.build()))
    return _LIB["L"]
from workloads.format import ALIGN, FLAG_HOST_INIT, FLAG_LIVE_OUT, KIND_PARAM


def plan_ctx(tensors, kernels, M, variant=4, lookahead=0, affinity_w=1, placement=0, roofs=None,
             guard=None, bucket=None, object_bytes=0):
    """Register a trace (oracle-style dicts) in a plan-only context and plan it.

    Kernels that carry a measured time (time_ns) hand the whole list to
    set_kernel_times before planning.
    """
    ctx = Context(-1, library=plan_library())
    off = 0
    offs = []
    for t in tensors:
        offs.append(off)
        off += (t["nbytes"] + ALIGN - 1) // ALIGN * ALIGN
    ctx.arena_init(max(off, ALIGN))
    for t, o in zip(tensors, offs):
        flags = FLAG_HOST_INIT if (t["host_init"] and t["kind"] != KIND_PARAM) else 0
        flags |= FLAG_LIVE_OUT if t.get("live_out") else 0
        ctx.register_tensor(o, t["nbytes"], t["dtype"], t["kind"], flags)
    for k in kernels:
        ctx.add_kernel(k["op"], k["shape"], k["operands"], k.get("flops", 0), k.get("hbm_bytes", 0))
    ctx.set_budget(M)
    if roofs is not None:
        ctx.set_roofs(*roofs)
    ctx.set_policy(variant, lookahead, affinity_w, placement, guard=guard, bucket=bucket,
                   object_bytes=object_bytes)
    times = [k.get("time_ns", 0) for k in kernels]
    if any(times):
        ctx.set_kernel_times(times)
    ctx.plan()
    return ctx


def assert_same_plan(ctx, r):
    """C++ plan in ctx equals oracle Result r field by field."""
    sched = ctx.get_schedule()
    assert len(sched) == len(r.schedule)
    for i, (a, b) in enumerate(zip(sched, r.schedule)):
        assert tuple(a) == tuple(b), f"schedule entry {i}: lib {a} oracle {b}"
    assert [tuple(x) for x in ctx.get_residency()] == [tuple(x) for x in r.residency]
    cls = ctx.get_classes()
    assert [c[0] for c in cls] == list(r.static_cls)
    assert [c[1] for c in cls] == list(r.dyn_cls)
    assert [(c[2], c[3]) for c in cls] == [tuple(x) for x in r.costs]
    c = ctx.get_counters()
    for k, v in r.counters.items():
        assert c[k] == v, (k, c[k], v)
