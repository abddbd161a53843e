"""Semantic validation of a transfer schedule, independent of how it was made.

Replays a schedule of (op, tensor, dev_off, bytes, issue_k, need_k) entries
and checks the properties any correct schedule has under a device budget M:

* resident bytes never exceed M, and device windows stay inside [0, M) and
  never overlap (pool placement);
* at every LAUNCH all the kernel's operands are resident;
* every read sees the latest written value: each tensor carries a version;
  a launch that writes it creates a new version, a writeback copies the device
  version to the host, and a drop of a value that is still needed loses it;
* launches appear once each, in kernel order.
"""
from workloads.format import (ALIGN, KIND_PARAM, MODE_R, MODE_W, S_ALLOC,
                              S_D2H_WRITEBACK, S_DROP, S_H2D_DEMAND,
                              S_H2D_PREFETCH, S_LAUNCH)

LOST = object()


class ScheduleError(AssertionError):
    pass


def check(tensors, kernels, M, schedule, pool=True):
    nT = len(tensors)
    size = [(t["nbytes"] + ALIGN - 1) // ALIGN * ALIGN for t in tensors]
    host = [0 if (t["kind"] == KIND_PARAM or t["host_init"]) else None for t in tensors]
    latest = [0 if host[t] is not None else None for t in range(nT)]
    dev = {}                       # t -> (off, version)
    used = 0
    next_k = 0
    for i, (op, t, o, b, ik, nk) in enumerate(schedule):
        if op == S_LAUNCH:
            if ik != next_k:
                raise ScheduleError(f"entry {i}: launch {ik}, expected {next_k}")
            kd = kernels[ik]
            merged = {}
            for u, m in kd["operands"]:
                merged[u] = merged.get(u, 0) | m
            for u, m in merged.items():
                if u not in dev:
                    raise ScheduleError(f"launch {ik}: operand {u} not resident")
                if m & MODE_R:
                    v = dev[u][1]
                    if v is LOST or v is None or v != latest[u]:
                        raise ScheduleError(f"launch {ik}: stale read of tensor {u} "
                                            f"(has {v}, latest {latest[u]})")
            for u, m in merged.items():
                if m & MODE_W:
                    latest[u] = ("k", ik)
                    dev[u] = (dev[u][0], latest[u])
            next_k += 1
            continue
        if not 0 <= t < nT:
            raise ScheduleError(f"entry {i}: bad tensor {t}")
        if b != size[t]:
            raise ScheduleError(f"entry {i}: size {b} != {size[t]}")
        if op in (S_H2D_DEMAND, S_H2D_PREFETCH, S_ALLOC):
            if t in dev:
                raise ScheduleError(f"entry {i}: tensor {t} already resident")
            if pool:
                if o % ALIGN or o < 0 or o + size[t] > M:
                    raise ScheduleError(f"entry {i}: window [{o},{o + size[t]}) outside pool")
                for u, (ou, _) in dev.items():
                    if ou < o + size[t] and o < ou + size[u]:
                        raise ScheduleError(f"entry {i}: window of {t} overlaps {u}")
            if op == S_ALLOC:
                dev[t] = (o, None)
            else:
                if host[t] is None or host[t] is LOST:
                    raise ScheduleError(f"entry {i}: fetch of tensor {t} without a host value")
                dev[t] = (o, host[t])
            used += size[t]
            if used > M:
                raise ScheduleError(f"entry {i}: resident {used} > budget {M}")
        elif op in (S_D2H_WRITEBACK, S_DROP):
            if t not in dev or dev[t][0] != o:
                raise ScheduleError(f"entry {i}: evicting non-resident tensor {t}")
            v = dev.pop(t)[1]
            used -= size[t]
            if op == S_D2H_WRITEBACK:
                host[t] = v
            elif v != host[t]:
                host[t] = LOST           # device value differed from host: gone
        else:
            raise ScheduleError(f"entry {i}: unknown op {op}")
    if next_k != len(kernels):
        raise ScheduleError(f"{next_k} launches for {len(kernels)} kernels")
    return True


def check_workload(w, M, schedule, pool=True):
    tensors = [dict(nbytes=t.nbytes, kind=t.kind, host_init=t.host_init) for t in w.tensors]
    kernels = [dict(operands=k.operands) for k in w.kernels]
    return check(tensors, kernels, M, schedule, pool)
