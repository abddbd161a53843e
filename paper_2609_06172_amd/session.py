"""Load a workload (tensor list + kernel trace) into a runtime context.

Marshalling only: registers the workload's tensors and kernels through the C
interface, writes the seeded initial host contents into the context's arena,
lends the device pool (allocated with PyTorch) and plans.  The library runs
on streams of its own (one hardware queue each); all scheduling and every
kernel run inside it.
"""
import ctypes as C

import numpy as np

from workloads import init as winit
from workloads.format import DT_BF16, DT_F32, DT_I32, DT_U8, KIND_PARAM

from .capi import Context

NP_DTYPE = {DT_F32: np.float32, DT_I32: np.int32, DT_U8: np.uint8, DT_BF16: np.uint16}


def host_layout(w, pinned_limit=None):
    """Arena offsets of the workload's tensors and the pinned tier's size.

    Without a limit, or when the whole arena fits it, the workload's own
    offsets and a pinned arena (None).  Otherwise a tiered arena: first every
    tensor that is not a parameter or that some kernel writes (these must be
    pinned), then the read-only parameters in registration order, the pinned
    tier ending before the first tensor that would cross the limit."""
    from workloads.format import MODE_W
    if pinned_limit is None or w.arena_bytes <= pinned_limit:
        return [t.off for t in w.tensors], None
    written = {tid for k in w.kernels for tid, m in k.operands if m & MODE_W}
    pin = {t.tid for t in w.tensors if t.kind != KIND_PARAM or t.tid in written}
    must = [t for t in w.tensors if t.tid in pin]
    rest = [t for t in w.tensors if t.tid not in pin]
    offs, off, pinned = [0] * len(w.tensors), 0, None
    for t in must + rest:
        size = (t.nbytes + 255) // 256 * 256
        if pinned is None and t.tid not in pin and off + size > pinned_limit:
            pinned = off
        offs[t.tid] = off
        off += size
    if pinned is None:
        pinned = off
    if sum((t.nbytes + 255) // 256 * 256 for t in must) > pinned_limit:
        raise ValueError("the tensors that must be pinned exceed the pinned limit")
    return offs, pinned


class Session:
    def __init__(self, w, device=-1, M=None, variant=4, lookahead=0, affinity_w=1, placement=0,
                 validate=0, timing=0, roofs=None, fill=True, threads=16, guard=None, bucket=None,
                 object_bytes=0, pinned_limit=None):
        self.w = w
        self.device = device
        self.ctx = Context(device)
        ctx = self.ctx
        offs, pinned = host_layout(w, pinned_limit)
        if pinned is None:
            ctx.arena_init(w.arena_bytes)
        else:
            ctx.arena_init_tiered(w.arena_bytes, pinned)
        self.pinned_bytes = w.arena_bytes if pinned is None else pinned
        for t in w.tensors:
            tid = ctx.register_tensor(offs[t.tid], t.nbytes, t.dtype, t.kind, t.flags)
            assert tid == t.tid
        if device >= 0 and fill:
            winit.fill_host(w, self.host_view, threads=threads)
        for k in w.kernels:
            ctx.add_kernel(k.op, k.shape, k.operands, layer=k.layer)
        self.M = w.budget() if M is None else M
        self._torch_refs = []
        if device >= 0:
            import torch
            pool = torch.empty(self.M, dtype=torch.uint8, device=f"cuda:{device}")
            self._torch_refs.append(pool)
            ctx.set_budget(self.M, pool.data_ptr())
        else:
            ctx.set_budget(self.M)
        if roofs is not None:
            ctx.set_roofs(*roofs)
        self.set_policy(variant, lookahead, affinity_w, placement, validate, timing, guard, bucket,
                        object_bytes)

    def set_budget(self, M, plan=True):
        """The same trace under a new device budget (a new pool); plans again
        unless plan is False (then set_policy plans)."""
        import torch
        pool = torch.empty(M, dtype=torch.uint8, device=f"cuda:{self.device}")
        self.ctx.set_budget(M, pool.data_ptr())
        self._torch_refs = [pool]          # the old pool is idle once set_budget returned
        self.M = M
        if plan:
            self.ctx.plan()

    def set_policy(self, variant=4, lookahead=0, affinity_w=1, placement=0, validate=0, timing=0,
                   guard=None, bucket=None, object_bytes=0):
        self.ctx.set_policy(variant, lookahead, affinity_w, placement, validate, timing, guard, bucket,
                            object_bytes)
        self.ctx.plan()

    def measured_kernel_times_ns(self):
        """Duration of every kernel in the last timed run, integer ns (at least 1)."""
        dur, _ = self.ctx.get_kernel_times()
        if len(dur) != len(self.w.kernels):
            raise RuntimeError(f"{len(dur)} of {len(self.w.kernels)} kernels timed: "
                               "run every kernel with the timing policy on first")
        return [max(1, int(round(d * 1e6))) for d in dur]

    def replan_measured(self, times_ns=None):
        """Runtime monitor (Sec. IV, Online Executor): classify the kernels
        again from measured durations (default: the last timed run's) and
        plan again; the executor restarts from an empty pool."""
        t = self.measured_kernel_times_ns() if times_ns is None else times_ns
        self.ctx.set_kernel_times(t)
        self.ctx.plan()
        return t

    def retrace(self, w):
        """Replace the trace by the kernels of ``w``, a workload over the same
        tensors (for routed experts: the trace a profiling run recorded), and
        plan again.  Execution restarts from an empty pool."""
        same = [(t.nbytes, t.dtype, t.kind, t.off) for t in w.tensors]
        if same != [(t.nbytes, t.dtype, t.kind, t.off) for t in self.w.tensors]:
            raise ValueError("retrace needs a workload over the same tensors")
        self.ctx.clear_kernels()
        for k in w.kernels:
            self.ctx.add_kernel(k.op, k.shape, k.operands, layer=k.layer)
        self.w = w
        self.ctx.plan()

    def routing_counts(self):
        """Per-expert row counts logged by the MoE dispatch kernels, [seg][layer][expert]."""
        c = self.w.cfg
        return self.read("moe_counts").reshape(1 + c.decode_steps, c.n_layers, c.n_experts)

    # -- host arena access ----------------------------------------------------
    def host_view(self, t):
        """uint8 numpy view of tensor t's host arena window."""
        addr = self.ctx.tensor_host_ptr(t.tid)
        return np.ctypeslib.as_array((C.c_uint8 * t.nbytes).from_address(addr))

    def restore_inputs(self, threads=16):
        """Rewrite the initial host contents of non-parameter inputs (a rerun
        after reset must start from them; write-backs may have changed them)."""
        todo = [t for t in self.w.tensors if t.host_init and t.kind != KIND_PARAM]
        for t in todo:
            self.host_view(t)[: t.nbytes] = winit.tensor_bytes(self.w, t)

    def write(self, name, value):
        t = self.w.tensors[self.w.id(name)]
        src = np.ascontiguousarray(value, NP_DTYPE[t.dtype]).view(np.uint8).reshape(-1)
        self.host_view(t)[:] = src

    def read(self, name):
        """Current value of a tensor (fp32 for bf16 tensors), shaped."""
        t = self.w.tensors[self.w.id(name)]
        buf = np.empty(t.nbytes, np.uint8)
        self.ctx.read_tensor(t.tid, buf.ctypes.data, t.nbytes)
        v = buf.view(NP_DTYPE[t.dtype])
        if t.dtype == DT_BF16:
            v = winit.bf16_to_f32(v)
        return v.reshape(t.shape)

    # -- execution --------------------------------------------------------------
    def run(self, first_k, n_k):
        self.ctx.run(first_k, n_k)

    def run_all(self):
        self.ctx.run(0, len(self.w.kernels))

    def close(self):
        self.ctx.destroy()
        self._torch_refs.clear()
