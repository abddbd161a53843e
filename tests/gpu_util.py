"""Helpers for GPU tests: single-kernel traces, touch-trace expectations, errors."""
import numpy as np

from workloads import init as winit
from workloads.format import (DT_BF16, DT_F32, DT_I32, DT_U8, FLAG_HOST_INIT,
                              KIND_ACT, KIND_PARAM, MODE_R, MODE_W)
from workloads.trace import Workload


def rel_l2(a, b):
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def bf16_round(x):
    """fp32 values of the bf16 (RNE) rounding of x."""
    return winit.bf16_to_f32(winit.bf16_bits(np.asarray(x, np.float32))).reshape(np.shape(x))


def single_kernel(op, shape, operands):
    """operands: list of (name, shape, dtype, mode, value or None).

    Returns (workload, values) where values holds the (dtype-rounded) fp64
    inputs the kernel sees, by name.
    """
    w = Workload(None)
    vals = {}
    ops = []
    for name, shp, dt, mode, value in operands:
        if name in w.by_name:
            ops.append((w.id(name), mode))
            continue
        host = value is not None
        kind = KIND_PARAM if (host and not (mode & 2)) else KIND_ACT
        tid = w.tensor(name, shp, dt, kind, host_init=host)
        if host:
            v = np.asarray(value)
            if dt == DT_BF16:
                v = bf16_round(v)
            vals[name] = v.astype(np.float64) if dt in (DT_F32, DT_BF16) else v
        ops.append((tid, mode))
    w.kernel(op, shape, ops)
    return w, vals


def write_inputs(s, w, vals):
    for name, v in vals.items():
        t = w.tensors[w.id(name)]
        if t.dtype == DT_BF16:
            s.host_view(t)[:] = winit.bf16_bits(np.asarray(v, np.float32)).view(np.uint8).reshape(-1)
        else:
            s.write(name, v)


def touch_expectations(tensors, kernels, init_words):
    """Expected (min, max) log words of every touch read, replaying versions."""
    ver = dict(init_words)
    exp = []
    for kd in kernels:
        slot = kd["shape"][0]
        for i, (t, m) in enumerate(kd["operands"][1:], start=1):
            if m & MODE_R:
                exp.append((slot, i, ver[t]))
        for t, m in kd["operands"][1:]:
            if m & MODE_W:
                ver[t] = slot + 1
    return exp
