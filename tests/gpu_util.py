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


# Per-element bounds |got - ref| <= r*|ref| + c*rms(ref), by what the kernel
# rounds (derivations with the tolerances in the design notes).  bf16 keeps 8
# significant bits, so one round-to-nearest-even is off by at most 2^-8
# relative (half an ulp just above a power of two):
# * one bf16 rounding of an fp32 result, taken twice; c covers fp32
#   accumulation (about 2^-24 * sqrt(K) of rms) and epilogue approximations
#   near zero outputs;
ELEM_BF16 = (2.0 ** -7, 2.0 ** -8)
# * fp32 results: accumulation order only;
ELEM_F32 = (1e-5, 1e-5)
# * attention with probabilities rounded to bf16 before P.V: each term p*v is
#   off by up to 2^-8 relative, so the absolute error of an output scales with
#   sum p|v|, several times |o| when o averages many values (random signs:
#   about 2^-8 / sqrt(3) of rms, ~5 sigma at the largest element);
ELEM_ATTN = (2.0 ** -7, 2.0 ** -6)
# * a whole decoder layer (norm, projections, attention, FFN), every stage
#   stored in bf16: independent roundings (rms 2^-8 / sqrt(3) relative each)
#   at about six stages, a few 1e-3 of the rms of the layer's increment, with
#   its largest elements ~5 sigma out.
ELEM_LAYER = (2.0 ** -6, 2.0 ** -5)


def assert_close(got, ref, tol, elem, what=""):
    """rel-L2 below tol, and every element within the per-element bound."""
    g = np.asarray(got, np.float64)
    f = np.asarray(ref, np.float64)
    assert g.shape == f.shape, f"{what}: shape {g.shape} != {f.shape}"
    assert np.isfinite(g).all(), f"{what}: {np.count_nonzero(~np.isfinite(g))} non-finite elements"
    e = rel_l2(g, f)
    assert e < tol, f"{what}: rel-L2 {e:.3e} >= {tol:.1e}"
    r, c = elem
    rms = float(np.sqrt(np.mean(f * f))) if f.size else 0.0
    d = np.abs(g - f)
    bound = r * np.abs(f) + c * rms
    bad = d > bound
    if bad.any():
        i = np.unravel_index(int(np.argmax(d - bound)), d.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {d.size} elements outside "
                             f"|got - ref| <= {r:.2e}|ref| + {c:.2e}*rms (rms {rms:.3e}); worst at {i}: "
                             f"got {g[i]:.6e}, ref {f[i]:.6e}")
    return e, float(np.max(d / max(rms, 1e-300))) if d.size else 0.0


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


def attention_backward_bounds(q, K, V, dO):
    """Per-element error bounds of a causal attention backward (one head, [S, d]
    fp64 inputs) whose kernel recomputes the probabilities P from the forward's
    log-sum-exp, takes D_i = sum_c dO_ic O_ic from the forward's bf16 output O,
    and rounds P and dS = P (dP - D) to bf16 before their products.  To first
    order each bf16 rounding is at most u = 2^-8 relative (the outputs' own
    rounding included), so with a factor 2:
    * dV_j = sum_i P_ij dO_i:        2^-7 (|dV| + (P^T |dO|))
    * dS_ij is off by P_ij |dD_i| + u |dS_ij| (its rounding) + u |dS_ij| (P's
      rounding), with |dD_i| <= u sum_c |dO_ic O_ic| (O's rounding);
    * dq_i = sc sum_j dS_ij K_j:     2^-7 (|dq| + sc (2 |dS| |K| + A P |K|)),
    * dK_j = sc sum_i dS_ij q_i:     2^-7 (|dK| + sc (2 |dS|^T |q| + P^T (A |q|))),
    where A_i = sum_c |dO_ic O_ic|.  The fp32 accumulations are far below these.
    Returns (dq, dK, dV) and their bounds."""
    S, d = q.shape
    sc = 1.0 / np.sqrt(d)
    s = (q @ K.T) * sc
    s = np.where(np.arange(S)[None, :] <= np.arange(S)[:, None], s, -np.inf)
    P = np.exp(s - s.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    O = P @ V
    dP = dO @ V.T
    D = (dO * O).sum(axis=1, keepdims=True)
    dS = P * (dP - D)
    dq, dK, dV = dS @ K * sc, dS.T @ q * sc, P.T @ dO
    A = np.abs(dO * O).sum(axis=1, keepdims=True)
    u = 2.0 ** -7
    bq = u * (np.abs(dq) + sc * (2 * np.abs(dS) @ np.abs(K) + A * (P @ np.abs(K))))
    bk = u * (np.abs(dK) + sc * (2 * np.abs(dS).T @ np.abs(q) + P.T @ (A * np.abs(q))))
    bv = u * (np.abs(dV) + P.T @ np.abs(dO))
    return (dq, dK, dV), (bq, bk, bv)


def assert_within(got, ref, bound, tol, what=""):
    """rel-L2 below tol and every element within its own bound."""
    g = np.asarray(got, np.float64)
    assert np.isfinite(g).all(), f"{what}: non-finite elements"
    e = rel_l2(g, ref)
    assert e < tol, f"{what}: rel-L2 {e:.3e} >= {tol:.1e}"
    d = np.abs(g - ref)
    bad = d > bound
    if bad.any():
        i = np.unravel_index(int(np.argmax(d / np.maximum(bound, 1e-300))), d.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {d.size} elements outside their bound; worst at {i}: "
                             f"got {g[i]:.6e}, ref {ref[i]:.6e}, bound {bound[i]:.3e}")
    return e, float(np.max(d / np.maximum(bound, 1e-300)))
