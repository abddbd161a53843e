"""ctypes binding of include/autouvm.h — argument marshalling only.

Every method of :class:`Context` is one C call of the same name (without the
``auvm_`` prefix); failures raise :class:`AuvmError` with the status code and
the library's message.  The library must have been built
(``python -m paper_2609_06172_amd.build``); importing fails loudly otherwise.
"""
import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libautouvm.so")

OK, E_INVAL, E_STATE, E_BUDGET, E_FRAG, E_HIP, E_NOMEM, E_RANGE = 0, -1, -2, -3, -4, -5, -6, -7

# every symbol the header declares
SYMBOLS = [
    "auvm_create", "auvm_destroy", "auvm_last_error", "auvm_arena_init", "auvm_arena_init_tiered",
    "auvm_register_tensor", "auvm_tensor_host_ptr", "auvm_add_kernel", "auvm_set_budget",
    "auvm_set_roofs", "auvm_set_policy", "auvm_set_kernel_times", "auvm_clear_kernels", "auvm_plan", "auvm_bind_streams", "auvm_run", "auvm_run_noalloc",
    "auvm_reset", "auvm_read_tensor", "auvm_get_counters", "auvm_get_schedule",
    "auvm_get_executed", "auvm_get_residency", "auvm_get_classes", "auvm_get_kernel_times",
    "auvm_get_timeline",
]


class KernelDesc(C.Structure):
    _fields_ = [("op", C.c_uint32), ("shape", C.c_int64 * 8), ("n", C.c_uint32),
                ("ids", C.POINTER(C.c_int32)), ("modes", C.POINTER(C.c_uint8)),
                ("flops", C.c_uint64), ("hbm_bytes", C.c_uint64), ("layer", C.c_uint32)]


class Policy(C.Structure):
    _fields_ = [("variant", C.c_uint32), ("lookahead", C.c_uint32), ("affinity_w", C.c_uint32),
                ("placement", C.c_uint32), ("validate", C.c_uint32), ("timing", C.c_uint32),
                ("guard", C.c_uint32), ("bucket", C.c_uint32), ("object_bytes", C.c_uint64)]


class SchedEntry(C.Structure):
    _fields_ = [("op", C.c_int32), ("tensor", C.c_int32), ("dev_off", C.c_uint64),
                ("bytes", C.c_uint64), ("issue_k", C.c_int32), ("need_k", C.c_int32)]


class Residency(C.Structure):
    _fields_ = [("k", C.c_int32), ("n_resident", C.c_int32), ("resident_bytes", C.c_uint64)]


class KernelClass(C.Structure):
    _fields_ = [("static_cls", C.c_uint8), ("dyn_cls", C.c_uint8), ("pad", C.c_uint8 * 6),
                ("flops", C.c_uint64), ("hbm_bytes", C.c_uint64)]


class TimelineEntry(C.Structure):
    _fields_ = [("kind", C.c_int32), ("segment", C.c_int32), ("index", C.c_int64), ("bytes", C.c_uint64),
                ("host_ms", C.c_double), ("start_ms", C.c_double), ("end_ms", C.c_double)]


TL_KERNEL, TL_H2D, TL_D2H, TL_H2D_B = 0, 1, 2, 3

POLICY_DEFAULT = 0xFFFFFFFF      # guard / bucket: the library's default for the variant


class Counters(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in (
        "h2d_prefetch_n", "h2d_prefetch_B", "h2d_demand_n", "h2d_demand_B", "d2h_wb_n",
        "d2h_wb_B", "drop_n", "alloc_n", "useless_prefetch_n", "useless_prefetch_B")] + [
        ("class_n", C.c_uint64 * 3), ("plan_ns", C.c_uint64), ("run_ns", C.c_uint64),
        ("kernels_run", C.c_uint64), ("stall_ns", C.c_uint64)]

    def as_dict(self):
        d = {n: getattr(self, n) for n, _ in self._fields_ if n != "class_n"}
        d["class_n"] = list(self.class_n)
        return d


class AuvmError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"[{code}] {msg}")
        self.code = code


_lib = None


def _hip_runtimes():
    """Distinct HIP runtime files mapped into this process."""
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                p = line.split()[-1] if line.strip() else ""
                if os.path.basename(p).startswith("libamdhip64.so"):
                    paths.add(os.path.realpath(p))
    except OSError:
        pass
    return paths


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2609_06172_amd.build`")
    # PyTorch ships its own HIP runtime with the same soname as the system
    # one.  Loading torch first makes the library bind to that runtime, so the
    # process has a single HIP runtime and torch's device buffers and streams
    # are valid handles for the library.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    L = C.CDLL(LIB_PATH)
    if len(_hip_runtimes()) > 1:
        raise ImportError(f"two HIP runtimes are loaded ({sorted(_hip_runtimes())}); "
                          "import torch before any other HIP library")
    _lib = bind_library(L)
    return _lib


def bind_library(L):
    """Declare the C ABI's argument and result types on a loaded library."""
    P = C.c_void_p
    st = C.c_int32
    sig = {
        "auvm_create": (st, [C.c_int, C.POINTER(P)]),
        "auvm_destroy": (None, [P]),
        "auvm_last_error": (C.c_char_p, [P]),
        "auvm_arena_init": (st, [P, C.c_uint64, P]),
        "auvm_arena_init_tiered": (st, [P, C.c_uint64, C.c_uint64]),
        "auvm_register_tensor": (st, [P, C.c_uint64, C.c_uint64, C.c_uint32, C.c_uint32,
                                      C.c_uint32, C.POINTER(C.c_int32)]),
        "auvm_tensor_host_ptr": (st, [P, C.c_int32, C.POINTER(P)]),
        "auvm_add_kernel": (st, [P, C.POINTER(KernelDesc), C.POINTER(C.c_int32)]),
        "auvm_set_budget": (st, [P, C.c_uint64, P]),
        "auvm_set_roofs": (st, [P, C.c_uint64, C.c_uint64, C.c_uint64]),
        "auvm_set_policy": (st, [P, C.POINTER(Policy)]),
        "auvm_set_kernel_times": (st, [P, C.POINTER(C.c_uint64), C.c_uint64]),
        "auvm_clear_kernels": (st, [P]),
        "auvm_plan": (st, [P]),
        "auvm_bind_streams": (st, [P, P, P, P]),
        "auvm_run": (st, [P, C.c_uint32, C.c_uint32]),
        "auvm_run_noalloc": (st, [P, C.c_uint32, C.c_uint32]),
        "auvm_reset": (st, [P]),
        "auvm_read_tensor": (st, [P, C.c_int32, P, C.c_uint64]),
        "auvm_get_counters": (st, [P, C.POINTER(Counters)]),
        "auvm_get_schedule": (st, [P, C.POINTER(SchedEntry), C.c_uint64, C.POINTER(C.c_uint64)]),
        "auvm_get_executed": (st, [P, C.POINTER(SchedEntry), C.c_uint64, C.POINTER(C.c_uint64)]),
        "auvm_get_residency": (st, [P, C.POINTER(Residency), C.c_uint64, C.POINTER(C.c_uint64)]),
        "auvm_get_classes": (st, [P, C.POINTER(KernelClass), C.c_uint64, C.POINTER(C.c_uint64)]),
        "auvm_get_kernel_times": (st, [P, C.POINTER(C.c_float), C.POINTER(C.c_float), C.c_uint64,
                                       C.POINTER(C.c_uint64)]),
        "auvm_get_timeline": (st, [P, C.POINTER(TimelineEntry), C.c_uint64, C.POINTER(C.c_uint64)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


class Context:
    """One auvm_ctx.  hip_device < 0 gives a plan-only context.  library: a
    library bound with bind_library (default: this package's)."""

    def __init__(self, hip_device=-1, library=None):
        self._L = lib() if library is None else library
        h = C.c_void_p()
        s = self._L.auvm_create(int(hip_device), C.byref(h))
        if s != OK:
            raise AuvmError(s, "auvm_create failed")
        self._h = h

    def _check(self, s):
        if s != OK:
            raise AuvmError(s, self.last_error())
        return s

    def last_error(self):
        m = self._L.auvm_last_error(self._h)
        return m.decode() if m else ""

    def destroy(self):
        if getattr(self, "_h", None):
            self._L.auvm_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def arena_init(self, arena_bytes, host_pinned=None):
        self._check(self._L.auvm_arena_init(self._h, int(arena_bytes), host_pinned))

    def arena_init_tiered(self, arena_bytes, pinned_bytes):
        self._check(self._L.auvm_arena_init_tiered(self._h, int(arena_bytes), int(pinned_bytes)))

    def register_tensor(self, arena_off, nbytes, dtype, kind, flags=0):
        out = C.c_int32()
        self._check(self._L.auvm_register_tensor(self._h, int(arena_off), int(nbytes), int(dtype),
                                                 int(kind), int(flags), C.byref(out)))
        return out.value

    def tensor_host_ptr(self, tid):
        out = C.c_void_p()
        self._check(self._L.auvm_tensor_host_ptr(self._h, int(tid), C.byref(out)))
        return out.value

    def add_kernel(self, op, shape, operands, flops=0, hbm_bytes=0, layer=0):
        n = len(operands)
        ids = (C.c_int32 * n)(*[int(t) for t, _ in operands])
        modes = (C.c_uint8 * n)(*[int(m) for _, m in operands])
        sh = (C.c_int64 * 8)(*([int(x) for x in shape] + [0] * (8 - len(shape))))
        d = KernelDesc(int(op), sh, n, ids, modes, int(flops), int(hbm_bytes), int(layer))
        out = C.c_int32()
        self._check(self._L.auvm_add_kernel(self._h, C.byref(d), C.byref(out)))
        return out.value

    def set_budget(self, device_bytes, device_pool=None):
        self._check(self._L.auvm_set_budget(self._h, int(device_bytes), device_pool))

    def set_roofs(self, peak_flops, hbm_Bps, link_Bps):
        self._check(self._L.auvm_set_roofs(self._h, int(peak_flops), int(hbm_Bps), int(link_Bps)))

    def set_policy(self, variant=4, lookahead=0, affinity_w=1, placement=0, validate=0, timing=0,
                   guard=None, bucket=None, object_bytes=0):
        """guard / bucket None: the library applies its own default for the variant."""
        p = Policy(variant, lookahead, affinity_w, placement, validate, timing,
                   POLICY_DEFAULT if guard is None else guard, POLICY_DEFAULT if bucket is None else bucket,
                   int(object_bytes))
        self._check(self._L.auvm_set_policy(self._h, C.byref(p)))

    def plan(self):
        self._check(self._L.auvm_plan(self._h))

    def clear_kernels(self):
        """Drop the trace and the plan (tensors and arena stay); resets execution."""
        self._check(self._L.auvm_clear_kernels(self._h))

    def set_kernel_times(self, t_ns):
        """Measured time per kernel in integer ns (0: analytic class); drops the plan."""
        arr = (C.c_uint64 * max(1, len(t_ns)))(*[int(t) for t in t_ns])
        self._check(self._L.auvm_set_kernel_times(self._h, arr, len(t_ns)))

    def bind_streams(self, compute=None, h2d=None, d2h=None):
        self._check(self._L.auvm_bind_streams(self._h, compute, h2d, d2h))

    def run(self, first_k, n_k):
        self._check(self._L.auvm_run(self._h, int(first_k), int(n_k)))

    def run_noalloc(self, first_k, n_k):
        """run with the kernels' workspaces in the library's static device scratch."""
        self._check(self._L.auvm_run_noalloc(self._h, int(first_k), int(n_k)))

    def reset(self):
        self._check(self._L.auvm_reset(self._h))

    def read_tensor(self, tid, dst_ptr, dst_bytes):
        self._check(self._L.auvm_read_tensor(self._h, int(tid), dst_ptr, int(dst_bytes)))

    def get_counters(self):
        c = Counters()
        self._check(self._L.auvm_get_counters(self._h, C.byref(c)))
        return c.as_dict()

    def _array(self, fn, T):
        n = C.c_uint64()
        self._check(fn(self._h, None, 0, C.byref(n)))
        buf = (T * max(1, n.value))()
        self._check(fn(self._h, buf, n.value, C.byref(n)))
        return buf, n.value

    def get_schedule(self):
        buf, n = self._array(self._L.auvm_get_schedule, SchedEntry)
        return [(e.op, e.tensor, e.dev_off, e.bytes, e.issue_k, e.need_k) for e in buf[:n]]

    def get_executed(self):
        buf, n = self._array(self._L.auvm_get_executed, SchedEntry)
        return [(e.op, e.tensor, e.dev_off, e.bytes, e.issue_k, e.need_k) for e in buf[:n]]

    def get_residency(self):
        buf, n = self._array(self._L.auvm_get_residency, Residency)
        return [(r.k, r.n_resident, r.resident_bytes) for r in buf[:n]]

    def get_classes(self):
        buf, n = self._array(self._L.auvm_get_classes, KernelClass)
        return [(c.static_cls, c.dyn_cls, c.flops, c.hbm_bytes) for c in buf[:n]]

    def get_kernel_times(self):
        n = C.c_uint64()
        self._check(self._L.auvm_get_kernel_times(self._h, None, None, 0, C.byref(n)))
        dur = (C.c_float * max(1, n.value))()
        gap = (C.c_float * max(1, n.value))()
        self._check(self._L.auvm_get_kernel_times(self._h, dur, gap, n.value, C.byref(n)))
        return list(dur[:n.value]), list(gap[:n.value])

    def get_timeline(self):
        """(kind, segment, index, bytes, host_ms, start_ms, end_ms) per kernel or copy, in issue order."""
        buf, n = self._array(self._L.auvm_get_timeline, TimelineEntry)
        return [(e.kind, e.segment, e.index, e.bytes, e.host_ms, e.start_ms, e.end_ms) for e in buf[:n]]
