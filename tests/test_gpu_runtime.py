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
