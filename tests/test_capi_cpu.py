"""CPU tests of the C-ABI library: exported symbols, argument checking, and
bit-exact agreement of the library's planner with the oracle replay."""
import os
import random
import re

import numpy as np
import pytest

import paper_2609_06172_amd as pkg
from paper_2609_06172_amd.capi import AuvmError, Context
from oracle import planner as op
from workloads import configs, trace
from workloads.format import (DT_BF16, DT_F32, DT_I32, DT_U8, KIND_ACT,
                              KIND_PARAM, MODE_R, MODE_RW, MODE_W, OP_LINEAR,
                              OP_TOUCH, PLACE_IDEAL, PLACE_POOL,
                              VAR_DEMAND_BELADY, VAR_DEMAND_LRU, VAR_T,
                              VAR_T_A, VAR_T_A_P)

from capi_util import assert_same_plan, plan_ctx
from planner_cases import golden_inputs, load_golden, random_trace

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "autouvm.h")


def test_library_exports_every_declared_symbol():
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(auvm_[a-z_]+)\s*\(", text))
    assert declared == set(pkg.SYMBOLS)
    L = pkg.lib()
    for name in declared:
        assert hasattr(L, name), name


def _tiny_ctx():
    ctx = Context(-1)
    ctx.arena_init(4096)
    a = ctx.register_tensor(0, 256, DT_U8, KIND_PARAM)
    b = ctx.register_tensor(256, 256, DT_U8, KIND_ACT)
    return ctx, a, b


def test_argument_errors():
    ctx, a, b = _tiny_ctx()
    with pytest.raises(AuvmError) as e:
        ctx.register_tensor(128, 256, DT_U8, KIND_PARAM)          # overlap
    assert e.value.code == -1
    with pytest.raises(AuvmError):
        ctx.register_tensor(3, 256, DT_U8, KIND_PARAM)            # unaligned
    with pytest.raises(AuvmError):
        ctx.register_tensor(3840, 512, DT_U8, KIND_PARAM)         # beyond the arena
    with pytest.raises(AuvmError) as e:
        ctx.add_kernel(OP_TOUCH, (0,), [(a, MODE_RW), (99, MODE_R)])  # unknown id
    assert e.value.code == -1
    with pytest.raises(AuvmError):
        ctx.add_kernel(77, (0,), [(a, MODE_RW)])                  # unknown op
    with pytest.raises(AuvmError):
        ctx.add_kernel(OP_TOUCH, (9,), [(a, MODE_RW), (b, MODE_R)])  # log slot too large
    with pytest.raises(AuvmError) as e:
        ctx.run(0, 1)                                             # plan-only context
    assert e.value.code == -2


def test_shape_validation_rejects_out_of_bounds_operands():
    ctx = Context(-1)
    ctx.arena_init(1 << 20)
    x = ctx.register_tensor(0, 16 * 64 * 2, DT_BF16, KIND_ACT, 1)
    W = ctx.register_tensor(4096, 32 * 64 * 2, DT_BF16, KIND_PARAM)
    c = ctx.register_tensor(12288, 16 * 32 * 2, DT_BF16, KIND_ACT)
    ctx.add_kernel(OP_LINEAR, (16, 32, 64), [(x, MODE_R), (W, MODE_R), (c, MODE_W)])
    with pytest.raises(AuvmError):       # N larger than the weight holds
        ctx.add_kernel(OP_LINEAR, (16, 64, 64), [(x, MODE_R), (W, MODE_R), (c, MODE_W)])
    with pytest.raises(AuvmError):       # K not a multiple of 32 for bf16
        ctx.add_kernel(OP_LINEAR, (16, 32, 48), [(x, MODE_R), (W, MODE_R), (c, MODE_W)])
    with pytest.raises(AuvmError):       # weight written
        ctx.add_kernel(OP_LINEAR, (16, 32, 64), [(x, MODE_R), (W, MODE_W), (c, MODE_W)])


def test_every_config_trace_is_accepted():
    for cfg in configs.CONFIGS.values():
        if cfg.name in ("llama-7b", "moe-8x14336"):
            continue          # covered (truncated) below
        w = trace.build(cfg)
        from paper_2609_06172_amd.session import Session
        s = Session(w, device=-1)
        assert len(s.ctx.get_classes()) == len(w.kernels)
        s.close()


@pytest.mark.parametrize("case", load_golden()["cases"], ids=lambda c: c["name"])
def test_golden_schedules_through_the_library(case):
    tensors, kernels = golden_inputs(case)
    # golden traces use plain touch ops without a log: give them one
    tensors = [dict(nbytes=64, dtype=DT_U8, kind=KIND_ACT, host_init=True)] + tensors
    ks = []
    for i, k in enumerate(kernels):
        ops = [(t + 1, m) for t, m in k["operands"]]
        ks.append(dict(op=OP_TOUCH, shape=(0,), operands=[(0, MODE_RW)] + ops, flops=k["flops"],
                       hbm_bytes=1, time_ns=k["time_ns"]))
    ob = case.get("object_bytes", 0)
    M = case["M"] + (768 if ob else 256)       # the log shares a block with a data tensor
    ctx = plan_ctx(tensors, ks, M, variant=case["variant"], affinity_w=case["affinity_w"],
                   placement=case["placement"], guard=case.get("guard"), bucket=case.get("bucket"),
                   object_bytes=ob)
    r = op.plan(tensors, ks, M, variant=case["variant"], affinity_w=case["affinity_w"],
                placement=case["placement"], guard=case.get("guard"), bucket=case.get("bucket"),
                object_bytes=ob)
    assert_same_plan(ctx, r)


@pytest.mark.parametrize("case", load_golden()["errors"], ids=lambda c: c["name"])
def test_golden_errors_through_the_library(case):
    tensors, kernels = golden_inputs(case)
    tensors = [dict(nbytes=64, dtype=DT_U8, kind=KIND_ACT, host_init=True)] + tensors
    ks = [dict(op=OP_TOUCH, shape=(0,), operands=[(0, MODE_RW)] + [(t + 1, m) for t, m in k["operands"]],
               flops=1, hbm_bytes=1) for k in kernels]
    with pytest.raises(AuvmError) as e:
        plan_ctx(tensors, ks, case["M"] + 256, variant=case["variant"])
    assert e.value.code == case["code"]


VARIANTS = [VAR_DEMAND_LRU, VAR_DEMAND_BELADY, VAR_T, VAR_T_A, VAR_T_A_P]


@pytest.mark.parametrize("seed", range(60))
def test_random_traces_bit_exact(seed):
    tensors, kernels = random_trace(seed, touch=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    rnd = random.Random(seed)
    for variant in VARIANTS:
        for placement in (PLACE_POOL, PLACE_IDEAL):
            M = max(1024, (fp * rnd.choice([1, 2, 3, 4]) // rnd.choice([2, 3, 4, 5])) // 256 * 256)
            kw = dict(variant=variant, placement=placement, affinity_w=rnd.choice([0, 1, 2, 3]),
                      lookahead=rnd.choice([0, 0, 1, 2, 5]), guard=rnd.choice([None, 0, 1, 3, 8]),
                      bucket=rnd.choice([None, 1, 2, 5, 40]))
            roofs = rnd.choice([None, (10**15, 10**13, 10**10), (10**9, 10**9, 10**9)])
            try:
                r = op.plan(tensors, kernels, M, roofs=roofs or op.DEFAULT_ROOFS, **kw)
            except op.PlanError as e:
                with pytest.raises(AuvmError) as ee:
                    plan_ctx(tensors, kernels, M, roofs=roofs, **kw)
                assert ee.value.code == e.code
                continue
            assert_same_plan(plan_ctx(tensors, kernels, M, roofs=roofs, **kw), r)


@pytest.mark.parametrize("name", ["tiny", "gpt-small", "llama-small", "gpt-1.3b", "train-small"])
@pytest.mark.parametrize("variant", VARIANTS)
def test_config_traces_bit_exact(name, variant):
    from paper_2609_06172_amd.session import Session
    cfg = configs.CONFIGS[name]
    w = trace.build(cfg)
    s = Session(w, device=-1, variant=variant)
    r = op.plan_workload(w, s.M, variant=variant)
    assert_same_plan(s.ctx, r)
    s.close()


@pytest.mark.parametrize("factor", [(5, 4), (3, 2), (2, 1)])
def test_llama7b_prefill_and_decode_bit_exact(factor):
    """The 7B-shape trace (prefill + 6 decode steps) at its full tensor sizes."""
    import dataclasses
    from paper_2609_06172_amd.session import Session
    cfg = dataclasses.replace(configs.LLAMA_7B, factor=factor)
    full = trace.build(cfg)
    M = full.budget()                    # budget from the whole 256-step job
    w = trace.build(dataclasses.replace(cfg, decode_steps=6))
    w_kernels = w.kernels
    # same tensors (gen rows differ): compare on the shorter trace with the full budget
    s = Session(w, device=-1, M=M)
    r = op.plan_workload(w, M)
    assert_same_plan(s.ctx, r)
    s.close()


def test_library_defines_every_kernel_launch_stub():
    """A kernel template whose host pass fails (a device-only builtin reachable
    from host-compiled code) loses its launch stub without a compile error; the
    library then fails to load on a GPU machine."""
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    path = pkg.lib()._name
    out = subprocess.run([nm, "-D", "--undefined-only", path], capture_output=True, text=True, check=True).stdout
    missing = [l.split()[-1] for l in out.splitlines() if "__device_stub__" in l]
    assert not missing, missing


@pytest.mark.parametrize("seed", range(40))
def test_random_timed_traces_bit_exact(seed):
    # per-kernel measured times (auvm_set_kernel_times) take the oracle's rule
    tensors, kernels = random_trace(seed, touch=True, timed=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    rnd = random.Random(1000 + seed)
    for variant in VARIANTS:
        M = max(1024, (fp * rnd.choice([1, 2, 3]) // rnd.choice([2, 3, 4])) // 256 * 256)
        kw = dict(variant=variant, affinity_w=rnd.choice([0, 1, 2]), guard=rnd.choice([None, 0, 3]))
        try:
            r = op.plan(tensors, kernels, M, **kw)
        except op.PlanError as e:
            with pytest.raises(AuvmError) as ee:
                plan_ctx(tensors, kernels, M, **kw)
            assert ee.value.code == e.code
            continue
        assert_same_plan(plan_ctx(tensors, kernels, M, **kw), r)


def test_set_kernel_times_checks_its_length_and_replans():
    tensors, kernels = random_trace(3, touch=True, timed=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    M = max(1024, fp * 3 // 4 // 256 * 256)
    untimed = [dict(k, time_ns=0) for k in kernels]
    ctx = plan_ctx(tensors, untimed, M)
    with pytest.raises(AuvmError) as e:
        ctx.set_kernel_times([1] * (len(kernels) - 1))
    assert e.value.code == op.E_INVAL
    with pytest.raises(AuvmError):
        ctx.set_kernel_times([1] * (len(kernels) + 1))
    ctx.set_kernel_times([k.get("time_ns", 0) for k in kernels])
    ctx.plan()
    assert_same_plan(ctx, op.plan(tensors, kernels, M))
    ctx.set_kernel_times([0] * len(kernels))        # back to the analytic classes
    ctx.plan()
    assert_same_plan(ctx, op.plan(tensors, untimed, M))
    ctx.destroy()


@pytest.mark.parametrize("name", ["gpt-small", "llama-small", "gpt-1.3b"])
def test_config_traces_with_measured_times_bit_exact(name):
    # times scattered around the link time of each kernel's read operands, so
    # that kernels change class both ways
    from paper_2609_06172_amd.session import Session
    cfg = configs.CONFIGS[name]
    w = trace.build(cfg)
    s = Session(w, device=-1)
    _, _, Bl = op.DEFAULT_ROOFS
    rnd = random.Random(7)
    times = []
    for k in w.kernels:
        X = sum(op.aligned(w.tensors[t].nbytes) for t, m in k.operands if m & MODE_R)
        times.append(max(1, int(X * 10**9 // Bl * rnd.choice([0.3, 0.9, 1.1, 3.0]))))
    s.replan_measured(times)
    r = op.plan_workload(w, s.M, times=times)
    assert_same_plan(s.ctx, r)
    base = op.plan_workload(w, s.M)
    assert any(a != b for a, b in zip(r.static_cls, base.static_cls))
    assert r.schedule != base.schedule
    s.close()


# ------------------------------------------------------- routed experts (MoE)
@pytest.mark.parametrize("variant", VARIANTS)
def test_moe_traces_bit_exact(variant):
    from planner_cases import oracle_routing_counts
    from paper_2609_06172_amd.session import Session
    cfg = configs.MOE_SMALL
    counts = oracle_routing_counts(cfg)
    for routing in (None, counts):
        w = trace.build(cfg, routing)
        s = Session(w, device=-1, variant=variant)
        assert_same_plan(s.ctx, op.plan_workload(w, s.M, variant=variant))
        s.close()


def test_full_shape_moe_trace_bit_exact_and_retrace():
    # the 8 x 14336 trace, prefill + 2 decode steps, under a seeded random routing
    import dataclasses
    from planner_cases import random_routing_counts
    from paper_2609_06172_amd.session import Session
    cfg = dataclasses.replace(configs.MOE_8X, decode_steps=2)
    full = trace.build(cfg)
    routed = trace.build(cfg, random_routing_counts(cfg, 5))
    assert len(routed.kernels) < len(full.kernels)
    s = Session(full, device=-1)
    s.retrace(routed)                    # the profiling trace swapped for the routed one
    assert_same_plan(s.ctx, op.plan_workload(routed, s.M))
    s.close()


def test_routed_trace_moves_only_routed_experts():
    # the profiling trace (every expert) against the recorded one: the same
    # kernels run, but unrouted experts' weights are never fetched
    from planner_cases import oracle_routing_counts
    cfg = configs.MOE_SMALL
    counts = oracle_routing_counts(cfg)
    assert (counts == 0).any()            # some expert idles in some decode layer
    full, routed = trace.build(cfg), trace.build(cfg, counts)
    M = full.budget()
    a, b = op.plan_workload(full, M), op.plan_workload(routed, M)
    fa = a.counters["h2d_prefetch_B"] + a.counters["h2d_demand_B"]
    fb = b.counters["h2d_prefetch_B"] + b.counters["h2d_demand_B"]
    assert fb < fa
    # every weight fetched under the routed trace belongs to a routed expert
    names = {t.tid: t.name for t in routed.tensors}
    routed_experts = set()
    for seg in range(counts.shape[0]):
        for l in range(cfg.n_layers):
            routed_experts |= {f"L{l}.x{e}." for e in np.nonzero(counts[seg, l])[0]}
    for e in b.schedule:
        if e[0] in (0, 1) and ".x" in names[e[1]]:
            assert names[e[1]].rsplit(".", 1)[0] + "." in routed_experts


def test_moe_op_validation():
    from workloads.format import OP_MOE_DISPATCH, OP_MOE_DOWN, OP_MOE_ROUTE, OP_MOE_UP
    ctx = Context(-1)
    ctx.arena_init(1 << 24)
    off = [0]

    def t(nbytes, dt, kind=KIND_ACT):
        i = ctx.register_tensor(off[0], nbytes, dt, kind, 1 if kind != KIND_PARAM else 0)
        off[0] += (nbytes + 255) // 256 * 256
        return i
    M, H, F, E, K = 32, 128, 192, 4, 2
    h = t(M * H * 2, DT_BF16)
    wr = t(E * H * 2, DT_BF16, KIND_PARAM)
    rte, rtw = t(M * K * 4, DT_I32), t(M * K * 4, DT_F32)
    lists, log = t(E * (M + 1) * 4, DT_I32), t(3 * E * 4, DT_I32)
    wg, wu, wd = t(F * H * 2, DT_BF16, KIND_PARAM), t(F * H * 2, DT_BF16, KIND_PARAM), t(H * F * 2, DT_BF16, KIND_PARAM)
    fe, x = t(M * F * 2, DT_BF16), t(M * H * 4, DT_F32)
    R, W = MODE_R, MODE_W
    ctx.add_kernel(OP_MOE_ROUTE, (M, H, E, K), [(h, R), (wr, R), (rte, W), (rtw, W)])
    ctx.add_kernel(OP_MOE_DISPATCH, (M, E, K, 2), [(rte, R), (lists, W), (log, MODE_RW)])
    ctx.add_kernel(OP_MOE_UP, (M, F, H, 3, M, K), [(h, R), (lists, R), (wg, R), (wu, R), (fe, W)])
    ctx.add_kernel(OP_MOE_DOWN, (M, H, F, 3, 5, K), [(fe, R), (lists, R), (rtw, R), (wd, R), (x, MODE_RW)])
    bad = [
        (OP_MOE_ROUTE, (M, H, E, 5), [(h, R), (wr, R), (rte, W), (rtw, W)]),            # K > E
        (OP_MOE_ROUTE, (M, H, 17, 2), [(h, R), (wr, R), (rte, W), (rtw, W)]),           # E > 16
        (OP_MOE_ROUTE, (M, 124, E, K), [(h, R), (wr, R), (rte, W), (rtw, W)]),          # H % 8
        (OP_MOE_DISPATCH, (M, E, K, 3), [(rte, R), (lists, W), (log, MODE_RW)]),         # log row beyond
        (OP_MOE_DISPATCH, (M, E, K, 1), [(rte, R), (lists, W), (log, W)]),               # log must be RW
        (OP_MOE_UP, (M, F, H, 4, M, K), [(h, R), (lists, R), (wg, R), (wu, R), (fe, W)]),   # expert beyond lists
        (OP_MOE_UP, (M, F, H, 0, M + 1, K), [(h, R), (lists, R), (wg, R), (wu, R), (fe, W)]),  # n > M
        (OP_MOE_UP, (M, F, 96, 0, M, K), [(h, R), (lists, R), (wg, R), (wu, R), (fe, W)]),  # K % 64
        (OP_MOE_DOWN, (M, H, F, 0, M, K), [(fe, R), (lists, R), (rtw, R), (wd, R), (x, W)]),  # x must be RW
    ]
    for o, sh, ops in bad:
        with pytest.raises(AuvmError) as e:
            ctx.add_kernel(o, sh, ops)
        assert e.value.code == op.E_INVAL, (o, sh)
    ctx.destroy()


def test_training_step_trace_bit_exact():
    # the 13B-shape training step, two layers, under the full method
    import dataclasses
    from paper_2609_06172_amd.session import Session
    cfg = dataclasses.replace(configs.LLAMA_13B_TRAIN, n_layers=2)
    w = trace.build(cfg)
    s = Session(w, device=-1)
    assert_same_plan(s.ctx, op.plan_workload(w, s.M))
    s.close()


@pytest.mark.parametrize("seed", range(30))
def test_random_live_out_traces_bit_exact(seed):
    tensors, kernels = random_trace(100 + seed, touch=True, live_out=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    rnd = random.Random(seed)
    for variant in VARIANTS:
        M = max(1024, (fp * rnd.choice([1, 2, 3]) // rnd.choice([2, 3, 4])) // 256 * 256)
        try:
            r = op.plan(tensors, kernels, M, variant=variant)
        except op.PlanError as e:
            with pytest.raises(AuvmError) as ee:
                plan_ctx(tensors, kernels, M, variant=variant)
            assert ee.value.code == e.code
            continue
        assert_same_plan(plan_ctx(tensors, kernels, M, variant=variant), r)


def test_linear_qkv_validation_and_cost():
    """LINEAR_QKV: three LINEARs of one input.  Its cost is theirs with the
    shared input read once; malformed operand lists are rejected."""
    from oracle.costs import kernel_cost
    from workloads.format import DT_SIZE, OP_LINEAR_QKV
    M, N, K = 16, 64, 96
    ctx = Context(-1)
    ctx.arena_init(1 << 22)
    off = [0]

    def t(nbytes, dt, kind=KIND_ACT):
        i = ctx.register_tensor(off[0], nbytes, dt, kind, 1 if kind != KIND_PARAM else 0)
        off[0] += (nbytes + 255) // 256 * 256
        return i
    a = t(M * K * 2, DT_BF16)
    wq, wk, wv = (t(N * K * 2, DT_BF16, KIND_PARAM) for _ in range(3))
    q, k, v = (t(M * N * 2, DT_BF16) for _ in range(3))
    w32 = t(N * K * 4, DT_F32, KIND_PARAM)
    q32 = t(M * N * 4, DT_F32)
    small = t(N * K, DT_BF16, KIND_PARAM)
    R, W = MODE_R, MODE_W
    good = [(a, R), (wq, R), (wk, R), (wv, R), (q, W), (k, W), (v, W)]
    ctx.add_kernel(OP_LINEAR_QKV, (M, N, K), good)

    def swap(i, e):
        ops = list(good)
        ops[i] = e
        return ops
    bad = [
        good[:6],                                # six operands
        swap(5, (q, W)),                         # k is q
        swap(6, (a, W)),                         # v is the input
        swap(2, (wk, W)),                        # a weight written
        swap(3, (w32, R)),                       # weight dtype differs from a
        swap(5, (q32, W)),                       # k's dtype differs from q's
        swap(3, (small, R)),                     # Wv too small for N x K
    ]
    for ops in bad:
        with pytest.raises(AuvmError) as e:
            ctx.add_kernel(OP_LINEAR_QKV, (M, N, K), ops)
        assert e.value.code == op.E_INVAL, ops
    with pytest.raises(AuvmError):               # bf16 needs K % 32 == 0
        ctx.add_kernel(OP_LINEAR_QKV, (M, N, 80), good)
    ctx.destroy()
    dtypes = {i: DT_BF16 for i in range(7)}
    nbytes = {i: 0 for i in range(7)}
    ops = [(i, m) for i, (_, m) in enumerate(good)]
    F3, B3 = kernel_cost(OP_LINEAR_QKV, (M, N, K), ops, dtypes, nbytes)
    F1, B1 = kernel_cost(OP_LINEAR, (M, N, K), [(0, R), (1, R), (4, W)], dtypes, nbytes)
    assert F3 == 3 * F1 == 6 * M * N * K
    assert B3 == 3 * B1 - 2 * M * K * DT_SIZE[DT_BF16]


def test_separate_qkv_trace_bit_exact():
    """The three-kernel q, k, v trace plans in the library exactly as in the oracle."""
    import dataclasses
    from paper_2609_06172_amd.session import Session
    cfg = dataclasses.replace(configs.LLAMA_SMALL, fuse_qkv=False)
    w = trace.build(cfg)
    for variant in VARIANTS:
        s = Session(w, device=-1, variant=variant)
        assert_same_plan(s.ctx, op.plan_workload(w, s.M, variant=variant))
        s.close()


@pytest.mark.parametrize("variant", VARIANTS)
def test_the_library_applies_its_own_policy_defaults(variant):
    """guard and bucket left unset travel as AUVM_POLICY_DEFAULT, and the
    library's defaults for the variant plan exactly what the oracle's do."""
    from paper_2609_06172_amd import capi
    seen = {}
    real = capi.Policy

    class Spy(real):
        def __init__(self, *a):
            super().__init__(*a)
            seen["guard"], seen["bucket"] = self.guard, self.bucket
    capi.Policy = Spy
    try:
        tensors, kernels = random_trace(4242 + variant, touch=True)
        fp = sum(op.aligned(t["nbytes"]) for t in tensors)
        for num, den in ((1, 2), (2, 3), (3, 4), (5, 6), (1, 1)):
            M = max(1024, fp * num // den // 256 * 256)
            try:
                ref = op.plan(tensors, kernels, M, variant=variant)
                break
            except op.PlanError:
                continue
        ctx = plan_ctx(tensors, kernels, M, variant=variant)
    finally:
        capi.Policy = real
    assert seen == {"guard": capi.POLICY_DEFAULT, "bucket": capi.POLICY_DEFAULT}
    assert_same_plan(ctx, ref)


@pytest.mark.parametrize("seed", range(40))
def test_object_granularity_bit_exact(seed):
    """Blocks of a pooling allocator (object_bytes > 0), every variant: the
    library's expanded member schedule, residency, classes and counters
    (useless member fetches included) equal the oracle's, and the schedule
    passes the checker."""
    from oracle import checker
    tensors, kernels = random_trace(seed, touch=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    rnd = random.Random(9000 + seed)
    for variant in VARIANTS:
        ob = rnd.choice([512, 2048, 4096, 16384])
        for num, den in ((1, 1), (5, 6), (3, 4), (2, 3)):
            M = max(1024, fp * num // den // 256 * 256)
            try:
                r = op.plan(tensors, kernels, M, variant=variant, object_bytes=ob)
            except op.PlanError as e:
                with pytest.raises(AuvmError) as x:
                    plan_ctx(tensors, kernels, M, variant=variant, object_bytes=ob)
                assert x.value.code == e.code
                continue
            checker.check(tensors, kernels, M, r.schedule)
            assert_same_plan(plan_ctx(tensors, kernels, M, variant=variant, object_bytes=ob), r)


@pytest.mark.parametrize("name", ["llama-small", "gpt-small", "moe-small", "train-small"])
def test_object_granularity_config_traces(name):
    from oracle import checker
    cfg = configs.CONFIGS[name]
    w = trace.build(cfg)
    tensors = [dict(nbytes=t.nbytes, dtype=t.dtype, kind=t.kind, host_init=t.host_init, live_out=t.live_out)
               for t in w.tensors]
    kernels = [dict(op=k.op, shape=k.shape, operands=k.operands) for k in w.kernels]
    ob = 1 << 20
    try:
        r = op.plan(tensors, kernels, w.budget(), object_bytes=ob)
    except op.PlanError:
        r = None
    if r is None:
        pytest.skip("blocks do not fit the budget")
    checker.check(tensors, kernels, w.budget(), r.schedule)
    assert_same_plan(plan_ctx(tensors, kernels, w.budget(), object_bytes=ob), r)


@pytest.mark.parametrize("seed", range(40))
def test_kv_tensors_bit_exact(seed):
    """Traces with KV-cache tensors, whose first writes pack at the top of
    the pool under farthest-next-use victims: the library plans exactly what
    the oracle plans, and the checker accepts it."""
    from oracle import checker
    tensors, kernels = random_trace(seed, touch=True, kv=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    rnd = random.Random(7000 + seed)
    for variant in VARIANTS:
        for num, den in ((1, 2), (2, 3), (5, 6)):
            M = max(1024, fp * num // den // 256 * 256)
            kw = dict(variant=variant, guard=rnd.choice([None, 0, 3]), bucket=rnd.choice([None, 1, 8]))
            try:
                r = op.plan(tensors, kernels, M, **kw)
            except op.PlanError as e:
                with pytest.raises(AuvmError) as x:
                    plan_ctx(tensors, kernels, M, **kw)
                assert x.value.code == e.code
                continue
            checker.check(tensors, kernels, M, r.schedule)
            assert_same_plan(plan_ctx(tensors, kernels, M, **kw), r)
