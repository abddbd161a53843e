"""Pins of the oracle planner: hand-derived schedules, closed forms, exhaustive
search, the schedule checker and the limits of the roofline gate."""
import dataclasses
import itertools
import random

import pytest

from oracle import brute, checker
from oracle import planner as op
from workloads import configs, trace
from workloads.format import (CLS_CGI, CLS_COMPUTE, CLS_MEMORY, DT_U8,
                              KIND_PARAM, OP_LINEAR, OP_TOUCH, PLACE_IDEAL,
                              PLACE_POOL, S_D2H_WRITEBACK, S_DROP,
                              S_H2D_DEMAND, S_H2D_PREFETCH, S_LAUNCH,
                              VAR_DEMAND_BELADY, VAR_DEMAND_LRU, VAR_T,
                              VAR_T_A, VAR_T_A_P)

from planner_cases import golden_inputs, load_golden, random_trace

VARIANTS = [VAR_DEMAND_LRU, VAR_DEMAND_BELADY, VAR_T, VAR_T_A, VAR_T_A_P]


@pytest.mark.parametrize("case", load_golden()["cases"], ids=lambda c: c["name"])
def test_golden_schedules(case):
    tensors, kernels = golden_inputs(case)
    r = op.plan(tensors, kernels, case["M"], variant=case["variant"],
                affinity_w=case["affinity_w"], placement=case["placement"], guard=case.get("guard"),
                bucket=case.get("bucket"), object_bytes=case.get("object_bytes", 0))
    assert [list(e) for e in r.schedule] == case["schedule"]
    if "residency" in case:
        assert [list(e) for e in r.residency] == case["residency"]
    if "dyn_cls" in case:
        assert r.dyn_cls == case["dyn_cls"]
    if "static_cls" in case:
        assert r.static_cls == case["static_cls"]
    for k, v in case.get("counters", {}).items():
        assert r.counters[k] == v, k
    checker.check(tensors, kernels, case["M"], r.schedule)


@pytest.mark.parametrize("case", load_golden()["errors"], ids=lambda c: c["name"])
def test_golden_errors(case):
    tensors, kernels = golden_inputs(dict(case, kernels=case["kernels"]))
    with pytest.raises(op.PlanError) as e:
        op.plan(tensors, kernels, case["M"], variant=case["variant"])
    assert e.value.code == case["code"]


def test_classify_hand_examples():
    roofs = op.DEFAULT_ROOFS          # P = 2.5e15, Bh = 8e12, Bl = 6.4e10
    # GEMM 4096^3: F/B = 2*4096^3 / (3*4096^2*2) = 1365 flop/B > 312.5 ridge
    F, B = 2 * 4096 ** 3, 3 * 4096 * 4096 * 2
    assert op.classify(F, B, 0, roofs) == CLS_COMPUTE
    # weight of 32 MiB missing: link 0.52 ms > compute 0.055 ms and HBM 12.6 us
    assert op.classify(F, B, 4096 * 4096 * 2, roofs) == CLS_CGI
    # decode GEMV 16x4096x4096: intensity 16 < 312.5
    F2, B2 = 2 * 16 * 4096 * 4096, 4096 * 4096 * 2 + 2 * 16 * 4096 * 2
    assert op.classify(F2, B2, 0, roofs) == CLS_MEMORY
    # a missing 8 KB gain on a 268 MB prefill norm: X/B below Bl/Bh, not CGI
    assert op.classify(4 * 16384 * 4096, 268_443_648, 8192, roofs) == CLS_MEMORY
    # exact ties are not CGI and go to COMPUTE
    assert op.classify(8, 8, 1, (1, 1, 8)) == CLS_COMPUTE      # X*P == F*Bl
    assert op.classify(1, 1, 0, (1, 1, 1)) == CLS_COMPUTE      # F*Bh == B*P


def _sched_counts(r):
    c = {}
    for e in r.schedule:
        c[e[0]] = c.get(e[0], 0) + 1
    return c


@pytest.mark.parametrize("seed", range(40))
def test_random_schedules_are_valid(seed):
    tensors, kernels = random_trace(seed)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    rnd = random.Random(seed)
    for variant in VARIANTS:
        for placement in (PLACE_POOL, PLACE_IDEAL):
            M = max(256, (fp * rnd.choice([1, 2, 3]) // rnd.choice([2, 3, 4, 5])) // 256 * 256)
            try:
                r = op.plan(tensors, kernels, M, variant=variant, placement=placement,
                            affinity_w=rnd.choice([0, 1, 2]), lookahead=rnd.choice([0, 1, 3]))
            except op.PlanError as e:
                if variant == VAR_T_A_P and placement == PLACE_IDEAL:
                    assert e.code == op.E_INVAL
                else:
                    assert e.code in (op.E_BUDGET, op.E_FRAG)
                continue
            checker.check(tensors, kernels, M, r.schedule, pool=(placement == PLACE_POOL))
            assert all(rb <= M for _, _, rb in r.residency)
            assert len(r.residency) == len(kernels)


def test_checker_catches_planted_mistakes():
    case = load_golden()["cases"][3]            # contains a writeback
    tensors, kernels = golden_inputs(case)
    good = [tuple(e) for e in case["schedule"]]
    checker.check(tensors, kernels, case["M"], good)
    wb = next(i for i, e in enumerate(good) if e[0] == S_D2H_WRITEBACK)
    bad = list(good)
    bad[wb] = (S_DROP,) + bad[wb][1:]           # lose a live dirty value
    with pytest.raises(checker.ScheduleError):
        checker.check(tensors, kernels, case["M"], bad)
    bad = [e for e in good if not (e[0] == S_H2D_PREFETCH and e[1] == 3)]
    with pytest.raises(checker.ScheduleError):     # operand missing at launch
        checker.check(tensors, kernels, case["M"], bad)
    bad = list(good)
    i = next(i for i, e in enumerate(good) if e[0] == S_H2D_PREFETCH)
    bad[i] = bad[i][:2] + (bad[i][2] + 256,) + bad[i][3:]
    with pytest.raises(checker.ScheduleError):     # overlapping / out-of-pool window
        checker.check(tensors, kernels, case["M"], bad)


@pytest.mark.parametrize("seed", range(15))
def test_no_pressure_is_compulsory_fetches_only(seed):
    tensors, kernels = random_trace(seed)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    read_host = set()
    state = {t: tensors[t]["host_init"] or tensors[t]["kind"] == KIND_PARAM
             for t in range(len(tensors))}
    for kd in kernels:          # distinct host tensors read before being overwritten
        merged = op.merge_operands(kd["operands"])
        for t, m in merged:
            if (m & 1) and state[t] is True:
                read_host.add(t)
            state[t] = "dev"
    for variant in VARIANTS:
        r = op.plan(tensors, kernels, fp, variant=variant)
        c = _sched_counts(r)
        assert c.get(S_DROP, 0) == 0 and c.get(S_D2H_WRITEBACK, 0) == 0
        n_h2d = c.get(S_H2D_DEMAND, 0) + c.get(S_H2D_PREFETCH, 0)
        assert n_h2d == len(read_host)


def _cyclic(n, cycles):
    tensors = [dict(nbytes=256, dtype=DT_U8, kind=KIND_PARAM, host_init=True) for _ in range(n)]
    kernels = [dict(op=OP_TOUCH, shape=(0,), operands=[(k % n, 1)], flops=1, hbm_bytes=1)
               for k in range(n * cycles)]
    return tensors, kernels


@pytest.mark.parametrize("n,c", [(3, 2), (5, 3), (8, 7), (6, 2)])
def test_lru_cyclic_pathology(n, c):
    tensors, kernels = _cyclic(n, 6)
    for placement in (PLACE_IDEAL, PLACE_POOL):
        r = op.plan(tensors, kernels, c * 256, variant=VAR_DEMAND_LRU, placement=placement)
        assert r.counters["h2d_demand_n"] == len(kernels)     # every access misses


@pytest.mark.parametrize("seed", range(60))
def test_demand_belady_is_optimal(seed):
    rnd = random.Random(1000 + seed)
    n = rnd.randint(2, 8)
    tensors, kernels = random_trace(seed, n_tensors=n, n_kernels=rnd.randint(4, 24),
                                    max_ops=2, equal=True, read_only=True)
    cap = rnd.randint(2, n)
    acc = [set(t for t, _ in k["operands"]) for k in kernels]
    opt = brute.min_demand_fetches(acc, cap)
    for placement in (PLACE_IDEAL, PLACE_POOL):
        r = op.plan(tensors, kernels, cap * 256, variant=VAR_DEMAND_BELADY,
                    affinity_w=0, placement=placement)
        assert r.counters["h2d_demand_n"] == opt
    # LRU is never better than the optimum
    r = op.plan(tensors, kernels, cap * 256, variant=VAR_DEMAND_LRU, placement=PLACE_IDEAL)
    assert r.counters["h2d_demand_n"] >= opt


def test_belady_cyclic_rate():
    # cyclic access of n equal pages with c frames: the optimum misses
    # (n-c)/(n-1) of the accesses in steady state
    n, c, cycles = 7, 4, 40
    tensors, kernels = _cyclic(n, cycles)
    r = op.plan(tensors, kernels, c * 256, variant=VAR_DEMAND_BELADY, affinity_w=0,
                placement=PLACE_IDEAL)
    misses = r.counters["h2d_demand_n"]
    steady = (n * cycles - n) * (n - c) / (n - 1)
    assert abs(misses - n - steady) <= n


@pytest.mark.parametrize("seed", range(20))
def test_gate_limits(seed):
    tensors, kernels = random_trace(seed)
    for kd in kernels:          # analytic costs everywhere: B >= X / 125000 holds
        kd["flops"], kd["hbm_bytes"] = 0, 0
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    M = max(256, fp // 2 // 256 * 256)
    fast_link = (op.DEFAULT_ROOFS[0], op.DEFAULT_ROOFS[1], 10 ** 18)
    try:
        a = op.plan(tensors, kernels, M, roofs=fast_link, variant=VAR_T_A_P, affinity_w=0, guard=0,
                    bucket=1)
        b = op.plan(tensors, kernels, M, roofs=fast_link, variant=VAR_DEMAND_BELADY, affinity_w=0)
    except op.PlanError:
        return
    assert a.counters["h2d_prefetch_n"] == 0
    assert a.schedule == b.schedule
    assert CLS_CGI not in a.dyn_cls
    slow_link = (op.DEFAULT_ROOFS[0], op.DEFAULT_ROOFS[1], 1)
    try:
        c = op.plan(tensors, kernels, M, roofs=slow_link, variant=VAR_T_A_P)
    except op.PlanError:
        return
    for k, kd in enumerate(kernels):
        reads = [t for t, m in op.merge_operands(kd["operands"]) if m & 1]
        assert (c.static_cls[k] == CLS_CGI) == (len(reads) > 0)


def test_plan_is_deterministic():
    tensors, kernels = random_trace(7)
    M = sum(op.aligned(t["nbytes"]) for t in tensors) * 9 // 10 // 256 * 256
    a = op.plan(tensors, kernels, M)
    b = op.plan(tensors, kernels, M)
    assert a.schedule == b.schedule and a.counters == b.counters
    assert a.counters["h2d_prefetch_n"] > 0


def test_ablation_ladder_directions_on_cyclic_decoder():
    """On a decode-like cyclic trace the full method moves no more bytes than
    demand LRU and never stalls a launch on a demand fetch in steady state."""
    cfg = configs.LLAMA_SMALL
    w = trace.build(cfg)
    M = w.budget()
    r_lru = op.plan_workload(w, M, variant=VAR_DEMAND_LRU)
    r_tap = op.plan_workload(w, M, variant=VAR_T_A_P)
    h2d = lambda r: r.counters["h2d_prefetch_B"] + r.counters["h2d_demand_B"]
    assert h2d(r_tap) <= h2d(r_lru)
    checker.check_workload(w, M, r_tap.schedule)
    checker.check_workload(w, M, r_lru.schedule)
    # L_min: per decode step at least (persistent bytes read per step - M) must move
    k0, n = w.segments["decode"][-2]
    first = {}                  # tensors whose first access in the step reads them
    for kd in w.kernels[k0:k0 + n]:
        for t, m in op.merge_operands(kd.operands):
            first.setdefault(t, m)
    persistent = sum(op.aligned(w.tensors[t].nbytes) for t, m in first.items() if m & 1)
    lmin = max(0, persistent - M)
    moved = sum(e[3] for e in r_tap.schedule
                if e[0] in (S_H2D_DEMAND, S_H2D_PREFETCH) and k0 <= e[4] < k0 + n)
    assert moved >= lmin


def test_link_lower_bound_hand_derived():
    """The benchmark's link bound on two hand-built units of 256-byte tensors
    (TOUCH kernels stand for any op; only the access modes matter).

    Unit 1, M = 768: every kernel also reads and writes a 256-byte log; k0
    writes a, k1 reads a and writes b, k2 reads a, b and the host-initialised
    c.  Before k2 all four are needed (1024 B): 256 B must be fetched; the
    unit writes the log, a and b but not c, so the shortfall can be met by c
    alone and no write-back is forced.  Before k1 the log, a and c are
    needed (b is written there): 768 B, no shortfall.  Bound (256, 0).

    Unit 2, M = 256: k0 writes a, k1 writes b, k2 reads a and b.  Before k2,
    512 B are needed, both written by the unit: 256 B must come back, and in
    a repeated unit they were rewritten since, so 256 B were written back.
    Bound (256, 256)."""
    import bench
    from workloads.format import MODE_R, MODE_RW, MODE_W
    w = trace.Workload(None)
    a = w.tensor("a", (256,), DT_U8, 1)
    b = w.tensor("b", (256,), DT_U8, 1)
    c = w.tensor("c", (256,), DT_U8, 1, host_init=True)
    log = w.tensor("log", (64,), DT_U8, 1)
    w.kernel(OP_TOUCH, (0,), [(log, MODE_RW), (a, MODE_W)])
    w.kernel(OP_TOUCH, (0,), [(log, MODE_RW), (a, MODE_R), (b, MODE_W)])
    w.kernel(OP_TOUCH, (0,), [(log, MODE_RW), (a, MODE_R), (b, MODE_R), (c, MODE_R)])
    assert bench.link_lower_bound(w, 0, 3, 512 + 256) == (256, 0)
    w2 = trace.Workload(None)
    a = w2.tensor("a", (256,), DT_U8, 1)
    b = w2.tensor("b", (256,), DT_U8, 1)
    w2.kernel(OP_TOUCH, (0,), [(a, MODE_W)])
    w2.kernel(OP_TOUCH, (0,), [(b, MODE_W)])
    w2.kernel(OP_TOUCH, (0,), [(a, MODE_R), (b, MODE_R)])
    assert bench.link_lower_bound(w2, 0, 3, 256) == (256, 256)
    # a larger budget removes both; a smaller one grows both by the same bytes
    assert bench.link_lower_bound(w2, 0, 3, 512) == (0, 0)
    assert bench.link_lower_bound(w2, 0, 3, 0) == (512, 512)


@pytest.mark.parametrize("name", ["train-small", "llama-small"])
def test_link_lower_bound_holds_for_every_variant(name):
    """The benchmark's link bound per repeated unit (training step, decode
    step) is met by every policy: H2D and D2H both at least the bound, and
    for training the write-back part is not trivially zero."""
    import bench
    cfg = dataclasses.replace(configs.CONFIGS[name], iterations=4) if name == "train-small" \
        else configs.CONFIGS[name]
    w = trace.build(cfg)
    M = w.budget()
    seg = "step" if name == "train-small" else "decode"
    units = w.segments[seg][1:-1]
    bounds = [bench.link_lower_bound(w, a, n, M) for a, n in units]
    assert all(b[0] > 0 for b in bounds)
    if name == "train-small":
        assert all(b[1] > 0 for b in bounds)
    else:
        assert all(b[1] == 0 for b in bounds)      # weights are never written at decode
    for variant in (VAR_DEMAND_LRU, VAR_DEMAND_BELADY, VAR_T_A_P):
        r = op.plan_workload(w, M, variant=variant)
        for (a, n), (h_min, d_min) in zip(units, bounds):
            h2d = sum(e[3] for e in r.schedule if e[0] in (S_H2D_DEMAND, S_H2D_PREFETCH) and a <= e[4] < a + n)
            d2h = sum(e[3] for e in r.schedule if e[0] == S_D2H_WRITEBACK and a <= e[4] < a + n)
            assert h2d >= h_min and d2h >= d_min, (variant, a, h2d, h_min, d2h, d_min)


# ---- measured kernel times (the runtime monitor's re-classification, Sec. IV)

def test_classify_measured_time_closed_form():
    roofs = op.DEFAULT_ROOFS          # Bl = 6.4e10 B/s: 64 bytes per ns on the link
    # link time of X bytes vs the measured time: a tie is not CGI
    assert op.classify(1, 1, 64_000, roofs, 1000) != CLS_CGI
    assert op.classify(1, 1, 64_001, roofs, 1000) == CLS_CGI
    # nothing missing is never CGI, however short the kernel
    assert op.classify(1, 1, 0, roofs, 1) == CLS_MEMORY
    # a measured time overrides the analytic roofs either way: a huge GEMM
    # (analytically COMPUTE) that ran in 1 us while 1 MB was missing ...
    F, B = 2 * 4096 ** 3, 3 * 4096 * 4096 * 2
    assert op.classify(F, B, 1 << 20, roofs) == CLS_COMPUTE
    assert op.classify(F, B, 1 << 20, roofs, 1000) == CLS_CGI
    # ... and a 1-flop kernel missing 32 MiB (analytically CGI) that took a second
    assert op.classify(1, 1, 32 << 20, roofs) == CLS_CGI
    assert op.classify(1, 1, 32 << 20, roofs, 10**9) == CLS_MEMORY
    # below the link time the fallback is the plain roofline comparison
    assert op.classify(F, B, 1 << 20, roofs, 10**9) == CLS_COMPUTE


def _with_times(kernels, t):
    return [dict(k, time_ns=t(i)) for i, k in enumerate(kernels)]


@pytest.mark.parametrize("seed", range(25))
def test_huge_times_leave_the_demand_timeline(seed):
    # no kernel is CGI when every kernel took longer than any transfer, so the
    # full method's second pass moves nothing: with guard 0, unit buckets and
    # no pins its plan is plain farthest-next-use demand paging
    tensors, kernels = random_trace(seed, touch=True)
    kernels = _with_times(kernels, lambda i: 10**15)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    for div in (1, 2, 3):
        M = max(1024, fp // div // 256 * 256)
        try:
            ref = op.plan(tensors, kernels, M, variant=VAR_DEMAND_BELADY)
        except op.PlanError:
            continue
        r = op.plan(tensors, kernels, M, variant=VAR_T_A_P, affinity_w=0, guard=0, bucket=1)
        assert r.schedule == ref.schedule
        assert r.residency == ref.residency
        assert r.dyn_cls == ref.dyn_cls
        assert CLS_CGI not in r.dyn_cls and CLS_CGI not in r.static_cls
        assert r.counters["h2d_prefetch_n"] == 0


@pytest.mark.parametrize("seed", range(25))
def test_one_ns_times_make_every_fetching_kernel_cgi(seed):
    # at 1 ns even one 256-byte block takes longer on the link, so under demand
    # paging a kernel is CGI exactly when the schedule fetches something for it
    tensors, kernels = random_trace(seed, touch=True)
    kernels = _with_times(kernels, lambda i: 1)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    M = max(1024, fp // 2 // 256 * 256)
    try:
        r = op.plan(tensors, kernels, M, variant=VAR_DEMAND_BELADY)
    except op.PlanError:
        return
    fetched = set(e[5] for e in r.schedule if e[0] == S_H2D_DEMAND)
    for k, c in enumerate(r.dyn_cls):
        assert (c == CLS_CGI) == (k in fetched), k


@pytest.mark.parametrize("seed", range(10))
def test_zero_times_are_the_analytic_plan(seed):
    tensors, kernels = random_trace(seed, touch=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    M = max(1024, fp // 2 // 256 * 256)
    try:
        ref = op.plan(tensors, kernels, M)
    except op.PlanError:
        return
    r = op.plan(tensors, _with_times(kernels, lambda i: 0), M)
    assert r.schedule == ref.schedule and r.dyn_cls == ref.dyn_cls


@pytest.mark.parametrize("seed", range(15))
def test_timed_plans_pass_the_checker(seed):
    tensors, kernels = random_trace(seed, touch=True, timed=True)
    fp = sum(op.aligned(t["nbytes"]) for t in tensors)
    for div in (1, 2, 3):
        M = max(1024, fp // div // 256 * 256)
        try:
            r = op.plan(tensors, kernels, M)
        except op.PlanError:
            continue
        checker.check(tensors, kernels, M, r.schedule)
