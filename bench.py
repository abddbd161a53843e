#!/usr/bin/env python3
"""Throughput of decoders whose tensors oversubscribe the device budget, with
tensor-granular roofline-gated prefetching.

Default (llama-7b config): one step = one greedy decode step of the whole
model at batch 16 (every layer's transfers and kernels, scheduled by the
planner).  The job is a 1024-token prompt (prefill, untimed, reported)
followed by up to 256 decode steps; W steps run untimed, then K steps are
timed between two device synchronisations.  --factor sets the
oversubscription (default 3/2); --sweep runs several factors in one job.

GPT-style configs (gpt-1.3b): one step = one prefill forward pass over the
same ids; one cold pass is reported separately, then --iterations passes are
timed back to back.

Reported next to the value (one JSON line on stdout):
  * path_roofline: max(F/P, B/Bh, L/Bl) for the timed steps, with L the
    tensor-granular lower bound on host-to-device bytes (bytes the steps read
    before writing minus the budget), at nominal MI355X roofs and at the host
    link measured in the same run;
  * roofline: the dominant compute kernels (decode: the projection GEMVs;
    prefill: the projection GEMMs), algorithmic bytes or flops over their
    average duration from HIP events on the compute stream;
  * transfers: host-to-device bytes against L, link busy and idle time from
    the executor's timeline, compute-stream stall time;
  * per_layer: wall and kernel time per layer and step;
  * no_prefetch_baseline and ablation: the same engine with fault-driven
    demand fetches (LRU, then Belady eviction) and with the paper's T and
    T+A policies;
  * cpu_baseline: the CPU oracle on a bounded sample of the same work, and
    the oracle's planner replay timed against the library's planner.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

NOMINAL = dict(P=2.5e15, Bh=8.0e12, Bl=64.0e9)
PREFILL_GUARD = 16
# LLaMA-style decode with fused q, k, v projections (9 kernels per layer):
# planned H2D per 7B step at 1.5x, guard 4 / 5 / 6 -> 7.579 / 7.528 / 7.528 GB
# (the separate projections at guard 4: 7.527 GB)
DECODE_GUARD = 5
# 13B-shape training step at 2x (5 layers), two timed steps, same box:
# guard 0 / 1 / 2 / 3 / 4 / 5 -> 697 / 672.3-672.7 / 699 / 1064 / 689-691 / 699
# ms per step (34.9 / 35.5 / 37.0 / 37.6 / 37.9 / 39.4 GB over the link)
TRAIN_GUARD = 1
POLICY_NAMES = {0: "DEMAND_LRU", 1: "DEMAND_BELADY", 2: "T", 3: "T+A", 4: "T+A+P"}


# pinned host memory a run may use for its arena (the GPU host grants about 64 GiB)
PINNED_LIMIT = 58 << 30


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed decode steps (default 256; 32 per factor with --sweep)")
    ap.add_argument("--warmup", type=int, default=0, help="untimed decode steps before")
    ap.add_argument("--config", default="llama-7b")
    ap.add_argument("--factor", default=None, help="oversubscription factor num/den (default: the "
                                                    "config's own, 3/2 for llama-7b)")
    ap.add_argument("--sweep", default=None, help="comma-separated factors, e.g. 5/4,3/2,7/4,2/1")
    ap.add_argument("--iterations", type=int, default=4, help="timed passes (gpt-style configs)")
    ap.add_argument("--baseline-steps", type=int, default=8)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-baseline", action="store_true")
    ap.add_argument("--no-ablation", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="default decode line: skip the factor sweep (5/4, 3/2, 7/4, 2/1, one session)")
    ap.add_argument("--no-prefill-leg", action="store_true",
                    help="default decode line: skip the 1.3B prefill leg (1 cold + 4 timed passes)")
    ap.add_argument("--layers", type=int, default=0,
                    help="MoE and training configs: layers to run (default: MoE all of them, on a tiered host "
                         "arena past the pinned limit; training as many as fit the pinned limit)")
    ap.add_argument("--guard", type=int, default=None,
                    help="victim guard of the T+A+P plan (default: 5 for LLaMA-style decode and the sweep, 16 for prefill configs, 1 for the training step, the library's 4 for MoE)")
    ap.add_argument("--separate-qkv", action="store_true",
                    help="LLaMA-style traces: q, k and v projections as three LINEAR kernels "
                         "instead of one LINEAR_QKV")
    ap.add_argument("--no-replan", action="store_true",
                    help="skip the rerun planned from the measured kernel times")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run one 256 MiB device-to-device copy kernel (a known-size "
                         "reference for hardware byte counters)")
    return ap.parse_args()


def factor_of(s):
    num, den = (int(x) for x in s.split("/"))
    return num, den


def metric(kind, num, den):
    return f"{kind}tokens/sec at {num / den:g}x oversubscription; fraction of max(compute,HBM,link) roofline"


def link_bandwidth():
    """Pinned host-to-device copy rate measured with torch (1 GiB, best of 6
    after two untimed copies)."""
    import torch
    n = 1 << 30
    h = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(n, dtype=torch.uint8, device="cuda")
    for _ in range(2):
        d.copy_(h, non_blocking=True)
    best = 0.0
    for _ in range(6):
        torch.cuda.synchronize()
        t = time.perf_counter()
        d.copy_(h, non_blocking=True)
        torch.cuda.synchronize()
        best = max(best, n / (time.perf_counter() - t))
    del h, d
    return best


def counted_traffic(profile, source):
    """HBM bytes per launch of a kernel from its committed counter runs, if the
    kernel source is unchanged since they were taken (else None)."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", profile)
    src = os.path.join(ROOT, "paper_2609_06172_amd", "csrc", "kernels", source)
    try:
        meta = json.load(open(prof))
        if hashlib.sha256(open(src, "rb").read()).hexdigest() != meta["kernel_source_sha256"]:
            return None
        return meta["traffic_bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        return None


def microbench_peaks():
    """Same-run peaks of the three roofs, measured with PyTorch's own kernels
    (not this package's), each after two warm-up calls, as the best of 3
    groups of back-to-back calls timed with events: a device-to-device copy of
    2 GiB (bytes read + written per second), a streaming read (a sum over
    4 GiB), and a bf16 GEMM 8192 x 8192 x 8192 through torch.matmul (the
    vendor BLAS)."""
    import torch

    def best_rate(fn, work, reps):
        for _ in range(2):
            fn()
        best = 0.0
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            torch.cuda.synchronize()
            best = max(best, work * reps / (a.elapsed_time(b) * 1e-3))
        return best

    out = {}
    n = 2 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    out["hbm_copy_GBps"] = round(best_rate(lambda: b.copy_(a), 2 * n, 5) / 1e9, 1)
    del a, b
    x = torch.ones((1 << 30,), dtype=torch.float32, device="cuda")
    out["hbm_read_GBps"] = round(best_rate(lambda: x.sum(), 4 * x.numel(), 5) / 1e9, 1)
    del x
    m = 8192
    A = torch.randn((m, m), dtype=torch.bfloat16, device="cuda")
    Bm = torch.randn((m, m), dtype=torch.bfloat16, device="cuda")
    out["mfma_bf16_TFLOPs"] = round(best_rate(lambda: torch.matmul(A, Bm), 2 * m ** 3, 10) / 1e12, 1)
    del A, Bm
    torch.cuda.empty_cache()
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def calibrate_copy():
    """One 256 MiB device-to-device copy kernel: a known-size reference for
    hardware byte counters taken over the same command."""
    import torch
    n = 256 << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def link_lower_bound(w, a, n, M):
    """(H2D, D2H) bytes kernels [a, a+n) must move over the host link at least.

    At the boundary before kernel k, every tensor whose next access in the
    unit is a read must be on the device when that kernel runs; at most M
    bytes are there at the boundary, so at least (needed - M) bytes must
    cross to the device after it.  Those off the device that the unit itself
    writes were rewritten within the last repetition of the unit (decode
    steps and training steps repeat the same trace), so each of them was
    also written back; only needed tensors the unit never writes (weights
    at inference, token ids) can be off the device with a current host copy.
    Both bounds are taken at the boundary where their sum is largest (the
    first boundary gives the bytes the unit reads before writing, minus M).
    """
    from workloads.format import MODE_R, MODE_W
    written = set()
    for kd in w.kernels[a:a + n]:
        for t, m in kd.operands:
            if m & MODE_W:
                written.add(t)
    needed, live, ro, best = set(), 0, 0, (0, 0)
    for kd in reversed(w.kernels[a:a + n]):
        merged = {}
        for t, m in kd.operands:
            merged[t] = merged.get(t, 0) | m
        for t, m in merged.items():
            size = (w.tensors[t].nbytes + 255) // 256 * 256
            if m & MODE_R:
                if t not in needed:
                    needed.add(t)
                    live += size
                    ro += 0 if t in written else size
            elif t in needed:
                needed.remove(t)
                live -= size
                ro -= 0 if t in written else size
        h2d = max(0, live - M)
        d2h = max(0, live - M - ro)
        if h2d + d2h > sum(best):
            best = (h2d, d2h)
    return best


def seg_stats(w, sched, classes, M, segs):
    """Work and transfers of whole units (decode steps or forward passes) segs."""
    k0 = segs[0][0]
    k1 = segs[-1][0] + segs[-1][1]
    F = sum(c[2] for c in classes[k0:k1])
    B = sum(c[3] for c in classes[k0:k1])
    bounds = [link_lower_bound(w, a, n, M) for a, n in segs]
    lmin = sum(b[0] for b in bounds)
    lmin_d2h = sum(b[1] for b in bounds)
    h2d = sum(e[3] for e in sched if e[0] in (0, 1) and k0 <= e[4] < k1)
    d2h = sum(e[3] for e in sched if e[0] == 2 and k0 <= e[4] < k1)
    demand = sum(1 for e in sched if e[0] == 1 and k0 <= e[4] < k1)
    return dict(flops=F, hbm_bytes=B, lmin_bytes=lmin, lmin_d2h_bytes=lmin_d2h, h2d_bytes=h2d, d2h_bytes=d2h,
                demand_fetches=demand)


def link_timeline(tl, K):
    """Host link over the timed run segment (the last one): host-to-device
    busy and idle time (those copies run on two streams: busy is the union of
    their intervals), the part of each idle gap during which the host had not
    yet issued the next copy (host and device clocks share the segment's
    start), and, where the plan writes back, the device-to-host busy time and
    how much of it ran while a host-to-device copy was also in flight (copies
    in the two directions share one rate when they overlap)."""
    from paper_2609_06172_amd.capi import TL_D2H, TL_H2D, TL_H2D_B
    seg = max(e[1] for e in tl)
    cur = [e for e in tl if e[1] == seg]
    h = sorted((e for e in cur if e[0] in (TL_H2D, TL_H2D_B)), key=lambda e: e[5])
    span = max(e[6] for e in cur)
    busy = late = 0.0
    prev = 0.0                      # end of the busy union so far
    for e in h:
        if e[5] > prev:             # a gap before this copy
            late += max(0.0, min(e[5], e[4]) - prev)
            busy += e[6] - e[5]
        else:
            busy += max(0.0, e[6] - prev)
        prev = max(prev, e[6])
    nbytes = sum(e[3] for e in h)
    out = {"h2d_busy_ms_per_step": round(busy / K, 3), "h2d_idle_ms_per_step": round((span - busy) / K, 3),
           "idle_before_host_issue_ms_per_step": round(late / K, 3),
           "h2d_GBps_while_busy": round(nbytes / (busy * 1e-3) / 1e9, 2) if busy > 0 else None,
           "copies_per_step": round(len(h) / K, 2)}
    d = sorted((e for e in cur if e[0] == TL_D2H), key=lambda e: e[5])
    if d:
        def union(es):
            u = []
            for e in es:
                if u and e[5] <= u[-1][1]:
                    u[-1][1] = max(u[-1][1], e[6])
                else:
                    u.append([e[5], e[6]])
            return u
        hu, du = union(h), union(d)
        dbusy = sum(b - a for a, b in du)
        both, i = 0.0, 0
        for a, b in du:
            while i < len(hu) and hu[i][1] <= a:
                i += 1
            j = i
            while j < len(hu) and hu[j][0] < b:
                both += max(0.0, min(b, hu[j][1]) - max(a, hu[j][0]))
                j += 1
        out.update({"d2h_busy_ms_per_step": round(dbusy / K, 3),
                    "d2h_GBps_while_busy": round(sum(e[3] for e in d) / (dbusy * 1e-3) / 1e9, 2) if dbusy > 0 else None,
                    "d2h_copies_per_step": round(len(d) / K, 2),
                    "both_directions_busy_ms_per_step": round(both / K, 3),
                    "link_busy_ms_per_step": round((busy + dbusy - both) / K, 3)})
    return out


def per_layer(w, tl, segs, n_layers):
    """Mean wall time per layer (first kernel of the layer to the first kernel
    after it) and mean kernel time per layer, over the units segs."""
    from paper_2609_06172_amd.capi import TL_KERNEL
    seg = max(e[1] for e in tl)
    start = {e[2]: e[5] for e in tl if e[0] == TL_KERNEL and e[1] == seg}
    end = {e[2]: e[6] for e in tl if e[0] == TL_KERNEL and e[1] == seg}
    wall = [0.0] * n_layers
    kern = [0.0] * n_layers
    for a, n in segs:
        first = {}
        for k in range(a, a + n):
            kd = w.kernels[k]
            if kd.tag == "embed":
                continue
            first.setdefault(kd.layer, k)
            if kd.layer < n_layers:
                kern[kd.layer] += end[k] - start[k]
        for l in range(n_layers):
            nxt = first.get(l + 1)
            if l in first and nxt is not None:
                wall[l] += start[nxt] - start[first[l]]
    u = len(segs)
    return {"wall_ms": [round(x / u, 3) for x in wall], "kernel_ms": [round(x / u, 3) for x in kern]}


def step_series(tl, segs, block=32):
    """Mean wall time per unit over consecutive blocks of units (start of a
    unit's first kernel to the start of the next unit's first kernel)."""
    from paper_2609_06172_amd.capi import TL_KERNEL
    seg = max(e[1] for e in tl)
    start = {e[2]: e[5] for e in tl if e[0] == TL_KERNEL and e[1] == seg}
    end = max(e[6] for e in tl if e[1] == seg)
    t = [start[a] for a, _ in segs] + [end]
    d = [t[i + 1] - t[i] for i in range(len(segs))]
    return [round(sum(d[i:i + block]) / len(d[i:i + block]), 2) for i in range(0, len(d), block)]


def run_decode(s, w, W, K):
    import torch
    steps = w.segments["decode"]
    k0, n = w.segments["prefill"][0]
    torch.cuda.synchronize()
    t = time.perf_counter()
    s.run(k0, n)
    torch.cuda.synchronize()
    prefill_s = time.perf_counter() - t
    for i in range(W):
        s.run(*steps[i])
    first = steps[W][0]
    last = steps[W + K - 1]
    nk = last[0] + last[1] - first
    stall0 = s.ctx.get_counters()["stall_ns"]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    s.run(first, nk)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    s.timed_stall_ns = s.ctx.get_counters()["stall_ns"] - stall0   # timing policy only
    return prefill_s, dt, first, first + nk


def decode_policy(s, w, M, variant, W, K, ref_gen, object_bytes=0, guard=None):
    """Rerun the decode under another policy (timing off) and summarise it."""
    s.set_policy(variant=variant, timing=0, object_bytes=object_bytes, guard=guard)
    s.ctx.reset()
    s.restore_inputs()
    pb, db, _, _ = run_decode(s, w, W, K)
    gen = s.read("gen")[: W + K + 1]
    st = seg_stats(w, s.ctx.get_schedule(), s.ctx.get_classes(), M, w.segments["decode"][W:W + K])
    b = w.cfg.batch
    return {"policy": POLICY_NAMES[variant], "steps": K, "value": round(b * K / db, 3), "unit": "tokens/s",
            "ms_per_step": round(db / K * 1e3, 3), "prefill_seconds": round(pb, 3),
            "h2d_bytes_per_step": st["h2d_bytes"] // K, "d2h_bytes_per_step": st["d2h_bytes"] // K,
            "demand_fetches_per_step": round(st["demand_fetches"] / K, 2),
            "tokens_identical": bool((gen == ref_gen[: W + K + 1]).all())}


def plan_only_sweeps(s, w, M, segs, guard):
    """Plans of the same session, not run: host-to-device bytes per timed step
    for T+A at several affinity windows, and for T+A+P on allocator blocks
    of several sizes, with the useless and useful fetched bytes of the whole
    plan (member fetches no kernel reads while resident, and the rest)."""
    a, n = segs[0][0], segs[-1][0] + segs[-1][1] - segs[0][0]
    K = len(segs)

    def step_bytes():
        sched = s.ctx.get_schedule()
        return sum(e[3] for e in sched if e[0] in (0, 1) and a <= e[4] < a + n) // K

    out = {"affinity_window": [], "allocator_blocks": []}
    for Wa in (1, 4, 16, 64):
        s.set_policy(variant=3, affinity_w=Wa)
        out["affinity_window"].append({"policy": "T+A", "W": Wa, "h2d_bytes_per_step": step_bytes()})
    for ob in (0, 64 << 20, 256 << 20, 1 << 30):
        try:
            s.set_policy(variant=4, guard=guard, object_bytes=ob)
        except Exception as e:       # blocks that do not fit the budget
            out["allocator_blocks"].append({"object_bytes": ob, "error": str(e)})
            continue
        c = s.ctx.get_counters()
        fetched = c["h2d_prefetch_B"] + c["h2d_demand_B"]
        out["allocator_blocks"].append({
            "object_bytes": ob, "h2d_bytes_per_step": step_bytes(),
            "useless_fetched_bytes": c["useless_prefetch_B"] if ob else 0,
            "useful_fetched_bytes": fetched - (c["useless_prefetch_B"] if ob else 0)})
    s.set_policy(variant=4, timing=0, guard=guard)
    return out


def measured_replan(s, w, dur, guard, rerun):
    """Runtime monitor: classify again from the kernel durations of the timed
    run (kernels it did not run keep the analytic class) and plan again.
    rerun() (which reads the outputs it needs: planning again resets the
    executor) runs once under the analytic plan and once under the measured
    one, both with timing off; the analytic plan is restored after.  Returns
    (static and dynamic class changes, schedule entries changed, analytic
    result, measured result)."""
    s.set_policy(variant=4, timing=0, guard=guard)
    analytic, a_sched = s.ctx.get_classes(), s.ctx.get_schedule()
    s.ctx.reset()
    s.restore_inputs()
    out_a = rerun()
    times = [max(1, int(round(d * 1e6))) for d in dur] + [0] * (len(w.kernels) - len(dur))
    s.ctx.set_kernel_times(times)
    s.ctx.plan()
    measured, sched = s.ctx.get_classes(), s.ctx.get_schedule()
    s.ctx.reset()
    s.restore_inputs()
    out_m = rerun()
    s.ctx.set_kernel_times([0] * len(w.kernels))
    s.ctx.plan()
    names = ("compute", "memory", "cgi")
    flips = [{}, {}]
    for a, m in zip(analytic[: len(dur)], measured[: len(dur)]):
        for f, x, y in ((flips[0], a[0], m[0]), (flips[1], a[1], m[1])):
            if x != y:
                key = f"{names[x]}->{names[y]}"
                f[key] = f.get(key, 0) + 1
    moved = sum(1 for x, y in zip(a_sched, sched) if x != y) + abs(len(a_sched) - len(sched))
    return flips, moved, out_a, out_m


def planner_replay(cfg, M, steps):
    """The oracle's planner and the library's on the prefill + `steps` decode
    steps of the same trace (same budget): wall times and schedule identity."""
    import dataclasses
    from oracle import planner as op
    from paper_2609_06172_amd.session import Session
    from workloads import trace
    w = trace.build(dataclasses.replace(cfg, decode_steps=steps))
    s = Session(w, device=-1, M=M)
    cxx_s = s.ctx.get_counters()["plan_ns"] / 1e9
    sched = s.ctx.get_schedule()
    s.close()
    t = time.perf_counter()
    r = op.plan_workload(w, M)
    oracle_s = time.perf_counter() - t
    same = [tuple(e) for e in sched] == [tuple(e) for e in r.schedule]
    return {"trace": f"prefill + {steps} decode steps ({len(w.kernels)} kernels)",
            "library_plan_s": round(cxx_s, 4), "oracle_plan_s": round(oracle_s, 3),
            "schedules_identical": bool(same)}


def blas_info():
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        threads = max((i.get("num_threads", 1) for i in info), default=1)
        vendor = ",".join(sorted(set(i.get("internal_api", "?") for i in info)))
    except Exception:
        threads, vendor = len(os.sched_getaffinity(0)), "unknown"
    return threads, vendor


def cpu_baseline_decode(cfg, w, seconds, pos, M):
    """fp32 oracle decode of a few layers at the timed position, scaled to the model."""
    import numpy as np
    from oracle import forward as of
    from workloads import init as winit
    threads, vendor = blas_info()
    from concurrent.futures import ThreadPoolExecutor
    L = 2
    B, nH, d, Lmax = cfg.batch, cfg.n_heads, cfg.head_dim, cfg.kv_len
    names = [f"L{l}.{nm}" for l in range(L) for nm in
             ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd")] + ["head", "norm_f"]

    def weight(nm):
        return nm, winit.tensor_value(w, w.tensors[w.id(nm)]).astype(np.float32)

    def cache(i):   # synthetic prefix of the KV cache (values do not change the timing)
        g = np.random.default_rng([7, i])
        return g.standard_normal((B, nH, Lmax, d), dtype=np.float32) * np.float32(0.5)

    with ThreadPoolExecutor(16) as ex:
        Wt = dict(ex.map(weight, names))
        kv = list(ex.map(cache, range(2 * L)))
    Wl = [({nm.split(".", 1)[1]: v for nm, v in Wt.items() if nm.startswith(f"L{l}.")},
           kv[2 * l], kv[2 * l + 1]) for l in range(L)]
    head, gf = Wt["head"], Wt["norm_f"]
    x0 = (np.random.default_rng(8).standard_normal((B, cfg.hidden)) * 0.02).astype(np.float32)
    t_layers, reps = 0.0, 0
    t_start = time.perf_counter()
    while reps == 0 or time.perf_counter() - t_start < seconds:
        x = x0
        t = time.perf_counter()
        for Lw, K, V in Wl:
            x = of.llama_layer(cfg, Lw, x, K, V, pos)
        t_layers += time.perf_counter() - t
        reps += 1
    t = time.perf_counter()
    of.linear(of.rmsnorm(x, gf), head)
    t_head = time.perf_counter() - t
    assert x.dtype == np.float32
    step_s = t_layers / reps / L * cfg.n_layers + t_head
    return {"value": B / step_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "blas": vendor, "cpu": cpu_model(), "precision": "fp32",
            "sample": f"fp32 numpy oracle decode step at position {pos}, batch {B}: {L} of "
                      f"{cfg.n_layers} layers timed over {reps} repetitions plus the LM head, "
                      f"scaled to {cfg.n_layers} layers ({step_s:.2f} s per step)",
            "planner": planner_replay(cfg, M, 16)}


def cpu_baseline_prefill(cfg, w, seconds):
    """fp64 oracle forward of one layer over the whole prompt, scaled to the model."""
    import numpy as np
    from oracle import forward as of
    from workloads import init as winit
    threads, vendor = blas_info()
    names = [n for n in ("L0.ln1.g", "L0.ln1.b", "L0.wqkv", "L0.wo", "L0.ln2.g", "L0.ln2.b", "L0.w1", "L0.w2")]
    Wt = {nm: winit.tensor_value(w, w.tensors[w.id(nm)]).astype(np.float32) for nm in names}
    x0 = (np.random.default_rng(8).standard_normal((cfg.tokens, cfg.hidden)) * 0.02).astype(np.float32)
    reps, t_layer = 0, 0.0
    t_start = time.perf_counter()
    while reps == 0 or time.perf_counter() - t_start < seconds:
        t = time.perf_counter()
        of.gpt_layer(cfg, Wt, 0, x0)
        t_layer += time.perf_counter() - t
        reps += 1
    pass_s = t_layer / reps * cfg.n_layers
    return {"value": cfg.tokens / pass_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "blas": vendor, "cpu": cpu_model(), "precision": "fp32",
            "sample": f"fp32 numpy oracle: 1 of {cfg.n_layers} layers over {cfg.batch} x {cfg.prompt_len} "
                      f"tokens timed over {reps} repetitions, scaled to {cfg.n_layers} layers (LM head "
                      f"not included; {pass_s:.1f} s per pass)"}


def cpu_baseline_moe(cfg, w, seconds, pos):
    """fp64 oracle MoE decode of one layer at the timed position, scaled to the model."""
    import numpy as np
    from oracle import forward as of
    from workloads import init as winit
    threads, vendor = blas_info()
    from concurrent.futures import ThreadPoolExecutor
    B, nH, d, Lmax = cfg.batch, cfg.n_heads, cfg.head_dim, cfg.kv_len
    names = [f"L0.{nm}" for nm in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "router")]
    names += [f"L0.x{e}.{nm}" for e in range(cfg.n_experts) for nm in ("wg", "wu", "wd")]

    def weight(nm):
        return nm.split(".", 1)[1], winit.tensor_value(w, w.tensors[w.id(nm)]).astype(np.float64)

    def cache(i):   # synthetic prefix of the KV cache (values do not change the timing)
        g = np.random.default_rng([7, i])
        return g.standard_normal((B, nH, Lmax, d), dtype=np.float32).astype(np.float64) * 0.5

    with ThreadPoolExecutor(16) as ex:
        Lw = dict(ex.map(weight, names))
        K, V = ex.map(cache, range(2))
    x0 = np.random.default_rng(8).standard_normal((B, cfg.hidden)) * 0.02
    t_layer, reps = 0.0, 0
    t_start = time.perf_counter()
    while reps == 0 or time.perf_counter() - t_start < seconds:
        t = time.perf_counter()
        of.llama_layer(cfg, Lw, x0, K, V, pos)
        t_layer += time.perf_counter() - t
        reps += 1
    step_s = t_layer / reps * cfg.n_layers
    return {"value": B / step_s, "unit": "tokens/s", "cores": threads, "kind": "oracle", "blas": vendor,
            "cpu": cpu_model(), "precision": "fp64",
            "sample": f"fp64 numpy oracle MoE decode step at position {pos}, batch {B}: 1 of "
                      f"{cfg.n_layers} layers (attention and the routed experts) timed over {reps} "
                      f"repetitions, scaled to {cfg.n_layers} layers; LM head not included "
                      f"({step_s:.2f} s per step)"}


def expert_fetches(w, sched, counts, k0, k1):
    """Bytes fetched for expert weights between kernels k0 and k1, split into
    fetches for experts that got rows and for experts that got none."""
    from workloads.format import OP_MOE_DOWN, OP_MOE_UP
    seg_of = {}
    for seg, (a, n) in enumerate(w.segments["prefill"] + w.segments["decode"]):
        for k in range(a, a + n):
            seg_of[k] = seg
    used = idle = 0
    for e in sched:
        if e[0] not in (0, 1) or not k0 <= e[5] < k1:
            continue
        kd = w.kernels[e[5]]
        if kd.op == OP_MOE_UP:
            weights = (kd.operands[2][0], kd.operands[3][0])
        elif kd.op == OP_MOE_DOWN:
            weights = (kd.operands[3][0],)
        else:
            continue
        if e[1] not in weights:
            continue
        if counts[seg_of[e[5]], kd.layer, kd.shape[3]] > 0:
            used += e[3]
        else:
            idle += e[3]
    return used, idle


def roofline_fields(st, seconds, bl_meas, units, peaks=None):
    """The path's roofline: max of compute, HBM and host-link times at the
    nominal roofs; the same with the measured link; and, with same-run
    microbenchmark peaks, the same against all three measured roofs."""
    import numpy as np
    t_comp = st["flops"] / NOMINAL["P"]
    t_hbm = st["hbm_bytes"] / NOMINAL["Bh"]
    # both directions share the host link (concurrent H2D and D2H copies
    # together reach the rate of one direction alone)
    link = st["lmin_bytes"] + st["lmin_d2h_bytes"]
    t_link = link / NOMINAL["Bl"]
    roof_s = max(t_comp, t_hbm, t_link)
    roof_meas = max(t_comp, t_hbm, link / bl_meas)
    extra = {}
    if peaks:
        hbm = max(peaks["hbm_copy_GBps"], peaks["hbm_read_GBps"]) * 1e9
        roof_peaks = max(st["flops"] / (peaks["mfma_bf16_TFLOPs"] * 1e12), st["hbm_bytes"] / hbm, link / bl_meas)
        extra = {"frac_measured_peaks": round(roof_peaks / seconds, 4)}
    return {"bound": ["mfma", "hbm", "link"][int(np.argmax([t_comp, t_hbm, t_link]))],
            "roofline_units_per_s": round(units / roof_s, 3),
            "frac": round(roof_s / seconds, 4),
            "frac_measured_link": round(roof_meas / seconds, 4), **extra,
            "link_GBps_nominal": NOMINAL["Bl"] / 1e9, "link_GBps_measured": round(bl_meas / 1e9, 2),
            "t_mfma_ms": round(t_comp * 1e3, 3), "t_hbm_ms": round(t_hbm * 1e3, 3),
            "t_link_ms": round(t_link * 1e3, 3), "t_measured_ms": round(seconds * 1e3, 3)}


def linear_kernels(w, k0, k1):
    from workloads.format import (OP_LINEAR, OP_LINEAR_GELU, OP_LINEAR_QKV, OP_LINEAR_RESID,
                                  OP_LINEAR_SWIGLU)
    return [k for k in range(k0, k1)
            if w.kernels[k].op in (OP_LINEAR, OP_LINEAR_GELU, OP_LINEAR_RESID, OP_LINEAR_SWIGLU,
                                   OP_LINEAR_QKV)]


def decode_main(args, cfg):
    import numpy as np
    import torch

    from paper_2609_06172_amd.session import Session
    from workloads import trace

    num, den = cfg.factor
    W, K = args.warmup, (256 if args.steps is None else args.steps)
    if W + K > cfg.decode_steps or K < 1:
        sys.exit(f"warmup + steps must be within 1..{cfg.decode_steps}")
    w = trace.build(cfg)
    M = w.budget()
    log(f"workload {cfg.name}: {len(w.tensors)} tensors, {len(w.kernels)} kernels, "
        f"footprint {w.footprint} B, budget {M} B")
    if args.calibrate_copy:
        calibrate_copy()
    bl_meas = link_bandwidth()
    log(f"measured pinned H2D: {bl_meas / 1e9:.1f} GB/s")
    peaks = microbench_peaks()
    log(f"same-run peaks: {peaks}")

    t = time.perf_counter()
    guard = DECODE_GUARD if args.guard is None else args.guard
    s = Session(w, device=0, M=M, variant=4, timing=1, guard=guard)
    log(f"session ready in {time.perf_counter() - t:.1f} s (plan {s.ctx.get_counters()['plan_ns'] / 1e9:.2f} s)")
    prefill_s, decode_s, k0, k1 = run_decode(s, w, W, K)
    log(f"prefill {prefill_s:.3f} s, decode {K} steps {decode_s:.3f} s")
    sched = s.ctx.get_schedule()
    classes = s.ctx.get_classes()
    dur, gap = s.ctx.get_kernel_times()
    tl = s.ctx.get_timeline()
    gen_tap = s.read("gen")[: W + K + 1].copy()
    segs = w.segments["decode"][W:W + K]
    st = seg_stats(w, sched, classes, M, segs)

    # dominant kernels: decode projections (M <= 16 rows) on the matrix cores
    lin = linear_kernels(w, k0, k1)
    g_bytes = sum(classes[k][3] for k in lin)
    g_time = sum(dur[k] for k in lin) * 1e-3
    g_achieved = g_bytes / g_time / 1e9
    per_op = {}
    for k in range(k0, k1):
        e = per_op.setdefault(w.kernels[k].tag, [0, 0.0])
        e[0] += 1
        e[1] += dur[k]
    stall_ms = s.timed_stall_ns / 1e6          # the library's counter over the timed segment
    busy_ms = sum(dur[k] for k in range(k0, k1))
    hbm_peak = max(peaks["hbm_copy_GBps"], peaks["hbm_read_GBps"])

    tok_s = cfg.batch * K / decode_s
    pr = roofline_fields(st, decode_s, bl_meas, cfg.batch * K, peaks)
    pr["roofline_tok_s"] = pr.pop("roofline_units_per_s")
    result = {
        "metric": metric("", num, den), "value": round(tok_s, 3), "unit": "tokens/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(decode_s / K * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shape decode: {cfg.n_layers} layers, hidden {cfg.hidden}, "
                               f"SwiGLU {cfg.ffn}, vocab {cfg.vocab}, batch {cfg.batch}, "
                               f"{cfg.prompt_len}-token prompt then greedy steps, "
                               f"budget = footprint*{den}/{num}",
                   "batch": cfg.batch, "prompt_len": cfg.prompt_len, "factor": f"{num}/{den}",
                   "footprint_bytes": w.footprint, "budget_bytes": M, "policy": "T+A+P",
                   "guard": guard, "qkv": "fused" if cfg.fuse_qkv else "separate"},
        "path_roofline": pr,
        "roofline": {"kernel": "decode projection GEMV (M=16, bf16 matrix cores)", "bound": "hbm",
                     "achieved": round(g_achieved, 1), "peak": 8000.0, "unit": "GB/s",
                     "frac": round(g_achieved / 8000.0, 4),
                     "frac_measured_peak": round(g_achieved / hbm_peak, 4),
                     "traffic": counted_traffic("gemv_mfma_traffic_llama7b_decode.json", "gemv.hip"),
                     "launches": len(lin), "avg_us": round(g_time / max(1, len(lin)) * 1e6, 2),
                     "avg_bytes": int(g_bytes / max(1, len(lin)))},
        "transfers": {"h2d_bytes_per_step": st["h2d_bytes"] // K, "d2h_bytes_per_step": st["d2h_bytes"] // K,
                      "lmin_bytes_per_step": st["lmin_bytes"] // K,
                      "h2d_over_lmin": round(st["h2d_bytes"] / max(1, st["lmin_bytes"]), 4),
                      "demand_fetches": st["demand_fetches"],
                      "achieved_h2d_GBps": round(st["h2d_bytes"] / decode_s / 1e9, 2),
                      "compute_busy_ms_per_step": round(busy_ms / K, 3),
                      "compute_stall_ms_per_step": round(stall_ms / K, 3),
                      "link_timeline": link_timeline(tl, K)},
        "prefill": {"seconds": round(prefill_s, 3), "tokens": cfg.batch * cfg.prompt_len},
        "microbench": {**peaks, "link_GBps": round(bl_meas / 1e9, 2)},
        "per_kernel_ms_per_step": {k: round(v[1] / K, 4) for k, v in sorted(per_op.items())},
        "per_layer": per_layer(w, tl, segs, cfg.n_layers),
        "step_ms_per_32_steps": step_series(tl, segs),
    }

    if not args.no_baseline:
        Bk = min(args.baseline_steps, K)
        b = decode_policy(s, w, M, 0, W, Bk, gen_tap)
        b["policy"] = "demand fetch at launch, LRU eviction"
        b["speedup_of_T+A+P"] = round(tok_s / b["value"], 3)
        result["no_prefetch_baseline"] = b
        log(f"baseline {Bk} steps {Bk / b['value'] * cfg.batch:.3f} s")
        if not args.no_ablation:
            result["ablation"] = [decode_policy(s, w, M, v, W, Bk, gen_tap) for v in (1, 2, 3)]
            # the object-level contrast: the full method on 1 GiB allocator blocks
            ob = 1 << 30
            row = decode_policy(s, w, M, 4, W, Bk, gen_tap, object_bytes=ob, guard=guard)
            c = s.ctx.get_counters()
            fetched = c["h2d_prefetch_B"] + c["h2d_demand_B"]
            row.update(policy="T+A+P on 1 GiB allocator blocks", object_bytes=ob,
                       useless_to_useful_fetched_bytes=round(c["useless_prefetch_B"] /
                                                             max(1, fetched - c["useless_prefetch_B"]), 4),
                       speedup_of_tensor_granularity=round(tok_s / row["value"], 3))
            result["ablation"].append(row)
            log("ablation: " + ", ".join(f"{a['policy']} {a['value']}" for a in result["ablation"]))
            result["plan_only"] = plan_only_sweeps(s, w, M, segs, guard)
    if not args.no_replan:
        Bk = min(args.baseline_steps, K)

        def rerun():
            r = run_decode(s, w, W, Bk)
            return r[1], s.read("gen")[: W + Bk + 1].copy()
        flips, moved, (da, ga), (dm, gm) = measured_replan(s, w, dur, guard, rerun)
        result["measured_replan"] = {
            "steps": Bk, "unit": "tokens/s", "kernels_timed": len(dur),
            "analytic_value": round(cfg.batch * Bk / da, 3), "value": round(cfg.batch * Bk / dm, 3),
            "analytic_ms_per_step": round(da / Bk * 1e3, 3), "ms_per_step": round(dm / Bk * 1e3, 3),
            "static_class_changes": flips[0], "dynamic_class_changes": flips[1],
            "schedule_entries_changed": moved,
            "tokens_identical": bool((gm == gen_tap[: W + Bk + 1]).all() and (ga == gm).all())}
        log(f"re-planned from measured times: {result['measured_replan']}")
    if not args.no_sweep:
        # the same session re-budgeted at each factor: 4 untimed, 16 timed steps
        rows = sweep_in_session(s, w, cfg, DEFAULT_SWEEP.split(","), 4, 16,
                                0 if args.no_baseline else 4, bl_meas, guard, peaks)
        result["factor_sweep"] = {"steps": 16, "warmup": 4, "demand_lru_steps": 0 if args.no_baseline else 4,
                                  "rows": rows}
    s.close()
    del s
    torch.cuda.empty_cache()

    if not args.no_prefill_leg:
        from workloads import configs
        pf = prefill_measure(configs.GPT_1P3B, 4, PREFILL_GUARD, bl_meas, peaks, baseline=not args.no_baseline,
                             replan=False)
        result["prefill_1p3b"] = {k: pf[k] for k in ("value", "unit", "ms_per_step", "path_roofline", "roofline",
                                                     "attention", "transfers", "cold_pass", "no_prefetch_baseline")
                                  if k in pf}
        result["prefill_1p3b"]["config"] = pf["config"]
        log(f"1.3b prefill: {pf['value']} tok/s, path frac {pf['path_roofline']['frac']}")
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_decode(cfg, w, args.cpu_seconds, cfg.prompt_len + W, M)
    emit(args, result)


DEFAULT_SWEEP = "5/4,3/2,7/4,2/1"


def sweep_in_session(s, w, cfg, factors, W, K, Bk, bl_meas, guard, peaks=None):
    """The decode at several oversubscription factors: the same session (host
    arena, tensors, trace) re-budgeted for each factor and planned again; W
    untimed and K timed steps of T+A+P each, then Bk steps of DEMAND_LRU."""
    rows = []
    for f in factors:
        num, den = factor_of(f)
        M = w.budget(num, den)
        s.set_budget(M, plan=False)
        s.set_policy(variant=4, timing=1, guard=guard)
        s.restore_inputs()
        _, decode_s, k0, k1 = run_decode(s, w, W, K)
        segs = w.segments["decode"][W:W + K]
        st = seg_stats(w, s.ctx.get_schedule(), s.ctx.get_classes(), M, segs)
        gen = s.read("gen")[: W + K + 1].copy()
        pr = roofline_fields(st, decode_s, bl_meas, cfg.batch * K, peaks)
        row = {"factor": f"{num}/{den}", "budget_bytes": M, "value": round(cfg.batch * K / decode_s, 3),
               "ms_per_step": round(decode_s / K * 1e3, 3), "roofline_tok_s": pr["roofline_units_per_s"],
               "bound": pr["bound"], "frac": pr["frac"], "frac_measured_link": pr["frac_measured_link"],
               "h2d_bytes_per_step": st["h2d_bytes"] // K, "lmin_bytes_per_step": st["lmin_bytes"] // K,
               "h2d_over_lmin": round(st["h2d_bytes"] / max(1, st["lmin_bytes"]), 4),
               "compute_stall_ms_per_step": round(s.timed_stall_ns / 1e6 / K, 3),
               "link_timeline": link_timeline(s.ctx.get_timeline(), K)}
        if Bk:
            b = decode_policy(s, w, M, 0, W, Bk, gen)
            row["demand_lru_value"] = b["value"]
            row["speedup_over_demand_lru"] = round(row["value"] / b["value"], 3)
            row["tokens_identical"] = b["tokens_identical"]
        log(f"factor {num}/{den}: {row['value']} tok/s, frac {row['frac']}")
        rows.append(row)
    return rows


def sweep_main(args, cfg):
    """The decode at several oversubscription factors in one session."""
    import torch

    from paper_2609_06172_amd.session import Session
    from workloads import trace

    W, K = args.warmup, (32 if args.steps is None else args.steps)
    bl_meas = link_bandwidth()
    w = trace.build(cfg)
    guard = DECODE_GUARD if args.guard is None else args.guard
    s = Session(w, device=0, variant=4, timing=1, guard=guard)
    rows = sweep_in_session(s, w, cfg, args.sweep.split(","), W, K,
                            0 if args.no_baseline else min(args.baseline_steps, K), bl_meas, guard)
    s.close()
    del s
    torch.cuda.empty_cache()
    out = {"metric": "tokens/sec per oversubscription factor; fraction of max(compute,HBM,link) roofline",
           "unit": "tokens/s", "n_gpus": 1, "steps": K, "warmup": W, "higher_is_better": True,
           "dtype": "bf16", "data": "synthetic", "link_GBps_measured": round(bl_meas / 1e9, 2),
           "config": {"workload": f"{cfg.name}-shape decode, batch {cfg.batch}, {cfg.prompt_len}-token prompt",
                      "policy": "T+A+P"},
           "sweep": rows}
    emit(args, out)


def prefill_main(args, cfg):
    """GPT-style prefill: one cold pass, then timed passes over the same ids."""
    if args.calibrate_copy:
        calibrate_copy()
    bl_meas = link_bandwidth()
    peaks = microbench_peaks()
    guard = PREFILL_GUARD if args.guard is None else args.guard
    result = prefill_measure(cfg, args.iterations, guard, bl_meas, peaks, baseline=not args.no_baseline,
                             replan=not args.no_replan)
    result["microbench"] = peaks
    if not args.no_cpu_baseline:
        from workloads import trace
        result["cpu_baseline"] = cpu_baseline_prefill(cfg, trace.build(cfg), args.cpu_seconds)
    emit(args, result)


def prefill_measure(cfg, I, guard, bl_meas, peaks=None, baseline=True, replan=True):
    """One cold pass, then I timed passes over the same ids under T+A+P, with
    the GEMM and attention rooflines; DEMAND_LRU over the same passes and the
    measured-time re-plan on request."""
    import dataclasses

    import torch

    from paper_2609_06172_amd.session import Session
    from workloads import trace

    num, den = cfg.factor
    cfg = dataclasses.replace(cfg, iterations=1 + I)
    w = trace.build(cfg)
    M = w.budget()
    its = w.segments["iterations"]
    log(f"workload {cfg.name}: {len(w.tensors)} tensors, {len(w.kernels)} kernels, "
        f"footprint {w.footprint} B, budget {M} B")
    # Prefill is compute-bound (the link idles most of a pass), so a longer
    # victim guard buys overlap with bytes the link has time for; measured on
    # the 1.3B prefill: guard 4 / 8 / 16 / 24 / 32 -> 32.8 / 31.5 / 30.4 / 30.4 /
    # 31.0 ms per pass.  The link-bound decode uses DECODE_GUARD.
    s = Session(w, device=0, M=M, variant=4, timing=1, guard=guard)

    def passes(sess):
        torch.cuda.synchronize()
        t = time.perf_counter()
        sess.run(*its[0])
        torch.cuda.synchronize()
        cold = time.perf_counter() - t
        k0 = its[1][0]
        k1 = its[-1][0] + its[-1][1]
        t = time.perf_counter()
        sess.run(k0, k1 - k0)
        torch.cuda.synchronize()
        return cold, time.perf_counter() - t, k0, k1

    cold_s, hot_s, k0, k1 = passes(s)
    sched, classes = s.ctx.get_schedule(), s.ctx.get_classes()
    dur, gap = s.ctx.get_kernel_times()
    tl = s.ctx.get_timeline()
    st = seg_stats(w, sched, classes, M, its[1:])
    st0 = seg_stats(w, sched, classes, M, its[:1])
    logits = s.read("logits").copy()
    lin = [k for k in linear_kernels(w, k0, k1) if w.kernels[k].shape[0] >= 512]   # the projection GEMMs
    g_flops = sum(classes[k][2] for k in lin)
    g_time = sum(dur[k] for k in lin) * 1e-3
    attn = [k for k in range(k0, k1) if w.kernels[k].tag == "attn"]
    a_flops = sum(classes[k][2] for k in attn)
    a_time = sum(dur[k] for k in attn) * 1e-3
    tok_s = cfg.tokens * I / hot_s
    pr = roofline_fields(st, hot_s, bl_meas, cfg.tokens * I, peaks)
    pr["roofline_tok_s"] = pr.pop("roofline_units_per_s")
    stall_ns = s.ctx.get_counters()["stall_ns"]
    result = {
        "metric": metric("prefill ", num, den), "value": round(tok_s, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": I, "warmup": 1, "ms_per_step": round(hot_s / I * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shape prefill: {cfg.n_layers} layers, hidden {cfg.hidden}, "
                               f"GELU {cfg.ffn}, vocab {cfg.vocab}, {cfg.batch} x {cfg.prompt_len} tokens, "
                               f"budget = footprint*{den}/{num}",
                   "tokens_per_pass": cfg.tokens, "factor": f"{num}/{den}", "footprint_bytes": w.footprint,
                   "budget_bytes": M, "policy": f"T+A+P (guard {guard})"},
        "path_roofline": pr,
        "roofline": {"kernel": "prefill projection GEMM (bf16 matrix cores)", "bound": "mfma",
                     "achieved": round(g_flops / g_time / 1e12, 1), "peak": 2500.0, "unit": "TFLOP/s",
                     "frac": round(g_flops / g_time / 2.5e15, 4),
                     **({"frac_measured_peak": round(g_flops / g_time / 1e12 / peaks["mfma_bf16_TFLOPs"], 4)}
                        if peaks else {}),
                     "traffic": counted_traffic("gemm_big_traffic_gpt1p3b_prefill.json", "gemm_big.hip"),
                     "launches": len(lin),
                     "avg_us": round(g_time / max(1, len(lin)) * 1e6, 2),
                     "avg_flops": int(g_flops / max(1, len(lin)))},
        "attention": {"launches": len(attn), "avg_us": round(a_time / max(1, len(attn)) * 1e6, 2),
                      "TFLOPs": round(a_flops / a_time / 1e12, 1) if a_time > 0 else None},
        "transfers": {"h2d_bytes_per_pass": st["h2d_bytes"] // I, "lmin_bytes_per_pass": st["lmin_bytes"] // I,
                      "h2d_over_lmin": round(st["h2d_bytes"] / max(1, st["lmin_bytes"]), 4),
                      "d2h_bytes_per_pass": st["d2h_bytes"] // I,
                      "compute_busy_ms_per_pass": round(sum(dur[k] for k in range(k0, k1)) / I, 3),
                      "compute_stall_ms_per_pass": round(sum(gap[k] for k in range(k0 + 1, k1)) / I, 3),
                      "compute_stall_ms_all_passes_counter": round(stall_ns / 1e6, 3),
                      "link_timeline": link_timeline(tl, I)},
        "cold_pass": {"seconds": round(cold_s, 4), "h2d_bytes": st0["h2d_bytes"]},
        "per_layer": per_layer(w, tl, [w.segments["iterations"][1]], cfg.n_layers),
    }
    if baseline:
        s.set_policy(variant=0, timing=0)
        s.ctx.reset()
        s.restore_inputs()
        _, hot_b, _, _ = passes(s)
        result["no_prefetch_baseline"] = {
            "policy": "demand fetch at launch, LRU eviction", "value": round(cfg.tokens * I / hot_b, 1),
            "unit": "tokens/s", "ms_per_pass": round(hot_b / I * 1e3, 3),
            "speedup_of_T+A+P": round(hot_b / hot_s, 3),
            "logits_identical": bool((s.read("logits") == logits).all())}
    if replan:
        def rerun():
            r = passes(s)
            return r[1], s.read("logits").copy()
        flips, moved, (ha, la), (hm, lm) = measured_replan(s, w, dur, guard, rerun)
        result["measured_replan"] = {
            "unit": "tokens/s", "kernels_timed": len(dur),
            "analytic_value": round(cfg.tokens * I / ha, 1), "value": round(cfg.tokens * I / hm, 1),
            "analytic_ms_per_pass": round(ha / I * 1e3, 3), "ms_per_pass": round(hm / I * 1e3, 3),
            "static_class_changes": flips[0], "dynamic_class_changes": flips[1],
            "schedule_entries_changed": moved,
            "logits_identical": bool((lm == logits).all() and (la == logits).all())}
        log(f"re-planned from measured times: {result['measured_replan']}")
    s.close()
    del s
    torch.cuda.empty_cache()
    return result


def cpu_baseline_train(cfg, seconds):
    """fp64 oracle training step (forward, backward, AdamW) of a one-layer
    model of the same width over one 2048-token sequence, split into the
    layer's share and the embedding/head share, scaled to the run's layers
    and batch."""
    import dataclasses

    import numpy as np
    from oracle import train as ot
    from workloads import init as winit
    from workloads import trace
    threads, vendor = blas_info()
    c1 = dataclasses.replace(cfg, n_layers=1, batch=1, iterations=1)
    w1 = trace.build(c1)
    names = winit.param_names(w1)
    P = winit.weights_f64(w1, names=names)
    ids = winit.token_ids(c1.seed, 1, c1.prompt_len, c1.vocab)
    labels = winit.next_token_labels(ids)
    reps, t_all, t_head = 0, 0.0, 0.0
    t_start = time.perf_counter()
    while reps == 0 or time.perf_counter() - t_start < seconds:
        t = time.perf_counter()
        lg, cache = ot.forward(c1, P, ids)
        loss, dl = ot.cross_entropy(lg, labels)
        ot.backward(c1, P, ids, cache, dl)
        t_all += time.perf_counter() - t
        t = time.perf_counter()           # the head's share: logits, loss, both head gradients
        hf = cache["hf"]
        lg2 = ot.linear(hf, P["head"])
        ot.cross_entropy(lg2, labels)
        _ = dl.T @ hf, dl @ P["head"]
        t_head += time.perf_counter() - t
        reps += 1
    t_all, t_head = t_all / reps, t_head / reps
    # AdamW over one layer's parameters
    lw = [n for n in names if n.startswith("L0.")]
    t = time.perf_counter()
    for n in lw:
        ot.adamw(P[n], P[n], P[n], np.abs(P[n]), 10, 1e-4, 0.9, 0.95, 1e-8, 0.1)
    t_adam_layer = time.perf_counter() - t
    seq_s = t_head + (t_all - t_head + t_adam_layer) * cfg.n_layers
    step_s = seq_s * cfg.batch
    return {"value": cfg.tokens / step_s, "unit": "tokens/s", "cores": threads, "kind": "oracle", "blas": vendor,
            "cpu": cpu_model(), "precision": "fp64",
            "sample": f"fp64 numpy oracle training step (forward, backward, AdamW) of a 1-layer model of the "
                      f"same width over one {cfg.prompt_len}-token sequence, timed over {reps} repetitions; "
                      f"the layer's share ({t_all - t_head + t_adam_layer:.2f} s) scaled to {cfg.n_layers} layers "
                      f"plus the head's ({t_head:.2f} s), times {cfg.batch} sequences ({step_s:.1f} s per step)"}


def train_main(args, cfg):
    """Training steps of the LLaMA-style model: warmup steps, then K timed."""
    import dataclasses

    import torch

    from paper_2609_06172_amd.session import Session
    from workloads import trace
    from workloads.format import OP_ATTN_BWD, OP_LINEAR, OP_LINEAR_RESID

    num, den = cfg.factor
    W = max(1, args.warmup)
    K = 2 if args.steps is None else args.steps
    n_layers = cfg.n_layers
    layers = args.layers or cfg.n_layers
    while layers > 1 and trace.build(dataclasses.replace(cfg, n_layers=layers)).footprint > PINNED_LIMIT:
        layers -= 1
    cfg = dataclasses.replace(cfg, n_layers=layers, iterations=W + K)
    w = trace.build(cfg)
    M = w.budget()
    steps = w.segments["step"]
    log(f"workload {cfg.name}: {layers} of {n_layers} layers, {len(w.tensors)} tensors, "
        f"{len(w.kernels)} kernels ({W + K} steps), footprint {w.footprint} B, budget {M} B")
    bl_meas = link_bandwidth()
    t = time.perf_counter()
    guard = TRAIN_GUARD if args.guard is None else args.guard
    s = Session(w, device=0, M=M, variant=4, timing=1, guard=guard)
    log(f"session ready in {time.perf_counter() - t:.1f} s")

    def run(sess):
        torch.cuda.synchronize()
        t = time.perf_counter()
        sess.run(steps[0][0], steps[W][0] - steps[0][0])
        torch.cuda.synchronize()
        cold = time.perf_counter() - t
        k0, k1 = steps[W][0], steps[-1][0] + steps[-1][1]
        t = time.perf_counter()
        sess.run(k0, k1 - k0)
        torch.cuda.synchronize()
        return cold, time.perf_counter() - t, k0, k1

    cold_s, hot_s, k0, k1 = run(s)
    log(f"{W} warmup step(s) {cold_s:.2f} s, {K} timed steps {hot_s:.2f} s")
    sched, classes = s.ctx.get_schedule(), s.ctx.get_classes()
    dur, gap = s.ctx.get_kernel_times()
    tl = s.ctx.get_timeline()
    loss = float(s.read("losses").astype("float64").mean())
    st = seg_stats(w, sched, classes, M, steps[W:])
    tokens = cfg.tokens * K
    lin = [k for k in range(k0, k1) if w.kernels[k].op in (OP_LINEAR, OP_LINEAR_RESID)
           and w.kernels[k].shape[2] % 64 == 0 and w.kernels[k].shape[0] >= 512]
    g_flops = sum(classes[k][2] for k in lin)
    g_time = sum(dur[k] for k in lin) * 1e-3
    ab = [k for k in range(k0, k1) if w.kernels[k].op == OP_ATTN_BWD]
    per_tag = {}
    for k in range(k0, k1):
        tag = w.kernels[k].tag.split(".")[-1] if "." in w.kernels[k].tag else w.kernels[k].tag
        per_tag[tag] = per_tag.get(tag, 0.0) + dur[k]
    pr = roofline_fields(st, hot_s, bl_meas, tokens)
    pr["roofline_tok_s"] = pr.pop("roofline_units_per_s")
    result = {
        "metric": metric("training ", num, den), "value": round(tokens / hot_s, 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": round(hot_s / K * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shape training step: {layers} of the model's {n_layers} layers (host "
                               f"backing limited to the pinned memory the host grants), hidden {cfg.hidden}, "
                               f"SwiGLU {cfg.ffn}, vocab {cfg.vocab}, {cfg.batch} x {cfg.prompt_len} tokens, bf16 "
                               f"weights with fp32 master weights and AdamW moments, budget = footprint*{den}/{num}",
                   "tokens_per_step": cfg.tokens, "layers": layers, "model_layers": n_layers,
                   "factor": f"{num}/{den}", "footprint_bytes": w.footprint, "budget_bytes": M,
                   "policy": f"T+A+P (guard {guard})"},
        "path_roofline": pr,
        "roofline": {"kernel": "GEMMs of the step (forward, data and weight gradients; bf16 matrix cores)",
                     "bound": "mfma", "achieved": round(g_flops / g_time / 1e12, 1), "peak": 2500.0,
                     "unit": "TFLOP/s", "frac": round(g_flops / g_time / 2.5e15, 4), "traffic": None,
                     "launches": len(lin), "avg_us": round(g_time / max(1, len(lin)) * 1e6, 2)},
        "attention_backward": {"launches": len(ab), "ms_per_step": round(sum(dur[k] for k in ab) / K, 2),
                               "TFLOPs": round(sum(classes[k][2] for k in ab) / max(1e-9, sum(dur[k] for k in ab) * 1e-3)
                                               / 1e12, 1)},
        "kernel_ms_per_step_by_tag": {t_: round(v / K, 2) for t_, v in sorted(per_tag.items(), key=lambda x: -x[1])[:12]},
        "transfers": {"h2d_bytes_per_step": st["h2d_bytes"] // K, "d2h_bytes_per_step": st["d2h_bytes"] // K,
                      "lmin_bytes_per_step": st["lmin_bytes"] // K,
                      "lmin_d2h_bytes_per_step": st["lmin_d2h_bytes"] // K,
                      "link_over_lmin": round((st["h2d_bytes"] + st["d2h_bytes"])
                                              / max(1, st["lmin_bytes"] + st["lmin_d2h_bytes"]), 4),
                      "compute_busy_ms_per_step": round(sum(dur[k] for k in range(k0, k1)) / K, 2),
                      "link_timeline": link_timeline(tl, K)},
        "loss_last_step": round(loss, 5),
        "warmup_seconds": round(cold_s, 3),
    }
    if not args.no_baseline:
        s.set_policy(variant=0, timing=0)
        s.ctx.reset()
        s.restore_inputs()
        _, hot_b, _, _ = run(s)
        result["no_prefetch_baseline"] = {"policy": "demand fetch at launch, LRU eviction",
                                          "value": round(tokens / hot_b, 1), "ms_per_step": round(hot_b / K * 1e3, 3),
                                          "speedup_of_T+A+P": round(hot_b / hot_s, 3)}
    s.close()
    del s
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_train(cfg, args.cpu_seconds)
    emit(args, result)


def moe_main(args, cfg):
    """Routed-expert decode: a profiling run with every expert in the trace,
    then the recorded trace (routed experts only), both timed."""
    import torch

    from paper_2609_06172_amd.session import Session
    from workloads import trace
    from workloads.format import OP_MOE_DOWN, OP_MOE_UP

    import dataclasses

    num, den = cfg.factor
    W, K = args.warmup, (4 if args.steps is None else args.steps)
    if W + K > cfg.decode_steps or K < 1:
        sys.exit(f"warmup + steps must be within 1..{cfg.decode_steps}")
    n = W + K
    # The GPU host pins about 64 GiB: a model whose host backing is larger
    # (115.6 GB for the 8 x 14336 model) keeps PINNED_LIMIT of it pinned and
    # the rest of its read-only weights in pageable memory, fetched through the
    # library's pinned staging ring (a tiered arena).
    n_layers = cfg.n_layers
    cfg = dataclasses.replace(cfg, n_layers=args.layers or cfg.n_layers)
    full = trace.build(cfg, steps=n)
    M = full.budget()
    log(f"workload {cfg.name}: {len(full.tensors)} tensors, {len(full.kernels)} kernels "
        f"(every expert), footprint {full.footprint} B, budget {M} B")
    bl_meas = link_bandwidth()
    t = time.perf_counter()
    s = Session(full, device=0, M=M, variant=4, timing=1, guard=args.guard, pinned_limit=PINNED_LIMIT)
    pinned = s.pinned_bytes
    log(f"session ready in {time.perf_counter() - t:.1f} s (host arena: {pinned} B pinned, "
        f"{full.arena_bytes - pinned} B pageable)")
    pf_prefill, pf_decode, a0, a1 = run_decode(s, full, W, K)
    counts = s.routing_counts().copy()
    gen_prof = s.read("gen")[: n + 1].copy()
    st_prof = seg_stats(full, s.ctx.get_schedule(), s.ctx.get_classes(), M, full.segments["decode"][W:n])
    used_p, idle_p = expert_fetches(full, s.ctx.get_schedule(), counts, a0, a1)
    log(f"profiling run: prefill {pf_prefill:.2f} s, decode {K} steps {pf_decode:.2f} s")

    routed = trace.build(cfg, counts, steps=n)
    s.retrace(routed)
    s.restore_inputs()
    prefill_s, decode_s, k0, k1 = run_decode(s, routed, W, K)
    log(f"recorded trace: prefill {prefill_s:.2f} s, decode {K} steps {decode_s:.2f} s")
    sched, classes = s.ctx.get_schedule(), s.ctx.get_classes()
    dur, gap = s.ctx.get_kernel_times()
    tl = s.ctx.get_timeline()
    gen = s.read("gen")[: n + 1].copy()
    same_routing = bool((s.routing_counts() == counts).all())
    st = seg_stats(routed, sched, classes, M, routed.segments["decode"][W:n])
    used_r, idle_r = expert_fetches(routed, sched, counts, k0, k1)
    ex = [k for k in range(k0, k1) if routed.kernels[k].op in (OP_MOE_UP, OP_MOE_DOWN)]
    g_bytes = sum(classes[k][3] for k in ex)
    g_time = sum(dur[k] for k in ex) * 1e-3
    tok_s = cfg.batch * K / decode_s
    pr = roofline_fields(st, decode_s, bl_meas, cfg.batch * K)
    pr["roofline_tok_s"] = pr.pop("roofline_units_per_s")
    routed_per_layer = float((counts[1 + W:1 + n] > 0).sum(axis=2).mean())
    result = {
        "metric": metric("", num, den), "value": round(tok_s, 3), "unit": "tokens/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(decode_s / K * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shape MoE decode: {cfg.n_layers} of the model's {n_layers} layers, "
                               f"hidden {cfg.hidden}, "
                               f"{cfg.n_experts} SwiGLU experts of {cfg.ffn}, top-{cfg.top_k} routing, "
                               f"vocab {cfg.vocab}, batch {cfg.batch}, {cfg.prompt_len}-token prompt then "
                               f"greedy steps, budget = footprint*{den}/{num}",
                   "batch": cfg.batch, "prompt_len": cfg.prompt_len, "factor": f"{num}/{den}",
                   "layers": cfg.n_layers, "model_layers": n_layers,
                   "footprint_bytes": full.footprint, "budget_bytes": M,
                   "host_arena": {"pinned_bytes": pinned, "pageable_bytes": full.arena_bytes - pinned},
                   "policy": "T+A+P on the recorded (routed-expert) trace"},
        "path_roofline": pr,
        "roofline": {"kernel": "routed-expert GEMV (M = 8 rows, routed rows only, bf16 matrix cores)",
                     "bound": "hbm", "achieved": round(g_bytes / g_time / 1e9, 1), "peak": 8000.0,
                     "unit": "GB/s", "frac": round(g_bytes / g_time / 8e12, 4), "traffic": None,
                     "launches": len(ex), "avg_us": round(g_time / max(1, len(ex)) * 1e6, 2),
                     "avg_bytes": int(g_bytes / max(1, len(ex)))},
        "transfers": {"h2d_bytes_per_step": st["h2d_bytes"] // K, "lmin_bytes_per_step": st["lmin_bytes"] // K,
                      "h2d_over_lmin": round(st["h2d_bytes"] / max(1, st["lmin_bytes"]), 4),
                      "d2h_bytes_per_step": st["d2h_bytes"] // K,
                      "achieved_h2d_GBps": round(st["h2d_bytes"] / decode_s / 1e9, 2),
                      "compute_busy_ms_per_step": round(sum(dur[k] for k in range(k0, k1)) / K, 3),
                      "link_timeline": link_timeline(tl, K)},
        "routing": {"experts_routed_per_layer": round(routed_per_layer, 3), "of": cfg.n_experts,
                    "expert_bytes_fetched_per_step": used_r // K,
                    "same_routing_as_profile": same_routing,
                    "tokens_identical": bool((gen == gen_prof).all())},
        "profiling_trace": {"policy": "T+A+P with every expert in the trace (each expert's weights fetched "
                                      "for each layer whether routed rows or not)",
                            "value": round(cfg.batch * K / pf_decode, 3), "ms_per_step": round(pf_decode / K * 1e3, 3),
                            "h2d_bytes_per_step": st_prof["h2d_bytes"] // K,
                            "expert_bytes_fetched_per_step": used_p // K,
                            "unrouted_expert_bytes_fetched_per_step": idle_p // K,
                            "speedup_of_recorded_trace": round(pf_decode / decode_s, 3)},
        "prefill": {"seconds": round(prefill_s, 3), "tokens": cfg.batch * cfg.prompt_len},
    }
    if not args.no_baseline:
        Bk = min(args.baseline_steps, K)
        b = decode_policy(s, routed, M, 0, W, Bk, gen)
        b["policy"] = "demand fetch at launch, LRU eviction (recorded trace)"
        b["speedup_of_T+A+P"] = round(tok_s / b["value"], 3)
        result["no_prefetch_baseline"] = b
    s.close()
    del s
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_moe(cfg, full, args.cpu_seconds, cfg.prompt_len + W)
    emit(args, result)


def emit(args, result):
    """Print the bench line; a victim guard or separate q, k, v projections set on
    the command line are part of its config."""
    if args.guard is not None:
        result.setdefault("config", {})["guard"] = args.guard
    if args.separate_qkv:
        result.setdefault("config", {})["qkv"] = "separate"
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU: the library has no multi-GPU path; it measures "
              "one GPU's share of the hot path (--gpus 1)", file=sys.stderr)
        sys.exit(2)
    import dataclasses

    from workloads import configs

    cfg = configs.CONFIGS[args.config]
    if args.factor:
        cfg = dataclasses.replace(cfg, factor=factor_of(args.factor))
    if args.separate_qkv:
        cfg = dataclasses.replace(cfg, fuse_qkv=False)
    if cfg.style == "gpt":
        prefill_main(args, cfg)
    elif cfg.style == "moe":
        moe_main(args, cfg)
    elif cfg.style == "train":
        train_main(args, cfg)
    elif args.sweep:
        sweep_main(args, cfg)
    else:
        decode_main(args, cfg)


if __name__ == "__main__":
    main()
