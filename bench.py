#!/usr/bin/env python3
"""Decode throughput of a 7B-shape decoder whose tensors oversubscribe the
device budget 1.5x, with tensor-granular roofline-gated prefetching.

One step = one greedy decode step of the whole model at batch 16 (every layer's
transfers and kernels, scheduled by the planner).  The job is a 1024-token
prompt (prefill, untimed, reported) followed by up to 256 decode steps; W steps
are run untimed, then K steps are timed between two device synchronisations.

Reported next to the value (one JSON line on stdout):
  * path_roofline: max(F/P, B/Bh, L/Bl) for the timed steps, with L the
    tensor-granular lower bound on host-to-device bytes (bytes the steps read
    before writing minus the budget), at nominal MI355X roofs and at the host
    link measured in the same run;
  * roofline: the decode projection GEMV kernels (the dominant compute
    kernels), algorithmic bytes over their average duration from HIP events;
  * no_prefetch_baseline: the same engine with fault-driven demand fetches and
    LRU eviction;
  * cpu_baseline: the CPU oracle on a bounded sample of the same decode.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tokens/sec at 1.5x oversubscription; fraction of max(compute,HBM,link) roofline"
NOMINAL = dict(P=2.5e15, Bh=8.0e12, Bl=64.0e9)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256, help="timed decode steps")
    ap.add_argument("--warmup", type=int, default=0, help="untimed decode steps before")
    ap.add_argument("--config", default="llama-7b")
    ap.add_argument("--factor", default="3/2", help="oversubscription factor num/den")
    ap.add_argument("--baseline-steps", type=int, default=8)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-baseline", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run one 256 MiB device-to-device copy kernel (a known-size "
                         "reference for hardware byte counters)")
    return ap.parse_args()


def link_bandwidth():
    """Pinned host-to-device copy rate measured with torch (1 GiB, best of 3)."""
    import torch
    n = 1 << 30
    h = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(n, dtype=torch.uint8, device="cuda")
    best = 0.0
    for _ in range(4):
        torch.cuda.synchronize()
        t = time.perf_counter()
        d.copy_(h, non_blocking=True)
        torch.cuda.synchronize()
        best = max(best, n / (time.perf_counter() - t))
    del h, d
    return best


def counted_traffic():
    """HBM bytes per GEMV launch from the committed counter runs, if the kernel
    source is unchanged since they were taken (else None)."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", "gemv_mfma_traffic_llama7b_decode.json")
    src = os.path.join(ROOT, "paper_2609_06172_amd", "csrc", "kernels", "gemv.hip")
    try:
        meta = json.load(open(prof))
        if hashlib.sha256(open(src, "rb").read()).hexdigest() != meta["kernel_source_sha256"]:
            return None
        return int(meta["traffic_bytes_per_launch"])
    except (OSError, ValueError, KeyError):
        return None


def step_stats(w, sched, classes, M, k0, k1):
    """Work and transfers of kernels k0..k1-1 (whole decode steps)."""
    from workloads.format import MODE_R
    F = sum(c[2] for c in classes[k0:k1])
    B = sum(c[3] for c in classes[k0:k1])
    lmin = 0
    for a, n in w.segments["decode"]:
        if a < k0 or a + n > k1:
            continue
        first = {}
        for kd in w.kernels[a:a + n]:
            merged = {}
            for t, m in kd.operands:
                merged[t] = merged.get(t, 0) | m
            for t, m in merged.items():
                first.setdefault(t, m)
        read = sum((w.tensors[t].nbytes + 255) // 256 * 256 for t, m in first.items() if m & MODE_R)
        lmin += max(0, read - M)
    h2d = sum(e[3] for e in sched if e[0] in (0, 1) and k0 <= e[4] < k1)
    d2h = sum(e[3] for e in sched if e[0] == 2 and k0 <= e[4] < k1)
    demand = sum(1 for e in sched if e[0] == 1 and k0 <= e[4] < k1)
    return dict(flops=F, hbm_bytes=B, lmin_bytes=lmin, h2d_bytes=h2d, d2h_bytes=d2h,
                demand_fetches=demand)


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
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    s.run(first, nk)
    torch.cuda.synchronize()
    return prefill_s, time.perf_counter() - t0, first, first + nk


def link_timeline(tl, K):
    """Host-to-device link over the timed run segment (the last one): busy and
    idle time, and the part of each idle gap during which the host had not yet
    issued the next copy (host and device clocks share the segment's start)."""
    from paper_2609_06172_amd.capi import TL_H2D
    seg = max(e[1] for e in tl)
    cur = [e for e in tl if e[1] == seg]
    h = sorted((e for e in cur if e[0] == TL_H2D), key=lambda e: e[5])
    span = max(e[6] for e in cur)
    busy = sum(e[6] - e[5] for e in h)
    late, prev = 0.0, 0.0
    for e in h:
        late += max(0.0, min(e[5], e[4]) - prev)
        prev = e[6]
    nbytes = sum(e[3] for e in h)
    return {"h2d_busy_ms_per_step": round(busy / K, 3), "h2d_idle_ms_per_step": round((span - busy) / K, 3),
            "idle_before_host_issue_ms_per_step": round(late / K, 3),
            "h2d_GBps_while_busy": round(nbytes / (busy * 1e-3) / 1e9, 2) if busy > 0 else None,
            "copies_per_step": round(len(h) / K, 2)}


def cpu_baseline(cfg, w, seconds, pos):
    """fp64 oracle decode of a few layers at the timed position, scaled to the model."""
    import numpy as np
    from oracle import forward as of
    from workloads import init as winit
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        threads = max((i.get("num_threads", 1) for i in info), default=1)
        vendor = ",".join(sorted(set(i.get("internal_api", "?") for i in info)))
    except Exception:
        threads, vendor = len(os.sched_getaffinity(0)), "unknown"
    from concurrent.futures import ThreadPoolExecutor
    L = 2
    B, nH, d, Lmax = cfg.batch, cfg.n_heads, cfg.head_dim, cfg.kv_len
    names = [f"L{l}.{nm}" for l in range(L) for nm in
             ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd")] + ["head", "norm_f"]

    def weight(nm):
        return nm, winit.tensor_value(w, w.tensors[w.id(nm)]).astype(np.float64)

    def cache(i):   # synthetic prefix of the KV cache (values do not change the timing)
        g = np.random.default_rng([7, i])
        return g.standard_normal((B, nH, Lmax, d), dtype=np.float32).astype(np.float64) * 0.5

    with ThreadPoolExecutor(16) as ex:
        Wt = dict(ex.map(weight, names))
        kv = list(ex.map(cache, range(2 * L)))
    Wl = [({nm.split(".", 1)[1]: v for nm, v in Wt.items() if nm.startswith(f"L{l}.")},
           kv[2 * l], kv[2 * l + 1]) for l in range(L)]
    head, gf = Wt["head"], Wt["norm_f"]
    x0 = np.random.default_rng(8).standard_normal((B, cfg.hidden)) * 0.02
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
    step_s = t_layers / reps / L * cfg.n_layers + t_head
    return {"value": B / step_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "blas": vendor,
            "sample": f"fp64 numpy oracle decode step at position {pos}, batch {B}: {L} of "
                      f"{cfg.n_layers} layers timed over {reps} repetitions plus the LM head, "
                      f"scaled to {cfg.n_layers} layers ({step_s:.2f} s per step)"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU: this build has no multi-GPU path "
              "(the per-GPU hot path is what it measures)", file=sys.stderr)
        sys.exit(2)
    import dataclasses

    import numpy as np
    import torch

    from paper_2609_06172_amd.session import Session
    from workloads import configs, trace
    from workloads.format import OP_LINEAR, OP_LINEAR_GELU, OP_LINEAR_RESID, OP_LINEAR_SWIGLU

    num, den = (int(x) for x in args.factor.split("/"))
    cfg = dataclasses.replace(configs.CONFIGS[args.config], factor=(num, den))
    W, K = args.warmup, args.steps
    if W + K > cfg.decode_steps or K < 1:
        sys.exit(f"warmup + steps must be within 1..{cfg.decode_steps}")
    w = trace.build(cfg)
    M = w.budget()
    log(f"workload {cfg.name}: {len(w.tensors)} tensors, {len(w.kernels)} kernels, "
        f"footprint {w.footprint} B, budget {M} B")
    if args.calibrate_copy:
        n = 256 << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    bl_meas = link_bandwidth()
    log(f"measured pinned H2D: {bl_meas / 1e9:.1f} GB/s")

    t = time.perf_counter()
    s = Session(w, device=0, M=M, variant=4, timing=1)
    log(f"session ready in {time.perf_counter() - t:.1f} s (plan {s.ctx.get_counters()['plan_ns'] / 1e9:.2f} s)")
    prefill_s, decode_s, k0, k1 = run_decode(s, w, W, K)
    log(f"prefill {prefill_s:.3f} s, decode {K} steps {decode_s:.3f} s")
    sched = s.ctx.get_schedule()
    classes = s.ctx.get_classes()
    dur, gap = s.ctx.get_kernel_times()
    link_tl = link_timeline(s.ctx.get_timeline(), K)
    gen_tap = s.read("gen")[: W + K + 1].copy()
    st = step_stats(w, sched, classes, M, k0, k1)

    # dominant kernels: decode projections (M <= 16 rows) on the matrix cores
    lin = [k for k in range(k0, k1)
           if w.kernels[k].op in (OP_LINEAR, OP_LINEAR_GELU, OP_LINEAR_RESID, OP_LINEAR_SWIGLU)]
    g_bytes = sum(classes[k][3] for k in lin)
    g_time = sum(dur[k] for k in lin) * 1e-3
    g_achieved = g_bytes / g_time / 1e9
    per_op = {}
    for k in range(k0, k1):
        tag = w.kernels[k].tag
        e = per_op.setdefault(tag, [0, 0.0, 0])
        e[0] += 1
        e[1] += dur[k]
        e[2] += classes[k][3]
    stall_ms = sum(gap[k] for k in range(k0 + 1, k1))
    busy_ms = sum(dur[k] for k in range(k0, k1))

    tok_s = cfg.batch * K / decode_s
    t_comp = st["flops"] / NOMINAL["P"]
    t_hbm = st["hbm_bytes"] / NOMINAL["Bh"]
    t_link = st["lmin_bytes"] / NOMINAL["Bl"]
    roof_s = max(t_comp, t_hbm, t_link)
    roof_meas = max(t_comp, t_hbm, st["lmin_bytes"] / bl_meas)
    result = {
        "metric": METRIC, "value": round(tok_s, 3), "unit": "tokens/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(decode_s / K * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shape decode: {cfg.n_layers} layers, hidden {cfg.hidden}, "
                               f"SwiGLU {cfg.ffn}, vocab {cfg.vocab}, batch {cfg.batch}, "
                               f"{cfg.prompt_len}-token prompt then greedy steps, "
                               f"budget = footprint*{den}/{num}",
                   "batch": cfg.batch, "prompt_len": cfg.prompt_len, "factor": f"{num}/{den}",
                   "footprint_bytes": w.footprint, "budget_bytes": M, "policy": "T+A+P"},
        "path_roofline": {
            "bound": ["mfma", "hbm", "link"][int(np.argmax([t_comp, t_hbm, t_link]))],
            "roofline_tok_s": round(cfg.batch * K / roof_s, 3),
            "frac": round(roof_s / decode_s, 4),
            "frac_measured_link": round(roof_meas / decode_s, 4),
            "link_GBps_nominal": NOMINAL["Bl"] / 1e9, "link_GBps_measured": round(bl_meas / 1e9, 2),
            "t_mfma_ms": round(t_comp * 1e3, 3), "t_hbm_ms": round(t_hbm * 1e3, 3),
            "t_link_ms": round(t_link * 1e3, 3), "t_measured_ms": round(decode_s * 1e3, 3)},
        "roofline": {"kernel": "decode projection GEMV (M=16, bf16 matrix cores)", "bound": "hbm",
                     "achieved": round(g_achieved, 1), "peak": 8000.0, "unit": "GB/s",
                     "frac": round(g_achieved / 8000.0, 4), "traffic": counted_traffic(),
                     "launches": len(lin), "avg_us": round(g_time / max(1, len(lin)) * 1e6, 2),
                     "avg_bytes": int(g_bytes / max(1, len(lin)))},
        "transfers": {"h2d_bytes_per_step": st["h2d_bytes"] // K, "d2h_bytes_per_step": st["d2h_bytes"] // K,
                      "lmin_bytes_per_step": st["lmin_bytes"] // K,
                      "h2d_over_lmin": round(st["h2d_bytes"] / max(1, st["lmin_bytes"]), 4),
                      "demand_fetches": st["demand_fetches"],
                      "achieved_h2d_GBps": round(st["h2d_bytes"] / decode_s / 1e9, 2),
                      "compute_busy_ms_per_step": round(busy_ms / K, 3),
                      "compute_stall_ms_per_step": round(stall_ms / K, 3),
                      "link_timeline": link_tl},
        "prefill": {"seconds": round(prefill_s, 3), "tokens": cfg.batch * cfg.prompt_len},
        "per_kernel_ms_per_step": {k: round(v[1] / K, 4) for k, v in sorted(per_op.items())},
    }

    if not args.no_baseline:
        Bk = min(args.baseline_steps, K)
        s.set_policy(variant=0, timing=0)
        s.ctx.reset()
        s.restore_inputs()
        pb, db, _, _ = run_decode(s, w, W, Bk)
        gen_lru = s.read("gen")[: W + Bk + 1]
        result["no_prefetch_baseline"] = {
            "policy": "demand fetch at launch, LRU eviction", "steps": Bk,
            "value": round(cfg.batch * Bk / db, 3), "unit": "tokens/s",
            "ms_per_step": round(db / Bk * 1e3, 3), "prefill_seconds": round(pb, 3),
            "speedup_of_T+A+P": round(tok_s / (cfg.batch * Bk / db), 3),
            "tokens_identical": bool(np.array_equal(gen_lru, gen_tap[: W + Bk + 1]))}
        log(f"baseline {Bk} steps {db:.3f} s")
    s.close()
    del s
    torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, w, args.cpu_seconds, cfg.prompt_len + W)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
