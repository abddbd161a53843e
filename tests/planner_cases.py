"""Trace helpers shared by the planner tests (oracle pins and C-ABI parity)."""
import json
import os
import random

from workloads.format import DT_U8, KIND_ACT, KIND_KV, KIND_PARAM, OP_TOUCH

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "planner_cases.json")


def load_golden():
    with open(GOLDEN) as f:
        return json.load(f)


def golden_inputs(case):
    kinds = {"param": KIND_PARAM, "act": KIND_ACT, "kv": KIND_KV}
    tensors = [dict(nbytes=e[0], dtype=DT_U8, kind=kinds[e[1]],
                    host_init=(e[1] == "param"), live_out=(len(e) > 2 and e[2] == "out"))
               for e in case["tensors"]]
    n = len(case["kernels"])
    flops = case.get("flops", [1] * n)
    times = case.get("times", [0] * n)
    kernels = [dict(op=OP_TOUCH, shape=(0,), operands=[tuple(o) for o in ops],
                    flops=f, hbm_bytes=1, time_ns=t)
               for ops, f, t in zip(case["kernels"], flops, times)]
    return tensors, kernels


def random_trace(seed, n_tensors=None, n_kernels=None, max_ops=4, equal=False,
                 read_only=False, unit=256, touch=False, timed=False, live_out=False, kv=False):
    """Random trace of touch kernels with explicit or analytic costs.

    touch=True makes every kernel a well-formed touch op: tensor 0 is a log
    (read-write operand 0 of every kernel, one 64-byte slot per kernel), data
    operands are distinct and their sizes are multiples of 4 bytes.
    timed=True gives most kernels a measured time (time_ns) drawn around the
    link time of a few hundred bytes, so both sides of the measured-time rule
    occur.  live_out=True marks about a third of the tensors live-out.
    kv=True makes about half of the non-parameter tensors KV-cache tensors.
    """
    r = random.Random(seed)
    nT = n_tensors or r.randint(1, 40)
    nK = n_kernels or r.randint(1, 200)
    tensors = []
    sizes = [4, 200, 256, 300, 512, 1000, 2048, 4096, 776] if touch else \
        [1, 200, 256, 300, 512, 1000, 2048, 4096, 777]
    for t in range(nT):
        kind = KIND_PARAM if (read_only or r.random() < 0.6) else KIND_ACT
        if kv and kind == KIND_ACT and r.random() < 0.5:
            kind = KIND_KV
        nbytes = unit if equal else r.choice(sizes)
        tensors.append(dict(nbytes=nbytes, dtype=DT_U8, kind=kind,
                            host_init=(kind == KIND_PARAM or r.random() < 0.3),
                            live_out=live_out and r.random() < 0.35))
    if touch:
        tensors.insert(0, dict(nbytes=64 * nK, dtype=DT_U8, kind=KIND_ACT, host_init=True))
    first = 1 if touch else 0
    written = set(t for t in range(len(tensors)) if tensors[t]["host_init"])
    kernels = []
    for k in range(nK):
        n = r.randint(1, max_ops)
        ops = []
        for _ in range(n):
            t = r.randrange(first, len(tensors))
            if touch and any(t == u for u, _ in ops):
                continue
            if read_only:
                m = 1
            elif t in written:
                m = r.choice([1, 1, 1, 2, 3])
            else:
                m = 2
            ops.append((t, m))
        written.update(t for t, m in ops if m & 2)
        if r.random() < 0.5:
            fl, hb = r.choice([(1, 1), (10**12, 10**6), (10**6, 10**9), (0, 0)])
        else:
            fl, hb = 0, 0
        if touch:
            ops = [(0, 3)] + ops
        kd = dict(op=OP_TOUCH, shape=(k if touch else 0,), operands=ops, flops=fl, hbm_bytes=hb)
        if timed and r.random() < 0.8:
            kd["time_ns"] = r.choice([1, 2, 3, 5, 8, 13, 40, 10**6])
        kernels.append(kd)
    return tensors, kernels


def oracle_routing_counts(cfg):
    """Per-expert row counts [seg][layer][expert] of the fp64 oracle's own
    greedy run of an MoE config (what the dispatch kernels would log)."""
    import numpy as np

    from oracle import forward as of
    from workloads import init, trace
    w = trace.build(cfg)
    Wt = init.weights_f64(w)
    ids = init.token_ids(cfg.seed, cfg.batch, cfg.prompt_len, cfg.vocab)
    gen = of.llama_generate(cfg, Wt, ids)
    counts = np.zeros((1 + cfg.decode_steps, cfg.n_layers, cfg.n_experts), np.int64)
    for seg, layers in enumerate(gen["routes"]):
        for l, (idx, _, _) in enumerate(layers):
            counts[seg, l] = np.bincount(idx.reshape(-1), minlength=cfg.n_experts)
    return counts


def random_routing_counts(cfg, seed):
    """Counts of a seeded random top-k choice per token (planning inputs only)."""
    import numpy as np
    rng = np.random.default_rng(seed)
    counts = np.zeros((1 + cfg.decode_steps, cfg.n_layers, cfg.n_experts), np.int64)
    for seg in range(1 + cfg.decode_steps):
        M = cfg.tokens if seg == 0 else cfg.batch
        for l in range(cfg.n_layers):
            pick = np.argsort(rng.random((M, cfg.n_experts)), axis=1)[:, :cfg.top_k]
            counts[seg, l] = np.bincount(pick.reshape(-1), minlength=cfg.n_experts)
    return counts
