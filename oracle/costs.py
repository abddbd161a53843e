"""Analytic flops F and algorithmic HBM bytes B of each kernel (oracle side).

The paper counts FLOP instructions and memory loads per kernel to place each
kernel on its multi-level roofline (Sec. III-C, Sec. IV-G).  Here the counts
are the algorithmic ones, written per op from its shape: every operand element
is read or written once, a read-modify-write counts twice, and a GEMM costs
2*M*N*K flops; elements an op does not touch (rows it does not gather, cache
positions past the valid prefix) do not count.  Integer arithmetic only.
"""
from workloads.format import (DT_SIZE, MODE_RW, OP_ARGMAX, OP_ATTN_CACHE,
                              OP_ATTN_QKV, OP_EMBED, OP_LAYERNORM, OP_LINEAR,
                              OP_LINEAR_GELU, OP_LINEAR_RESID,
                              OP_LINEAR_SWIGLU, OP_MOE_DISPATCH, OP_MOE_DOWN,
                              OP_MOE_ROUTE, OP_MOE_UP, OP_RMSNORM, OP_ROPE_KV,
                              OP_TOUCH, OP_COPY, OP_TRANSPOSE, OP_SWIGLU_ACT,
                              OP_SWIGLU_BWD, OP_RMSNORM_BWD, OP_ATTN_BWD,
                              OP_ROPE_BWD, OP_XENT, OP_EMBED_BWD, OP_ADAM,
                              OP_LINEAR_QKV)


def kernel_cost(op, shape, operands, dtypes, nbytes):
    """operands: list of (tid, mode) in positional order; dtypes/nbytes by tid.

    Returns (F, B) as Python ints.
    """
    es = [DT_SIZE[dtypes[t]] for t, _ in operands]
    sh = list(shape) + [0] * (8 - len(shape))
    if op == OP_TOUCH:
        seen = {}
        for t, m in operands:
            seen[t] = seen.get(t, 0) | m
        return 0, sum(nbytes[t] * (2 if m == MODE_RW else 1) for t, m in seen.items())
    if op == OP_EMBED:
        T, H = sh[0], sh[1]
        return 0, 4 * T + T * H * es[1] + T * H * es[2]
    if op == OP_LAYERNORM:
        T, H = sh[0], sh[1]
        return 8 * T * H, T * H * es[0] + H * es[1] + H * es[2] + T * H * es[3]
    if op == OP_RMSNORM:
        T, H = sh[0], sh[1]
        return 4 * T * H, T * H * es[0] + H * es[1] + T * H * es[2]
    if op in (OP_LINEAR, OP_LINEAR_GELU, OP_LINEAR_RESID):
        M, N, K = sh[0], sh[1], sh[2]
        F = 2 * M * N * K + {OP_LINEAR: 0, OP_LINEAR_GELU: 8 * M * N, OP_LINEAR_RESID: M * N}[op]
        out = M * N * es[2] * (2 if op == OP_LINEAR_RESID else 1)
        return F, M * K * es[0] + N * K * es[1] + out
    if op == OP_LINEAR_QKV:
        M, N, K = sh[0], sh[1], sh[2]
        return 6 * M * N * K, M * K * es[0] + N * K * (es[1] + es[2] + es[3]) + M * N * (es[4] + es[5] + es[6])
    if op == OP_LINEAR_SWIGLU:
        M, N, K = sh[0], sh[1], sh[2]
        return 4 * M * N * K + 4 * M * N, M * K * es[0] + N * K * (es[1] + es[2]) + M * N * es[3]
    if op == OP_ATTN_QKV:
        Bt, S, nH, d = sh[0], sh[1], sh[2], sh[3]
        pairs = S * (S + 1) // 2
        return Bt * nH * pairs * (4 * d + 4), Bt * S * nH * d * (3 * es[0] + es[1])
    if op == OP_ROPE_KV:
        Bt, S, nH, d = sh[0], sh[1], sh[2], sh[3]
        n = Bt * S * nH * d
        return 6 * n, n * (2 * es[0] + es[1] + es[2] + es[3] + es[4])
    if op == OP_ATTN_CACHE:
        Bt, S, nH, d, pos0 = sh[0], sh[1], sh[2], sh[3], sh[5]
        pairs = S * pos0 + S * (S + 1) // 2
        F = Bt * nH * pairs * (4 * d + 4)
        B = Bt * S * nH * d * (es[0] + es[3]) + Bt * nH * (pos0 + S) * d * (es[1] + es[2])
        if len(operands) > 4:            # row log-sum-exp for the backward pass
            B += 4 * Bt * nH * S
        return F, B
    if op == OP_ARGMAX:
        Bt, V = sh[0], sh[1]
        return Bt * V, Bt * V * es[0] + 4 * Bt + (4 * Bt if len(operands) > 2 else 0)
    # routed experts: n is the number of rows the trace expects expert e to see
    if op == OP_MOE_ROUTE:
        M, H, E, K = sh[0], sh[1], sh[2], sh[3]
        return 2 * M * H * E, M * H * es[0] + E * H * es[1] + 8 * M * K
    if op == OP_MOE_DISPATCH:
        M, E, K = sh[0], sh[1], sh[2]
        return 0, 4 * M * K + 4 * (M * K + E) + 8 * E
    if op == OP_MOE_UP:
        M, F, H, n = sh[0], sh[1], sh[2], sh[4]
        return 4 * n * F * H + 4 * n * F, n * H * es[0] + 4 * (n + 1) + F * H * (es[2] + es[3]) + n * F * es[4]
    if op == OP_MOE_DOWN:
        M, H, F, n = sh[0], sh[1], sh[2], sh[4]
        return 2 * n * H * F + 2 * n * H, n * F * es[0] + 4 * (n + 1) + 4 * n + H * F * es[3] + 8 * n * H
    # training step: every operand element read or written once
    if op == OP_COPY:
        return 0, 2 * sh[0]
    if op == OP_TRANSPOSE:
        return 0, 2 * sh[0] * sh[1] * es[0]
    if op == OP_SWIGLU_ACT:
        T, Fw = sh[0], sh[1]
        return 5 * T * Fw, T * Fw * (es[0] + es[1] + es[2])
    if op == OP_SWIGLU_BWD:
        T, Fw = sh[0], sh[1]
        return 10 * T * Fw, T * Fw * (es[0] + es[1] + es[2] + es[3] + es[4])
    if op == OP_RMSNORM_BWD:
        T, H, acc = sh[0], sh[1], sh[2]
        return (10 * T * H, T * H * (es[0] + es[2] + es[4]) + T * H * es[3] * (2 if acc else 1)
                + H * (es[1] + es[5]) + 4 * T)
    if op == OP_ATTN_BWD:
        Bt, S, nH, d = sh[0], sh[1], sh[2], sh[3]
        pairs = S * (S + 1) // 2
        return (Bt * nH * pairs * (10 * d + 8),
                Bt * S * nH * d * sum(es[i] for i in (0, 1, 2, 3, 5, 6, 7, 8)) + 12 * Bt * nH * S)
    if op == OP_ROPE_BWD:
        n = sh[0] * sh[1] * sh[2] * sh[3]
        return 6 * n, n * (2 * es[0] + es[1] + es[2] + es[3] + es[4])
    if op == OP_XENT:
        T, V = sh[0], sh[1]
        return 4 * T * V, T * V * (es[0] + es[3]) + 8 * T
    if op == OP_EMBED_BWD:
        T, H, V = sh[0], sh[1], sh[2]
        return T * H, 4 * T + T * H * es[1] + V * H * es[2]
    if op == OP_ADAM:
        n = sh[0]
        return 12 * n, n * (es[0] + 2 * es[1] + 2 * es[2] + 2 * es[3] + es[4])
    raise ValueError(f"unknown op {op}")
