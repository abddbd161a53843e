"""Numeric codes of the trace format (tensor dtypes, kinds, access modes, ops).

These are the wire values of the C interface in ``include/autouvm.h``; a trace
is a list of tensors and an ordered list of kernels, each kernel naming an op,
up to eight shape integers and its operand tensors with an access mode.  This
is the kernel--tensor access record that the paper's profiler collects
(Sec. IV-D, "Kernel--Tensor Access Tracing"); here the workload generator
writes it directly.
"""

# tensor element types
DT_F32, DT_BF16, DT_I32, DT_U8 = 0, 1, 2, 3
DT_SIZE = {DT_F32: 4, DT_BF16: 2, DT_I32: 4, DT_U8: 1}
DT_NAME = {DT_F32: "f32", DT_BF16: "bf16", DT_I32: "i32", DT_U8: "u8"}

# tensor kinds
KIND_PARAM, KIND_ACT, KIND_KV = 0, 1, 2

# registration flags
FLAG_HOST_INIT = 1
FLAG_LIVE_OUT = 2      # final value read after the trace: written back, never dropped

# operand access modes
MODE_R, MODE_W, MODE_RW = 1, 2, 3

# kernel ops (shape integers listed per op)
OP_TOUCH = 0          # (n_words_checked,)  operands: log RW, then data operands
OP_EMBED = 1          # (T, H, V)            ids R, E R, x W
OP_LAYERNORM = 2      # (T, H, row_stride, row_offset)  x R, g R, b R, h W
OP_RMSNORM = 3        # (T, H, row_stride, row_offset)  x R, g R, h W
OP_LINEAR = 4         # (M, N, K)            a R, W R, c W          c = a W^T
OP_LINEAR_GELU = 5    # (M, N, K)            a R, W R, c W          c = gelu(a W^T)
OP_LINEAR_RESID = 6   # (M, N, K)            a R, W R, x RW         x += a W^T
OP_LINEAR_SWIGLU = 7  # (M, N, K)            a R, Wg R, Wu R, c W   c = silu(a Wg^T) * (a Wu^T)
OP_ATTN_QKV = 8       # (B, S, nH, d)        qkv R, o W   causal, fused qkv rows
OP_ROPE_KV = 9        # (B, S, nH, d, Lmax, pos0)  q RW, k R, v R, Kc W|RW, Vc W|RW
OP_ATTN_CACHE = 10    # (B, S, nH, d, Lmax, pos0)  q R, Kc R, Vc R, o W
OP_ARGMAX = 11        # (B, V, gen_row)      logits R, tok W [, gen RW]
OP_MOE_ROUTE = 12     # (M, H, E, K)         h R, Wr R, rte W, rtw W    top-K of E router logits
OP_MOE_DISPATCH = 13  # (M, E, K, log_row)   rte R, lists W, log RW     per-expert ordered row lists
OP_MOE_UP = 14        # (M, F, H, e, n, K)   h R, lists R, Wg R, Wu R, fe W   routed rows of expert e
OP_MOE_DOWN = 15      # (M, H, F, e, n, K)   fe R, lists R, rtw R, Wd R, x RW  weighted scatter-add
# training step (backward and update)
OP_COPY = 16          # (nbytes,)            a R, b W
OP_TRANSPOSE = 17     # (R, C)               a R [R,C], b W [C,R]
OP_SWIGLU_ACT = 18    # (T, F)               G R, U R, F W          F = silu(G) * U
OP_SWIGLU_BWD = 19    # (T, F)               G R, U R, dF R, dG W, dU W
OP_RMSNORM_BWD = 20   # (T, H, acc)          x R, g R, dy R, dx W|RW, dxb W, dg W, rstd W
OP_ATTN_BWD = 21      # (B, S, nH, d)        q R, K R, V R, o R, lse R, do R, dq W, dK W, dV W, D W
OP_ROPE_BWD = 22      # (B, S, nH, d)        dq RW, dK R, dV R, dk W, dv W
OP_XENT = 23          # (T, V)               logits R, labels R, losses W, dlogits W
OP_EMBED_BWD = 24     # (T, H, V)            ids R, dx R, dE W
OP_ADAM = 25          # (n, step, lr*1e9, b1*1e6, b2*1e6, eps*1e12, wd*1e6)  g R, p32 RW, m RW, v RW, p W
OP_LINEAR_QKV = 26    # (M, N, K)            a R, Wq R, Wk R, Wv R, q W, k W, v W   q = a Wq^T (k, v alike)

OP_NAMES = {
    OP_TOUCH: "touch", OP_EMBED: "embed", OP_LAYERNORM: "layernorm",
    OP_RMSNORM: "rmsnorm", OP_LINEAR: "linear", OP_LINEAR_GELU: "linear_gelu",
    OP_LINEAR_RESID: "linear_resid", OP_LINEAR_SWIGLU: "linear_swiglu",
    OP_ATTN_QKV: "attn_qkv", OP_ROPE_KV: "rope_kv", OP_ATTN_CACHE: "attn_cache",
    OP_ARGMAX: "argmax", OP_MOE_ROUTE: "moe_route", OP_MOE_DISPATCH: "moe_dispatch",
    OP_MOE_UP: "moe_up", OP_MOE_DOWN: "moe_down", OP_COPY: "copy", OP_TRANSPOSE: "transpose",
    OP_SWIGLU_ACT: "swiglu_act", OP_SWIGLU_BWD: "swiglu_bwd", OP_RMSNORM_BWD: "rmsnorm_bwd",
    OP_ATTN_BWD: "attn_bwd", OP_ROPE_BWD: "rope_bwd", OP_XENT: "xent", OP_EMBED_BWD: "embed_bwd",
    OP_ADAM: "adam", OP_LINEAR_QKV: "linear_qkv",
}

# planner policy variants (paper's ablation ladder plus the two demand baselines)
VAR_DEMAND_LRU, VAR_DEMAND_BELADY, VAR_T, VAR_T_A, VAR_T_A_P = 0, 1, 2, 3, 4
PLACE_POOL, PLACE_IDEAL = 0, 1

# schedule entry ops
S_H2D_PREFETCH, S_H2D_DEMAND, S_D2H_WRITEBACK, S_DROP, S_ALLOC, S_LAUNCH = 0, 1, 2, 3, 4, 5
S_NAMES = {S_H2D_PREFETCH: "H2D_PREFETCH", S_H2D_DEMAND: "H2D_DEMAND",
           S_D2H_WRITEBACK: "D2H_WRITEBACK", S_DROP: "DROP", S_ALLOC: "ALLOC",
           S_LAUNCH: "LAUNCH"}

# roofline classes
CLS_COMPUTE, CLS_MEMORY, CLS_CGI = 0, 1, 2

ALIGN = 256
