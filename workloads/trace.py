"""Tensor lists and kernel access traces of the synthetic decoders.

A workload is what the paper's offline profiler would have recorded for one
inference run (Sec. IV-D): every tensor with its byte size, and the ordered
kernel list where each kernel names the tensors it accesses.  Tensors are
sub-allocations of one pooled arena (Sec. II-B): each gets an arena offset
aligned to 256 bytes, in registration order.

No arithmetic of the method lives here: this module only describes the model's
structure (which kernel touches which tensor, with which mode and shape).
"""
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

from .configs import DecoderConfig
from .format import (ALIGN, DT_F32, DT_I32, DT_SIZE, FLAG_HOST_INIT, FLAG_LIVE_OUT, KIND_ACT,
                     KIND_KV, KIND_PARAM, MODE_R, MODE_RW, MODE_W, OP_ARGMAX,
                     OP_ATTN_CACHE, OP_ATTN_QKV, OP_EMBED, OP_LAYERNORM,
                     OP_LINEAR, OP_LINEAR_GELU, OP_LINEAR_RESID,
                     OP_LINEAR_SWIGLU, OP_LINEAR_QKV, OP_MOE_DISPATCH, OP_MOE_DOWN,
                     OP_MOE_ROUTE, OP_MOE_UP, OP_RMSNORM, OP_ROPE_KV, OP_ADAM,
                     OP_ATTN_BWD, OP_COPY, OP_EMBED_BWD, OP_RMSNORM_BWD,
                     OP_ROPE_BWD, OP_SWIGLU_ACT, OP_SWIGLU_BWD, OP_TRANSPOSE,
                     OP_XENT, DT_BF16)


def align_up(n: int, a: int = ALIGN) -> int:
    return (n + a - 1) // a * a


@dataclass
class TensorSpec:
    name: str
    shape: Tuple[int, ...]
    dtype: int
    kind: int
    host_init: bool
    init: str = "none"       # "normal" (weights), "ones" (norm gains), "zeros", "ids", ...
    off: int = 0             # arena offset
    tid: int = -1
    live_out: bool = False   # final value read after the trace (carried state)

    @property
    def nbytes(self) -> int:
        n = DT_SIZE[self.dtype]
        for s in self.shape:
            n *= s
        return n

    @property
    def flags(self) -> int:
        f = FLAG_HOST_INIT if (self.host_init and self.kind != KIND_PARAM) else 0
        return f | (FLAG_LIVE_OUT if self.live_out else 0)


@dataclass
class KernelSpec:
    op: int
    shape: Tuple[int, ...]
    operands: List[Tuple[int, int]]      # (tensor id, mode) in the op's positional order
    layer: int = 0
    tag: str = ""


@dataclass
class Workload:
    cfg: Optional[DecoderConfig]
    tensors: List[TensorSpec] = field(default_factory=list)
    kernels: List[KernelSpec] = field(default_factory=list)
    by_name: Dict[str, int] = field(default_factory=dict)
    segments: Dict[str, List[Tuple[int, int]]] = field(default_factory=dict)
    arena_bytes: int = 0

    # -- construction helpers -------------------------------------------------
    def tensor(self, name, shape, dtype, kind, host_init=False, init="none", live_out=False) -> int:
        t = TensorSpec(name, tuple(int(s) for s in shape), dtype, kind,
                       host_init or kind == KIND_PARAM, init, live_out=live_out)
        t.tid = len(self.tensors)
        t.off = self.arena_bytes
        self.arena_bytes += align_up(t.nbytes)
        self.tensors.append(t)
        self.by_name[name] = t.tid
        return t.tid

    def kernel(self, op, shape, operands, layer=0, tag="") -> int:
        self.kernels.append(KernelSpec(op, tuple(int(s) for s in shape),
                                       [(int(t), int(m)) for t, m in operands],
                                       layer, tag))
        return len(self.kernels) - 1

    def id(self, name: str) -> int:
        return self.by_name[name]

    # -- derived ---------------------------------------------------------------
    @property
    def footprint(self) -> int:
        """Sum of 256-aligned tensor sizes (what a pooling allocator would hold)."""
        return sum(align_up(t.nbytes) for t in self.tensors)

    def budget(self, num: Optional[int] = None, den: Optional[int] = None) -> int:
        """Device bytes for oversubscription factor num/den, floored to 256."""
        if num is None:
            num, den = self.cfg.factor
        return (self.footprint * den // num) // ALIGN * ALIGN


def build(cfg: DecoderConfig, routing=None, steps=None, keep_grads=False) -> Workload:
    """The workload of a config.

    ``steps`` traces only the first decode steps of a LLaMA-style or MoE
    config; the tensors (KV cache length, logs) stay those of the full run.
    ``keep_grads`` marks a training step's gradients live-out, so that they
    can be read after the step (they are otherwise dead once applied).

    For MoE configs ``routing`` is the per-expert row count of every MoE layer
    in every run segment (prefill, then each decode step), as the dispatch
    kernels log it (``routing[seg][layer][expert]``).  The trace then holds the
    expert kernels of routed experts only.  Without it every expert of every
    layer gets its kernels (the profiling trace), each expected to see all
    rows.
    """
    if cfg.style == "gpt":
        return _build_gpt(cfg)
    if cfg.style in ("llama", "moe"):
        return _build_llama(cfg, routing, cfg.decode_steps if steps is None else steps)
    if cfg.style == "train":
        return _build_train(cfg, keep_grads)
    raise ValueError(cfg.style)


def _build_gpt(c: DecoderConfig) -> Workload:
    w = Workload(c)
    H, F, V, T, B, S = c.hidden, c.ffn, c.vocab, c.tokens, c.batch, c.prompt_len
    dt = c.dtype
    E = w.tensor("E", (V, H), dt, KIND_PARAM, init="normal")
    layers = []
    for l in range(c.n_layers):
        p = f"L{l}."
        layers.append(dict(
            g1=w.tensor(p + "ln1.g", (H,), dt, KIND_PARAM, init="ones"),
            b1=w.tensor(p + "ln1.b", (H,), dt, KIND_PARAM, init="zeros"),
            wqkv=w.tensor(p + "wqkv", (3 * H, H), dt, KIND_PARAM, init="normal"),
            wo=w.tensor(p + "wo", (H, H), dt, KIND_PARAM, init="normal"),
            g2=w.tensor(p + "ln2.g", (H,), dt, KIND_PARAM, init="ones"),
            b2=w.tensor(p + "ln2.b", (H,), dt, KIND_PARAM, init="zeros"),
            w1=w.tensor(p + "w1", (F, H), dt, KIND_PARAM, init="normal"),
            w2=w.tensor(p + "w2", (H, F), dt, KIND_PARAM, init="normal"),
        ))
    gf = w.tensor("lnf.g", (H,), dt, KIND_PARAM, init="ones")
    bf = w.tensor("lnf.b", (H,), dt, KIND_PARAM, init="zeros")
    ids = w.tensor("ids", (T,), DT_I32, KIND_ACT, host_init=True, init="ids")
    x = w.tensor("x", (T, H), DT_F32, KIND_ACT)
    h = w.tensor("h", (T, H), dt, KIND_ACT)
    qkv = w.tensor("qkv", (T, 3 * H), dt, KIND_ACT)
    attn = w.tensor("attn", (T, H), dt, KIND_ACT)
    ffn = w.tensor("ffn", (T, F), dt, KIND_ACT)
    if c.logits_all:
        logits = w.tensor("logits", (T, V), DT_F32, KIND_ACT)
    else:
        hl = w.tensor("hl", (B, H), dt, KIND_ACT)
        logits = w.tensor("logits", (B, V), DT_F32, KIND_ACT)

    R, W_, RW = MODE_R, MODE_W, MODE_RW
    w.segments["iterations"] = []
    for it in range(c.iterations):
        i0 = len(w.kernels)
        segs = _gpt_forward(w, c, layers, E, gf, bf, ids, x, h, qkv, attn, ffn, logits,
                            None if c.logits_all else hl)
        if it == 0:
            w.segments["forward"] = segs       # embed, one entry per layer, head (first pass)
        w.segments["iterations"].append((i0, len(w.kernels) - i0))
    return w


def _gpt_forward(w, c, layers, E, gf, bf, ids, x, h, qkv, attn, ffn, logits, hl):
    H, F, V, T, B, S = c.hidden, c.ffn, c.vocab, c.tokens, c.batch, c.prompt_len
    R, W_, RW = MODE_R, MODE_W, MODE_RW
    segs = []
    k0 = w.kernel(OP_EMBED, (T, H, V), [(ids, R), (E, R), (x, W_)], tag="embed")
    segs.append((k0, 1))
    for l, L in enumerate(layers):
        k0 = len(w.kernels)
        w.kernel(OP_LAYERNORM, (T, H, 1, 0), [(x, R), (L["g1"], R), (L["b1"], R), (h, W_)], l, "ln1")
        w.kernel(OP_LINEAR, (T, 3 * H, H), [(h, R), (L["wqkv"], R), (qkv, W_)], l, "qkv")
        w.kernel(OP_ATTN_QKV, (B, S, c.n_heads, c.head_dim), [(qkv, R), (attn, W_)], l, "attn")
        w.kernel(OP_LINEAR_RESID, (T, H, H), [(attn, R), (L["wo"], R), (x, RW)], l, "o")
        w.kernel(OP_LAYERNORM, (T, H, 1, 0), [(x, R), (L["g2"], R), (L["b2"], R), (h, W_)], l, "ln2")
        w.kernel(OP_LINEAR_GELU, (T, F, H), [(h, R), (L["w1"], R), (ffn, W_)], l, "w1")
        w.kernel(OP_LINEAR_RESID, (T, H, F), [(ffn, R), (L["w2"], R), (x, RW)], l, "w2")
        segs.append((k0, len(w.kernels) - k0))
    k0 = len(w.kernels)
    if c.logits_all:
        w.kernel(OP_LAYERNORM, (T, H, 1, 0), [(x, R), (gf, R), (bf, R), (h, W_)], c.n_layers, "lnf")
        w.kernel(OP_LINEAR, (T, V, H), [(h, R), (E, R), (logits, W_)], c.n_layers, "head")
    else:
        w.kernel(OP_LAYERNORM, (B, H, S, S - 1), [(x, R), (gf, R), (bf, R), (hl, W_)], c.n_layers, "lnf")
        w.kernel(OP_LINEAR, (B, V, H), [(hl, R), (E, R), (logits, W_)], c.n_layers, "head")
    segs.append((k0, len(w.kernels) - k0))
    return segs


def _build_llama(c: DecoderConfig, routing=None, n_steps=0) -> Workload:
    w = Workload(c)
    H, F, V, B, S = c.hidden, c.ffn, c.vocab, c.batch, c.prompt_len
    nH, d, Lmax, T = c.n_heads, c.head_dim, c.kv_len, c.tokens
    dt = c.dtype
    moe = c.style == "moe"
    nE, topk = c.n_experts, c.top_k
    E = w.tensor("E", (V, H), dt, KIND_PARAM, init="normal")
    layers = []
    for l in range(c.n_layers):
        p = f"L{l}."
        L = dict(
            g1=w.tensor(p + "attn_norm", (H,), dt, KIND_PARAM, init="ones"),
            wq=w.tensor(p + "wq", (H, H), dt, KIND_PARAM, init="normal"),
            wk=w.tensor(p + "wk", (H, H), dt, KIND_PARAM, init="normal"),
            wv=w.tensor(p + "wv", (H, H), dt, KIND_PARAM, init="normal"),
            wo=w.tensor(p + "wo", (H, H), dt, KIND_PARAM, init="normal"),
            g2=w.tensor(p + "ffn_norm", (H,), dt, KIND_PARAM, init="ones"),
        )
        if moe:
            L["wr"] = w.tensor(p + "router", (nE, H), dt, KIND_PARAM, init="normal")
            L["experts"] = [dict(
                wg=w.tensor(p + f"x{e}.wg", (F, H), dt, KIND_PARAM, init="normal"),
                wu=w.tensor(p + f"x{e}.wu", (F, H), dt, KIND_PARAM, init="normal"),
                wd=w.tensor(p + f"x{e}.wd", (H, F), dt, KIND_PARAM, init="normal"),
            ) for e in range(nE)]
        else:
            L["wg"] = w.tensor(p + "wg", (F, H), dt, KIND_PARAM, init="normal")
            L["wu"] = w.tensor(p + "wu", (F, H), dt, KIND_PARAM, init="normal")
            L["wd"] = w.tensor(p + "wd", (H, F), dt, KIND_PARAM, init="normal")
        layers.append(L)
    gf = w.tensor("norm_f", (H,), dt, KIND_PARAM, init="ones")
    head = w.tensor("head", (V, H), dt, KIND_PARAM, init="normal")
    for l in range(c.n_layers):
        layers[l]["K"] = w.tensor(f"L{l}.K", (B, nH, Lmax, d), dt, KIND_KV)
        layers[l]["V"] = w.tensor(f"L{l}.V", (B, nH, Lmax, d), dt, KIND_KV)
    # prefill activations
    ids_p = w.tensor("ids_p", (T,), DT_I32, KIND_ACT, host_init=True, init="ids")
    xp = w.tensor("x_p", (T, H), DT_F32, KIND_ACT)
    hp = w.tensor("h_p", (T, H), dt, KIND_ACT)
    qp = w.tensor("q_p", (T, H), dt, KIND_ACT)
    kp = w.tensor("k_p", (T, H), dt, KIND_ACT)
    vp = w.tensor("v_p", (T, H), dt, KIND_ACT)
    ap = w.tensor("a_p", (T, H), dt, KIND_ACT)
    fp = w.tensor("f_p", (T, F), dt, KIND_ACT)
    # shared head activations and the generated-token record
    hl = w.tensor("hl", (B, H), dt, KIND_ACT)
    logits = w.tensor("logits", (B, V), DT_F32, KIND_ACT)
    tok = w.tensor("tok", (B,), DT_I32, KIND_ACT)
    gen = w.tensor("gen", (c.decode_steps + 1, B), DT_I32, KIND_ACT, host_init=True, init="zeros")
    # decode activations
    xd = w.tensor("x_d", (B, H), DT_F32, KIND_ACT)
    hd = w.tensor("h_d", (B, H), dt, KIND_ACT)
    qd = w.tensor("q_d", (B, H), dt, KIND_ACT)
    kd = w.tensor("k_d", (B, H), dt, KIND_ACT)
    vd = w.tensor("v_d", (B, H), dt, KIND_ACT)
    ad = w.tensor("a_d", (B, H), dt, KIND_ACT)
    fd = w.tensor("f_d", (B, F), dt, KIND_ACT)
    if moe:
        # routing results and per-expert row lists of each phase, and the log
        # of per-expert row counts (one row of n_experts per segment and layer)
        rt = {ph: (w.tensor(f"rte_{ph}", (M, topk), DT_I32, KIND_ACT),
                   w.tensor(f"rtw_{ph}", (M, topk), DT_F32, KIND_ACT),
                   w.tensor(f"lists_{ph}", (nE, M + 1), DT_I32, KIND_ACT))
              for ph, M in (("p", T), ("d", B))}
        log = w.tensor("moe_counts", ((1 + c.decode_steps) * c.n_layers, nE), DT_I32, KIND_ACT,
                       host_init=True, init="zeros")

    R, W_, RW = MODE_R, MODE_W, MODE_RW

    def moe_ffn(l, L, x, h, f, M, seg):
        rte, rtw, lists = rt["p" if seg == 0 else "d"]
        w.kernel(OP_MOE_ROUTE, (M, H, nE, topk), [(h, R), (L["wr"], R), (rte, W_), (rtw, W_)], l, "route")
        w.kernel(OP_MOE_DISPATCH, (M, nE, topk, seg * c.n_layers + l),
                 [(rte, R), (lists, W_), (log, RW)], l, "dispatch")
        for e, X in enumerate(L["experts"]):
            n = M if routing is None else int(routing[seg][l][e])
            if n == 0:
                continue
            w.kernel(OP_MOE_UP, (M, F, H, e, n, topk), [(h, R), (lists, R), (X["wg"], R), (X["wu"], R), (f, W_)],
                     l, "expert_up")
            w.kernel(OP_MOE_DOWN, (M, H, F, e, n, topk),
                     [(f, R), (lists, R), (rtw, R), (X["wd"], R), (x, RW)], l, "expert_down")

    def block(l, L, x, h, q, k, v, a, f, M, s_len, pos0, kv_mode, seg=0):
        w.kernel(OP_RMSNORM, (M, H, 1, 0), [(x, R), (L["g1"], R), (h, W_)], l, "attn_norm")
        if c.fuse_qkv:
            w.kernel(OP_LINEAR_QKV, (M, H, H), [(h, R), (L["wq"], R), (L["wk"], R), (L["wv"], R),
                                                (q, W_), (k, W_), (v, W_)], l, "wqkv")
        else:
            w.kernel(OP_LINEAR, (M, H, H), [(h, R), (L["wq"], R), (q, W_)], l, "wq")
            w.kernel(OP_LINEAR, (M, H, H), [(h, R), (L["wk"], R), (k, W_)], l, "wk")
            w.kernel(OP_LINEAR, (M, H, H), [(h, R), (L["wv"], R), (v, W_)], l, "wv")
        w.kernel(OP_ROPE_KV, (B, s_len, nH, d, Lmax, pos0),
                 [(q, RW), (k, R), (v, R), (L["K"], kv_mode), (L["V"], kv_mode)], l, "rope_kv")
        w.kernel(OP_ATTN_CACHE, (B, s_len, nH, d, Lmax, pos0),
                 [(q, R), (L["K"], R), (L["V"], R), (a, W_)], l, "attn")
        w.kernel(OP_LINEAR_RESID, (M, H, H), [(a, R), (L["wo"], R), (x, RW)], l, "wo")
        w.kernel(OP_RMSNORM, (M, H, 1, 0), [(x, R), (L["g2"], R), (h, W_)], l, "ffn_norm")
        if moe:
            moe_ffn(l, L, x, h, f, M, seg)
            return
        w.kernel(OP_LINEAR_SWIGLU, (M, F, H), [(h, R), (L["wg"], R), (L["wu"], R), (f, W_)], l, "gate_up")
        w.kernel(OP_LINEAR_RESID, (M, H, F), [(f, R), (L["wd"], R), (x, RW)], l, "wd")

    # prefill: the KV cache is first written here (positions 0..S-1 of Lmax),
    # so its mode is a pure write; the unwritten tail is never read.
    k0 = len(w.kernels)
    w.kernel(OP_EMBED, (T, H, V), [(ids_p, R), (E, R), (xp, W_)], 0, "embed")
    for l, L in enumerate(layers):
        block(l, L, xp, hp, qp, kp, vp, ap, fp, T, S, 0, W_)
    w.kernel(OP_RMSNORM, (B, H, S, S - 1), [(xp, R), (gf, R), (hl, W_)], c.n_layers, "norm_f")
    w.kernel(OP_LINEAR, (B, V, H), [(hl, R), (head, R), (logits, W_)], c.n_layers, "head")
    w.kernel(OP_ARGMAX, (B, V, 0), [(logits, R), (tok, W_), (gen, RW)], c.n_layers, "argmax")
    w.segments["prefill"] = [(k0, len(w.kernels) - k0)]
    steps = []
    if not 0 <= n_steps <= c.decode_steps:
        raise ValueError("steps beyond the config's decode steps")
    for s in range(n_steps):
        k0 = len(w.kernels)
        pos = S + s
        w.kernel(OP_EMBED, (B, H, V), [(tok, R), (E, R), (xd, W_)], 0, "embed")
        for l, L in enumerate(layers):
            block(l, L, xd, hd, qd, kd, vd, ad, fd, B, 1, pos, RW, seg=s + 1)
        w.kernel(OP_RMSNORM, (B, H, 1, 0), [(xd, R), (gf, R), (hl, W_)], c.n_layers, "norm_f")
        w.kernel(OP_LINEAR, (B, V, H), [(hl, R), (head, R), (logits, W_)], c.n_layers, "head")
        w.kernel(OP_ARGMAX, (B, V, s + 1), [(logits, R), (tok, W_), (gen, RW)], c.n_layers, "argmax")
        steps.append((k0, len(w.kernels) - k0))
    w.segments["decode"] = steps
    return w


def adam_shape(n, hp):
    """Shape integers of an ADAM kernel: the hyperparameters in fixed point."""
    return (n, hp["step"], round(hp["lr"] * 1e9), round(hp["b1"] * 1e6), round(hp["b2"] * 1e6),
            round(hp["eps"] * 1e12), round(hp["wd"] * 1e6))


def _build_train(c: DecoderConfig, keep_grads=False) -> Workload:
    """One training step of the LLaMA-style decoder: forward keeping every
    layer's activations, cross-entropy against next-token targets, backward,
    and AdamW on fp32 master weights (bf16 copies feed the GEMMs).  Backward
    GEMMs run as C = A W^T over explicit transposes of their operands."""
    w = Workload(c)
    H, F, V, B, S = c.hidden, c.ffn, c.vocab, c.batch, c.prompt_len
    nH, d, T = c.n_heads, c.head_dim, c.tokens
    dt = c.dtype
    R, W_, RW = MODE_R, MODE_W, MODE_RW
    params = []

    # weights, master weights and moments are carried to the next step: live-out
    def param(name, shape, init):
        t = w.tensor(name, shape, dt, KIND_PARAM, init=init, live_out=True)
        params.append(name)
        return t
    E = param("E", (V, H), "normal")
    layers = []
    for l in range(c.n_layers):
        p = f"L{l}."
        layers.append(dict(
            g1=param(p + "attn_norm", (H,), "ones"), wq=param(p + "wq", (H, H), "normal"),
            wk=param(p + "wk", (H, H), "normal"), wv=param(p + "wv", (H, H), "normal"),
            wo=param(p + "wo", (H, H), "normal"), g2=param(p + "ffn_norm", (H,), "ones"),
            wg=param(p + "wg", (F, H), "normal"), wu=param(p + "wu", (F, H), "normal"),
            wd=param(p + "wd", (H, F), "normal")))
    gf = param("norm_f", (H,), "ones")
    head = param("head", (V, H), "normal")
    opt = {}
    for n in params:
        shp = w.tensors[w.id(n)].shape
        opt[n] = dict(master=w.tensor(n + ".master", shp, DT_F32, KIND_PARAM, init="master", live_out=True),
                      m=w.tensor(n + ".m", shp, DT_F32, KIND_PARAM, init="adam_m", live_out=True),
                      v=w.tensor(n + ".v", shp, DT_F32, KIND_PARAM, init="adam_v", live_out=True),
                      grad=w.tensor(n + ".grad", shp, DT_F32, KIND_ACT, live_out=keep_grads))
    ids = w.tensor("ids", (T,), DT_I32, KIND_ACT, host_init=True, init="ids")
    labels = w.tensor("labels", (T,), DT_I32, KIND_ACT, host_init=True, init="labels")
    # activations kept for the backward pass
    for l, L in enumerate(layers):
        p = f"L{l}."
        for nm, shp, ty in (("x", (T, H), DT_F32), ("h1", (T, H), dt), ("q", (T, H), dt),
                            ("K", (B, nH, S, d), dt), ("V", (B, nH, S, d), dt), ("o", (T, H), dt),
                            ("lse", (B, nH, S), DT_F32), ("xm", (T, H), DT_F32), ("h2", (T, H), dt),
                            ("G", (T, F), dt), ("U", (T, F), dt), ("F", (T, F), dt)):
            L[nm] = w.tensor(p + nm, shp, ty, KIND_ACT)
    xL = w.tensor("xL", (T, H), DT_F32, KIND_ACT)
    hf = w.tensor("hf", (T, H), dt, KIND_ACT)
    logits = w.tensor("logits", (T, V), DT_F32, KIND_ACT)
    losses = w.tensor("losses", (T,), DT_F32, KIND_ACT)
    dlogits = w.tensor("dlogits", (T, V), dt, KIND_ACT)
    # temporaries shared by the layers
    k_t = w.tensor("k_tmp", (T, H), dt, KIND_ACT)
    v_t = w.tensor("v_tmp", (T, H), dt, KIND_ACT)
    dx = w.tensor("dx", (T, H), DT_F32, KIND_ACT)
    dxb = w.tensor("dxb", (T, H), dt, KIND_ACT)
    dh = w.tensor("dh", (T, H), DT_F32, KIND_ACT)
    dF = w.tensor("dF", (T, F), dt, KIND_ACT)
    dG = w.tensor("dG", (T, F), dt, KIND_ACT)
    dU = w.tensor("dU", (T, F), dt, KIND_ACT)
    do_ = w.tensor("do", (T, H), dt, KIND_ACT)
    dq = w.tensor("dq", (T, H), dt, KIND_ACT)
    dK = w.tensor("dK", (B, nH, S, d), dt, KIND_ACT)
    dV = w.tensor("dV", (B, nH, S, d), dt, KIND_ACT)
    dk = w.tensor("dk", (T, H), dt, KIND_ACT)
    dv = w.tensor("dv", (T, H), dt, KIND_ACT)
    WT = w.tensor("WT", (max(F, V), H), dt, KIND_ACT)
    AT1 = w.tensor("AT1", (max(F, V, H), T), dt, KIND_ACT)
    AT2 = w.tensor("AT2", (max(F, H), T), dt, KIND_ACT)
    rstd = w.tensor("rstd", (T,), DT_F32, KIND_ACT)
    Dws = w.tensor("attn_D", (B, nH, S), DT_F32, KIND_ACT)

    g = dict(E=E, gf=gf, head=head, ids=ids, labels=labels, xL=xL, hf=hf, logits=logits, losses=losses,
             dlogits=dlogits, k_t=k_t, v_t=v_t, dx=dx, dxb=dxb, dh=dh, dF=dF, dG=dG, dU=dU, do_=do_, dq=dq,
             dK=dK, dV=dV, dk=dk, dv=dv, WT=WT, AT1=AT1, AT2=AT2, rstd=rstd, Dws=Dws)
    for it in range(c.iterations):
        _train_step(w, c, it, layers, params, opt, g)
    return w


def _train_step(w, c, it, layers, params, opt, g):
    """Kernels of training step it (the AdamW step number advances with it);
    g holds the tensors the layers share."""
    from .init import TRAIN_HP
    H, F, V, B, S = c.hidden, c.ffn, c.vocab, c.batch, c.prompt_len
    nH, d, T = c.n_heads, c.head_dim, c.tokens
    dt = c.dtype
    R, W_, RW = MODE_R, MODE_W, MODE_RW
    E, gf, head, ids, labels = g["E"], g["gf"], g["head"], g["ids"], g["labels"]
    xL, hf, logits, losses, dlogits = g["xL"], g["hf"], g["logits"], g["losses"], g["dlogits"]
    k_t, v_t, dx, dxb, dh = g["k_t"], g["v_t"], g["dx"], g["dxb"], g["dh"]
    dF, dG, dU, do_, dq, dK, dV, dk, dv = (g[n] for n in ("dF", "dG", "dU", "do_", "dq", "dK", "dV", "dk", "dv"))
    WT, AT1, AT2, rstd, Dws = g["WT"], g["AT1"], g["AT2"], g["rstd"], g["Dws"]

    def lin(a, Wt, out, M, N, K, l, tag, op=OP_LINEAR):
        w.kernel(op, (M, N, K), [(a, R), (Wt, R), (out, RW if op == OP_LINEAR_RESID else W_)], l, tag)

    def tr(a, b, rows, cols, l, tag):
        w.kernel(OP_TRANSPOSE, (rows, cols), [(a, R), (b, W_)], l, tag)

    def dlin(dy, Wt, dX, X, gW, M, N, K, l, tag, acc=False):
        """y[M,N] = X[M,K] W[N,K]^T: dX (+)= dy W (dy [M,N] bf16), gW = dy^T X."""
        tr(Wt, WT, N, K, l, tag + ".wT")
        lin(dy, WT, dX, M, K, N, l, tag + ".dX", OP_LINEAR_RESID if acc else OP_LINEAR)
        tr(dy, AT1, M, N, l, tag + ".dyT")
        if X is not None:
            tr(X, AT2, M, K, l, tag + ".xT")
        lin(AT1, AT2, gW, N, K, M, l, tag + ".dW")

    kf = len(w.kernels)
    # ---- forward
    w.kernel(OP_EMBED, (T, H, V), [(ids, R), (E, R), (layers[0]["x"], W_)], 0, "embed")
    for l, L in enumerate(layers):
        x_next = layers[l + 1]["x"] if l + 1 < len(layers) else xL
        w.kernel(OP_RMSNORM, (T, H, 1, 0), [(L["x"], R), (L["g1"], R), (L["h1"], W_)], l, "attn_norm")
        lin(L["h1"], L["wq"], L["q"], T, H, H, l, "wq")
        lin(L["h1"], L["wk"], k_t, T, H, H, l, "wk")
        lin(L["h1"], L["wv"], v_t, T, H, H, l, "wv")
        w.kernel(OP_ROPE_KV, (B, S, nH, d, S, 0), [(L["q"], RW), (k_t, R), (v_t, R), (L["K"], W_), (L["V"], W_)],
                 l, "rope")
        w.kernel(OP_ATTN_CACHE, (B, S, nH, d, S, 0), [(L["q"], R), (L["K"], R), (L["V"], R), (L["o"], W_),
                                                      (L["lse"], W_)], l, "attn")
        w.kernel(OP_COPY, (T * H * 4,), [(L["x"], R), (L["xm"], W_)], l, "copy")
        lin(L["o"], L["wo"], L["xm"], T, H, H, l, "wo", OP_LINEAR_RESID)
        w.kernel(OP_RMSNORM, (T, H, 1, 0), [(L["xm"], R), (L["g2"], R), (L["h2"], W_)], l, "ffn_norm")
        lin(L["h2"], L["wg"], L["G"], T, F, H, l, "wg")
        lin(L["h2"], L["wu"], L["U"], T, F, H, l, "wu")
        w.kernel(OP_SWIGLU_ACT, (T, F), [(L["G"], R), (L["U"], R), (L["F"], W_)], l, "swiglu")
        w.kernel(OP_COPY, (T * H * 4,), [(L["xm"], R), (x_next, W_)], l, "copy")
        lin(L["F"], L["wd"], x_next, T, H, F, l, "wd", OP_LINEAR_RESID)
    nl = c.n_layers
    w.kernel(OP_RMSNORM, (T, H, 1, 0), [(xL, R), (gf, R), (hf, W_)], nl, "norm_f")
    lin(hf, head, logits, T, V, H, nl, "head")
    w.kernel(OP_XENT, (T, V), [(logits, R), (labels, R), (losses, W_), (dlogits, W_)], nl, "xent")
    kb = len(w.kernels)
    # ---- backward
    dlin(dlogits, head, dh, hf, opt["head"]["grad"], T, V, H, nl, "head")
    w.kernel(OP_RMSNORM_BWD, (T, H, 0), [(xL, R), (gf, R), (dh, R), (dx, W_), (dxb, W_),
                                          (opt["norm_f"]["grad"], W_), (rstd, W_)], nl, "norm_f.bwd")
    for l in reversed(range(c.n_layers)):
        L = layers[l]
        p = f"L{l}."
        dlin(dxb, L["wd"], dF, L["F"], opt[p + "wd"]["grad"], T, H, F, l, "wd")
        w.kernel(OP_SWIGLU_BWD, (T, F), [(L["G"], R), (L["U"], R), (dF, R), (dG, W_), (dU, W_)], l, "swiglu.bwd")
        dlin(dG, L["wg"], dh, L["h2"], opt[p + "wg"]["grad"], T, F, H, l, "wg")
        dlin(dU, L["wu"], dh, None, opt[p + "wu"]["grad"], T, F, H, l, "wu", acc=True)
        w.kernel(OP_RMSNORM_BWD, (T, H, 1), [(L["xm"], R), (L["g2"], R), (dh, R), (dx, RW), (dxb, W_),
                                              (opt[p + "ffn_norm"]["grad"], W_), (rstd, W_)], l, "ffn_norm.bwd")
        dlin(dxb, L["wo"], do_, L["o"], opt[p + "wo"]["grad"], T, H, H, l, "wo")
        w.kernel(OP_ATTN_BWD, (B, S, nH, d), [(L["q"], R), (L["K"], R), (L["V"], R), (L["o"], R), (L["lse"], R),
                                              (do_, R), (dq, W_), (dK, W_), (dV, W_), (Dws, W_)], l, "attn.bwd")
        w.kernel(OP_ROPE_BWD, (B, S, nH, d), [(dq, RW), (dK, R), (dV, R), (dk, W_), (dv, W_)], l, "rope.bwd")
        dlin(dq, L["wq"], dh, L["h1"], opt[p + "wq"]["grad"], T, H, H, l, "wq")
        dlin(dk, L["wk"], dh, None, opt[p + "wk"]["grad"], T, H, H, l, "wk", acc=True)
        dlin(dv, L["wv"], dh, None, opt[p + "wv"]["grad"], T, H, H, l, "wv", acc=True)
        w.kernel(OP_RMSNORM_BWD, (T, H, 1), [(L["x"], R), (L["g1"], R), (dh, R), (dx, RW), (dxb, W_),
                                              (opt[p + "attn_norm"]["grad"], W_), (rstd, W_)], l, "attn_norm.bwd")
    w.kernel(OP_EMBED_BWD, (T, H, V), [(ids, R), (dx, R), (opt["E"]["grad"], W_)], 0, "embed.bwd")
    ka = len(w.kernels)
    # ---- update
    hp = dict(TRAIN_HP, step=TRAIN_HP["step"] + it)
    for n in params:
        o = opt[n]
        nel = w.tensors[w.id(n)].nbytes // DT_SIZE[dt]
        w.kernel(OP_ADAM, adam_shape(nel, hp), [(o["grad"], R), (o["master"], RW), (o["m"], RW),
                                                (o["v"], RW), (w.id(n), W_)], 0, "adam")
    for name, seg in (("forward", (kf, kb - kf)), ("backward", (kb, ka - kb)),
                      ("update", (ka, len(w.kernels) - ka)), ("step", (kf, len(w.kernels) - kf))):
        w.segments.setdefault(name, []).append(seg)
