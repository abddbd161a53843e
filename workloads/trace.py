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
from .format import (ALIGN, DT_F32, DT_I32, DT_SIZE, FLAG_HOST_INIT, KIND_ACT,
                     KIND_KV, KIND_PARAM, MODE_R, MODE_RW, MODE_W, OP_ARGMAX,
                     OP_ATTN_CACHE, OP_ATTN_QKV, OP_EMBED, OP_LAYERNORM,
                     OP_LINEAR, OP_LINEAR_GELU, OP_LINEAR_RESID,
                     OP_LINEAR_SWIGLU, OP_MOE_DISPATCH, OP_MOE_DOWN,
                     OP_MOE_ROUTE, OP_MOE_UP, OP_RMSNORM, OP_ROPE_KV)


def align_up(n: int, a: int = ALIGN) -> int:
    return (n + a - 1) // a * a


@dataclass
class TensorSpec:
    name: str
    shape: Tuple[int, ...]
    dtype: int
    kind: int
    host_init: bool
    init: str = "none"       # "normal" (weights), "ones" (norm gains), "zeros", "ids"
    off: int = 0             # arena offset
    tid: int = -1

    @property
    def nbytes(self) -> int:
        n = DT_SIZE[self.dtype]
        for s in self.shape:
            n *= s
        return n

    @property
    def flags(self) -> int:
        return FLAG_HOST_INIT if (self.host_init and self.kind != KIND_PARAM) else 0


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
    def tensor(self, name, shape, dtype, kind, host_init=False, init="none") -> int:
        t = TensorSpec(name, tuple(int(s) for s in shape), dtype, kind,
                       host_init or kind == KIND_PARAM, init)
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


def build(cfg: DecoderConfig, routing=None, steps=None) -> Workload:
    """The workload of a config.

    ``steps`` traces only the first decode steps of a LLaMA-style or MoE
    config; the tensors (KV cache length, logs) stay those of the full run.

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
