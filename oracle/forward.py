"""fp64 reference forward of the synthetic decoders.

The paper runs unmodified Hugging Face decoders (Sec. V, Table II) and does not
restate their math; the definitions below are the textbook ones for the two
architecture families the workloads use:

* GPT style: LayerNorm (eps 1e-5), fused q/k/v projection, causal softmax
  attention, exact-erf GELU MLP, residual adds, tied LM head.
* LLaMA style: RMSNorm (eps 1e-6), separate q/k/v/o projections, rotate-half
  RoPE with base 10000, KV cache, SwiGLU MLP, untied LM head, greedy argmax.
* MoE style: the LLaMA block with its MLP replaced by a routed mixture of
  SwiGLU experts: router logits h Wr^T, the top-k experts of each token (ties
  to the lower index), weights the softmax over the selected logits, output
  the weighted sum of the selected experts' MLPs.

Weights are stored [out, in]; a projection is ``y = x @ W.T``.  Everything is
computed in the precision of the inputs (fp64 by default), with no blocking or
fusion, so each function can be read against its definition.
"""
import math

import numpy as np
from scipy.special import erf

LN_EPS = 1e-5
RMS_EPS = 1e-6
ROPE_BASE = 10000.0


def linear(x, W):
    """y[m, n] = sum_k x[m, k] W[n, k]."""
    return x @ W.T


def layernorm(x, g, b, eps=LN_EPS):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def rmsnorm(x, g, eps=RMS_EPS):
    ms = (x * x).mean(axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def gelu(z):
    """Exact GELU: z * Phi(z) with Phi the standard normal CDF."""
    return z * 0.5 * (1.0 + erf(z / math.sqrt(2.0)))


def silu(z):
    return z / (1.0 + np.exp(-z))


def softmax(s):
    """Row-wise softmax with max subtraction; -inf entries get weight 0."""
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def causal_attention(q, k, v, pos0=0):
    """One head: q [S, d] at positions pos0..pos0+S-1; k, v [L, d] at 0..L-1.

    Query i attends to keys 0..pos0+i with scores q.k / sqrt(d).
    """
    S, d = q.shape
    L = k.shape[0]
    s = (q @ k.T) / math.sqrt(d)
    qpos = pos0 + np.arange(S)[:, None]
    kpos = np.arange(L)[None, :]
    s = np.where(kpos <= qpos, s, -np.inf)
    return softmax(s) @ v


def rope(x, pos):
    """Rotate-half RoPE on the last axis of x [..., d] at integer positions pos [...].

    Pair (i, i + d/2) is rotated by angle pos * base^(-2i/d).
    """
    d = x.shape[-1]
    half = d // 2
    inv = ROPE_BASE ** (-2.0 * np.arange(half) / d)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv
    c, s = np.cos(ang).astype(x.dtype), np.sin(ang).astype(x.dtype)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


# ---------------------------------------------------------------- GPT style
def gpt_layer(cfg, Wt, l, x):
    """One pre-norm GPT block on x [B*S, H] (sequences of cfg.prompt_len)."""
    B, S, H, nH, d = cfg.batch, cfg.prompt_len, cfg.hidden, cfg.n_heads, cfg.head_dim
    p = f"L{l}."
    h = layernorm(x, Wt[p + "ln1.g"], Wt[p + "ln1.b"])
    qkv = linear(h, Wt[p + "wqkv"])
    q, k, v = qkv[:, :H], qkv[:, H:2 * H], qkv[:, 2 * H:]
    o = np.empty_like(q)
    for b in range(B):
        rows = slice(b * S, (b + 1) * S)
        for i in range(nH):
            cols = slice(i * d, (i + 1) * d)
            o[rows, cols] = causal_attention(q[rows, cols], k[rows, cols], v[rows, cols])
    x = x + linear(o, Wt[p + "wo"])
    h = layernorm(x, Wt[p + "ln2.g"], Wt[p + "ln2.b"])
    return x + linear(gelu(linear(h, Wt[p + "w1"])), Wt[p + "w2"])


def gpt_forward(cfg, Wt, ids):
    """Returns (list of x after each layer, logits).

    ids [B, S]; logits at every position if cfg.logits_all else at the last
    position of each sequence.
    """
    B, S = cfg.batch, cfg.prompt_len
    x = Wt["E"][np.asarray(ids).reshape(-1)]
    outs = []
    for l in range(cfg.n_layers):
        x = gpt_layer(cfg, Wt, l, x)
        outs.append(x)
    if not cfg.logits_all:
        x = x[np.arange(B) * S + S - 1]
    h = layernorm(x, Wt["lnf.g"], Wt["lnf.b"])
    return outs, linear(h, Wt["E"])


# -------------------------------------------------------------- LLaMA style
def route_topk(logits, k):
    """Top-k routing of router logits [M, E].

    Returns (idx [M, k] int32, weights [M, k]): per row the k largest logits
    in descending order, equal logits taken by increasing expert index, and
    the softmax over the selected logits.
    """
    M, E = logits.shape
    idx = np.empty((M, k), np.int32)
    wts = np.empty((M, k), logits.dtype)
    for m in range(M):
        order = sorted(range(E), key=lambda e: (-logits[m, e], e))[:k]
        sel = logits[m, order]
        ex = np.exp(sel - sel.max())
        idx[m] = order
        wts[m] = ex / ex.sum()
    return idx, wts


def expert_mlp(h, Xw):
    """One SwiGLU expert: (silu(h Wg^T) * (h Wu^T)) Wd^T."""
    return linear(silu(linear(h, Xw["wg"])) * linear(h, Xw["wu"]), Xw["wd"])


def moe_mlp(cfg, Lw, h, forced=None):
    """Routed mixture of experts on rows h [M, H].

    ``forced`` [M, k] replaces the expert choice (the weights are still the
    softmax over this layer's logits at the forced experts).  Returns
    (output [M, H], idx, weights, logits).
    """
    logits = linear(h, Lw["router"])
    if forced is None:
        idx, wts = route_topk(logits, cfg.top_k)
    else:
        idx = np.asarray(forced, np.int32)
        sel = np.take_along_axis(logits, idx, axis=1)
        ex = np.exp(sel - sel.max(axis=1, keepdims=True))
        wts = ex / ex.sum(axis=1, keepdims=True)
    y = np.zeros_like(h)
    for e in range(cfg.n_experts):
        rows, slots = np.nonzero(idx == e)
        if rows.size == 0:
            continue
        Xw = {n: Lw[f"x{e}.{n}"] for n in ("wg", "wu", "wd")}
        y[rows] += wts[rows, slots][:, None] * expert_mlp(h[rows], Xw)
    return y, idx, wts, logits


def llama_layer(cfg, Lw, x, K, V, pos0, forced_route=None, route_log=None):
    """One LLaMA (or MoE) block for S new tokens per sequence.

    x [B*S, H]; K, V [B, nH, Lmax, d] caches, updated in place at positions
    pos0..pos0+S-1.  Lw holds the layer's tensors by short name.  For MoE
    configs the routing (idx, weights, logits) is appended to route_log.
    """
    B, nH, d = cfg.batch, cfg.n_heads, cfg.head_dim
    S = x.shape[0] // B
    h = rmsnorm(x, Lw["attn_norm"])
    q = linear(h, Lw["wq"]).reshape(B, S, nH, d)
    k = linear(h, Lw["wk"]).reshape(B, S, nH, d)
    v = linear(h, Lw["wv"]).reshape(B, S, nH, d)
    pos = pos0 + np.arange(S)
    q = rope(q, pos[None, :, None])
    k = rope(k, pos[None, :, None])
    K[:, :, pos0:pos0 + S, :] = k.transpose(0, 2, 1, 3)
    V[:, :, pos0:pos0 + S, :] = v.transpose(0, 2, 1, 3)
    o = np.empty((B, S, nH, d), dtype=x.dtype)
    for b in range(B):
        for i in range(nH):
            L = pos0 + S
            o[b, :, i, :] = causal_attention(q[b, :, i, :], K[b, i, :L], V[b, i, :L], pos0)
    x = x + linear(o.reshape(B * S, nH * d), Lw["wo"])
    h = rmsnorm(x, Lw["ffn_norm"])
    if cfg.style == "moe":
        y, idx, wts, logits = moe_mlp(cfg, Lw, h, forced_route)
        if route_log is not None:
            route_log.append((idx, wts, logits))
        return x + y
    return x + linear(silu(linear(h, Lw["wg"])) * linear(h, Lw["wu"]), Lw["wd"])


def layer_weights(Wt, l):
    p = f"L{l}."
    return {k[len(p):]: v for k, v in Wt.items() if k.startswith(p)}


def new_cache(cfg, dtype=np.float64):
    shape = (cfg.batch, cfg.n_heads, cfg.kv_len, cfg.head_dim)
    return [(np.zeros(shape, dtype), np.zeros(shape, dtype)) for _ in range(cfg.n_layers)]


def llama_step(cfg, Wt, cache, x, pos0, forced_routes=None, route_log=None):
    """Run all layers on embedded tokens x [B*S, H] at positions pos0..; returns
    (per-layer outputs, logits at the last position of each sequence).
    forced_routes[l] forces layer l's expert choice (MoE)."""
    B = cfg.batch
    S = x.shape[0] // B
    outs = []
    for l in range(cfg.n_layers):
        K, V = cache[l]
        fr = None if forced_routes is None else forced_routes[l]
        x = llama_layer(cfg, layer_weights(Wt, l), x, K, V, pos0, fr, route_log)
        outs.append(x)
    last = x[np.arange(B) * S + S - 1]
    return outs, linear(rmsnorm(last, Wt["norm_f"]), Wt["head"])


def argmax_lowest(logits):
    """Greedy token: the lowest index among the maxima of each row."""
    return np.argmax(logits, axis=-1).astype(np.int32)


def llama_generate(cfg, Wt, ids, forced=None, dtype=np.float64, forced_routes=None):
    """Prefill ids [B, S] then cfg.decode_steps greedy steps.

    If ``forced`` [steps+1, B] is given, step s consumes forced[s] instead of
    its own argmax (teacher forcing); the chosen ids are still returned.
    For MoE configs ``forced_routes[seg][l]`` ([M, k]; seg 0 is the prefill)
    likewise forces the expert choice.  Returns dict(outs, logits=[per step],
    tokens=[per step], routes=[per segment: per layer (idx, weights, logits)]).
    """
    B, S = cfg.batch, cfg.prompt_len
    cache = new_cache(cfg, dtype)
    E = Wt["E"]

    def fr(seg):
        return None if forced_routes is None else forced_routes[seg]
    log = []
    outs, lg = llama_step(cfg, Wt, cache, E[np.asarray(ids).reshape(-1)], 0, fr(0), log)
    logits, tokens, step_outs, routes = [lg], [argmax_lowest(lg)], [outs], [log]
    for s in range(cfg.decode_steps):
        t = tokens[-1] if forced is None else np.asarray(forced[s], np.int32)
        log = []
        outs, lg = llama_step(cfg, Wt, cache, E[t], S + s, fr(s + 1), log)
        logits.append(lg)
        tokens.append(argmax_lowest(lg))
        step_outs.append(outs)
        routes.append(log)
    return dict(outs=step_outs, logits=logits, tokens=tokens, cache=cache, routes=routes)
