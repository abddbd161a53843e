"""fp64 reference of one training step of the LLaMA-style decoder.

Test infrastructure: only the tests, the smoke check and the benchmark's CPU
baseline use this module; the HIP path never does.

The paper motivates its memory system with training and inference jobs whose
working set exceeds device memory (Sec. I, Sec. II-A); it does not restate
the training arithmetic.  The definitions here are the textbook ones:

* forward as in ``forward.llama_layer`` (RMSNorm, q/k/v projections,
  rotate-half RoPE, causal softmax attention, SwiGLU MLP, residual adds), all
  activations kept for the backward pass;
* loss: mean over all tokens of the cross-entropy of the untied head's
  logits against integer targets;
* backward: the chain rule written out per op (no automatic differentiation);
* update: AdamW (decoupled weight decay) on fp32 master weights with first
  and second moments and bias correction, in the form
  p <- p (1 - lr wd);  m <- b1 m + (1 - b1) g;  v <- b2 v + (1 - b2) g^2;
  p <- p - lr / (1 - b1^t) * m / (sqrt(v / (1 - b2^t)) + eps).

Everything is fp64 and unblocked, so each function can be read against its
definition.  Parameter names follow the workload's tensors ("E", "L{l}.wq",
..., "norm_f", "head").
"""
import math

import numpy as np

from .forward import (RMS_EPS, causal_attention, linear, rmsnorm, rope, silu,
                      softmax)


# ------------------------------------------------------------- forward
def forward(cfg, P, ids):
    """Forward over ids [B, S]; returns (logits [T, V], cache for backward)."""
    B, S, H, nH, d = cfg.batch, cfg.prompt_len, cfg.hidden, cfg.n_heads, cfg.head_dim
    T = B * S
    pos = np.tile(np.arange(S), B)
    x = P["E"][np.asarray(ids).reshape(-1)].copy()
    layers = []
    for l in range(cfg.n_layers):
        p = f"L{l}."
        c = {"x": x}
        c["h1"] = h1 = rmsnorm(x, P[p + "attn_norm"])
        q = rope(linear(h1, P[p + "wq"]).reshape(T, nH, d), pos[:, None])
        k = rope(linear(h1, P[p + "wk"]).reshape(T, nH, d), pos[:, None])
        v = linear(h1, P[p + "wv"]).reshape(T, nH, d)
        o = np.empty_like(q)
        for b in range(B):
            rows = slice(b * S, (b + 1) * S)
            for h in range(nH):
                o[rows, h] = causal_attention(q[rows, h], k[rows, h], v[rows, h])
        c.update(q=q, k=k, v=v, o=o.reshape(T, H))
        x = x + linear(c["o"], P[p + "wo"])
        c["x_mid"] = x
        c["h2"] = h2 = rmsnorm(x, P[p + "ffn_norm"])
        c["G"] = G = linear(h2, P[p + "wg"])
        c["U"] = U = linear(h2, P[p + "wu"])
        c["F"] = F = silu(G) * U
        x = x + linear(F, P[p + "wd"])
        layers.append(c)
    hf = rmsnorm(x, P["norm_f"])
    logits = linear(hf, P["head"])
    return logits, dict(layers=layers, x_last=x, hf=hf)


def cross_entropy(logits, labels):
    """(mean loss, dlogits) of softmax cross-entropy over all rows."""
    T = logits.shape[0]
    pr = softmax(logits)
    lbl = np.asarray(labels).reshape(-1)
    loss = float(np.mean(-np.log(pr[np.arange(T), lbl])))
    g = pr.copy()
    g[np.arange(T), lbl] -= 1.0
    return loss, g / T


# ------------------------------------------------------------ backward
def rmsnorm_backward(x, g, dy, eps=RMS_EPS):
    """y = x / r * g with r = sqrt(mean(x^2) + eps): returns (dx, dg)."""
    H = x.shape[-1]
    r = np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps)
    gdy = g * dy
    dx = gdy / r - x * (gdy * x).sum(axis=-1, keepdims=True) / (H * r ** 3)
    dg = (dy * x / r).sum(axis=0)
    return dx, dg


def silu_grad(z):
    s = 1.0 / (1.0 + np.exp(-z))
    return s * (1.0 + z * (1.0 - s))


def attention_backward(q, k, v, do):
    """One head, causal over one sequence: q, k, v, do [S, d] -> dq, dk, dv.

    Scores s = q k^T / sqrt(d) with key j <= query i; p = softmax(s); o = p v.
    """
    S, d = q.shape
    sc = 1.0 / math.sqrt(d)
    s = (q @ k.T) * sc
    mask = np.arange(S)[None, :] <= np.arange(S)[:, None]
    s = np.where(mask, s, -np.inf)
    p = softmax(s)
    dv = p.T @ do
    dp = do @ v.T
    ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True))
    dq = ds @ k * sc
    dk = ds.T @ q * sc
    return dq, dk, dv


def backward(cfg, P, ids, cache, dlogits):
    """Gradients of every parameter, by name."""
    B, S, H, nH, d = cfg.batch, cfg.prompt_len, cfg.hidden, cfg.n_heads, cfg.head_dim
    T = B * S
    pos = np.tile(np.arange(S), B)
    gr = {}
    gr["head"] = dlogits.T @ cache["hf"]
    dhf = dlogits @ P["head"]
    dx, gr["norm_f"] = rmsnorm_backward(cache["x_last"], P["norm_f"], dhf)
    for l in reversed(range(cfg.n_layers)):
        p = f"L{l}."
        c = cache["layers"][l]
        # x_next = x_mid + F Wd^T
        gr[p + "wd"] = dx.T @ c["F"]
        dF = dx @ P[p + "wd"]
        dG = dF * c["U"] * silu_grad(c["G"])
        dU = dF * silu(c["G"])
        gr[p + "wg"] = dG.T @ c["h2"]
        gr[p + "wu"] = dU.T @ c["h2"]
        dh2 = dG @ P[p + "wg"] + dU @ P[p + "wu"]
        dxn, gr[p + "ffn_norm"] = rmsnorm_backward(c["x_mid"], P[p + "ffn_norm"], dh2)
        dx = dx + dxn
        # x_mid = x + o Wo^T
        gr[p + "wo"] = dx.T @ c["o"]
        do = (dx @ P[p + "wo"]).reshape(T, nH, d)
        dq = np.empty_like(c["q"])
        dk = np.empty_like(c["k"])
        dv = np.empty_like(c["v"])
        for b in range(B):
            rows = slice(b * S, (b + 1) * S)
            for h in range(nH):
                dq[rows, h], dk[rows, h], dv[rows, h] = attention_backward(
                    c["q"][rows, h], c["k"][rows, h], c["v"][rows, h], do[rows, h])
        # RoPE is a rotation: its transpose rotates by the opposite angle
        dq = rope(dq, -pos[:, None]).reshape(T, H)
        dk = rope(dk, -pos[:, None]).reshape(T, H)
        dv = dv.reshape(T, H)
        h1 = c["h1"]
        gr[p + "wq"] = dq.T @ h1
        gr[p + "wk"] = dk.T @ h1
        gr[p + "wv"] = dv.T @ h1
        dh1 = dq @ P[p + "wq"] + dk @ P[p + "wk"] + dv @ P[p + "wv"]
        dxn, gr[p + "attn_norm"] = rmsnorm_backward(c["x"], P[p + "attn_norm"], dh1)
        dx = dx + dxn
    dE = np.zeros_like(P["E"])
    np.add.at(dE, np.asarray(ids).reshape(-1), dx)
    gr["E"] = dE
    return gr


# -------------------------------------------------------------- update
def adamw(p, g, m, v, step, lr, b1, b2, eps, wd):
    """One AdamW step at step number `step` (1-based); returns (p, m, v)."""
    p = p * (1.0 - lr * wd)
    m = b1 * m + (1.0 - b1) * g
    v = b2 * v + (1.0 - b2) * g * g
    bc1 = 1.0 - b1 ** step
    bc2 = 1.0 - b2 ** step
    p = p - (lr / bc1) * m / (np.sqrt(v / bc2) + eps)
    return p, m, v


def train_step(cfg, P, ids, labels, state, hp, master=None):
    """One step: forward, loss, backward, AdamW on every parameter.

    P: the weights the forward and backward use, by name (fp64 values of
    the bf16 weights for bf16 configs); master: the fp32 master weights the
    update applies to (default P); state: name -> (m, v); hp: dict with step,
    lr, b1, b2, eps, wd.  Returns dict(loss, grads, params (new master),
    state, logits).
    """
    master = P if master is None else master
    logits, cache = forward(cfg, P, ids)
    loss, dlogits = cross_entropy(logits, labels)
    grads = backward(cfg, P, ids, cache, dlogits)
    newP, newS = {}, {}
    for n, w in master.items():
        m, v = state[n]
        newP[n], m2, v2 = adamw(w, grads[n], m, v, hp["step"], hp["lr"], hp["b1"], hp["b2"],
                                hp["eps"], hp["wd"])
        newS[n] = (m2, v2)
    return dict(loss=loss, grads=grads, params=newP, state=newS, logits=logits)
