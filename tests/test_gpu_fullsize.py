"""Parity at full size, in the launch configuration the benchmark times: the
7B decode at 1.5x, the 1.3B prefill at 1.25x and the MoE decode at 2x run
through the C-ABI under T+A+P, and sampled outputs are checked against the
fp64 oracle one layer at a time.  The oracle takes the GPU's layer input
(and, for attention over a cache, the GPU's cache prefix; for MoE, the
GPU's expert choice) and must reproduce what the layer adds to the residual
stream (its output minus its input) at the bf16 tolerance (rel-L2 2e-2),
with every element within a per-element bound for a layer of bf16 stages."""
import dataclasses

import numpy as np
import pytest

from oracle import forward as of
from workloads import configs, init, trace
from workloads.format import OP_MOE_DOWN, OP_MOE_ROUTE

from gpu_util import (ELEM_BF16, ELEM_LAYER, assert_close, assert_within, attention_backward_bounds,
                      rel_l2)

pytestmark = pytest.mark.gpu

TOL = 2e-2
DECODE_GUARD = 5          # the decode benchmark's victim guard
PREFILL_GUARD = 16        # the prefill benchmark's


class Walker:
    """Runs a session's trace forward in contiguous pieces."""

    def __init__(self, s):
        self.s, self.pos = s, 0

    def to(self, k):
        assert k >= self.pos, f"kernel {k} already ran (at {self.pos})"
        if k > self.pos:
            self.s.run(self.pos, k - self.pos)
            self.pos = k


def _layer_range(w, seg, layer):
    a, n = seg
    ks = [k for k in range(a, a + n) if w.kernels[k].layer == layer and w.kernels[k].tag not in ("embed",)]
    return ks[0], ks[-1] + 1


def _weights(w, prefix, names):
    Wt = init.weights_f64(w, names=[prefix + n for n in names])
    return {k[len(prefix):]: v for k, v in Wt.items()}


def test_llama7b_decode_layer_and_head_sampled():
    from paper_2609_06172_amd.session import Session
    cfg = configs.LLAMA_7B
    w = trace.build(cfg, steps=2)
    step, l, bs = 1, 17, [0, 9, 15]
    print(f"llama-7b decode at 1.5x: step {step}, layer {l}, sequences {bs}", flush=True)
    s = Session(w, device=0, guard=DECODE_GUARD)  # budget footprint/1.5, T+A+P
    walk = Walker(s)
    seg = w.segments["decode"][step]
    a, b = _layer_range(w, seg, l)
    walk.to(a)
    x_in = s.read("x_d").astype(np.float64)
    walk.to(b)
    x_out = s.read("x_d")
    K, V = s.read(f"L{l}.K"), s.read(f"L{l}.V")
    walk.to(seg[0] + seg[1] - 3)                 # through the last layer, before norm_f / head / argmax
    x_last = s.read("x_d").astype(np.float64)
    walk.to(seg[0] + seg[1])
    logits = s.read("logits")
    s.close()
    pos = cfg.prompt_len + step
    Lw = _weights(w, f"L{l}.", ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd"))
    c1 = dataclasses.replace(cfg, batch=len(bs))
    Kc, Vc = K[bs].astype(np.float64), V[bs].astype(np.float64)
    ref = of.llama_layer(c1, Lw, x_in[bs], Kc, Vc, pos)
    e = assert_close(x_out[bs] - x_in[bs], ref - x_in[bs], TOL, ELEM_LAYER, "layer increment")
    print(f"layer {l} increment: rel-L2 {e[0]:.2e}, max |error| / rms {e[1]:.2e}")
    assert_close(K[bs][:, :, pos], Kc[:, :, pos], TOL, ELEM_LAYER, "new K row")
    assert_close(V[bs][:, :, pos], Vc[:, :, pos], TOL, ELEM_LAYER, "new V row")
    Hd = _weights(w, "", ("norm_f", "head"))
    lg = of.linear(of.rmsnorm(x_last[bs], Hd["norm_f"]), Hd["head"])
    e = assert_close(logits[bs], lg, TOL, ELEM_LAYER, "logits")
    print(f"logits: rel-L2 {e[0]:.2e}, max |error| / rms {e[1]:.2e}")


def test_gpt1p3b_prefill_layer_and_head_sampled():
    from paper_2609_06172_amd.session import Session
    cfg = configs.GPT_1P3B
    w = trace.build(cfg)
    l, b = 11, 2
    print(f"gpt-1.3b prefill at 1.25x: layer {l}, sequence {b}", flush=True)
    s = Session(w, device=0, guard=PREFILL_GUARD)   # the prefill benchmark's policy
    walk = Walker(s)
    a, n = w.segments["forward"][1 + l]
    walk.to(a)
    x_in = s.read("x").astype(np.float64)
    walk.to(a + n)
    x_out = s.read("x")
    h0, hn = w.segments["forward"][-1]
    walk.to(h0)
    x_last = s.read("x").astype(np.float64)
    walk.to(h0 + hn)
    logits = s.read("logits")
    s.close()
    S = cfg.prompt_len
    rows = slice(b * S, (b + 1) * S)
    names = ("ln1.g", "ln1.b", "wqkv", "wo", "ln2.g", "ln2.b", "w1", "w2")
    Wt = init.weights_f64(w, names=[f"L{l}.{x}" for x in names] + ["lnf.g", "lnf.b", "E"])
    ref = of.gpt_layer(dataclasses.replace(cfg, batch=1), Wt, l, x_in[rows])
    e = assert_close(x_out[rows] - x_in[rows], ref - x_in[rows], TOL, ELEM_LAYER, "layer increment")
    print(f"layer {l} increment: rel-L2 {e[0]:.2e}, max |error| / rms {e[1]:.2e}")
    last = x_last[np.arange(cfg.batch) * S + S - 1]
    lg = of.linear(of.layernorm(last, Wt["lnf.g"], Wt["lnf.b"]), Wt["E"])
    assert_close(logits, lg, TOL, ELEM_LAYER, "logits")


def _moe_bench_config():
    """The MoE benchmark's configuration: full per-layer shape, the layers
    whose host backing fits the pinned memory of the GPU host (16 of 32)."""
    return dataclasses.replace(configs.MOE_8X, n_layers=16)


def test_moe_decode_and_prefill_layers_sampled():
    from paper_2609_06172_amd.session import Session
    cfg = _moe_bench_config()
    w = trace.build(cfg, steps=1)                # every expert in the trace
    l, bs = 9, [1, 6]
    rows = np.array([0, 4097, 20000, 32767])
    print(f"moe 8 x 14336, {cfg.n_layers} layers at 2x: prefill rows {list(rows)} and decode "
          f"sequences {bs} of layer {l}", flush=True)
    s = Session(w, device=0)                     # budget footprint/2, T+A+P
    walk = Walker(s)
    # prefill: the routed FFN of layer l on sampled rows
    pseg = w.segments["prefill"][0]
    a, b = _layer_range(w, pseg, l)
    route = next(k for k in range(a, b) if w.kernels[k].op == OP_MOE_ROUTE)
    last_down = max(k for k in range(a, b) if w.kernels[k].op == OP_MOE_DOWN)
    walk.to(route)
    h_p, x_mid = s.read("h_p")[rows].astype(np.float64), s.read("x_p")[rows].astype(np.float64)
    walk.to(route + 1)
    rte_p = s.read("rte_p")[rows]
    walk.to(last_down + 1)
    x_ffn = s.read("x_p")[rows]
    # decode step 0: the whole block of layer l for sampled sequences
    dseg = w.segments["decode"][0]
    a, b = _layer_range(w, dseg, l)
    route = next(k for k in range(a, b) if w.kernels[k].op == OP_MOE_ROUTE)
    walk.to(a)
    x_in = s.read("x_d").astype(np.float64)
    walk.to(route + 1)
    rte_d = s.read("rte_d")
    walk.to(b)
    x_out = s.read("x_d")
    K, V = s.read(f"L{l}.K"), s.read(f"L{l}.V")
    s.close()
    experts = sorted(set(rte_p.ravel()) | set(rte_d[bs].ravel()))
    names = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "router"]
    names += [f"x{e}.{n}" for e in experts for n in ("wg", "wu", "wd")]
    Lw = _weights(w, f"L{l}.", names)
    y, _, _, _ = of.moe_mlp(cfg, Lw, h_p, forced=rte_p)
    assert_close(x_ffn - x_mid, y, TOL, ELEM_LAYER, "routed FFN increment")
    pos = cfg.prompt_len
    c1 = dataclasses.replace(cfg, batch=len(bs))
    Kc, Vc = K[bs].astype(np.float64), V[bs].astype(np.float64)
    ref = of.llama_layer(c1, Lw, x_in[bs], Kc, Vc, pos, forced_route=rte_d[bs])
    assert_close(x_out[bs] - x_in[bs], ref - x_in[bs], TOL, ELEM_LAYER, "layer increment")


def test_training_step_13b_shape_sampled():
    # two layers of the 13B shape at full width, 8 x 2048 tokens, 2x: each
    # stage is checked on the GPU's own inputs, read at the point it runs
    from oracle import train as ot
    from paper_2609_06172_amd.session import Session
    from workloads.format import OP_ADAM, OP_ATTN_BWD, OP_XENT
    cfg = dataclasses.replace(configs.LLAMA_13B_TRAIN, n_layers=2)
    w = trace.build(cfg)
    T, H, F, V, S, nH = cfg.tokens, cfg.hidden, cfg.ffn, cfg.vocab, cfg.prompt_len, cfg.n_heads
    print(f"13b-shape training step, 2 layers, {T} tokens at 2x", flush=True)
    kb = w.segments["backward"][0][0]
    ks = lambda pred: [k for k, kd in enumerate(w.kernels) if pred(k, kd)]
    fwd1 = ks(lambda k, kd: k < kb and kd.layer == 1)
    xent = ks(lambda k, kd: kd.op == OP_XENT)[0]
    ab1 = ks(lambda k, kd: kd.op == OP_ATTN_BWD and kd.layer == 1)[0]
    wd_tags = {kd.tag: k for k, kd in enumerate(w.kernels) if k > kb and kd.layer == 1 and kd.tag.startswith("wd.")}
    adam = ks(lambda k, kd: kd.op == OP_ADAM and kd.operands[4][0] == w.id("L1.wd"))[0]
    s = Session(w, device=0)
    walk = Walker(s)
    f64 = lambda n: s.read(n).astype(np.float64)
    # forward of layer 1 on sequence 5
    walk.to(fwd1[0])
    x_in = f64("L1.x")
    walk.to(fwd1[-1] + 1)
    x_out = s.read("xL")
    # loss and its gradient on sampled rows
    walk.to(xent)
    rows = np.array([0, 2047, 9000, 16383])
    logits = s.read("logits")[rows].astype(np.float64)
    walk.to(xent + 1)
    losses, dlog = s.read("losses")[rows], s.read("dlogits")[rows]
    # layer 1's down projection (the first of its backward): data gradient
    # rows and weight gradient rows
    walk.to(wd_tags["wd.wT"])
    dxb, Fl = f64("dxb"), f64("L1.F")
    walk.to(wd_tags["wd.dW"] + 1)
    dF, gwd = s.read("dF"), s.read("L1.wd.grad")
    # attention backward of layer 1 (the last of its backward), (b, h) = (3, 17)
    walk.to(ab1)
    b, h = 3, 17
    tok = slice(b * S, (b + 1) * S)
    q = f64("L1.q")[tok].reshape(S, nH, 128)[:, h]
    K, Vv = f64("L1.K")[b, h], f64("L1.V")[b, h]
    do = f64("do")[tok].reshape(S, nH, 128)[:, h]
    walk.to(ab1 + 1)
    dq = s.read("dq")[tok].reshape(S, nH, 128)[:, h]
    dK, dV = s.read("dK")[b, h], s.read("dV")[b, h]
    # AdamW of L1.wd
    walk.to(adam)
    before = {n: f64("L1.wd" + n) for n in (".grad", ".master", ".m", ".v")}
    walk.to(adam + 1)
    after = {n: s.read("L1.wd" + n) for n in (".master", ".m", ".v", "")}
    s.close()

    names = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd")
    Lw = _weights(w, "L1.", names)
    c1 = dataclasses.replace(cfg, n_layers=1, batch=1)
    seq = slice(5 * S, 6 * S)
    # the layer on the GPU's input for one whole sequence (its own K/V, positions 0..S-1)
    ref = of.llama_layer(dataclasses.replace(c1, style="llama"), Lw, x_in[seq],
                         np.zeros((1, nH, S, 128)), np.zeros((1, nH, S, 128)), 0)
    assert_close(x_out[seq] - x_in[seq], ref - x_in[seq], TOL, ELEM_LAYER, "layer increment")
    labels = init.next_token_labels(init.token_ids(cfg.seed, cfg.batch, S, V)).reshape(-1)[rows]
    lse = np.log(np.exp(logits - logits.max(1, keepdims=True)).sum(1)) + logits.max(1)
    assert np.abs(losses - (lse - logits[np.arange(len(rows)), labels])).max() < 1e-4
    _, dl = ot.cross_entropy(logits, labels)
    assert_close(dlog, dl * len(rows) / T, TOL, ELEM_BF16, "dlogits")
    rdq, rdk, rdv = ot.attention_backward(q, K, Vv, do)
    refs, bounds = attention_backward_bounds(q, K, Vv, do)
    for name, got, want, alt, bd in zip(("dq", "dK", "dV"), (dq, dK, dV), (rdq, rdk, rdv), refs, bounds):
        assert rel_l2(alt, want) < 1e-12                  # the bound's own recompute is the oracle's
        e = assert_within(got, want, bd, TOL, name)
        print(f"attention backward {name}: rel-L2 {e[0]:.2e}, max |error| / bound {e[1]:.2f}")
    for n in (0, 777, H - 1):
        assert_close(gwd[n], dxb[:, n] @ Fl, TOL, ELEM_LAYER, f"weight gradient row {n}")
    for t in (1, 8191, T - 1):
        assert_close(dF[t], dxb[t] @ Lw["wd"], TOL, ELEM_LAYER, f"data gradient row {t}")
    hp = dict(init.TRAIN_HP)
    p2, m2, v2 = ot.adamw(before[".master"], before[".grad"], before[".m"], before[".v"], hp["step"], hp["lr"],
                          hp["b1"], hp["b2"], hp["eps"], hp["wd"])
    assert rel_l2(after[".master"], p2) < 2e-6
    assert rel_l2(after[".m"], m2) < 1e-6 and rel_l2(after[".v"], v2) < 1e-6
    assert rel_l2(after[""], p2) < 4e-3
