"""Pins of the fp64 training-step oracle: gradients against transformers'
LLaMA under torch autograd and against central finite differences, the
attention and RMSNorm backward against finite differences, and the update
against torch.optim.AdamW."""
import dataclasses

import numpy as np
import pytest

from oracle import forward as of
from oracle import train as ot
from workloads import configs, init, trace


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


CFG = dataclasses.replace(configs.TRAIN_SMALL, n_layers=2)


def _setup(cfg=CFG, seed=3):
    w = trace.build(cfg)
    P = init.weights_f64(w, names=init.param_names(w))
    rng = np.random.default_rng(seed)
    for k in list(P):                   # random gains so a dropped gain shows
        if k.endswith("norm") or k == "norm_f":
            P[k] = 1 + 0.1 * rng.standard_normal(P[k].shape)
    ids = init.token_ids(cfg.seed, cfg.batch, cfg.prompt_len, cfg.vocab)
    return w, P, ids, init.next_token_labels(ids)


def test_loss_and_gradients_match_transformers_autograd():
    torch = pytest.importorskip("torch")
    tf = pytest.importorskip("transformers")
    cfg = CFG
    w, P, ids, labels = _setup()
    logits, cache = ot.forward(cfg, P, ids)
    loss, dl = ot.cross_entropy(logits, labels)
    grads = ot.backward(cfg, P, ids, cache, dl)
    hc = tf.LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.hidden, intermediate_size=cfg.ffn,
                        num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                        num_key_value_heads=cfg.n_heads, max_position_embeddings=cfg.prompt_len,
                        rms_norm_eps=1e-6, rope_theta=10000.0, tie_word_embeddings=False,
                        attention_bias=False, mlp_bias=False)
    hc._attn_implementation = "eager"
    m = tf.LlamaForCausalLM(hc).to(torch.float64)
    names = dict(attn_norm="input_layernorm.weight", wq="self_attn.q_proj.weight",
                 wk="self_attn.k_proj.weight", wv="self_attn.v_proj.weight",
                 wo="self_attn.o_proj.weight", ffn_norm="post_attention_layernorm.weight",
                 wg="mlp.gate_proj.weight", wu="mlp.up_proj.weight", wd="mlp.down_proj.weight")
    ours = {"E": "model.embed_tokens.weight", "norm_f": "model.norm.weight", "head": "lm_head.weight"}
    for l in range(cfg.n_layers):
        for a, b in names.items():
            ours[f"L{l}.{a}"] = f"model.layers.{l}.{b}"
    m.load_state_dict({ours[k]: torch.from_numpy(np.ascontiguousarray(v)) for k, v in P.items()}, strict=False)
    lg = m(torch.from_numpy(ids.astype(np.int64))).logits.reshape(-1, cfg.vocab)
    tl = torch.nn.functional.cross_entropy(lg, torch.from_numpy(labels.reshape(-1).astype(np.int64)))
    tl.backward()
    assert abs(loss - tl.item()) < 1e-6 * abs(loss)
    sd = dict(m.named_parameters())
    for k, g in grads.items():
        # transformers evaluates the RoPE angles in fp32, hence ~1e-6 and not 1e-14
        assert rel_l2(g, sd[ours[k]].grad.numpy()) < 2e-6, k


def test_gradients_match_central_differences():
    cfg = dataclasses.replace(CFG, n_layers=1)
    w, P, ids, labels = _setup(cfg)
    logits, cache = ot.forward(cfg, P, ids)
    _, dl = ot.cross_entropy(logits, labels)
    grads = ot.backward(cfg, P, ids, cache, dl)
    rng = np.random.default_rng(9)
    eps = 1e-5
    for name in ("E", "L0.attn_norm", "L0.wq", "L0.wk", "L0.wv", "L0.wo", "L0.ffn_norm", "L0.wg",
                 "L0.wu", "L0.wd", "norm_f", "head"):
        dirn = rng.standard_normal(P[name].shape)

        def loss_at(t):
            Q = dict(P)
            Q[name] = P[name] + t * dirn
            lg, _ = ot.forward(cfg, Q, ids)
            return ot.cross_entropy(lg, labels)[0]
        fd = (loss_at(eps) - loss_at(-eps)) / (2 * eps)
        an = float((grads[name] * dirn).sum())
        assert abs(fd - an) < 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_attention_and_rmsnorm_backward_by_differences():
    rng = np.random.default_rng(4)
    S, d = 9, 8
    q, k, v, do = (rng.standard_normal((S, d)) for _ in range(4))
    dq, dk, dv = ot.attention_backward(q, k, v, do)
    eps = 1e-6
    for arg, g in ((0, dq), (1, dk), (2, dv)):
        dirn = rng.standard_normal((S, d))
        xs = [q, k, v]

        def f(t):
            ys = list(xs)
            ys[arg] = xs[arg] + t * dirn
            return float((of.causal_attention(*ys) * do).sum())
        assert abs((f(eps) - f(-eps)) / (2 * eps) - (g * dirn).sum()) < 1e-7
    x, g, dy = rng.standard_normal((5, 12)), rng.standard_normal(12), rng.standard_normal((5, 12))
    dx, dg = ot.rmsnorm_backward(x, g, dy)
    for arr, grad in ((0, dx), (1, dg)):
        dirn = rng.standard_normal(x.shape if arr == 0 else g.shape)

        def f(t):
            xx, gg = (x + t * dirn, g) if arr == 0 else (x, g + t * dirn)
            return float((of.rmsnorm(xx, gg) * dy).sum())
        assert abs((f(eps) - f(-eps)) / (2 * eps) - (grad * dirn).sum()) < 1e-7


def test_adamw_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(6)
    p, g = rng.standard_normal(50), rng.standard_normal(50) * 1e-3
    m, v = rng.standard_normal(50) * 1e-4, (rng.standard_normal(50) * 1e-4) ** 2
    hp = dict(step=10, lr=1e-3, b1=0.9, b2=0.95, eps=1e-8, wd=0.1)
    p2, m2, v2 = ot.adamw(p, g, m, v, **hp)
    tp = torch.nn.Parameter(torch.from_numpy(p.copy()))
    opt = torch.optim.AdamW([tp], lr=hp["lr"], betas=(hp["b1"], hp["b2"]), eps=hp["eps"],
                            weight_decay=hp["wd"])
    tp.grad = torch.from_numpy(g.copy())
    opt.state[tp] = {"step": torch.tensor(float(hp["step"] - 1), dtype=torch.float64),
                     "exp_avg": torch.from_numpy(m.copy()), "exp_avg_sq": torch.from_numpy(v.copy())}
    opt.step()
    assert np.allclose(tp.detach().numpy(), p2, rtol=0, atol=1e-15)
    assert np.allclose(opt.state[tp]["exp_avg"].numpy(), m2, rtol=0, atol=1e-18)
    assert np.allclose(opt.state[tp]["exp_avg_sq"].numpy(), v2, rtol=0, atol=1e-21)


def test_train_step_updates_every_parameter():
    cfg = CFG
    w, P, ids, labels = _setup()
    state = init.adam_state_f64(w)
    hp = init.TRAIN_HP
    r = ot.train_step(cfg, P, ids, labels, state, hp)
    assert set(r["params"]) == set(P)
    for n in P:
        assert not np.array_equal(r["params"][n], P[n]), n
    # a second step from the new state lowers the loss on the same batch
    r2 = ot.train_step(cfg, r["params"], ids, labels, r["state"], dict(hp, step=hp["step"] + 1))
    assert r2["loss"] < r["loss"]
