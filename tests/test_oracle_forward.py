"""Pins of the fp64 oracle forward against hand results, closed forms,
invariants and independent library implementations (torch, transformers)."""
import numpy as np
import pytest

from oracle import forward as of
from workloads import configs, init, trace


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


# ---------------------------------------------------------------- GEMM
def test_linear_hand_2x2_and_3x3():
    x = np.array([[1., 2.], [3., 4.]])
    W = np.array([[5., 6.], [7., 8.]])          # [out, in]
    # y[m, n] = sum_k x[m,k] W[n,k]
    assert np.array_equal(of.linear(x, W), [[17., 23.], [39., 53.]])
    x3 = np.array([[1., 0., 2.], [0., 1., 0.], [-1., 3., 1.]])
    W3 = np.array([[2., 1., 0.], [0., 0., 1.], [1., -1., 4.]])
    assert np.array_equal(of.linear(x3, W3), [[2., 2., 9.], [1., 0., -1.], [1., 1., 0.]])


def test_linear_out_in_layout_permutation():
    P = np.eye(4)[[2, 0, 3, 1]]                 # output n takes input perm[n]
    x = np.arange(8.).reshape(2, 4)
    assert np.array_equal(of.linear(x, P), x[:, [2, 0, 3, 1]])


# ------------------------------------------------------ softmax / attention
def test_softmax_rows_sum_to_one():
    s = np.random.default_rng(0).standard_normal((7, 11)) * 10
    p = of.softmax(s)
    assert np.allclose(p.sum(-1), 1.0, atol=1e-12)
    assert (p >= 0).all()


def test_attention_causal_weights_and_special_cases():
    rng = np.random.default_rng(1)
    S, d = 6, 4
    q, k = rng.standard_normal((S, d)), rng.standard_normal((S, d))
    # with v = identity the output rows are the attention weights
    P = of.causal_attention(q, k, np.eye(S))
    assert np.allclose(np.triu(P, 1), 0.0)
    assert np.allclose(P.sum(-1), 1.0, atol=1e-12)
    # a single key: output is that value row
    v1 = rng.standard_normal((1, d))
    assert np.allclose(of.causal_attention(q[:1], k[:1], v1), v1)
    # zero queries give uniform scores: causal running mean of v
    v = rng.standard_normal((S, d))
    mean = np.cumsum(v, 0) / np.arange(1, S + 1)[:, None]
    assert np.allclose(of.causal_attention(np.zeros((S, d)), k, v), mean)
    # offset queries (decode): query at position pos0 sees keys 0..pos0
    out = of.causal_attention(np.zeros((1, d)), k, v, pos0=3)
    assert np.allclose(out, v[:4].mean(0))


# --------------------------------------------------------------- norms
def test_layernorm_moments_and_rmsnorm_rms():
    x = np.random.default_rng(2).standard_normal((5, 64)) * 3 + 1
    y = of.layernorm(x, np.ones(64), np.zeros(64))
    assert np.allclose(y.mean(-1), 0, atol=1e-12)
    assert np.allclose(y.var(-1), 1, atol=1e-5)
    r = of.rmsnorm(x, np.ones(64))
    assert np.allclose(np.sqrt((r * r).mean(-1)), 1, atol=1e-5)


def test_activations():
    z = np.linspace(-5, 5, 101)
    assert of.gelu(np.array(0.0)) == 0.0
    assert np.allclose(of.gelu(z) - of.gelu(-z), z, atol=1e-12)
    # Phi(1) = 0.8413447460685429 (standard normal CDF)
    assert abs(of.gelu(np.array(1.0)) - 0.8413447460685429) < 1e-15
    assert of.silu(np.array(0.0)) == 0.0
    assert abs(of.silu(np.array(1.0)) - 1 / (1 + np.exp(-1))) < 1e-15


# ---------------------------------------------------------------- RoPE
def test_rope_properties():
    rng = np.random.default_rng(3)
    d = 16
    x = rng.standard_normal((3, d))
    assert np.allclose(of.rope(x, np.zeros(3)), x)
    y = of.rope(x, np.array([5, 17, 123]))
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1))
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    a = of.rope(q, 7) @ of.rope(k, 3)
    b = of.rope(q, 104) @ of.rope(k, 100)
    assert abs(a - b) < 1e-12
    # rotate-half pairing: (x_i, x_{i+d/2}) rotated by pos * 10000^(-2i/d)
    e = np.zeros(d)
    e[1] = 1.0
    ang = 2.0 * 10000 ** (-2 * 1 / d)
    y = of.rope(e, 2)
    assert abs(y[1] - np.cos(ang)) < 1e-15 and abs(y[1 + d // 2] - np.sin(ang)) < 1e-15


# -------------------------------------------------- whole-model pins
def _weights(cfg):
    return init.weights_f64(trace.build(cfg))


def test_gpt_layer_matches_torch_encoder_layer():
    torch = pytest.importorskip("torch")
    cfg = configs.TINY
    Wt = _weights(cfg)
    H, nH, F = cfg.hidden, cfg.n_heads, cfg.ffn
    layer = torch.nn.TransformerEncoderLayer(H, nH, F, dropout=0.0, activation="gelu",
                                             norm_first=True, bias=False, batch_first=True,
                                             layer_norm_eps=1e-5, dtype=torch.float64)
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(torch.from_numpy(Wt["L0.wqkv"]))
        layer.self_attn.out_proj.weight.copy_(torch.from_numpy(Wt["L0.wo"]))
        layer.linear1.weight.copy_(torch.from_numpy(Wt["L0.w1"]))
        layer.linear2.weight.copy_(torch.from_numpy(Wt["L0.w2"]))
    x = np.random.default_rng(4).standard_normal((cfg.batch * cfg.prompt_len, H))
    mask = torch.nn.Transformer.generate_square_subsequent_mask(cfg.prompt_len, dtype=torch.float64)
    with torch.no_grad():
        ref = layer(torch.from_numpy(x).reshape(cfg.batch, cfg.prompt_len, H),
                    src_mask=mask, is_causal=True).reshape(-1, H).numpy()
    assert rel_l2(of.gpt_layer(cfg, Wt, 0, x), ref) < 1e-12


def test_gpt_causality_and_batch_independence():
    import dataclasses
    cfg = dataclasses.replace(configs.TINY, batch=2)
    Wt = _weights(cfg)
    ids = init.token_ids(0, 2, cfg.prompt_len, cfg.vocab)
    _, lg = of.gpt_forward(cfg, Wt, ids)
    ids2 = ids.copy()
    ids2[0, 20:] = (ids2[0, 20:] + 1) % cfg.vocab
    _, lg2 = of.gpt_forward(cfg, Wt, ids2)
    S = cfg.prompt_len
    assert np.array_equal(lg[:20], lg2[:20])           # earlier positions unchanged
    assert not np.allclose(lg[20:S], lg2[20:S])
    assert np.array_equal(lg[S:], lg2[S:])             # other sequence unchanged


def test_gpt_identity_layers_reduce_to_tied_head():
    cfg = configs.TINY
    Wt = _weights(cfg)
    for l in range(cfg.n_layers):
        Wt[f"L{l}.wo"][:] = 0
        Wt[f"L{l}.w2"][:] = 0
    ids = init.token_ids(0, 1, cfg.prompt_len, cfg.vocab)
    _, lg = of.gpt_forward(cfg, Wt, ids)
    x = Wt["E"][ids.reshape(-1)]
    xn = (x - x.mean(-1, keepdims=True)) / np.sqrt(x.var(-1, keepdims=True) + 1e-5)
    assert rel_l2(lg, xn @ Wt["E"].T) < 1e-13


def test_fp32_oracle_close_to_fp64():
    cfg = configs.TINY
    Wt = _weights(cfg)
    ids = init.token_ids(0, 1, cfg.prompt_len, cfg.vocab)
    o64, lg64 = of.gpt_forward(cfg, Wt, ids)
    W32 = {k: v.astype(np.float32) for k, v in Wt.items()}
    o32, lg32 = of.gpt_forward(cfg, W32, ids)
    assert lg32.dtype == np.float32
    assert rel_l2(lg32, lg64) < 1e-5
    for a, b in zip(o32, o64):
        assert rel_l2(a, b) < 1e-5


def _hf_llama(cfg, Wt):
    torch = pytest.importorskip("torch")
    tf = pytest.importorskip("transformers")
    hc = tf.LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.hidden,
                        intermediate_size=cfg.ffn, num_hidden_layers=cfg.n_layers,
                        num_attention_heads=cfg.n_heads, num_key_value_heads=cfg.n_heads,
                        max_position_embeddings=cfg.kv_len, rms_norm_eps=1e-6,
                        rope_theta=10000.0, tie_word_embeddings=False,
                        attention_bias=False, mlp_bias=False)
    hc._attn_implementation = "eager"
    m = tf.LlamaForCausalLM(hc).to(torch.float64).eval()
    sd = {"model.embed_tokens.weight": Wt["E"], "model.norm.weight": Wt["norm_f"],
          "lm_head.weight": Wt["head"]}
    names = dict(attn_norm="input_layernorm.weight", wq="self_attn.q_proj.weight",
                 wk="self_attn.k_proj.weight", wv="self_attn.v_proj.weight",
                 wo="self_attn.o_proj.weight", ffn_norm="post_attention_layernorm.weight",
                 wg="mlp.gate_proj.weight", wu="mlp.up_proj.weight", wd="mlp.down_proj.weight")
    for l in range(cfg.n_layers):
        for ours, theirs in names.items():
            sd[f"model.layers.{l}.{theirs}"] = Wt[f"L{l}.{ours}"]
    m.load_state_dict({k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in sd.items()},
                      strict=False)
    return m


def test_llama_matches_transformers_and_kv_cache():
    torch = pytest.importorskip("torch")
    cfg = configs.LLAMA_SMALL
    Wt = _weights(cfg)
    ids = init.token_ids(0, cfg.batch, cfg.prompt_len, cfg.vocab)
    # randomise the norm gains so a dropped gain would show
    rng = np.random.default_rng(5)
    for k in list(Wt):
        if k.endswith("norm") or k == "norm_f":
            Wt[k] = 1 + 0.1 * rng.standard_normal(Wt[k].shape)
    gen = of.llama_generate(cfg, Wt, ids)
    toks = np.stack(gen["tokens"])                      # [steps+1, B]
    full = np.concatenate([ids, toks[:-1].T], axis=1)   # prompt + consumed tokens
    m = _hf_llama(cfg, Wt)
    with torch.no_grad():
        ref = m(torch.from_numpy(full.astype(np.int64))).logits.numpy()
    S = cfg.prompt_len
    # transformers evaluates the RoPE angles in fp32, hence ~1e-7 and not 1e-15
    for s in range(cfg.decode_steps + 1):
        assert rel_l2(gen["logits"][s], ref[:, S - 1 + s]) < 1e-6, s


def test_llama_decode_equals_recompute_and_is_causal():
    import dataclasses
    cfg = configs.LLAMA_SMALL
    Wt = _weights(cfg)
    ids = init.token_ids(0, cfg.batch, cfg.prompt_len, cfg.vocab)
    gen = of.llama_generate(cfg, Wt, ids)
    # recompute: prefill the prompt plus the first generated token as one sequence
    ext = np.concatenate([ids, gen["tokens"][0][:, None]], axis=1)
    c2 = dataclasses.replace(cfg, prompt_len=cfg.prompt_len + 1, decode_steps=0)
    _, lg = of.llama_step(c2, Wt, of.new_cache(c2), Wt["E"][ext.reshape(-1)], 0)
    assert rel_l2(gen["logits"][1], lg) < 1e-12
    # teacher forcing with different future tokens leaves earlier logits unchanged
    forced = np.stack(gen["tokens"]).copy()
    forced[2] = (forced[2] + 7) % cfg.vocab
    g2 = of.llama_generate(cfg, Wt, ids, forced=forced)
    for s in range(3):
        assert np.array_equal(g2["logits"][s], gen["logits"][s])
    assert not np.allclose(g2["logits"][3], gen["logits"][3])


# -------------------------------------------------------------- MoE pins
def test_route_topk_against_brute_force():
    import itertools
    rng = np.random.default_rng(11)
    for E, k in ((4, 2), (8, 2), (5, 3), (3, 3), (6, 1)):
        lg = rng.integers(-3, 4, size=(200, E)).astype(np.float64)   # many ties
        idx, wts = of.route_topk(lg, k)
        for m in range(lg.shape[0]):
            # the chosen set is the best k-subset under (value, then lower index)
            def key(sub):
                return sorted(((-lg[m, e], e) for e in sub))
            best = min(itertools.combinations(range(E), k), key=key)
            assert sorted(idx[m]) == sorted(best)
            # listed by decreasing logit, ties by increasing index
            assert [tuple(x) for x in key(idx[m])] == [(-lg[m, e], e) for e in idx[m]]
            ex = np.exp(lg[m, idx[m]] - lg[m, idx[m]].max())
            assert np.allclose(wts[m], ex / ex.sum(), rtol=0, atol=1e-15)
            assert abs(wts[m].sum() - 1) < 1e-15 and np.all(np.diff(wts[m]) <= 0)


def _moe_weights(cfg, seed=3):
    Wt = _weights(cfg)
    rng = np.random.default_rng(seed)
    for k in list(Wt):                 # randomise the gains so a dropped gain shows
        if k.endswith("norm") or k == "norm_f":
            Wt[k] = 1 + 0.1 * rng.standard_normal(Wt[k].shape)
    return Wt


def test_moe_matches_transformers_mixtral():
    torch = pytest.importorskip("torch")
    tf = pytest.importorskip("transformers")
    cfg = configs.MOE_SMALL
    Wt = _moe_weights(cfg)
    ids = init.token_ids(0, cfg.batch, cfg.prompt_len, cfg.vocab)
    gen = of.llama_generate(cfg, Wt, ids)
    toks = np.stack(gen["tokens"])
    full = np.concatenate([ids, toks[:-1].T], axis=1)
    hc = tf.MixtralConfig(vocab_size=cfg.vocab, hidden_size=cfg.hidden, intermediate_size=cfg.ffn,
                          num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                          num_key_value_heads=cfg.n_heads, num_local_experts=cfg.n_experts,
                          num_experts_per_tok=cfg.top_k, max_position_embeddings=cfg.kv_len,
                          rms_norm_eps=1e-6, rope_theta=10000.0, tie_word_embeddings=False,
                          sliding_window=None, router_jitter_noise=0.0)
    hc._attn_implementation = "eager"
    hc._experts_implementation = "eager"     # per-expert loop (the grouped GEMM has no fp64)
    m = tf.MixtralForCausalLM(hc).to(torch.float64).eval()
    sd = {"model.embed_tokens.weight": Wt["E"], "model.norm.weight": Wt["norm_f"],
          "lm_head.weight": Wt["head"]}
    names = dict(attn_norm="input_layernorm.weight", wq="self_attn.q_proj.weight",
                 wk="self_attn.k_proj.weight", wv="self_attn.v_proj.weight",
                 wo="self_attn.o_proj.weight", ffn_norm="post_attention_layernorm.weight",
                 router="mlp.gate.weight")
    E = cfg.n_experts
    for l in range(cfg.n_layers):
        for ours, theirs in names.items():
            sd[f"model.layers.{l}.{theirs}"] = Wt[f"L{l}.{ours}"]
        sd[f"model.layers.{l}.mlp.experts.gate_up_proj"] = np.stack(
            [np.concatenate([Wt[f"L{l}.x{e}.wg"], Wt[f"L{l}.x{e}.wu"]], axis=0) for e in range(E)])
        sd[f"model.layers.{l}.mlp.experts.down_proj"] = np.stack([Wt[f"L{l}.x{e}.wd"] for e in range(E)])
    missing, unexpected = m.load_state_dict(
        {k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in sd.items()}, strict=False)
    assert not unexpected and all("rotary" in k for k in missing), (missing, unexpected)
    with torch.no_grad():
        ref = m(torch.from_numpy(full.astype(np.int64))).logits.numpy()
    S = cfg.prompt_len
    for s in range(cfg.decode_steps + 1):
        assert rel_l2(gen["logits"][s], ref[:, S - 1 + s]) < 1e-6, s


def _dense_twin(cfg, Wt, expert=0):
    """LLaMA config and weights whose MLP is expert `expert` of each layer."""
    import dataclasses
    dc = dataclasses.replace(cfg, style="llama", n_experts=0, top_k=0)
    Wd = {k: v for k, v in Wt.items() if ".x" not in k and "router" not in k}
    for l in range(cfg.n_layers):
        for n in ("wg", "wu", "wd"):
            Wd[f"L{l}.{n}"] = Wt[f"L{l}.x{expert}.{n}"]
    return dc, Wd


def test_moe_with_one_expert_is_the_dense_mlp():
    import dataclasses
    cfg = dataclasses.replace(configs.MOE_SMALL, n_experts=1, top_k=1)
    Wt = _moe_weights(cfg)
    ids = init.token_ids(0, cfg.batch, cfg.prompt_len, cfg.vocab)
    a = of.llama_generate(cfg, Wt, ids)
    dc, Wd = _dense_twin(cfg, Wt)
    b = of.llama_generate(dc, Wd, ids)
    for x, y in zip(a["logits"], b["logits"]):
        assert rel_l2(x, y) < 1e-13


def test_moe_with_identical_experts_ignores_the_router():
    cfg = configs.MOE_SMALL
    Wt = _moe_weights(cfg)
    for l in range(cfg.n_layers):
        for e in range(1, cfg.n_experts):
            for n in ("wg", "wu", "wd"):
                Wt[f"L{l}.x{e}.{n}"] = Wt[f"L{l}.x0.{n}"]
    ids = init.token_ids(0, cfg.batch, cfg.prompt_len, cfg.vocab)
    a = of.llama_generate(cfg, Wt, ids)
    dc, Wd = _dense_twin(cfg, Wt)
    b = of.llama_generate(dc, Wd, ids)
    for x, y in zip(a["logits"], b["logits"]):
        assert rel_l2(x, y) < 1e-13
    # every token still picks top_k distinct experts
    for seg in a["routes"]:
        for idx, wts, _ in seg:
            assert all(len(set(r)) == cfg.top_k for r in idx)


def test_moe_all_experts_with_a_flat_router_average_them():
    import dataclasses
    cfg = dataclasses.replace(configs.MOE_SMALL, top_k=configs.MOE_SMALL.n_experts)
    Wt = _moe_weights(cfg)
    h = np.random.default_rng(2).standard_normal((7, cfg.hidden))
    Lw = of.layer_weights(Wt, 0)
    Lw["router"] = np.zeros_like(Lw["router"])
    y, idx, wts, _ = of.moe_mlp(cfg, Lw, h)
    assert np.array_equal(idx, np.tile(np.arange(cfg.n_experts, dtype=np.int32), (7, 1)))
    mean = sum(of.expert_mlp(h, {n: Lw[f"x{e}.{n}"] for n in ("wg", "wu", "wd")})
               for e in range(cfg.n_experts)) / cfg.n_experts
    assert rel_l2(y, mean) < 1e-14


def test_moe_is_invariant_to_expert_order():
    cfg = configs.MOE_SMALL
    Wt = _moe_weights(cfg)
    h = np.random.default_rng(4).standard_normal((9, cfg.hidden))
    Lw = of.layer_weights(Wt, 1)
    y, idx, wts, _ = of.moe_mlp(cfg, Lw, h)
    perm = np.array([2, 0, 3, 1])
    Lp = dict(Lw)
    Lp["router"] = Lw["router"][perm]
    for new, old in enumerate(perm):
        for n in ("wg", "wu", "wd"):
            Lp[f"x{new}.{n}"] = Lw[f"x{old}.{n}"]
    yp, idxp, wtsp, _ = of.moe_mlp(cfg, Lp, h)
    assert rel_l2(yp, y) < 1e-14
    assert np.array_equal(perm[idxp], idx) and np.allclose(wtsp, wts, atol=1e-15)


def test_forced_routes_reproduce_or_change_the_run():
    cfg = configs.MOE_SMALL
    Wt = _moe_weights(cfg)
    ids = init.token_ids(0, cfg.batch, cfg.prompt_len, cfg.vocab)
    a = of.llama_generate(cfg, Wt, ids)
    own = [[idx for idx, _, _ in seg] for seg in a["routes"]]
    b = of.llama_generate(cfg, Wt, ids, forced_routes=own)
    for x, y in zip(a["logits"], b["logits"]):
        assert np.array_equal(x, y)
    other = [[(idx + 1) % cfg.n_experts for idx in seg] for seg in own]
    c = of.llama_generate(cfg, Wt, ids, forced_routes=other)
    assert not np.allclose(c["logits"][0], a["logits"][0])
