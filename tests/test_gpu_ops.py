"""Per-op parity of the HIP kernels with the fp64 oracle, each op run as a
one-kernel trace through the C-ABI (budget = footprint).  Shapes cover several
tiles and ragged tails; bf16 results are compared at bf16 output precision."""
import numpy as np
import pytest

from oracle import forward as of
from workloads.format import (DT_BF16, DT_F32, DT_I32, MODE_R, MODE_RW, MODE_W,
                              OP_ARGMAX, OP_ATTN_CACHE, OP_ATTN_QKV, OP_EMBED,
                              OP_LAYERNORM, OP_LINEAR, OP_LINEAR_GELU,
                              OP_LINEAR_QKV, OP_LINEAR_RESID,
                              OP_LINEAR_SWIGLU, OP_RMSNORM, OP_ROPE_KV)

from gpu_util import (ELEM_ATTN, ELEM_BF16, ELEM_F32, assert_close, attention_backward_bounds, rel_l2,
                      single_kernel, write_inputs)

pytestmark = pytest.mark.gpu

# fp32 kernels differ from fp64 only by accumulation order; bf16 outputs are
# rounded once to 8 significant bits (relative error <= 2^-8 per element, a
# rel-L2 of about 1.1e-3 on average over a binade)
TOL = {DT_F32: 1e-5, DT_BF16: 4e-3}
ELEM = {DT_F32: ELEM_F32, DT_BF16: ELEM_BF16}


def close(got, ref, dt, scale=1, elem=None, what=""):
    """rel-L2 within the dtype's tolerance (times scale) and every element
    within its per-element bound."""
    return assert_close(got, ref, TOL[dt] * scale, elem or ELEM[dt], what)


def _run(op_, shape, operands, out):
    from paper_2609_06172_amd.session import Session
    w, vals = single_kernel(op_, shape, operands)
    print(f"op={op_} shape={shape}", flush=True)
    s = Session(w, device=0, M=w.footprint, fill=False)
    write_inputs(s, w, vals)
    s.run_all()
    res = {n: s.read(n) for n in out}
    s.close()
    return vals, res


RNG = np.random.default_rng(1234)


def rnd(*shape, scale=1.0):
    return RNG.standard_normal(shape).astype(np.float32) * scale


# bf16 kernels by shape: M <= 16 matrix-core GEMV (K % 64 == 32 ends on a half
# chunk); M >= 512 with K % 64 == 0 the
# 256 x 256 direct-LDS GEMM (one exact tile, ragged edges, several tiles);
# otherwise the 128 x 128 GEMM (including M >= 512 with K % 64 != 0)
LIN_SHAPES = [(1, 64, 32), (5, 100, 64), (7, 130, 160), (16, 33, 96), (16, 4096 + 16, 256), (17, 96, 96), (100, 130, 160),
              (257, 300, 512), (512, 256, 64), (600, 300, 128), (1030, 520, 192), (777, 1000, 256),
              (520, 130, 96), (640, 333, 128), (544, 130, 128)]
# the last two in the 256 x 256 epilogue: odd N (single columns) and N % 4 == 2
# (column pairs, no four-column stores); the other 256 x 256 cases have N % 4 == 0


@pytest.mark.parametrize("dt", [DT_F32, DT_BF16])
@pytest.mark.parametrize("M,N,K", LIN_SHAPES)
@pytest.mark.parametrize("op_", [OP_LINEAR, OP_LINEAR_GELU, OP_LINEAR_RESID, OP_LINEAR_SWIGLU])
def test_linear_family(op_, M, N, K, dt):
    a, W, W2 = rnd(M, K), rnd(N, K, scale=K ** -0.5), rnd(N, K, scale=K ** -0.5)
    out_dt = DT_F32 if op_ == OP_LINEAR_RESID else dt
    x0 = rnd(M, N)
    ops = [("a", (M, K), dt, MODE_R, a), ("W", (N, K), dt, MODE_R, W)]
    if op_ == OP_LINEAR_SWIGLU:
        ops.append(("W2", (N, K), dt, MODE_R, W2))
    if op_ == OP_LINEAR_RESID:
        ops.append(("c", (M, N), DT_F32, MODE_RW, x0))
    else:
        ops.append(("c", (M, N), out_dt, MODE_W, None))
    vals, res = _run(op_, (M, N, K), ops, ["c"])
    y = of.linear(vals["a"], vals["W"])
    if op_ == OP_LINEAR_GELU:
        y = of.gelu(y)
    elif op_ == OP_LINEAR_RESID:
        y = vals["c"] + y
    elif op_ == OP_LINEAR_SWIGLU:
        y = of.silu(y) * of.linear(vals["a"], vals["W2"])
    close(res["c"], y, out_dt, what=f"op {op_} ({M}, {N}, {K})")


@pytest.mark.parametrize("dt", [DT_F32, DT_BF16])
@pytest.mark.parametrize("M,N,K", LIN_SHAPES)
def test_linear_qkv(M, N, K, dt):
    """Grouped q, k, v projections: each output matches the oracle, and is bit
    for bit the output of the same product run as its own LINEAR."""
    a = rnd(M, K)
    Ws = [rnd(N, K, scale=K ** -0.5) for _ in range(3)]
    ops = [("a", (M, K), dt, MODE_R, a)] + [(f"W{i}", (N, K), dt, MODE_R, Ws[i]) for i in range(3)] + \
          [(f"c{i}", (M, N), dt, MODE_W, None) for i in range(3)]
    vals, res = _run(OP_LINEAR_QKV, (M, N, K), ops, ["c0", "c1", "c2"])
    for i in range(3):
        close(res[f"c{i}"], of.linear(vals["a"], vals[f"W{i}"]), dt, what=f"output {i}")
        _, one = _run(OP_LINEAR, (M, N, K), [("a", (M, K), dt, MODE_R, a), ("W", (N, K), dt, MODE_R, Ws[i]),
                                             ("c", (M, N), dt, MODE_W, None)], ["c"])
        assert np.array_equal(res[f"c{i}"].view(np.uint8), one["c"].view(np.uint8)), i


# The benchmark models' own shapes: the 7B decode projections at batch 16
# (the GEMV's K loop over 64 to 172 chunks, with a short last pass at
# K = 11008; the grouped q, k, v launch at N = K = 4096; the 32000-wide head)
# and the 1.3B prefill GEMMs (32 to 128 K steps of the 256 x 256 tile).  The
# prefill outputs are checked on every 61st row and the last one (several
# rows of every row tile, every column).
MODEL_SHAPES = [
    (OP_LINEAR_QKV, 16, 4096, 4096), (OP_LINEAR_RESID, 16, 4096, 4096),
    (OP_LINEAR_SWIGLU, 16, 11008, 4096), (OP_LINEAR_RESID, 16, 4096, 11008), (OP_LINEAR, 16, 32000, 4096),
    (OP_LINEAR, 8192, 6144, 2048), (OP_LINEAR_GELU, 8192, 8192, 2048), (OP_LINEAR_RESID, 8192, 2048, 2048),
    (OP_LINEAR_RESID, 8192, 2048, 8192),
]


@pytest.mark.parametrize("op_,M,N,K", MODEL_SHAPES)
def test_linear_at_model_shapes(op_, M, N, K):
    dt = DT_BF16
    g = np.random.default_rng(M * 7 + N * 3 + K)
    nw = {OP_LINEAR_QKV: 3, OP_LINEAR_SWIGLU: 2}.get(op_, 1)
    a = g.standard_normal((M, K), np.float32)
    Ws = [g.standard_normal((N, K), np.float32) * np.float32(0.02) for _ in range(nw)]
    ops = [("a", (M, K), dt, MODE_R, a)] + [(f"W{i}", (N, K), dt, MODE_R, Ws[i]) for i in range(nw)]
    if op_ == OP_LINEAR_QKV:
        outs = ["c0", "c1", "c2"]
        ops += [(c, (M, N), dt, MODE_W, None) for c in outs]
    elif op_ == OP_LINEAR_RESID:
        outs = ["c"]
        ops.append(("c", (M, N), DT_F32, MODE_RW, g.standard_normal((M, N), np.float32)))
    else:
        outs = ["c"]
        ops.append(("c", (M, N), dt, MODE_W, None))
    vals, res = _run(op_, (M, N, K), ops, outs)
    rows = np.arange(M) if M <= 16 else np.unique(np.r_[np.arange(0, M, 61), M - 1])
    ar = vals["a"][rows]
    if op_ == OP_LINEAR_QKV:
        for i in range(3):
            close(res[f"c{i}"][rows], of.linear(ar, vals[f"W{i}"]), dt, what=f"output {i}")
        return
    y = of.linear(ar, vals["W0"])
    out_dt = dt
    if op_ == OP_LINEAR_GELU:
        y = of.gelu(y)
    elif op_ == OP_LINEAR_SWIGLU:
        y = of.silu(y) * of.linear(ar, vals["W1"])
    elif op_ == OP_LINEAR_RESID:
        y = vals["c"][rows] + y
        out_dt = DT_F32
    # an fp32 result of a K-deep fp32 accumulation: rounding errors random-walk
    # to about 2^-24 * sqrt(K / 2) of the result's rms, ~5 sigma at the
    # largest of a million elements; 8 * 2^-24 * sqrt(K) leaves a 2x margin
    elem = (1e-5, max(1e-5, 8 * 2.0 ** -24 * np.sqrt(K))) if out_dt == DT_F32 else None
    close(res["c"][rows], y, out_dt, elem=elem, what=f"op {op_} ({M}, {N}, {K})")


@pytest.mark.parametrize("dt", [DT_F32, DT_BF16])
@pytest.mark.parametrize("T,H,stride,offset", [(7, 128, 1, 0), (3, 4096, 5, 4), (33, 2048, 1, 0),
                                              (5, 8192, 2, 1), (4, 130, 1, 0), (2, 8196, 1, 0),
                                              (9, 12, 3, 2), (16, 2052, 1, 0)])
def test_norms(T, H, stride, offset, dt):
    rows = (T - 1) * stride + offset + 1
    x = rnd(rows, H) * 3 + 0.5
    g, b = rnd(H) * 0.5 + 1, rnd(H) * 0.1
    vals, res = _run(OP_LAYERNORM, (T, H, stride, offset),
                     [("x", (rows, H), DT_F32, MODE_R, x), ("g", (H,), dt, MODE_R, g),
                      ("b", (H,), dt, MODE_R, b), ("h", (T, H), dt, MODE_W, None)], ["h"])
    sel = vals["x"][np.arange(T) * stride + offset]
    close(res["h"], of.layernorm(sel, vals["g"], vals["b"]), dt, 2, what="layernorm")
    vals, res = _run(OP_RMSNORM, (T, H, stride, offset),
                     [("x", (rows, H), DT_F32, MODE_R, x), ("g", (H,), dt, MODE_R, g),
                      ("h", (T, H), dt, MODE_W, None)], ["h"])
    close(res["h"], of.rmsnorm(sel, vals["g"]), dt, 2, what="rmsnorm")


@pytest.mark.parametrize("dt", [DT_F32, DT_BF16])
def test_embed(dt):
    V, H, T = 1000, 256, 37
    E = rnd(V, H)
    ids = RNG.integers(0, V, T).astype(np.int32)
    vals, res = _run(OP_EMBED, (T, H, V), [("ids", (T,), DT_I32, MODE_R, ids),
                                           ("E", (V, H), dt, MODE_R, E),
                                           ("x", (T, H), DT_F32, MODE_W, None)], ["x"])
    assert np.array_equal(res["x"], vals["E"][ids].astype(np.float32))


@pytest.mark.parametrize("dt", [DT_F32, DT_BF16])
@pytest.mark.parametrize("B,S,nH,d", [(1, 32, 4, 32), (2, 75, 3, 64), (1, 130, 2, 128), (2, 12, 2, 128),
                                     (2, 75, 3, 128), (1, 257, 2, 128)])
def test_attention_fused_qkv(B, S, nH, d, dt):
    Hd = nH * d
    qkv = rnd(B * S, 3 * Hd)
    vals, res = _run(OP_ATTN_QKV, (B, S, nH, d), [("qkv", (B * S, 3 * Hd), dt, MODE_R, qkv),
                                                  ("o", (B * S, Hd), dt, MODE_W, None)], ["o"])
    q = vals["qkv"]
    ref = np.empty((B * S, Hd))
    for b in range(B):
        r = slice(b * S, (b + 1) * S)
        for h in range(nH):
            c = slice(h * d, (h + 1) * d)
            ref[r, c] = of.causal_attention(q[r, c], q[r, Hd + h * d:Hd + (h + 1) * d],
                                            q[r, 2 * Hd + h * d:2 * Hd + (h + 1) * d])
    close(res["o"], ref, dt, 2, elem=ELEM_ATTN if dt == DT_BF16 else None, what="attention")


@pytest.mark.parametrize("B,S,nH,d,Lmax,pos0", [(2, 1, 2, 128, 300, 257), (3, 40, 2, 128, 64, 0),
                                                (1, 5, 4, 64, 20, 9), (16, 1, 2, 128, 1280, 1100),
                                                (2, 7, 2, 128, 64, 20), (1, 1, 1, 128, 8, 0),
                                                (4, 16, 2, 128, 300, 131), (2, 33, 2, 128, 100, 50),
                                                (1, 200, 1, 128, 256, 0), (2, 64, 2, 128, 192, 64)])
def test_rope_kv_and_cached_attention(B, S, nH, d, Lmax, pos0):
    dt = DT_BF16
    Hd = nH * d
    q, k, v = rnd(B * S, Hd), rnd(B * S, Hd), rnd(B * S, Hd)
    Kc, Vc = rnd(B, nH, Lmax, d), rnd(B, nH, Lmax, d)
    shape = (B, S, nH, d, Lmax, pos0)
    vals, res = _run(OP_ROPE_KV, shape,
                     [("q", (B * S, Hd), dt, MODE_RW, q), ("k", (B * S, Hd), dt, MODE_R, k),
                      ("v", (B * S, Hd), dt, MODE_R, v), ("Kc", (B, nH, Lmax, d), dt, MODE_RW, Kc),
                      ("Vc", (B, nH, Lmax, d), dt, MODE_RW, Vc)], ["q", "Kc", "Vc"])
    pos = pos0 + np.arange(S)
    qr = of.rope(vals["q"].reshape(B, S, nH, d), pos[None, :, None])
    kr = of.rope(vals["k"].reshape(B, S, nH, d), pos[None, :, None])
    Kref, Vref = vals["Kc"].copy(), vals["Vc"].copy()
    Kref[:, :, pos0:pos0 + S] = kr.transpose(0, 2, 1, 3)
    Vref[:, :, pos0:pos0 + S] = vals["v"].reshape(B, S, nH, d).transpose(0, 2, 1, 3)
    close(res["q"], qr.reshape(B * S, Hd), dt, 2, what="roped q")
    close(res["Kc"][:, :, pos0:pos0 + S], Kref[:, :, pos0:pos0 + S], dt, 2, what="new K rows")
    assert np.array_equal(res["Vc"], Vref.astype(np.float32))
    untouched = np.ones(Lmax, bool)
    untouched[pos0:pos0 + S] = False
    assert np.array_equal(res["Kc"][:, :, untouched], Kref[:, :, untouched].astype(np.float32))
    # attention of the roped queries over the updated cache
    vals2, res2 = _run(OP_ATTN_CACHE, shape,
                       [("q", (B * S, Hd), dt, MODE_R, res["q"]), ("Kc", (B, nH, Lmax, d), dt, MODE_R, res["Kc"]),
                        ("Vc", (B, nH, Lmax, d), dt, MODE_R, res["Vc"]), ("o", (B * S, Hd), dt, MODE_W, None)], ["o"])
    qq = vals2["q"].reshape(B, S, nH, d)
    ref = np.empty((B, S, nH, d))
    for b in range(B):
        for h in range(nH):
            L = pos0 + S
            ref[b, :, h] = of.causal_attention(qq[b, :, h], vals2["Kc"][b, h, :L], vals2["Vc"][b, h, :L], pos0)
    close(res2["o"], ref.reshape(B * S, Hd), dt, 2, elem=ELEM_ATTN, what="cached attention")


@pytest.mark.parametrize("B,V", [(1, 1000), (16, 32000), (3, 50000)])
def test_argmax_lowest_index(B, V):
    logits = rnd(B, V)
    logits[0, 5] = logits[0, 900] = 50.0          # tie: lowest index wins
    row = 2
    vals, res = _run(OP_ARGMAX, (B, V, row), [("logits", (B, V), DT_F32, MODE_R, logits),
                                             ("tok", (B,), DT_I32, MODE_W, None),
                                             ("gen", (row + 1, B), DT_I32, MODE_RW,
                                              np.zeros((row + 1, B), np.int32))], ["tok", "gen"])
    ref = of.argmax_lowest(vals["logits"])
    assert ref[0] == 5
    assert np.array_equal(res["tok"], ref)
    assert np.array_equal(res["gen"][row], ref)
    assert np.array_equal(res["gen"][:row], np.zeros((row, B), np.int32))


# ------------------------------------------------------- routed experts (MoE)
from workloads.format import OP_MOE_DISPATCH, OP_MOE_DOWN, OP_MOE_ROUTE, OP_MOE_UP  # noqa: E402


def _topk_rows(logits, k):
    idx, wts = of.route_topk(logits, k)
    srt = -np.sort(-logits, axis=1)
    gap = srt[:, k - 1] - srt[:, k] if k < logits.shape[1] else np.full(len(logits), np.inf)
    return idx, wts, gap


@pytest.mark.parametrize("dt", [DT_F32, DT_BF16])
@pytest.mark.parametrize("M,H,E,K", [(1, 64, 4, 2), (37, 256, 4, 2), (300, 4096, 8, 2), (5, 128, 16, 4),
                                     (9, 520, 3, 3), (64, 64, 8, 1), (2049, 1024, 8, 2)])
def test_moe_route_topk(M, H, E, K, dt):
    h, wr = rnd(M, H), rnd(E, H, scale=H ** -0.5)
    ops = [("h", (M, H), dt, MODE_R, h), ("wr", (E, H), dt, MODE_R, wr),
           ("rte", (M, K), DT_I32, MODE_W, None), ("rtw", (M, K), DT_F32, MODE_W, None)]
    vals, res = _run(OP_MOE_ROUTE, (M, H, E, K), ops, ["rte", "rtw"])
    logits = of.linear(vals["h"], vals["wr"])
    idx, wts, gap = _topk_rows(logits, K)
    # fp32 accumulation moves a logit by ~1e-6 of its scale: rows whose k-th and
    # (k+1)-th logits are further apart must pick exactly the oracle's experts
    clear = gap > 1e-4
    assert clear.mean() > 0.9
    assert np.array_equal(res["rte"][clear], idx[clear])
    assert np.allclose(res["rtw"][clear], wts[clear], rtol=0, atol=2e-5)
    # every row: distinct experts, descending logits, weights summing to 1
    for m in range(M):
        assert len(set(res["rte"][m])) == K and all(0 <= e < E for e in res["rte"][m])
        assert np.all(np.diff(logits[m, res["rte"][m]]) <= 1e-4)
    assert np.allclose(res["rtw"].sum(axis=1), 1, atol=1e-6)


def test_moe_route_ties_go_to_the_lower_index():
    M, H, E, K = 40, 256, 6, 3
    h, wr = rnd(M, H), rnd(E, H, scale=H ** -0.5)
    wr[4] = wr[1]                     # experts 1 and 4 tie exactly, so do 2 and 5
    wr[5] = wr[2]
    ops = [("h", (M, H), DT_BF16, MODE_R, h), ("wr", (E, H), DT_BF16, MODE_R, wr),
           ("rte", (M, K), DT_I32, MODE_W, None), ("rtw", (M, K), DT_F32, MODE_W, None)]
    vals, res = _run(OP_MOE_ROUTE, (M, H, E, K), ops, ["rte", "rtw"])
    for m in range(M):
        sel = list(res["rte"][m])
        for lo, hi in ((1, 4), (2, 5)):
            if hi in sel:
                assert lo in sel and sel.index(lo) < sel.index(hi)


def _routes(M, E, K, seed, skip=()):
    """Random top-K choices (distinct per row) avoiding the experts in skip."""
    g = np.random.default_rng(seed)
    pool = [e for e in range(E) if e not in skip]
    return np.stack([g.permutation(pool)[:K] for _ in range(M)]).astype(np.int32)


@pytest.mark.parametrize("M,E,K,row,skip", [(1, 4, 2, 0, ()), (7, 4, 2, 1, (3,)), (600, 8, 2, 2, ()),
                                            (3000, 8, 2, 0, (5,)), (32768, 8, 2, 3, ()), (100, 16, 4, 1, (0, 9))])
def test_moe_dispatch_lists_are_exact(M, E, K, row, skip):
    rte = _routes(M, E, K, M + E, skip)
    log0 = np.arange((row + 2) * E, dtype=np.int32).reshape(row + 2, E) + 7
    ops = [("rte", (M, K), DT_I32, MODE_R, rte), ("lists", (E, M + 1), DT_I32, MODE_W, None),
           ("log", (row + 2, E), DT_I32, MODE_RW, log0)]
    vals, res = _run(OP_MOE_DISPATCH, (M, E, K, row), ops, ["lists", "log"])
    flat = rte.reshape(-1)
    for e in range(E):
        want = np.nonzero(flat == e)[0]
        assert res["lists"][e, 0] == len(want)
        assert np.array_equal(res["lists"][e, 1:1 + len(want)], want)
    exp_log = log0.copy()
    exp_log[row] = [np.count_nonzero(flat == e) for e in range(E)]
    assert np.array_equal(res["log"], exp_log)     # other rows of the log untouched


def _lists(M, E, K, rte):
    L = np.zeros((E, M + 1), np.int32)
    flat = rte.reshape(-1)
    for e in range(E):
        j = np.nonzero(flat == e)[0]
        L[e, 0] = len(j)
        L[e, 1:1 + len(j)] = j
    return L


# M <= 16: the routed-row GEMV; larger M: the 256 x 256 GEMM (tiles past the
# count exit).  Expert 1 of 3; some shapes leave it with no rows.
MOE_GEMM = [(1, 64, 64, ()), (8, 384, 256, ()), (16, 128, 64, (1,)), (80, 384, 256, ()),
            (600, 192, 128, ()), (2048, 256, 512, ()), (300, 128, 64, (1,))]


@pytest.mark.parametrize("M,F,H,skip", MOE_GEMM)
def test_moe_expert_up(M, F, H, skip):
    E, K, e = 3, 2, 1
    rte = _routes(M, E, K, 3 * M + F, skip)
    lists = _lists(M, E, K, rte)
    n = int(lists[e, 0])
    h, wg, wu = rnd(M, H), rnd(F, H, scale=H ** -0.5), rnd(F, H, scale=H ** -0.5)
    ops = [("h", (M, H), DT_BF16, MODE_R, h), ("lists", (E, M + 1), DT_I32, MODE_R, lists),
           ("wg", (F, H), DT_BF16, MODE_R, wg), ("wu", (F, H), DT_BF16, MODE_R, wu),
           ("fe", (M, F), DT_BF16, MODE_W, None)]
    vals, res = _run(OP_MOE_UP, (M, F, H, e, max(n, 1), K), ops, ["fe"])
    tok = lists[e, 1:1 + n] // K
    hr = vals["h"][tok]
    want = of.silu(of.linear(hr, vals["wg"])) * of.linear(hr, vals["wu"])
    if n:
        close(res["fe"][:n], want, DT_BF16, what="expert up")


@pytest.mark.parametrize("M,F,H,skip", MOE_GEMM)
def test_moe_expert_down(M, F, H, skip):
    E, K, e = 3, 2, 1
    rte = _routes(M, E, K, 5 * M + H, skip)
    lists = _lists(M, E, K, rte)
    n = int(lists[e, 0])
    fe, wd = rnd(M, F), rnd(H, F, scale=F ** -0.5)
    rtw, x0 = RNG.random((M, K)).astype(np.float32), rnd(M, H)
    ops = [("fe", (M, F), DT_BF16, MODE_R, fe), ("lists", (E, M + 1), DT_I32, MODE_R, lists),
           ("rtw", (M, K), DT_F32, MODE_R, rtw), ("wd", (H, F), DT_BF16, MODE_R, wd),
           ("x", (M, H), DT_F32, MODE_RW, x0)]
    vals, res = _run(OP_MOE_DOWN, (M, H, F, e, max(n, 1), K), ops, ["x"])
    j = lists[e, 1:1 + n]
    want = vals["x"].copy()
    want[j // K] += vals["rtw"].reshape(-1)[j][:, None] * of.linear(vals["fe"][:n], vals["wd"])
    routed = np.zeros(M, bool)
    routed[j // K] = True
    assert np.array_equal(res["x"][~routed], vals["x"][~routed])     # other rows untouched
    if n:
        close(res["x"][routed], want[routed], DT_F32, what="expert down")


# ------------------------------------------------------- training step ops
from oracle import train as ot  # noqa: E402
from workloads.format import (OP_ADAM, OP_ATTN_BWD, OP_COPY, OP_EMBED_BWD,  # noqa: E402
                              OP_RMSNORM_BWD, OP_ROPE_BWD, OP_SWIGLU_ACT, OP_SWIGLU_BWD,
                              OP_TRANSPOSE, OP_XENT)
from workloads.trace import adam_shape  # noqa: E402


@pytest.mark.parametrize("dt", [DT_F32, DT_BF16])
@pytest.mark.parametrize("R,C", [(1, 1), (64, 64), (100, 37), (130, 2049), (1024, 160)])
def test_transpose_and_copy(R, C, dt):
    a = rnd(R, C)
    vals, res = _run(OP_TRANSPOSE, (R, C), [("a", (R, C), dt, MODE_R, a), ("b", (C, R), dt, MODE_W, None)], ["b"])
    assert np.array_equal(res["b"], vals["a"].T)
    nb = R * C * (4 if dt == DT_F32 else 2)
    vals, res = _run(OP_COPY, (nb,), [("a", (R, C), dt, MODE_R, a), ("b", (R, C), dt, MODE_W, None)], ["b"])
    assert np.array_equal(res["b"], vals["a"])


@pytest.mark.parametrize("T,F", [(3, 5), (160, 384), (777, 1000)])
def test_swiglu_act_and_backward(T, F):
    G, U, dF = rnd(T, F, scale=3), rnd(T, F), rnd(T, F)
    ops = [("G", (T, F), DT_BF16, MODE_R, G), ("U", (T, F), DT_BF16, MODE_R, U), ("F", (T, F), DT_BF16, MODE_W, None)]
    vals, res = _run(OP_SWIGLU_ACT, (T, F), ops, ["F"])
    close(res["F"], of.silu(vals["G"]) * vals["U"], DT_BF16, what="swiglu")
    ops = [("G", (T, F), DT_BF16, MODE_R, G), ("U", (T, F), DT_BF16, MODE_R, U), ("dF", (T, F), DT_BF16, MODE_R, dF),
           ("dG", (T, F), DT_BF16, MODE_W, None), ("dU", (T, F), DT_BF16, MODE_W, None)]
    vals, res = _run(OP_SWIGLU_BWD, (T, F), ops, ["dG", "dU"])
    g = vals["G"]
    close(res["dG"], vals["dF"] * vals["U"] * ot.silu_grad(g), DT_BF16, what="dG")
    close(res["dU"], vals["dF"] * of.silu(g), DT_BF16, what="dU")


@pytest.mark.parametrize("acc", [0, 1])
@pytest.mark.parametrize("T,H", [(1, 64), (37, 256), (300, 5120), (5, 130)])
def test_rmsnorm_backward(T, H, acc):
    x, g, dy, dx0 = rnd(T, H), 1 + 0.1 * rnd(H), rnd(T, H), rnd(T, H)
    ops = [("x", (T, H), DT_F32, MODE_R, x), ("g", (H,), DT_BF16, MODE_R, g), ("dy", (T, H), DT_F32, MODE_R, dy),
           ("dx", (T, H), DT_F32, MODE_RW if acc else MODE_W, dx0 if acc else None),
           ("dxb", (T, H), DT_BF16, MODE_W, None), ("dg", (H,), DT_F32, MODE_W, None),
           ("rstd", (T,), DT_F32, MODE_W, None)]
    vals, res = _run(OP_RMSNORM_BWD, (T, H, acc), ops, ["dx", "dxb", "dg"])
    dx, dg = ot.rmsnorm_backward(vals["x"], vals["g"], vals["dy"])
    if acc:
        dx = dx + vals["dx"]
    close(res["dx"], dx, DT_F32, what="dx")
    close(res["dxb"], dx, DT_BF16, what="dx (bf16)")
    close(res["dg"], dg, DT_F32, what="dg")


def _attn_fwd_bwd_ref(q, K, V, dO, B, S, nH):
    """Oracle attention (per head, causal) on the GPU's cache layout."""
    d = 128
    qh = q.reshape(B, S, nH, d)
    do = dO.reshape(B, S, nH, d)
    o = np.empty_like(qh)
    lse = np.empty((B, nH, S))
    dq, dK, dV = np.empty_like(qh), np.empty_like(K), np.empty_like(V)
    for b in range(B):
        for h in range(nH):
            s = (qh[b, :, h] @ K[b, h].T) / np.sqrt(d)
            s = np.where(np.arange(S)[None, :] <= np.arange(S)[:, None], s, -np.inf)
            m = s.max(axis=1, keepdims=True)
            lse[b, h] = (m + np.log(np.exp(s - m).sum(axis=1, keepdims=True)))[:, 0]
            o[b, :, h] = of.causal_attention(qh[b, :, h], K[b, h], V[b, h])
            dq[b, :, h], dK[b, h], dV[b, h] = ot.attention_backward(qh[b, :, h], K[b, h], V[b, h], do[b, :, h])
    return o.reshape(B * S, nH * d), lse, dq.reshape(B * S, nH * d), dK, dV


# (1, 160, 80) and (2, 130, 40): 80 (batch, head) pairs, ten per XCD, taken in
# groups of four, the last group of two (the flash kernels' workgroup order)
@pytest.mark.parametrize("B,S,nH", [(1, 1, 1), (1, 70, 2), (2, 160, 2), (1, 300, 1), (1, 160, 80), (2, 130, 40)])
def test_attention_lse_and_backward(B, S, nH):
    d = 128
    q, K, V, dO = rnd(B * S, nH * d), rnd(B, nH, S, d), rnd(B, nH, S, d), rnd(B * S, nH * d)
    o_ref = None
    # forward with the log-sum-exp output (flash kernel)
    ops = [("q", (B * S, nH * d), DT_BF16, MODE_R, q), ("K", (B, nH, S, d), DT_BF16, MODE_R, K),
           ("V", (B, nH, S, d), DT_BF16, MODE_R, V), ("o", (B * S, nH * d), DT_BF16, MODE_W, None),
           ("lse", (B, nH, S), DT_F32, MODE_W, None)]
    vals, res = _run(OP_ATTN_CACHE, (B, S, nH, d, S, 0), ops, ["o", "lse"])
    o_ref, lse_ref, _, _, _ = _attn_fwd_bwd_ref(vals["q"], vals["K"], vals["V"], np.zeros_like(vals["q"]), B, S, nH)
    close(res["o"], o_ref, DT_BF16, elem=ELEM_ATTN, what="attention with lse")
    assert np.abs(res["lse"] - lse_ref).max() < 1e-3
    # backward from the GPU's own o and lse (the forward's outputs)
    o_b = res["o"]
    ops = [("q", (B * S, nH * d), DT_BF16, MODE_R, q), ("K", (B, nH, S, d), DT_BF16, MODE_R, K),
           ("V", (B, nH, S, d), DT_BF16, MODE_R, V), ("o", (B * S, nH * d), DT_BF16, MODE_R, o_b),
           ("lse", (B, nH, S), DT_F32, MODE_R, res["lse"]), ("do", (B * S, nH * d), DT_BF16, MODE_R, dO),
           ("dq", (B * S, nH * d), DT_BF16, MODE_W, None), ("dK", (B, nH, S, d), DT_BF16, MODE_W, None),
           ("dV", (B, nH, S, d), DT_BF16, MODE_W, None), ("D", (B, nH, S), DT_F32, MODE_W, None)]
    vals, res = _run(OP_ATTN_BWD, (B, S, nH, d), ops, ["dq", "dK", "dV"])
    _, _, dq, dK, dV = _attn_fwd_bwd_ref(vals["q"], vals["K"], vals["V"], vals["do"], B, S, nH)
    # relative, with an absolute floor of 1e-4 per element: a single key gives
    # dq = dK = 0 exactly, and the GPU's rounding leaves ~1e-7 there
    for got, want in ((res["dq"], dq), (res["dK"], dK), (res["dV"], dV)):
        err = np.linalg.norm(np.asarray(got, np.float64) - want)
        assert err < 1e-2 * np.linalg.norm(want) + 1e-4 * np.sqrt(want.size)
    # every element within its first-order rounding bound (plus 1e-6 absolute
    # for the exact zeros of a one-key row)
    qh = vals["q"].reshape(B, S, nH, d)
    doh = vals["do"].reshape(B, S, nH, d)
    gq = np.asarray(res["dq"], np.float64).reshape(B, S, nH, d)
    rq = dq.reshape(B, S, nH, d)
    for b in range(B):
        for h in range(nH):
            _, (bq, bk, bv) = attention_backward_bounds(qh[b, :, h], vals["K"][b, h], vals["V"][b, h], doh[b, :, h])
            for name, g, r, bd in (("dq", gq[b, :, h], rq[b, :, h], bq), ("dK", res["dK"][b, h], dK[b, h], bk),
                                   ("dV", res["dV"][b, h], dV[b, h], bv)):
                bad = np.abs(np.asarray(g, np.float64) - r) > bd + 1e-6
                assert not bad.any(), f"{name} ({b}, {h}): {int(bad.sum())} elements outside their bound"


@pytest.mark.parametrize("B,S,nH,d", [(1, 1, 1, 128), (2, 75, 3, 64), (1, 200, 2, 128)])
def test_rope_backward_is_the_inverse_rotation(B, S, nH, d):
    dq, dK, dV = rnd(B * S, nH * d), rnd(B, nH, S, d), rnd(B, nH, S, d)
    ops = [("dq", (B * S, nH * d), DT_F32, MODE_RW, dq), ("dK", (B, nH, S, d), DT_F32, MODE_R, dK),
           ("dV", (B, nH, S, d), DT_F32, MODE_R, dV), ("dk", (B * S, nH * d), DT_F32, MODE_W, None),
           ("dv", (B * S, nH * d), DT_F32, MODE_W, None)]
    vals, res = _run(OP_ROPE_BWD, (B, S, nH, d), ops, ["dq", "dk", "dv"])
    pos = np.tile(np.arange(S), B)[:, None]
    want_q = of.rope(vals["dq"].reshape(B * S, nH, d), -pos).reshape(B * S, nH * d)
    kt = vals["dK"].transpose(0, 2, 1, 3).reshape(B * S, nH, d)
    want_k = of.rope(kt, -pos).reshape(B * S, nH * d)
    # fp32 angles pos * 10000^(-2i/d): ~1e-5 rad of error at position 200
    assert_close(res["dq"], want_q, 5e-5, (1e-4, 1e-4), "dq")
    assert_close(res["dk"], want_k, 5e-5, (1e-4, 1e-4), "dk")
    assert np.array_equal(res["dv"], vals["dV"].transpose(0, 2, 1, 3).reshape(B * S, nH * d))


@pytest.mark.parametrize("T,V", [(1, 7), (33, 1024), (160, 32000)])
def test_cross_entropy_rows_and_gradient(T, V):
    lg = rnd(T, V, scale=2)
    labels = RNG.integers(0, V, T).astype(np.int32)
    ops = [("logits", (T, V), DT_F32, MODE_R, lg), ("labels", (T,), DT_I32, MODE_R, labels),
           ("losses", (T,), DT_F32, MODE_W, None), ("dlogits", (T, V), DT_BF16, MODE_W, None)]
    vals, res = _run(OP_XENT, (T, V), ops, ["losses", "dlogits"])
    loss, dl = ot.cross_entropy(vals["logits"], labels)
    assert abs(res["losses"].astype(np.float64).mean() - loss) < 1e-5 * max(1, abs(loss))
    close(res["dlogits"], dl, DT_BF16, what="dlogits")


@pytest.mark.parametrize("T,H,V", [(1, 64, 5), (160, 256, 1024), (2000, 130, 70)])
def test_embedding_backward_sums_in_token_order(T, H, V):
    ids = RNG.integers(0, V, T).astype(np.int32)
    dx = rnd(T, H)
    ops = [("ids", (T,), DT_I32, MODE_R, ids), ("dx", (T, H), DT_F32, MODE_R, dx), ("dE", (V, H), DT_F32, MODE_W, None)]
    vals, res = _run(OP_EMBED_BWD, (T, H, V), ops, ["dE"])
    want = np.zeros((V, H))
    np.add.at(want, ids, vals["dx"])
    assert_close(res["dE"], want, 1e-6, ELEM_F32, "dE")
    assert np.all(res["dE"][np.setdiff1d(np.arange(V), ids)] == 0)


@pytest.mark.parametrize("dt", [DT_F32, DT_BF16])
@pytest.mark.parametrize("n", [1, 1000, 70001])
def test_adamw_update(n, dt):
    from workloads.init import TRAIN_HP as hp
    g, p = rnd(n, scale=1e-3), rnd(n, scale=0.02)
    m, v = rnd(n, scale=1e-4), np.square(rnd(n, scale=1e-4))
    ops = [("g", (n,), DT_F32, MODE_R, g), ("p32", (n,), DT_F32, MODE_RW, p), ("m", (n,), DT_F32, MODE_RW, m),
           ("v", (n,), DT_F32, MODE_RW, v), ("p", (n,), dt, MODE_W, None)]
    vals, res = _run(OP_ADAM, adam_shape(n, hp), ops, ["p32", "m", "v", "p"])
    p2, m2, v2 = ot.adamw(vals["p32"], vals["g"], vals["m"], vals["v"], hp["step"], hp["lr"], hp["b1"], hp["b2"],
                          hp["eps"], hp["wd"])
    # weights at fp32 precision: the update (lr-sized, ~1% of a weight) shows at 1e-6
    assert rel_l2(res["p32"], p2) < 2e-6
    # and the update itself, elementwise, up to one fp32 rounding of the weight
    dg, dr = res["p32"] - vals["p32"], p2 - vals["p32"]
    assert np.all(np.abs(dg - dr) <= 1e-3 * np.abs(dr) + 2.4e-7 * np.abs(p2))
    assert_close(res["m"], m2, 1e-6, ELEM_F32, "m")
    assert_close(res["v"], v2, 1e-6, ELEM_F32, "v")
    close(res["p"], p2, dt, what="weight")
