"""Pins of the oracle's cost model (flops F and algorithmic HBM bytes B per
kernel), which places every kernel on the roofline (paper Sec. III-C; the
paper counts each kernel's flops and loads, Sec. IV-G).

The expected numbers are written out by hand from each op's definition (the
operand table of the trace format), under the counting rules stated with the
per-op table of the design notes:

* bytes: every operand element the op reads or writes counts once at its
  element size; an element that is read and then written (RW) counts twice;
  elements an op does not touch (rows it does not gather, cache positions
  past the prefix) do not count;
* flops: 2 per multiply-add of a contraction, plus the stated per-element
  cost of the epilogue or elementwise op.

Shapes use distinct small factors and mixed element types, so that a
transposed factor, a wrong operand's element size, a dropped operand or an
RW counted once changes the result.  A second group counts the causal
query--key pairs of the attention ops by enumeration, and a third checks
whole-unit totals (a 7B decode step, a 1.3B prefill pass) against closed
forms worked out from the model dimensions alone.
"""
import pytest

from oracle.costs import kernel_cost
from workloads.format import (DT_BF16, DT_F32, DT_I32, DT_U8, MODE_R, MODE_RW, MODE_W,
                              OP_ADAM, OP_ARGMAX, OP_ATTN_BWD, OP_ATTN_CACHE, OP_ATTN_QKV,
                              OP_COPY, OP_EMBED, OP_EMBED_BWD, OP_LAYERNORM, OP_LINEAR,
                              OP_LINEAR_GELU, OP_LINEAR_QKV, OP_LINEAR_RESID,
                              OP_LINEAR_SWIGLU, OP_MOE_DISPATCH, OP_MOE_DOWN, OP_MOE_ROUTE,
                              OP_MOE_UP, OP_NAMES, OP_RMSNORM, OP_RMSNORM_BWD, OP_ROPE_BWD,
                              OP_ROPE_KV, OP_SWIGLU_ACT, OP_SWIGLU_BWD, OP_TOUCH, OP_TRANSPOSE,
                              OP_XENT)

f32, bf16, i32, u8 = DT_F32, DT_BF16, DT_I32, DT_U8
R, W, RW = MODE_R, MODE_W, MODE_RW
ES = {f32: 4, bf16: 2, i32: 4, u8: 1}


def _cost(op, shape, ops):
    """ops: (element type, element count, mode) per operand, positional;
    a repeated tensor is given as ("dup", index of the first operand, mode)."""
    operands, dtypes, nbytes = [], [], []
    for o in ops:
        if o[0] == "dup":
            operands.append((operands[o[1]][0], o[2]))
            continue
        dt, n, m = o
        operands.append((len(dtypes), m))
        dtypes.append(dt)
        nbytes.append(n * ES[dt])
    return kernel_cost(op, shape, operands, dtypes, nbytes)


# (op, shape, operands, F, B, how B is made up)
CASES = [
    (OP_TOUCH, (2,), [(u8, 64, RW), (u8, 100, R), (u8, 256, W), ("dup", 1, W), (u8, 40, RW)], 0, 664,
     "log RW 2*64; t1 read then written (modes merge to RW) 2*100; t2 256; t3 RW 2*40"),
    (OP_EMBED, (3, 5, 11), [(i32, 3, R), (bf16, 55, R), (f32, 15, W)], 0, 102,
     "3 ids 12; the 3 gathered rows of E 3*5*2 = 30 (not all 11); x 3*5*4 = 60"),
    (OP_LAYERNORM, (3, 8, 2, 1), [(f32, 48, R), (bf16, 8, R), (bf16, 8, R), (bf16, 24, W)], 192, 176,
     "3 of the 6 strided rows of x 3*8*4 = 96; g 16; b 16; h 48.  F: 8 per element (mean, variance "
     "3, centre, scale, gain, bias) * 24"),
    (OP_RMSNORM, (3, 8, 2, 1), [(f32, 48, R), (bf16, 8, R), (bf16, 24, W)], 96, 160,
     "x rows 96; g 16; h 48.  F: 4 per element (square, sum, scale, gain) * 24"),
    (OP_LINEAR, (3, 5, 7), [(bf16, 21, R), (bf16, 35, R), (f32, 15, W)], 210, 172,
     "a 3*7*2 = 42; W 5*7*2 = 70; c 3*5*4 = 60.  F: 2*3*5*7"),
    (OP_LINEAR_GELU, (3, 5, 7), [(f32, 21, R), (f32, 35, R), (f32, 15, W)], 330, 284,
     "a 84; W 140; c 60.  F: 210 + 8 per output (GELU) * 15"),
    (OP_LINEAR_RESID, (3, 5, 7), [(bf16, 21, R), (bf16, 35, R), (f32, 15, RW)], 225, 232,
     "a 42; W 70; x read and written 2*60.  F: 210 + one add per output"),
    (OP_LINEAR_SWIGLU, (3, 5, 7), [(bf16, 21, R), (bf16, 35, R), (bf16, 35, R), (bf16, 15, W)], 480, 212,
     "a 42 (read once for both products); Wg 70; Wu 70; c 3*5*2 = 30.  F: two products 4*105 + 4 per "
     "output (silu and the gating multiply) * 15"),
    (OP_LINEAR_QKV, (3, 5, 7), [(bf16, 21, R), (bf16, 35, R), (bf16, 35, R), (bf16, 35, R),
                                (bf16, 15, W), (bf16, 15, W), (f32, 15, W)], 630, 372,
     "a 42 once; three weights 3*70; q, k 30 each, v (fp32) 60.  F: 3*210"),
    (OP_ATTN_QKV, (2, 3, 2, 4), [(bf16, 6 * 24, R), (bf16, 6 * 8, W)], 480, 384,
     "q, k, v rows of the fused tensor 3 * 6*8*2 = 288; o 96.  F: 2 sequences * 2 heads * 6 causal "
     "pairs (1+2+3) * (2d for q.k + 2d for p.v + 4 for the softmax) = 4*6*20"),
    (OP_ROPE_KV, (2, 3, 2, 4, 10, 5), [(bf16, 48, RW), (bf16, 48, R), (bf16, 48, R),
                                       (bf16, 2 * 2 * 10 * 4, RW), (bf16, 2 * 2 * 10 * 4, RW)], 288, 576,
     "q read and written 2*96; k 96; v 96; the 3 new rows of each cache 96 + 96 (the other 7 "
     "positions untouched).  F: 3 per rotated element of q and of k, 6*48"),
    (OP_ATTN_CACHE, (2, 3, 2, 4, 10, 5), [(bf16, 48, R), (bf16, 160, R), (bf16, 160, R), (bf16, 48, W)],
     1680, 704,
     "q 96; o 96; the 8 valid cache positions (5 cached + 3 new) of K and V 2 * 2*2*8*4*2 = 512 (not "
     "the 10 of Lmax).  F: 4 * (6+7+8 = 21 pairs) * 20"),
    (OP_ATTN_CACHE, (2, 3, 2, 4, 3, 0), [(bf16, 48, R), (bf16, 48, R), (bf16, 48, R), (bf16, 48, W),
                                         (f32, 12, W)], 480, 432,
     "no cached prefix: q 96; K, V 96 each; o 96; the row log-sum-exp 2*2*3*4 = 48.  F: 4*6*20"),
    (OP_ARGMAX, (3, 7, 1), [(f32, 21, R), (i32, 3, W), (i32, 6, RW)], 21, 108,
     "logits 84; tok 12; one row of gen written 12 (the other row untouched).  F: a compare per logit"),
    (OP_ARGMAX, (3, 7, 0), [(f32, 21, R), (i32, 3, W)], 21, 96, "logits 84; tok 12"),
    (OP_MOE_ROUTE, (3, 8, 4, 2), [(bf16, 24, R), (bf16, 32, R), (i32, 6, W), (f32, 6, W)], 192, 160,
     "h 48; router 64; expert ids 24; weights 24.  F: 2*3*8*4"),
    (OP_MOE_DISPATCH, (3, 4, 2, 0), [(i32, 6, R), (i32, 4 * 4, W), (i32, 2 * 4, RW)], 0, 96,
     "routes 24; per-expert counts and the 6 row entries 4*(4+6) = 40; one log row read and "
     "written 2*16"),
    (OP_MOE_UP, (5, 6, 4, 1, 3, 2), [(bf16, 20, R), (i32, 3 * 6, R), (bf16, 24, R), (bf16, 24, R),
                                     (bf16, 30, W)], 360, 172,
     "3 routed rows of h 3*4*2 = 24; the expert's count and 3 entries 16; Wg 48; Wu 48; 3 output "
     "rows 3*6*2 = 36.  F: 4*3*6*4 + 4*3*6"),
    (OP_MOE_DOWN, (5, 4, 6, 1, 3, 2), [(bf16, 30, R), (i32, 3 * 6, R), (f32, 10, R), (bf16, 24, R),
                                       (f32, 20, RW)], 168, 208,
     "3 rows of fe 36; count and entries 16; 3 routing weights 12; Wd 48; 3 rows of x read and "
     "written 2*3*4*4 = 96.  F: 2*3*4*6 + scale and add 2*3*4"),
    (OP_COPY, (40,), [(u8, 40, R), (u8, 40, W)], 0, 80, "40 read, 40 written"),
    (OP_TRANSPOSE, (3, 5), [(bf16, 15, R), (bf16, 15, W)], 0, 60, "15 elements read and written, 2 B"),
    (OP_SWIGLU_ACT, (3, 5), [(bf16, 15, R), (bf16, 15, R), (bf16, 15, W)], 75, 90,
     "G, U, F 3*30.  F: 5 per element"),
    (OP_SWIGLU_BWD, (3, 5), [(bf16, 15, R), (bf16, 15, R), (bf16, 15, R), (bf16, 15, W), (bf16, 15, W)],
     150, 150, "five bf16 operands 5*30.  F: 10 per element"),
    (OP_RMSNORM_BWD, (3, 8, 1), [(f32, 24, R), (bf16, 8, R), (f32, 24, R), (f32, 24, RW), (bf16, 24, W),
                                 (f32, 8, W), (f32, 3, W)], 240, 492,
     "x 96; g 16; dy 96; dx accumulated 2*96; dxb 48; dg 32; rstd 12.  F: 10 per element"),
    (OP_RMSNORM_BWD, (3, 8, 0), [(f32, 24, R), (bf16, 8, R), (f32, 24, R), (f32, 24, W), (bf16, 24, W),
                                 (f32, 8, W), (f32, 3, W)], 240, 396, "as above with dx written once 96"),
    (OP_ATTN_BWD, (2, 3, 2, 4), [(bf16, 48, R), (bf16, 48, R), (bf16, 48, R), (bf16, 48, R), (f32, 12, R),
                                 (bf16, 48, R), (bf16, 48, W), (bf16, 48, W), (bf16, 48, W), (f32, 12, W)],
     1152, 912,
     "q, K, V, o, dO read and dq, dK, dV written 8*96 = 768; lse read 48; D written and read back "
     "2*48.  F: 4 * 6 pairs * (5 products of 2d + 8)"),
    (OP_ROPE_BWD, (2, 3, 2, 4), [(f32, 48, RW), (f32, 48, R), (f32, 48, R), (f32, 48, W), (f32, 48, W)],
     288, 1152, "dq read and written 2*192; dK 192; dV 192; dk 192; dv 192.  F: 6*48"),
    (OP_XENT, (3, 7), [(f32, 21, R), (i32, 3, R), (f32, 3, W), (bf16, 21, W)], 84, 150,
     "logits 84; labels 12; losses 12; dlogits 42.  F: 4 per logit"),
    (OP_EMBED_BWD, (3, 4, 5), [(i32, 3, R), (f32, 12, R), (f32, 20, W)], 12, 140,
     "ids 12; dx 48; the whole of dE written (zeros included) 5*4*4 = 80.  F: one add per dx element"),
    (OP_ADAM, (10, 10, 100000, 900000, 950000, 10000, 100000),
     [(f32, 10, R), (f32, 10, RW), (f32, 10, RW), (f32, 10, RW), (bf16, 10, W)], 120, 300,
     "g 40; master, m, v read and written 3*80; bf16 weight 20.  F: 12 per element"),
]


@pytest.mark.parametrize("op,shape,ops,F,B,why", CASES, ids=[f"{OP_NAMES[c[0]]}{i}" for i, c in enumerate(CASES)])
def test_kernel_cost_by_hand(op, shape, ops, F, B, why):
    assert _cost(op, shape, ops) == (F, B), why


def test_every_op_has_a_hand_case():
    assert {c[0] for c in CASES} == set(OP_NAMES)


def _causal_pairs(S, pos0):
    """Query--key pairs a causal attention over a cached prefix evaluates,
    counted one by one: query i sits at position pos0 + i and sees keys
    0 .. pos0 + i."""
    return sum(1 for i in range(S) for j in range(pos0 + S) if j <= pos0 + i)


@pytest.mark.parametrize("S,pos0", [(1, 0), (1, 1100), (5, 0), (7, 9), (16, 300), (33, 1)])
def test_attention_pairs_by_enumeration(S, pos0):
    Bt, nH, d = 3, 2, 8
    n = Bt * S * nH * d
    pairs = _causal_pairs(S, pos0)
    F, _ = _cost(OP_ATTN_CACHE, (Bt, S, nH, d, pos0 + S, pos0),
                 [(bf16, n, R), (bf16, Bt * nH * (pos0 + S) * d, R), (bf16, Bt * nH * (pos0 + S) * d, R),
                  (bf16, n, W)])
    assert F == Bt * nH * pairs * (4 * d + 4)
    if pos0 == 0:
        F, _ = _cost(OP_ATTN_QKV, (Bt, S, nH, d), [(bf16, 3 * n, R), (bf16, n, W)])
        assert F == Bt * nH * pairs * (4 * d + 4)
        F, _ = _cost(OP_ATTN_BWD, (Bt, S, nH, d), [(bf16, n, R)] * 4 + [(f32, Bt * nH * S, R)] +
                     [(bf16, n, R)] + [(bf16, n, W)] * 3 + [(f32, Bt * nH * S, W)])
        assert F == Bt * nH * pairs * (10 * d + 8)


def _unit_total(w, seg):
    a, n = seg
    dt = [t.dtype for t in w.tensors]
    nb = [t.nbytes for t in w.tensors]
    F = B = 0
    for k in range(a, a + n):
        kd = w.kernels[k]
        f, b = kernel_cost(kd.op, kd.shape, kd.operands, dt, nb)
        F, B = F + f, B + b
    return F, B


def test_llama7b_decode_step_totals():
    """One decode step of the 7B shape (H 4096, FFN 11008, vocab 32000, batch
    16, 32 heads of 128) at position p.  Per layer, without attention:
    F 6,477,758,464 (two RMSNorms 2*262,144; q, k, v 1,610,612,736; RoPE
    393,216; o 536,936,448; gate/up 2,886,385,664; down 1,442,906,112) and
    B 409,141,248 (norms 2*401,408; q, k, v 101,187,584; RoPE 786,432;
    attention's q and o 262,144; o 34,209,792; gate/up 180,838,400; down
    91,054,080).  Attention adds 264,192 flops and 262,144 cache bytes per
    layer per valid position (p + 1).  Once per step: embed B 393,280; final
    norm F 262,144, B 401,408; head F 4,194,304,000, B 264,323,072; argmax
    F 512,000, B 2,048,128."""
    from workloads import configs, trace
    w = trace.build(configs.LLAMA_7B, steps=2)
    want = [(220_148_846_592, 21_958_009_024),      # p = 1024: 32*6,477,758,464 + 32*264,192*1025 + 4,195,078,144
            (220_157_300_736, 21_966_397_632)]      # p = 1025
    assert [_unit_total(w, s) for s in w.segments["decode"]] == want


def test_gpt1p3b_prefill_pass_totals():
    """One 1.3B prefill pass (24 layers, H 2048, FFN 8192, vocab 50000, 4 x
    2048 tokens, 16 heads of 128).  Per layer F 894,762,745,856: two
    LayerNorms 2*134,217,728; qkv 206,158,430,208; attention 4*16*2,098,176
    pairs*516 = 69,290,164,224; o 68,736,253,952; w1 + GELU 275,414,777,856;
    w2 274,894,684,160.  Per layer B 1,174,421,504: LayerNorms 2*100,671,488;
    qkv 159,383,552; attention 134,217,728; o 176,160,768; w1 201,326,592;
    w2 301,989,888.  Once: embed B 100,696,064; final LayerNorm on the 4 last
    rows F 65,536, B 57,344; head F 819,200,000, B 205,616,384."""
    from workloads import configs, trace
    w = trace.build(configs.GPT_1P3B)
    assert _unit_total(w, w.segments["iterations"][0]) == (21_475_125_166_080, 28_492_485_888)
