"""Synthetic decoder configurations (random-init stand-ins for the paper's LLMs).

The paper evaluates ten Hugging Face decoders of 12-32 layers, sequence length
1.9k-4.0k and 1.4-11.4 GB footprint (Sec. V, Table II).  Those checkpoints are
not used; seeded random-init decoders of the shapes below stand in for them.
The oversubscription factor is allocated bytes over device capacity
(Sec. II-A); a config's device budget is footprint * den / num.
"""
from dataclasses import dataclass, replace
from typing import Tuple

from .format import DT_F32, DT_BF16


@dataclass(frozen=True)
class DecoderConfig:
    name: str
    style: str              # "gpt": LayerNorm + GELU FFN + fused qkv, tied head
                            # "llama": RMSNorm + SwiGLU + RoPE + KV cache, untied head
                            # "moe": llama attention, then top-k of n_experts SwiGLU experts
                            # "train": llama, one training step (forward, backward, AdamW)
    n_layers: int
    hidden: int
    n_heads: int
    ffn: int
    vocab: int
    dtype: int              # storage type of weights and activations (DT_F32 / DT_BF16)
    batch: int
    prompt_len: int
    decode_steps: int = 0   # greedy steps after the prompt (llama style only)
    factor: Tuple[int, int] = (3, 2)   # oversubscription factor num/den
    logits_all: bool = False           # gpt style: logits at every position (else last only)
    seed: int = 0
    iterations: int = 1                # gpt style: forward passes over the same ids
    n_experts: int = 0                 # moe style: experts per layer (ffn is each expert's width)
    top_k: int = 0                     # moe style: experts routed per token
    fuse_qkv: bool = True              # llama/moe style: q, k, v projections as one LINEAR_QKV kernel

    @property
    def head_dim(self) -> int:
        return self.hidden // self.n_heads

    @property
    def tokens(self) -> int:
        return self.batch * self.prompt_len

    @property
    def kv_len(self) -> int:
        return self.prompt_len + self.decode_steps

    def with_factor(self, num: int, den: int) -> "DecoderConfig":
        return replace(self, factor=(num, den))


# Tiny parity decoder: 2 layers, hidden 128, 4 heads of 32, GELU FFN 512,
# LayerNorm, vocab 1000, fp32; prefill 1 x 32; budget 50% of the footprint.
TINY = DecoderConfig("tiny", "gpt", 2, 128, 4, 512, 1000, DT_F32, 1, 32,
                     factor=(2, 1), logits_all=True)

# 1.3B-shape GPT-style decoder, prefill 4 x 2048, bf16, 1.25x oversubscription.
GPT_1P3B = DecoderConfig("gpt-1.3b", "gpt", 24, 2048, 16, 8192, 50000, DT_BF16,
                         4, 2048, factor=(5, 4))

# 7B-shape LLaMA-style decoder: 1024-token prompt then 256 greedy steps at batch
# 16 with a growing KV cache, bf16, 1.5x oversubscription.
LLAMA_7B = DecoderConfig("llama-7b", "llama", 32, 4096, 32, 11008, 32000, DT_BF16,
                         16, 1024, decode_steps=256, factor=(3, 2))

# Small variants used by parity tests (same structure, seconds on the CPU).
LLAMA_SMALL = DecoderConfig("llama-small", "llama", 2, 256, 2, 512, 1000, DT_BF16,
                            2, 40, decode_steps=6, factor=(3, 2))
GPT_SMALL = DecoderConfig("gpt-small", "gpt", 2, 256, 2, 640, 1000, DT_BF16,
                          2, 160, factor=(5, 4))

# MoE decoder: 32 layers, hidden 4096, 32 heads, 8 SwiGLU experts of width
# 14336 per layer with top-2 routing from a seeded random router, bf16; prefill
# 8 x 4096 tokens then 128 greedy steps; budget = footprint / 2.
MOE_8X = DecoderConfig("moe-8x14336", "moe", 32, 4096, 32, 14336, 32000, DT_BF16,
                       8, 4096, decode_steps=128, factor=(2, 1), n_experts=8, top_k=2)

# Small MoE for parity tests (4 experts, top-2).
MOE_SMALL = DecoderConfig("moe-small", "moe", 2, 256, 2, 384, 1000, DT_BF16,
                          2, 40, decode_steps=6, factor=(2, 1), n_experts=4, top_k=2)

# 13B-shape LLaMA-style training step: 40 layers, hidden 5120, 40 heads,
# SwiGLU 13824, RMSNorm, vocab 32k; batch 8 x 2048 random tokens (next-token
# targets); bf16 weights with fp32 master weights and Adam moments; forward
# and backward with all activations kept; budget = footprint / 2.
LLAMA_13B_TRAIN = DecoderConfig("llama-13b-train", "train", 40, 5120, 40, 13824, 32000, DT_BF16,
                                8, 2048, factor=(2, 1))

# Small training step for parity tests (head dim 128).
TRAIN_SMALL = DecoderConfig("train-small", "train", 2, 256, 2, 384, 1024, DT_BF16,
                            2, 80, factor=(2, 1))

CONFIGS = {c.name: c for c in (TINY, GPT_1P3B, LLAMA_7B, LLAMA_SMALL, GPT_SMALL, MOE_8X, MOE_SMALL,
                               LLAMA_13B_TRAIN, TRAIN_SMALL)}
