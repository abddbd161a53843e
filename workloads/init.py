"""Seeded synthetic contents: random-init weights and uniform random token ids.

Tensor i of a workload with init "normal" draws
``default_rng([seed, i]).standard_normal(shape, float32) * 0.02``; bf16
configurations keep the round-to-nearest-even bf16 value of that draw, so every
consumer sees identical parameters.  Norm gains are 1 and biases 0.  Token ids
of sequence b are ``default_rng([seed, 1_000_000 + b]).integers(0, vocab, S)``.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .format import DT_BF16, DT_F32, DT_I32
from .trace import TensorSpec, Workload


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16), round to nearest even (no NaNs here)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_f32(seed: int, tid: int, shape) -> np.ndarray:
    g = np.random.default_rng([seed, tid])
    return g.standard_normal(shape, dtype=np.float32) * np.float32(0.02)


def token_ids(seed: int, batch: int, seq: int, vocab: int) -> np.ndarray:
    out = np.empty((batch, seq), dtype=np.int32)
    for b in range(batch):
        out[b] = np.random.default_rng([seed, 1_000_000 + b]).integers(0, vocab, seq)
    return out


def tensor_value(w: Workload, t: TensorSpec) -> np.ndarray:
    """Initial value of a host-initialised tensor as fp32 (int32 for ids).

    For bf16 tensors this is the exact bf16 value widened to fp32.
    """
    c = w.cfg
    if t.init == "normal":
        v = normal_f32(c.seed, t.tid, t.shape)
        if t.dtype == DT_BF16:
            v = bf16_to_f32(bf16_bits(v)).reshape(t.shape)
        return v
    if t.init == "ones":
        return np.ones(t.shape, np.float32)
    if t.init == "zeros":
        return np.zeros(t.shape, np.float32 if t.dtype != DT_I32 else np.int32)
    if t.init == "ids":
        return token_ids(c.seed, c.batch, c.prompt_len, c.vocab).reshape(t.shape)
    raise ValueError(f"tensor {t.name} has no initial value")


def tensor_bytes(w: Workload, t: TensorSpec) -> np.ndarray:
    """Initial value of a host-initialised tensor in its storage encoding (uint8)."""
    c = w.cfg
    if t.init == "normal" and t.dtype == DT_BF16:
        return bf16_bits(normal_f32(c.seed, t.tid, t.shape)).view(np.uint8).reshape(-1)
    v = tensor_value(w, t)
    if t.dtype == DT_BF16:
        return bf16_bits(v).view(np.uint8).reshape(-1)
    if t.dtype == DT_F32:
        return np.ascontiguousarray(v, np.float32).view(np.uint8).reshape(-1)
    if t.dtype == DT_I32:
        return np.ascontiguousarray(v, np.int32).view(np.uint8).reshape(-1)
    raise ValueError(t.dtype)


def fill_host(w: Workload, view_of, threads: int = 16, chunk_rows: int = 0) -> None:
    """Write every host-initialised tensor through ``view_of(tensor) -> uint8 array``.

    Tensors are generated in parallel (numpy's generators release the GIL).
    """
    todo = [t for t in w.tensors if t.host_init]

    def one(t):
        dst = view_of(t)
        dst[: t.nbytes] = tensor_bytes(w, t)

    # largest first so the pool stays busy
    todo.sort(key=lambda t: -t.nbytes)
    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(one, todo))


def weights_f64(w: Workload, names=None) -> dict:
    """Named initial values widened to fp64 (for the oracle)."""
    out = {}
    for t in w.tensors:
        if not t.host_init or t.init == "ids":
            continue
        if names is not None and t.name not in names:
            continue
        out[t.name] = tensor_value(w, t).astype(np.float64)
    return out
