"""Seeded synthetic contents: random-init weights and uniform random token ids.

Tensor i of a workload with init "normal" draws
``default_rng([seed, i]).standard_normal(shape, float32) * 0.02``; bf16
configurations keep the round-to-nearest-even bf16 value of that draw, so every
consumer sees identical parameters.  Norm gains are 1 and biases 0.  Token ids
of sequence b are ``default_rng([seed, 1_000_000 + b]).integers(0, vocab, S)``.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .format import DT_BF16, DT_F32, DT_I32, KIND_PARAM
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


# AdamW hyperparameters of the training step (a mid-run step: the moments are
# seeded non-zero and the bias corrections are those of step 10)
TRAIN_HP = dict(step=10, lr=1e-4, b1=0.9, b2=0.95, eps=1e-8, wd=0.1)


def next_token_labels(ids: np.ndarray) -> np.ndarray:
    """Targets of a training batch: the next token of each sequence, the
    last position wrapping to the first."""
    return np.roll(np.asarray(ids), -1, axis=-1).astype(np.int32)


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
    if t.init == "labels":
        return next_token_labels(token_ids(c.seed, c.batch, c.prompt_len, c.vocab)).reshape(t.shape)
    if t.init == "master":       # the fp32 draw the bf16 weight was rounded from
        src = w.tensors[w.id(t.name[: -len(".master")])]
        if src.init == "normal":
            return normal_f32(c.seed, src.tid, t.shape)
        return tensor_value(w, src)
    if t.init == "adam_m":       # seeded first moment of a step in mid-run
        return normal_f32(c.seed + 101, t.tid, t.shape) * np.float32(1e-4 / 0.02)
    if t.init == "adam_v":       # seeded second moment, bounded away from zero as in mid-run:
        # (1e-4 (0.5 + |N(0,1)|))^2, so the update m / sqrt(v) stays well conditioned
        z = np.abs(normal_f32(c.seed + 202, t.tid, t.shape) * np.float32(50.0))
        return np.square(np.float32(1e-4) * (np.float32(0.5) + z))
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


def param_names(w: Workload) -> list:
    """Names of a training workload's model parameters (the bf16 weights)."""
    return [t.name for t in w.tensors if t.kind == KIND_PARAM and t.init in ("normal", "ones")]


def master_f64(w: Workload) -> dict:
    """fp32 master weights widened to fp64, by parameter name."""
    return {n: tensor_value(w, w.tensors[w.id(n + ".master")]).astype(np.float64) for n in param_names(w)}


def adam_state_f64(w: Workload) -> dict:
    """Adam moments (m, v) widened to fp64, by parameter name."""
    return {n: (tensor_value(w, w.tensors[w.id(n + ".m")]).astype(np.float64),
                tensor_value(w, w.tensors[w.id(n + ".v")]).astype(np.float64)) for n in param_names(w)}


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
