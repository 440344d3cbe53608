"""Seeded synthetic inputs and workload shapes, shared by the tests, the bench and the oracle.

This module draws random numbers and encodes them for storage; it holds none of the method's
arithmetic.  Every draw comes from numpy's counter-based Philox4x32-10 bit generator keyed by a
SeedSequence built from (workload seed, tensor name, step, microbatch, chunk), so any tensor of any
step can be regenerated on its own, on any host, without replaying earlier draws.

Distributions follow the workloads the paper trains on, as synthetic stand-ins (the paper's corpus
is not available): weight matrices N(0, 0.02) (second argument is the standard deviation), RMSNorm
gains 1, token ids uniform over the vocabulary, stage-boundary activations N(0, 1) and upstream
gradients N(0, 1e-3).
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field, replace
from typing import Dict, List, Tuple

import numpy as np

CHUNK = 1 << 22  # elements per independently keyed chunk of a long flat draw


# --------------------------------------------------------------------------------------------
# keyed generators
# --------------------------------------------------------------------------------------------
def _key_word(k) -> int:
    if isinstance(k, (int, np.integer)):
        return int(k) & 0xFFFFFFFF
    return zlib.crc32(str(k).encode())


def rng(seed: int, *keys) -> np.random.Generator:
    """Philox4x32-10 generator for the stream named by (seed, *keys)."""
    words = [_key_word(seed)] + [_key_word(k) for k in keys]
    return np.random.Generator(np.random.Philox(np.random.SeedSequence(words)))


def normal(seed: int, name: str, shape, std: float, step: int = 0, micro: int = 0) -> np.ndarray:
    """float32 draws from N(0, std^2); small tensors (one chunk)."""
    g = rng(seed, name, step, micro)
    return (g.standard_normal(size=shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


def normal_flat_chunk(seed: int, name: str, chunk: int, count: int, std: float) -> np.ndarray:
    g = rng(seed, name, 0, 0, chunk)
    return (g.standard_normal(size=count, dtype=np.float32) * np.float32(std)).astype(np.float32)


def normal_flat(seed: int, name: str, n: int, std: float) -> np.ndarray:
    """Long flat float32 N(0, std^2) vector, drawn chunk by chunk (chunk i has its own key)."""
    out = np.empty(n, dtype=np.float32)
    for c in range((n + CHUNK - 1) // CHUNK):
        lo = c * CHUNK
        hi = min(n, lo + CHUNK)
        out[lo:hi] = normal_flat_chunk(seed, name, c, hi - lo, std)
    return out


def normal_flat_slice(seed: int, name: str, n: int, start: int, count: int, std: float) -> np.ndarray:
    """Elements [start, start+count) of normal_flat(seed, name, n, std), regenerated alone."""
    assert 0 <= start and start + count <= n
    parts = []
    c0, c1 = start // CHUNK, (start + count - 1) // CHUNK
    for c in range(c0, c1 + 1):
        lo = c * CHUNK
        hi = min(n, lo + CHUNK)
        chunk = normal_flat_chunk(seed, name, c, hi - lo, std)
        a = max(start, lo) - lo
        b = min(start + count, hi) - lo
        parts.append(chunk[a:b])
    return np.concatenate(parts)


def uniform_tokens(seed: int, name: str, shape, vocab: int, step: int = 0, micro: int = 0) -> np.ndarray:
    """int32 token ids uniform over [0, vocab)."""
    g = rng(seed, name, step, micro)
    return g.integers(0, vocab, size=shape, dtype=np.int64).astype(np.int32)


# --------------------------------------------------------------------------------------------
# bf16 storage encoding (round to nearest even), used to hand bf16 inputs to both sides
# --------------------------------------------------------------------------------------------
def bf16_bits(a: np.ndarray) -> np.ndarray:
    """uint16 bf16 encodings of float32 values, round-to-nearest-even; NaN stays NaN (quiet)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r = ((u + (np.uint32(0x7FFF) + ((u >> 16) & 1))) >> 16).astype(np.uint16)
    r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_values(a: np.ndarray) -> np.ndarray:
    """float32 values exactly representable in bf16 (the RNE image of a)."""
    return bf16_to_f32(bf16_bits(a))


# --------------------------------------------------------------------------------------------
# workload shapes
# --------------------------------------------------------------------------------------------
@dataclass(frozen=True)
class Workload:
    name: str
    n_blocks: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int            # 0: no embedding and no head on this stage
    first_stage: bool
    last_stage: bool
    tie_embedding: bool
    seq_len: int
    micro_batch: int
    microbatches_per_step: int
    dtype: str            # "f32" or "bf16" (bf16 compute, fp32 master weights)
    steps: int
    seed: int
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1
    clip_norm: float = 1.0
    ef_lambda: float = 1.0
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    max_inflight: int = 1

    @property
    def tokens_per_micro(self) -> int:
        return self.seq_len * self.micro_batch

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = Workload("tiny-fp32: 2 blocks d128 h4 ffn512 vocab512 tied seq64 mb2", 2, 128, 4, 4, 32, 512,
                512, True, True, True, 64, 2, 1, "f32", 20, 1)
SMALL = Workload("small-bf16: 3 blocks d768 h12 ffn3072 seq1024 mb8 vocab32000 first stage",
                 3, 768, 12, 12, 64, 3072, 32000, True, False, False, 1024, 8, 1, "bf16", 100, 2)
MID = Workload("mid-bf16: 4 blocks d2048 h16 hd128 ffn8192 seq2048 mb4 middle stage",
               4, 2048, 16, 16, 128, 8192, 0, False, False, False, 2048, 4, 1, "bf16", 100, 3)
LARGE = Workload("large-bf16: 4 blocks d4096 h32/kv8 hd128 ffn14336 seq4096 mb2 1F1B x8",
                 4, 4096, 32, 8, 128, 14336, 0, False, False, False, 4096, 2, 8, "bf16", 100, 4,
                 max_inflight=4)
UPDATE_N = 1_000_000_000
UPDATE_SEED = 5
UPDATE_STEPS = 50

LAST = Workload("last-bf16: 3 blocks d768 h12 ffn3072 seq1024 mb8 vocab49152 last stage, untied head",
                3, 768, 12, 12, 64, 3072, 49152, False, True, False, 1024, 8, 1, "bf16", 100, 6)

WORKLOADS = {"tiny": TINY, "small": SMALL, "mid": MID, "large": LARGE, "last": LAST}


# --------------------------------------------------------------------------------------------
# logical parameter list and initial values
# --------------------------------------------------------------------------------------------
def param_specs(w: Workload) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, init) for every parameter of the stage, in a fixed order.

    init is "normal" (N(0, 0.02)) or "ones" (RMSNorm gains)."""
    d, hd, f = w.d_model, w.head_dim, w.d_ffn
    out: List[Tuple[str, Tuple[int, ...], str]] = []
    if w.vocab > 0 and w.first_stage:
        out.append(("embed", (w.vocab, d), "normal"))
    for i in range(w.n_blocks):
        p = f"blk{i}."
        out += [
            (p + "attn_norm", (d,), "ones"),
            (p + "wq", (w.n_heads * hd, d), "normal"),
            (p + "wk", (w.n_kv_heads * hd, d), "normal"),
            (p + "wv", (w.n_kv_heads * hd, d), "normal"),
            (p + "wo", (d, w.n_heads * hd), "normal"),
            (p + "ffn_norm", (d,), "ones"),
            (p + "wgate", (f, d), "normal"),
            (p + "wup", (f, d), "normal"),
            (p + "wdown", (d, f), "normal"),
        ]
    if w.last_stage:
        out.append(("final_norm", (d,), "ones"))
        if not w.tie_embedding:
            out.append(("head", (w.vocab, d), "normal"))
    return out


def init_params(w: Workload) -> Dict[str, np.ndarray]:
    """float32 initial master weights: matrices N(0, 0.02), gains 1."""
    out = {}
    for name, shape, init in param_specs(w):
        if init == "ones":
            out[name] = np.ones(shape, dtype=np.float32)
        else:
            out[name] = normal(w.seed, "param:" + name, shape, 0.02)
    return out


def step_inputs(w: Workload, step: int, micro: int = 0) -> Dict[str, np.ndarray]:
    """Inputs of one microbatch of one step, as float32 values / int32 ids.

    First stage: tokens [B, s] (and, on a last stage, next-token targets [B, s], drawn as s+1
    tokens per row).  Other stages: x_in [B, s, d] ~ N(0, 1); a last stage among them gets
    targets [B, s] uniform over the vocabulary.  Any stage without a head: dy [B, s, d] ~
    N(0, 1e-3).  bf16 workloads get bf16-representable values."""
    B, s, d = w.micro_batch, w.seq_len, w.d_model
    out: Dict[str, np.ndarray] = {}
    if w.first_stage:
        toks = uniform_tokens(w.seed, "tokens", (B, s + 1), w.vocab, step, micro)
        out["tokens"] = np.ascontiguousarray(toks[:, :s])
        if w.last_stage:
            out["targets"] = np.ascontiguousarray(toks[:, 1:])
    else:
        x = normal(w.seed, "x_in", (B, s, d), 1.0, step, micro)
        out["x_in"] = bf16_values(x) if w.dtype == "bf16" else x
        if w.last_stage:
            out["targets"] = uniform_tokens(w.seed, "targets", (B, s), w.vocab, step, micro)
    if not w.last_stage:
        dy = normal(w.seed, "dy", (B, s, d), 1e-3, step, micro)
        out["dy"] = bf16_values(dy) if w.dtype == "bf16" else dy
    return out
