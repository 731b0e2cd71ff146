"""Seeded synthetic inputs for the Decode-Branch decode path.

This module is the only code shared by the GPU-side harness and the CPU
oracle.  It draws random numbers and lays them out; it holds none of the
method's arithmetic (no norms, no projections, no attention, no readout).

Every tensor comes from ``numpy.random.default_rng(SeedSequence([seed,
tensor_id]))`` so that any single tensor can be regenerated on its own.
Matrices and embeddings are N(0, std) drawn in float32; for bfloat16
workloads they are then rounded to bfloat16 (round to nearest, ties to
even) and both sides receive exactly those values: the device gets the
16-bit patterns, the oracle gets the same values widened to float64.

Tensor ids (fixed, documented order):
    0 E1 (primary embedding)   1 E2 (branch embedding)   2 W_out (LM head)
    10 + j: E_j, the embedding of decode branch j - 1 for j >= 3 (more branches)
    per layer l, base = 1000 + 100*l:
    +0 W_Q  +1 W_K  +2 W_V  +3 W_O  +4 W_gate  +5 W_up  +6 W_down
    +7 a    +8 b    +9 c    +10 W_router
    +11 expert W_gate  +12 expert W_up  +13 expert W_down
    +14 shared W_gate  +15 shared W_up  +16 shared W_down
    +20 g_A  +21 g_G   (gates of the compute-matched variant)
Norm gains are ones.  Data tensors use other seeds (see the helpers).
"""
from __future__ import annotations

import dataclasses
import numpy as np

__all__ = [
    "ModelShape", "WORKLOADS", "workload", "bf16_bits", "bf16_values",
    "normal", "make_weights", "make_tokens", "make_hidden", "make_kv",
    "make_lengths", "Weights",
]


# --------------------------------------------------------------------------
# bfloat16 storage helpers (data-type conversion of generated inputs only)
# --------------------------------------------------------------------------

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> uint16 bfloat16 bit patterns, round to nearest even.

    Finite inputs only (generated data is finite)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = u >> np.uint32(16)          # in place from here: (u + 0x7FFF + lsb) >> 16
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_values(bits: np.ndarray) -> np.ndarray:
    """uint16 bfloat16 bit patterns -> float32 values (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(seed), int(tensor_id)]))


def normal(seed: int, tensor_id: int, shape, std: float = 1.0) -> np.ndarray:
    """float32 N(0, std^2) array for (seed, tensor_id)."""
    x = _rng(seed, tensor_id).standard_normal(size=tuple(shape), dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


# --------------------------------------------------------------------------
# Workload shapes
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int                   # dense SwiGLU width (0 for MoE layers)
    vocab: int                  # 0: no LM head
    dtype: str                  # "f32" or "bf16" (weights and KV cache)
    has_embeddings: bool        # token inputs (else hidden-state inputs)
    n_experts: int = 0
    d_ff_expert: int = 0
    n_shared_experts: int = 0
    d_ff_shared: int = 0
    top_k1: int = 0
    top_k2: int = 0
    replay: bool = False        # router replay (branch reuses primary indices)
    compute_matched: bool = False  # App. B.3 variant (gated copies)
    n_branches: int = 1         # decode branches (App. C.1 allows more)
    std: float = 0.02           # weight std
    coupling_std: float = 0.02  # std of a, b, c
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    page_size: int = 16

    @property
    def d_q(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def d_kv(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def is_moe(self) -> bool:
        return self.n_experts > 0


# The five workloads and one tensor-parallel shard: shapes and run recipes
# (one GPU each).
WORKLOADS = {
    "tiny_f32": dict(
        shape=ModelShape(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=4, head_dim=64,
                         d_ff=683, vocab=1024, dtype="f32", has_embeddings=True),
        batch=1, prompt_len=128, steps=16),
    "layer8b_bf16": dict(
        shape=ModelShape(n_layers=1, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                         d_ff=14336, vocab=128256, dtype="bf16", has_embeddings=False),
        batch=32, cache_len=4096, steps=1),
    "longctx_bf16": dict(
        shape=ModelShape(n_layers=1, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                         d_ff=14336, vocab=0, dtype="bf16", has_embeddings=False),
        batch=8, len_lo=16384, len_hi=32768, steps=64),
    "moe_bf16": dict(
        shape=ModelShape(n_layers=1, d_model=2048, n_q_heads=16, n_kv_heads=4, head_dim=128,
                         d_ff=0, vocab=0, dtype="bf16", has_embeddings=False,
                         n_experts=64, d_ff_expert=1408, n_shared_experts=1, d_ff_shared=1408,
                         top_k1=2, top_k2=4),
        batch=64, cache_len=8192, steps=1),
    # one GPU's share of the 8B-shape layer under eight-way tensor parallelism
    # (one KV-head group: 4 query heads and 1 KV head, d_ff / 8, the vocabulary
    # split eight ways and rounded up to a multiple of 64); run as one GPU's
    # step, without the exchanges between the shards
    "tp8shard_bf16": dict(
        shape=ModelShape(n_layers=1, d_model=4096, n_q_heads=4, n_kv_heads=1, head_dim=128,
                         d_ff=1792, vocab=16064, dtype="bf16", has_embeddings=False),
        batch=32, cache_len=4096, steps=1),
    "full24_bf16": dict(
        shape=ModelShape(n_layers=24, d_model=2048, n_q_heads=16, n_kv_heads=4, head_dim=128,
                         d_ff=5632, vocab=32000, dtype="bf16", has_embeddings=True),
        batch=64, prompt_len=8192, steps=256),
}


def workload(name: str, **shape_overrides):
    """Copy of a workload recipe, optionally with shape fields replaced."""
    w = dict(WORKLOADS[name])
    if shape_overrides:
        w["shape"] = dataclasses.replace(w["shape"], **shape_overrides)
    return w


# --------------------------------------------------------------------------
# Weights
# --------------------------------------------------------------------------

class Weights:
    """Generated parameters.

    ``values[name]`` is a float32 array holding the exact parameter values
    (already bf16-representable for bf16 shapes).  ``bits[name]`` holds the
    uint16 patterns for bf16 matrices.  Layer tensors are named
    ``"L{l}.{name}"``; vectors a, b, c, gains and gates are always float32.
    """

    def __init__(self, shape: ModelShape):
        self.shape = shape
        self.values: dict[str, np.ndarray] = {}
        self.bits: dict[str, np.ndarray] = {}

    def _matrix(self, name, seed, tid, shp, std):
        x = normal(seed, tid, shp, std)
        if self.shape.dtype == "bf16":
            b = bf16_bits(x)
            self.bits[name] = b
            self.values[name] = bf16_values(b)
        else:
            self.values[name] = x

    def _vector(self, name, seed, tid, n, std):
        self.values[name] = normal(seed, tid, (n,), std)

    def _ones(self, name, n):
        self.values[name] = np.ones((n,), dtype=np.float32)

    def __getitem__(self, name):
        return self.values[name]

    def device_array(self, name):
        """Array in the on-device storage type (uint16 bits for bf16 matrices)."""
        return self.bits.get(name, self.values[name])


def make_weights(shape: ModelShape, seed: int = 0, coupling_std=None, skip_lm_head=False) -> Weights:
    s = shape
    w = Weights(s)
    cstd = s.coupling_std if coupling_std is None else coupling_std
    if s.has_embeddings:
        w._matrix("E1", seed, 0, (s.vocab, s.d_model), s.std)
        w._matrix("E2", seed, 1, (s.vocab, s.d_model), s.std)
        for j in range(3, s.n_branches + 2):
            w._matrix(f"E{j}", seed, 10 + j, (s.vocab, s.d_model), s.std)
        w._ones("g_emb", s.d_model)
    if s.vocab > 0:
        if not skip_lm_head:
            w._matrix("W_out", seed, 2, (s.vocab, s.d_model), s.std)
        w._ones("g_final", s.d_model)
    for l in range(s.n_layers):
        base = 1000 + 100 * l
        p = f"L{l}."
        w._ones(p + "g_attn", s.d_model)
        w._ones(p + "g_mlp", s.d_model)
        w._matrix(p + "W_Q", seed, base + 0, (s.d_q, s.d_model), s.std)
        w._matrix(p + "W_K", seed, base + 1, (s.d_kv, s.d_model), s.std)
        w._matrix(p + "W_V", seed, base + 2, (s.d_kv, s.d_model), s.std)
        w._matrix(p + "W_O", seed, base + 3, (s.d_model, s.d_q), s.std)
        w._vector(p + "a", seed, base + 7, s.d_q, cstd)
        w._vector(p + "c", seed, base + 9, s.d_model, cstd)
        if not s.is_moe:
            w._matrix(p + "W_gate", seed, base + 4, (s.d_ff, s.d_model), s.std)
            w._matrix(p + "W_up", seed, base + 5, (s.d_ff, s.d_model), s.std)
            w._matrix(p + "W_down", seed, base + 6, (s.d_model, s.d_ff), s.std)
            w._vector(p + "b", seed, base + 8, s.d_ff, cstd)
        else:
            E, fe = s.n_experts, s.d_ff_expert
            w._matrix(p + "W_router", seed, base + 10, (E, s.d_model), s.std)
            w._matrix(p + "X_gate", seed, base + 11, (E, fe, s.d_model), s.std)
            w._matrix(p + "X_up", seed, base + 12, (E, fe, s.d_model), s.std)
            w._matrix(p + "X_down", seed, base + 13, (E, s.d_model, fe), s.std)
            if s.n_shared_experts > 0:
                fs = s.d_ff_shared * s.n_shared_experts
                w._matrix(p + "S_gate", seed, base + 14, (fs, s.d_model), s.std)
                w._matrix(p + "S_up", seed, base + 15, (fs, s.d_model), s.std)
                w._matrix(p + "S_down", seed, base + 16, (s.d_model, fs), s.std)
                w._vector(p + "b", seed, base + 8, fs, cstd)
            if s.compute_matched:
                w._ones(p + "g_A", s.d_model)
                w._ones(p + "g_G", s.d_model)
    return w


# --------------------------------------------------------------------------
# Data
# --------------------------------------------------------------------------

def make_tokens(seed: int, tensor_id: int, shape, vocab: int) -> np.ndarray:
    """int32 tokens uniform in [0, vocab)."""
    return _rng(seed, tensor_id).integers(0, vocab, size=tuple(shape), dtype=np.int64).astype(np.int32)


def make_hidden(shape: ModelShape, batch: int, step: int = 0, seed: int = 2, paths: int = 2):
    """Residual-stream inputs for layer-only workloads: float32 N(0,1) [paths][batch][d]."""
    return normal(seed, 10 * step, (paths, batch, shape.d_model), 1.0)


def make_lengths(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    """int32 per-sequence cache lengths uniform in [lo, hi]."""
    return _rng(seed, 7).integers(lo, hi + 1, size=(batch,), dtype=np.int64).astype(np.int32)


def make_kv(shape: ModelShape, layer: int, seq: int, length: int, seed: int = 3):
    """Pre-filled cache contents for one (layer, sequence): N(0,1) K and V,
    each [length][n_kv][head_dim], returned as (values_f32, bits_or_None) pairs."""
    tid = 100000 * (layer + 1) + 2 * seq
    out = []
    for j in range(2):
        x = normal(seed, tid + j, (length, shape.n_kv_heads, shape.head_dim), 1.0)
        if shape.dtype == "bf16":
            b = bf16_bits(x)
            out.append((bf16_values(b), b))
        else:
            out.append((x, None))
    return out[0], out[1]
