"""Tiny model shapes shared by the oracle pins and the GPU parity tests."""
import dataclasses

import numpy as np

import synth


def tiny_shape(**kw):
    base = dict(n_layers=2, d_model=48, n_q_heads=4, n_kv_heads=2, head_dim=16,
                d_ff=96, vocab=64, dtype="f32", has_embeddings=True, coupling_std=0.5,
                std=0.2)
    base.update(kw)
    return synth.ModelShape(**base)


def tiny_moe_shape(**kw):
    base = dict(n_layers=1, d_model=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                d_ff=0, vocab=0, dtype="f32", has_embeddings=False, coupling_std=0.5,
                std=0.2, n_experts=8, d_ff_expert=32, n_shared_experts=1, d_ff_shared=32,
                top_k1=2, top_k2=3)
    base.update(kw)
    return synth.ModelShape(**base)


def params(shape, seed=0, **kw):
    return synth.make_weights(shape, seed=seed, **kw).values


def with_shape(shape, **kw):
    return dataclasses.replace(shape, **kw)


def rel_err(g, o):
    """max |g - o| / max |o| over the compared tensor."""
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    den = np.max(np.abs(o))
    return float(np.max(np.abs(g - o)) / (den if den > 0 else 1.0))
