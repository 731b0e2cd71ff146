"""Helpers for the GPU tests: sessions built from the seeded inputs, and
comparison helpers (no method arithmetic here)."""
import numpy as np

import synth


def device_params(weights):
    return {k: weights.device_array(k) for k in weights.values}


def make_session(shape, weights, max_batch, max_pos, max_prompt=0, num_pages=None):
    from paper_2608_12385_amd import Session
    return Session(shape, device_params(weights), max_batch=max_batch, max_pos=max_pos,
                   max_prompt=max_prompt, num_pages=num_pages)


def fill_cache(sess, orc, shape, lengths, seed=3):
    """Same seeded K/V into the GPU pages and the oracle cache."""
    for b, L in enumerate(lengths):
        ks, vs, kd, vd = [], [], [], []
        for l in range(shape.n_layers):
            (kv_, kb), (vv_, vb) = synth.make_kv(shape, l, b, int(L), seed=seed)
            ks.append(kv_)
            vs.append(vv_)
            kd.append(kb if kb is not None else kv_)
            vd.append(vb if vb is not None else vv_)
        if orc is not None:
            orc.kv_fill(b, int(L), ks, vs)
        if sess is not None and L > 0:
            sess.reserve_fill(b, kd, vd)


def row_err(g, o):
    """Per-row max |g - o| / max |o| (rows = leading index)."""
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    num = np.max(np.abs(g - o).reshape(g.shape[0], -1), axis=1)
    den = np.max(np.abs(o).reshape(o.shape[0], -1), axis=1)
    return num / np.where(den > 0, den, 1.0)


def near_tie_ok(m_oracle, tok, tol):
    """GPU token acceptable: its oracle mixture value is within tol of the max."""
    return m_oracle[tok] >= np.max(m_oracle) - tol
