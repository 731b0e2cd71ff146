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


def to_np(t):
    return t if isinstance(t, np.ndarray) else t.detach().cpu().numpy()


def check_readout(t, outs, tol, tag, branch=True):
    """Logits (per-row relative error), alpha, and greedy tokens (equal, or a
    certified near-tie of the oracle's mixture) of a step against the oracle."""
    z1 = np.stack([o["z1"] for o in outs])
    assert row_err(to_np(t["logits1"]), z1).max() <= tol, (tag, row_err(to_np(t["logits1"]), z1))
    if branch:
        z2 = np.stack([o["z2"] for o in outs])
        assert row_err(to_np(t["logits2"]), z2).max() <= tol, (tag, row_err(to_np(t["logits2"]), z2))
    alpha = np.array([o["alpha"] for o in outs])
    np.testing.assert_allclose(to_np(t["alpha"]), alpha, rtol=max(tol, 1e-6), atol=1e-7, err_msg=tag)
    for i, o in enumerate(outs):
        tok = int(to_np(t["next_token"])[i])
        if tok != o["next"]:
            assert near_tie_ok(o["m"], tok, 10 * tol * np.max(o["m"])), (tag, i, tok, o["next"])

