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


def softmax64(z):
    z = np.asarray(z, np.float64)
    e = np.exp(z - z.max())
    return e / e.sum()


def alpha_bound(alpha, eps1):
    """How far sum p^2 (clipped) can move when every primary logit moves by at
    most eps1: each p_v by a factor within e^(+-2 eps1), sum p^2 by one within
    e^(+-4 eps1)."""
    return alpha * (np.exp(4 * eps1) - 1)


def tie_margin(o, eps, eps1):
    """Certified near-tie margin of the mixture (Eqs. (17)-(18)) from the
    measured logit errors: with every logit within eps of the oracle's
    (eps1 for the primary), m_v = alpha p_v + (1 - alpha) q_v moves by at
    most max(m) (e^(2 eps) - 1) + |d alpha| per entry, so a token the GPU
    prefers can trail the oracle's maximum by at most twice that (plus
    float32 rounding of the GPU's own mixture)."""
    mm = float(np.max(o["m"]))
    return 2 * (mm * (np.exp(2 * eps) - 1) + alpha_bound(o["alpha"], eps1)) + 1e-6 * mm


def check_readout(t, outs, tol, tag, branch=True, alpha_own_tol=None):
    """Logits (per-row relative error), alpha, and greedy tokens of a step
    against the oracle.

    alpha: against the oracle within the bound the measured primary-logit
    error allows (alpha_bound), and, when alpha_own_tol is given, against
    sum p^2 (clipped) of the GPU's own logits in float64 at that relative
    tolerance.  Tokens: equal to the oracle's, or a certified near-tie
    (tie_margin from the measured logit errors)."""
    z1g = to_np(t["logits1"])
    z1 = np.stack([o["z1"] for o in outs])
    assert row_err(z1g, z1).max() <= tol, (tag, row_err(z1g, z1))
    zbs = []
    if branch:
        z2 = np.stack([o["z2"] for o in outs])
        g2 = to_np(t["logits2"])
        if g2.ndim == 3:          # several branches: [n_branches][batch][vocab]
            for j in range(g2.shape[0]):
                zj = np.stack([(o["zb"][j] if "zb" in o else o["z2"]) for o in outs])
                assert row_err(g2[j], zj).max() <= tol, (tag, j, row_err(g2[j], zj))
                zbs.append((g2[j], zj))
        else:
            assert row_err(g2, z2).max() <= tol, (tag, row_err(g2, z2))
            zbs.append((g2, z2))
    ag = to_np(t["alpha"]).astype(np.float64)
    nt = to_np(t["next_token"])
    for i, o in enumerate(outs):
        eps1 = float(np.max(np.abs(z1g[i].astype(np.float64) - o["z1"])))
        eps = max([eps1] + [float(np.max(np.abs(g[i].astype(np.float64) - z[i]))) for g, z in zbs])
        assert abs(ag[i] - o["alpha"]) <= alpha_bound(o["alpha"], eps1) + 1e-6, (tag, i, ag[i], o["alpha"], eps1)
        if alpha_own_tol is not None:
            own = 1.0 if o.get("z2") is None else np.clip(np.sum(softmax64(z1g[i]) ** 2), 0.5, 1.0)
            assert abs(ag[i] - own) <= alpha_own_tol * own, (tag, i, ag[i], own)
        tok = int(nt[i])
        if tok != o["next"]:
            assert near_tie_ok(o["m"], tok, tie_margin(o, eps, eps1)), (tag, i, tok, o["next"], eps)
