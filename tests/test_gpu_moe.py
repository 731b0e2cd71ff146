"""GPU parity of the MoE decode layer (Sec. 3.2, Sec. 4.3 router replay,
Sec. 5 independent fan-outs k1/k2) against the CPU oracle.

Routing indices must match the oracle exactly, except where the oracle's
own k-th and (k+1)-th router logits are closer than the stated margin
(then either choice is correct and the rest is checked for validity)."""
import numpy as np
import pytest

import synth
from oracle import Oracle
from tests.gpu_util import check_readout, fill_cache, make_session, row_err

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


def _np(t):
    return t.detach().cpu().numpy()


def _moe_shape(**kw):
    base = dict(n_layers=1, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=0, vocab=512,
                dtype="bf16", has_embeddings=False, n_experts=16, d_ff_expert=256, n_shared_experts=1,
                d_ff_shared=256, top_k1=2, top_k2=3, std=0.05, coupling_std=0.5)
    base.update(kw)
    return synth.ModelShape(**base)


def _check_routing(t, outs, shape, tag):
    """Indices equal the oracle's, or differ only where the oracle's router
    logits are within the margin that the bf16-level error of the router
    input allows (then the GPU choice is a valid top-k under that margin).
    Returns, per path, the rows whose indices equal the oracle's."""
    k2 = shape.top_k1 if shape.replay else shape.top_k2
    gi1, gw1 = _np(t["route_idx1"])[0], _np(t["route_w1"])[0]
    gi2, gw2 = _np(t["route_idx2"])[0], _np(t["route_w2"])[0]
    same = ([], [])
    for b, o in enumerate(outs):
        rec = o["layers"][0]
        for path, (gi, gw, oi, ow, r, k) in enumerate(
                ((gi1[b], gw1[b], rec["idx1"], rec["w1"], rec["r1"], shape.top_k1),
                 (gi2[b], gw2[b], rec["idx2"], rec["w2"], rec.get("r2"), k2))):
            assert len(set(gi.tolist())) == k
            if np.array_equal(gi, oi):
                np.testing.assert_allclose(gw, ow, rtol=BF16_TOL, atol=1e-4, err_msg=tag)
                same[path].append(b)
                continue
            r = np.asarray(r)
            rs = np.sort(r)[::-1]
            margin = BF16_TOL * np.max(np.abs(r))
            for j in range(k):
                assert abs(r[gi[j]] - rs[j]) <= margin, (tag, b, j, gi, oi, r[gi[j]], rs[j])
            if set(gi.tolist()) == set(oi.tolist()):
                og = dict(zip(oi.tolist(), ow.tolist()))
                np.testing.assert_allclose(gw, [og[e] for e in gi.tolist()], rtol=BF16_TOL, atol=1e-4)
                same[path].append(b)
    return same


def _check_outputs(t, outs, shape, tag, logits=True):
    """Routing first; then residual outputs (and logits) of a path are
    compared on the rows whose expert choice matches the oracle's.  A row
    the GPU routed differently at a certified near-tie takes other experts,
    so its outputs differ legitimately; such rows must stay rare."""
    same1, same2 = _check_routing(t, outs, shape, tag)
    both = sorted(set(same1) & set(same2))
    assert len(same1) >= len(outs) - 1 and len(both) >= len(outs) - 1, (tag, same1, same2)
    h1 = np.stack([o["h1"] for o in outs])
    h2 = np.stack([o["h2"] for o in outs])
    assert row_err(_np(t["h1_out"])[same1], h1[same1]).max() <= BF16_TOL, tag
    assert row_err(_np(t["h2_out"])[both], h2[both]).max() <= BF16_TOL, tag
    if logits:
        z1 = np.stack([o["z1"] for o in outs])
        z2 = np.stack([o["z2"] for o in outs])
        assert row_err(_np(t["logits1"])[same1], z1[same1]).max() <= BF16_TOL, tag
        assert row_err(_np(t["logits2"])[both], z2[both]).max() <= BF16_TOL, tag


def _gated(W, shape):
    """Compute-matched gates away from their initial value one, so a gate
    applied to the wrong row or not at all shows (seeded, N(1, 0.5))."""
    for l in range(shape.n_layers):
        for j, nm in enumerate(("g_A", "g_G")):
            W.values[f"L{l}.{nm}"] = 1.0 + synth.normal(5, 100 * l + j, (shape.d_model,), 0.5)
    return W


def _run(shape, lengths, steps=2, grouped=True, branch_on=True):
    W = synth.make_weights(shape, seed=0)
    if shape.compute_matched:
        W = _gated(W, shape)
    B = len(lengths)
    orc = Oracle(shape, W.values)
    sess = make_session(shape, W, max_batch=B, max_pos=max(lengths) + steps + 1)
    sess.k_pages.zero_()
    sess.v_pages.zero_()
    fill_cache(sess, orc, shape, lengths)
    res = []
    for step in range(steps):
        h = synth.make_hidden(shape, B, step=step, seed=2)
        outs = orc.decode_step(h1=h[0], h2=h[1], branch_on=branch_on)
        t = sess.decode(h1=h[0], h2=h[1], grouped=grouped, branch_on=branch_on)
        res.append((t, outs))
    return sess, res


@pytest.mark.parametrize("k2,replay", [(3, False), (8, False), (2, True)])
def test_moe_layer_parity(k2, replay):
    shape = _moe_shape(top_k2=k2, replay=replay)
    sess, res = _run(shape, [1, 17, 300, 64, 529])
    for step, (t, outs) in enumerate(res):
        _check_outputs(t, outs, shape, f"k2={k2} replay={replay} step {step}")
    sess.close()


def test_moe_no_shared_expert():
    shape = _moe_shape(n_shared_experts=0, d_ff_shared=0, top_k2=4)
    sess, res = _run(shape, [5, 40, 200], steps=1)
    t, outs = res[0]
    _check_outputs(t, outs, shape, "no shared")
    sess.close()


def test_moe_primary_bitwise_on_off_and_grouped_equals_ungrouped():
    shape = _moe_shape(top_k2=4)
    lengths = [3, 40, 530, 16]
    got = {}
    for mode in ("on", "off", "ungrouped"):
        sess, res = _run(shape, lengths, steps=1, grouped=(mode != "ungrouped"), branch_on=(mode != "off"))
        t = res[0][0]
        got[mode] = {k: _np(v).copy() for k, v in t.items()}
        got[mode]["k"] = _np(sess.k_pages).copy()
        sess.close()
    on, off, ug = got["on"], got["off"], got["ungrouped"]
    for k in ("h1_out", "logits1", "route_idx1", "route_w1", "k"):
        np.testing.assert_array_equal(on[k], off[k], err_msg=k)
    for k in ("h1_out", "h2_out", "logits1", "logits2", "alpha", "next_token", "route_idx1", "route_idx2",
              "route_w1", "route_w2", "k"):
        np.testing.assert_array_equal(on[k], ug[k], err_msg=k)


@pytest.mark.parametrize("k1,k2", [(2, 2), (1, 3), (3, 1)])
def test_moe_compute_matched_parity(k1, k2):
    """Compute-matched variant (App. B.3), k1 + k2 = 4: the branch evaluates
    no attention and no shared expert; it takes g_A * A1 and g_G * G(N1)."""
    shape = _moe_shape(compute_matched=True, top_k1=k1, top_k2=k2)
    sess, res = _run(shape, [1, 17, 300, 64, 529])
    for step, (t, outs) in enumerate(res):
        _check_outputs(t, outs, shape, f"compute-matched k1={k1} k2={k2} step {step}")
    sess.close()


def test_moe_compute_matched_bitwise_modes():
    """Compute-matched variant: primary outputs and cache bit-identical with
    the branch on or off; grouped equals the two-pass step (which hands the
    branch the kept A1 and G1) bit for bit."""
    shape = _moe_shape(compute_matched=True, top_k1=2, top_k2=2)
    lengths = [3, 40, 530, 16]
    got = {}
    for mode in ("on", "off", "ungrouped"):
        sess, res = _run(shape, lengths, steps=1, grouped=(mode != "ungrouped"), branch_on=(mode != "off"))
        t = res[0][0]
        got[mode] = {k: _np(v).copy() for k, v in t.items()}
        got[mode]["k"] = _np(sess.k_pages).copy()
        sess.close()
    on, off, ug = got["on"], got["off"], got["ungrouped"]
    for k in ("h1_out", "logits1", "route_idx1", "route_w1", "k"):
        np.testing.assert_array_equal(on[k], off[k], err_msg=k)
    for k in ("h1_out", "h2_out", "logits1", "logits2", "alpha", "next_token", "route_idx1", "route_idx2",
              "route_w1", "route_w2", "k"):
        np.testing.assert_array_equal(on[k], ug[k], err_msg=k)


@pytest.mark.slow
@pytest.mark.parametrize("k2", [2, 4, 8])
def test_moe_full_size_sampled(k2):
    """64 experts x 1408 + shared 1408, d 2048, batch 64, cache 8192."""
    _full_size(k2, compute_matched=False)


@pytest.mark.slow
def test_moe_compute_matched_full_size_sampled():
    """The compute-matched variant at the MoE workload's full size, k1 = k2 = 2."""
    _full_size(2, compute_matched=True)


def _full_size(k2, compute_matched):
    w = synth.workload("moe_bf16")
    shape = synth.ModelShape(**{**w["shape"].__dict__, "top_k2": k2, "compute_matched": compute_matched})
    B, L = w["batch"], w["cache_len"]
    W = synth.make_weights(shape, seed=0)
    if compute_matched:
        W = _gated(W, shape)
    sess = make_session(shape, W, max_batch=B, max_pos=L + 16)
    fill_cache(sess, None, shape, [L] * B)
    h = synth.make_hidden(shape, B, step=0, seed=2)
    t = sess.decode(h1=h[0], h2=h[1])
    sample = [0, 33, 63]
    orc = Oracle(shape, W.values)
    for b in sample:
        (kv_, _), (vv_, _) = synth.make_kv(shape, 0, b, L, seed=3)
        orc.kv_fill(b, L, [kv_], [vv_])
    outs = [orc.step_one(b, h1=h[0, b], h2=h[1, b], readout=False) for b in sample]
    sub = {k: (v[:, sample] if k.startswith("route") else v[sample]) for k, v in t.items()}
    _check_outputs(sub, outs, shape, f"full k2={k2} compute_matched={compute_matched}", logits=False)
    # every row: k distinct valid experts, weights positive summing to one
    for key, k in (("route_idx1", shape.top_k1), ("route_idx2", k2)):
        idx = _np(t[key])[0]
        assert idx.shape == (B, k)
        assert all(len(set(r.tolist())) == k for r in idx)
        assert np.all((idx >= 0) & (idx < shape.n_experts))
    for key in ("route_w1", "route_w2"):
        wts = _np(t[key])[0]
        np.testing.assert_allclose(wts.sum(axis=1), 1.0, rtol=1e-5)
    sess.close()


@pytest.mark.parametrize("compute_matched", [False, True])
def test_moe_prefill_boundary_and_steps(compute_matched):
    """Prompts through a two-layer MoE model with token embeddings: the
    prefill routes every prompt position on the primary path (Sec. 4.4,
    step 1; the 600-position prompt has 4800 assignments per layer, more
    than the chunked dispatch sorts, so its layers take the scanning
    dispatch), the boundary routes the branch once (step 2), then two
    grouped steps.  Cache pages are poisoned with NaN first."""
    shape = _moe_shape(n_layers=2, has_embeddings=True, top_k2=3, compute_matched=compute_matched)
    W = synth.make_weights(shape, seed=0)
    if compute_matched:
        W = _gated(W, shape)
    lens = [37, 300, 1, 600]
    prompts = [synth.make_tokens(1, 70 + i, (L,), shape.vocab) for i, L in enumerate(lens)]
    orc = Oracle(shape, W.values)
    obs = orc.prefill(prompts, run_boundary=True)
    sess = make_session(shape, W, max_batch=len(lens), max_pos=610, max_prompt=600)
    sess.k_pages.fill_(0xFF)
    sess.v_pages.fill_(0xFF)
    tag = f"moe prefill cm={compute_matched}"
    t = sess.prefill(prompts, run_boundary=True)
    check_readout(t, obs, BF16_TOL, tag + " boundary")
    toks = [o["next"] for o in obs]
    for step in range(2):
        outs = orc.decode_step(tokens=toks)
        t = sess.decode(tokens=toks)
        _check_outputs(t, outs, shape, f"{tag} step {step}")
        toks = [o["next"] for o in outs]
    sess.close()
