"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself through a retyped formula:
each test uses a closed form, a hand-worked value (tests/golden), a
library routine for a special case, brute force on tiny inputs, or a
structural property the paper states for the decode path.
"""
import cmath
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import synth
from oracle import (Oracle, PageAllocator, attend, mixture_readout, rmsnorm, rope,
                    round_bf16, route, silu, softmax, topk)
from oracle.dbt_oracle import expert_assignments
from tests.tiny import params, rel_err, tiny_moe_shape, tiny_shape, with_shape

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ----------------------------------------------------------------------------
# Elementary operations
# ----------------------------------------------------------------------------

def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 37))
    y = rmsnorm(x, np.ones(37), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-14)
    np.testing.assert_allclose(rmsnorm(7.5 * x, np.ones(37), 0.0), y, rtol=1e-13)
    g = rng.standard_normal(37)
    np.testing.assert_allclose(rmsnorm(x, g, 0.0), y * g, rtol=1e-13)
    # eps enters under the square root: constant row c gives c / sqrt(c^2 + eps)
    c = np.full((1, 4), 0.5)
    np.testing.assert_allclose(rmsnorm(c, np.ones(4), 0.25), 0.5 / math.sqrt(0.5), rtol=1e-14)


def test_rope_closed_forms():
    # position 0 is the identity
    rng = np.random.default_rng(1)
    v = rng.standard_normal((3, 16))
    np.testing.assert_array_equal(rope(v, 0, 10000.0), v)
    # d_h = 4, theta = 100: pair (0, 2) turns by pos * 1, pair (1, 3) by pos * 100^(-1/2)
    for pos in (1, 5, 123):
        x = np.array([0.3, -1.1, 0.7, 0.25])
        r = rope(x, pos, 100.0)
        z0 = complex(0.3, 0.7) * cmath.exp(1j * pos * 1.0)
        z1 = complex(-1.1, 0.25) * cmath.exp(1j * pos * 0.1)
        np.testing.assert_allclose(r, [z0.real, z1.real, z0.imag, z1.imag], rtol=1e-12, atol=1e-14)
    # norm-preserving; scores depend on the position difference only
    q, k = rng.standard_normal(64), rng.standard_normal(64)
    np.testing.assert_allclose(np.linalg.norm(rope(q, 77, 10000.0)), np.linalg.norm(q), rtol=1e-13)
    s1 = rope(q, 300, 10000.0) @ rope(k, 290, 10000.0)
    s2 = rope(q, 10, 10000.0) @ k
    assert abs(s1 - s2) < 1e-10 * max(1.0, abs(s2))


def test_silu_and_softmax_vs_library():
    u = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(silu(u), u * scipy.special.expit(u), rtol=1e-13, atol=1e-300)
    assert silu(np.array(0.0)) == 0.0
    z = np.random.default_rng(2).standard_normal((4, 50)) * 10
    np.testing.assert_allclose(softmax(z), scipy.special.softmax(z, axis=-1), rtol=1e-13)


def test_attend_special_cases_and_brute_force():
    rng = np.random.default_rng(3)
    d = 16
    q = rng.standard_normal(d)
    V = rng.standard_normal((9, d))
    # one key: the output is that key's value
    np.testing.assert_allclose(attend(q, rng.standard_normal((1, d)), V[:1]), V[0], rtol=1e-15)
    # identical keys: plain mean of the values
    K = np.tile(rng.standard_normal(d), (9, 1))
    np.testing.assert_allclose(attend(q, K, V), V.mean(axis=0), rtol=1e-13)
    # two keys, closed form with the 1/sqrt(d_h) scale
    e = np.zeros(d); e[0] = 1.0
    K2 = np.stack([3.0 * e, np.zeros(d)])
    w0 = math.exp(3.0 / 4.0) / (math.exp(3.0 / 4.0) + 1.0)
    np.testing.assert_allclose(attend(e, K2, V[:2]), w0 * V[0] + (1 - w0) * V[1], rtol=1e-14)
    # brute force with python floats (no max shift)
    K = rng.standard_normal((9, d))
    sc = [sum(q[i] * K[j, i] for i in range(d)) / math.sqrt(d) for j in range(9)]
    ex = [math.exp(s) for s in sc]
    ref = [sum(ex[j] * V[j, i] for j in range(9)) / sum(ex) for i in range(d)]
    np.testing.assert_allclose(attend(q, K, V), ref, rtol=1e-12)


def test_round_bf16_golden_and_vs_bit_rounding():
    for c in _golden("bf16_cases.json")["cases"]:
        assert round_bf16(float(c["x"])) == float(c["expect"]), c
    # float32 inputs: same result as integer rounding of the bit pattern
    x = np.random.default_rng(4).standard_normal(100000).astype(np.float32) * 3
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)),
                                  synth.bf16_values(synth.bf16_bits(x)).astype(np.float64))


def test_mixture_readout_golden():
    for c in _golden("mixture_cases.json")["cases"]:
        z1, z2 = np.log(c["p"]), np.log(c["q"])
        alpha, m, nxt = mixture_readout(z1, z2)
        assert abs(float(np.sum(softmax(z1) ** 2)) - c["sum_p2"]) < 1e-12
        assert abs(alpha - c["alpha"]) < 1e-12
        np.testing.assert_allclose(m, c["m"], rtol=1e-12, atol=1e-15)
        assert nxt == c["next"]
        assert abs(np.sum(m) - 1.0) < 1e-12


def test_mixture_with_several_branches_golden():
    """App. C.1: hand-worked cases of the averaged branch distribution."""
    for c in _golden("mixture_branches_cases.json")["cases"]:
        z1 = np.log(c["p"])
        zb = [np.log(q) for q in c["q"]]
        alpha, m, nxt = mixture_readout(z1, zb[0], z_branches=zb)
        assert abs(alpha - c["alpha"]) < 1e-12
        np.testing.assert_allclose(np.mean([softmax(z) for z in zb], axis=0), c["q_bar"], rtol=1e-12)
        np.testing.assert_allclose(m, c["m"], rtol=1e-12, atol=1e-15)
        assert nxt == c["next"]


def test_mixture_readout_limits():
    V = 1000
    # near one-hot primary: alpha -> 1, prediction -> p
    z1 = np.zeros(V); z1[17] = 60.0
    alpha, m, nxt = mixture_readout(z1, np.random.default_rng(5).standard_normal(V))
    assert alpha == pytest.approx(1.0, abs=1e-12) and nxt == 17
    # branch off: alpha = 1 and the token is argmax z1 regardless of z2
    z1 = np.random.default_rng(6).standard_normal(V)
    z2 = np.zeros(V); z2[3] = 100.0
    alpha, m, nxt = mixture_readout(z1, z2, branch_on=False)
    assert alpha == 1.0 and nxt == int(np.argmax(z1))
    # with the branch on, a confident branch can move the token when p is flat
    alpha, m, nxt = mixture_readout(np.zeros(V), z2)
    assert alpha == 0.5 and nxt == 3
    # two dominant equal primary logits: sum p^2 -> 0.5
    z1 = np.full(V, -50.0); z1[[4, 9]] = 10.0
    alpha, _, nxt = mixture_readout(z1, np.zeros(V))
    assert alpha == pytest.approx(0.5, abs=1e-12) and nxt == 4


def test_topk_brute_force_and_ties():
    rng = np.random.default_rng(7)
    for _ in range(50):
        r = rng.standard_normal(8)
        for k in (1, 2, 3, 5):
            best = max(itertools.combinations(range(8), k), key=lambda c: sum(r[i] for i in c))
            got = topk(r, k)
            assert sorted(got.tolist()) == sorted(best)
            assert all(r[got[i]] >= r[got[i + 1]] for i in range(k - 1))
            np.testing.assert_array_equal(got, np.argsort(-r, kind="stable")[:k])
    r = np.array([0.5, 2.0, 0.5, 2.0, 1.0])
    assert topk(r, 3).tolist() == [1, 3, 4]
    assert topk(r, 4).tolist() == [1, 3, 4, 0]


def test_route_normalize_identity_and_replay():
    rng = np.random.default_rng(8)
    r = rng.standard_normal(16)
    idx, w = route(r, 4)
    np.testing.assert_allclose(w, scipy.special.softmax(r[idx]), rtol=1e-13)
    assert abs(w.sum() - 1.0) < 1e-14
    idx2, w2 = route(r, 4, replay_idx=idx)
    np.testing.assert_array_equal(idx2, idx)
    np.testing.assert_allclose(w2, w, rtol=1e-15)
    # replay gathers the branch's own probabilities at the primary's indices
    r2 = rng.standard_normal(16)
    idx3, w3 = route(r2, 4, replay_idx=idx)
    np.testing.assert_allclose(w3, scipy.special.softmax(r2[idx]), rtol=1e-13)


def test_page_allocator_script():
    g = _golden("page_script.json")
    a = PageAllocator(g["num_pages"], 16)
    for op in g["ops"]:
        if op["op"] == "reserve":
            a.reserve(op["b"], op["len"])
        elif op["op"] == "append":
            assert a.append_one(op["b"]) == op["pos"]
        else:
            a.truncate(op["b"], op["len"])
        for b, tab in op["expect"].items():
            assert a.table[int(b)] == tab, (op, a.table)
    with pytest.raises(MemoryError):
        PageAllocator(2, 16).reserve(0, 33)


# ----------------------------------------------------------------------------
# Structural properties of the decode path (Sec. 4.1, Sec. 4.4, Sec. 4.5)
# ----------------------------------------------------------------------------

def _decode_all(orc, x, branch_on=True, grouped=True):
    """Token-by-token continuation steps from an empty cache."""
    outs = []
    for t in range(len(x)):
        outs.append(orc.decode_step(tokens=[x[t]], branch_on=branch_on, grouped=grouped)[0])
    return outs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_primary_bit_identical_branch_on_off(dtype):
    shape = tiny_shape(dtype=dtype)
    P = params(shape)
    x = synth.make_tokens(1, 0, (12,), shape.vocab)
    on, off = Oracle(shape, P), Oracle(shape, P)
    o_on = _decode_all(on, x, True)
    o_off = _decode_all(off, x, False)
    for a, b in zip(o_on, o_off):
        np.testing.assert_array_equal(a["h1"], b["h1"])
        np.testing.assert_array_equal(a["z1"], b["z1"])
    for l in range(shape.n_layers):
        np.testing.assert_array_equal(on.K[l][0], off.K[l][0])
        np.testing.assert_array_equal(on.V[l][0], off.V[l][0])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decode_equals_full_masked_forward(dtype):
    """Branch-off decode equals the one-flow causal forward; the branch at t
    equals the two-path training graph at t (Sec. 4.4)."""
    shape = tiny_shape(dtype=dtype)
    P = params(shape)
    x = synth.make_tokens(1, 1, (20,), shape.vocab)
    full = Oracle(shape, P).forward_full(x)
    dec = _decode_all(Oracle(shape, P), x, True)
    z1 = np.stack([o["z1"] for o in dec])
    z2 = np.stack([o["z2"] for o in dec])
    assert rel_err(z1, full["z1"]) < 1e-12
    assert rel_err(z2, full["z2"]) < 1e-12
    off = _decode_all(Oracle(shape, P), x, False)
    assert rel_err(np.stack([o["z1"] for o in off]), full["z1"]) < 1e-12


def test_grouped_equals_ungrouped_exactly():
    shape = tiny_shape()
    P = params(shape)
    x = synth.make_tokens(1, 2, (10,), shape.vocab)
    g = _decode_all(Oracle(shape, P), x, True, grouped=True)
    u = _decode_all(Oracle(shape, P), x, True, grouped=False)
    for a, b in zip(g, u):
        for k in ("h1", "h2", "z1", "z2", "m"):
            np.testing.assert_array_equal(a[k], b[k])
        assert a["next"] == b["next"] and a["alpha"] == b["alpha"]


def test_cache_grows_by_one_and_branch_writes_nothing():
    shape = tiny_shape()
    P = params(shape)
    orc = Oracle(shape, P)
    x = synth.make_tokens(1, 3, (9,), shape.vocab)
    orc.prefill([x[:5]], run_boundary=False)
    before = [orc.K[l][0].copy() for l in range(shape.n_layers)]
    orc.boundary(0)            # branch-only: must not touch the cache
    for l in range(shape.n_layers):
        np.testing.assert_array_equal(orc.K[l][0], before[l])
    for t in range(5, 9):
        orc.decode_step(tokens=[x[t]])
        for l in range(shape.n_layers):
            assert orc.K[l][0].shape[0] == t + 1 and orc.V[l][0].shape[0] == t + 1
            np.testing.assert_array_equal(orc.K[l][0][:5], before[l])
    assert orc.alloc.length[0] == 9


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_boundary_equals_decode_step(dtype):
    """prefill(x[:S]) + boundary == prefill(x[:S-1]) + one continuation step
    with x[S-1] (Sec. 4.4: the boundary is one token-level decode evaluation);
    batched prefill keys equal token-by-token keys."""
    shape = tiny_shape(dtype=dtype)
    P = params(shape)
    x = synth.make_tokens(1, 4, (15,), shape.vocab)
    a = Oracle(shape, P)
    ra = a.prefill([x], run_boundary=True)[0]
    b = Oracle(shape, P)
    b.prefill([x[:-1]], run_boundary=False)
    rb = b.decode_step(tokens=[x[-1]])[0]
    for k in ("z1", "z2", "h1", "h2"):
        assert rel_err(ra[k], rb[k]) < 1e-12, k
    assert ra["next"] == rb["next"]
    assert abs(ra["alpha"] - rb["alpha"]) < 1e-12
    c = Oracle(shape, P)
    _decode_all(c, x, False)
    for l in range(shape.n_layers):
        assert rel_err(a.K[l][0], c.K[l][0]) < 1e-12
        assert rel_err(a.V[l][0], c.V[l][0]) < 1e-12


def test_branch_reduces_to_primary():
    """E2 := E1 and a = b = c = 0: the branch recomputes the primary, so
    z2 = z1 and the mixture is p."""
    shape = tiny_shape()
    P = dict(params(shape))
    P["E2"] = P["E1"]
    for l in range(shape.n_layers):
        for v in "abc":
            P[f"L{l}.{v}"] = np.zeros_like(P[f"L{l}.{v}"])
    x = synth.make_tokens(1, 5, (8,), shape.vocab)
    for o in _decode_all(Oracle(shape, P), x):
        np.testing.assert_array_equal(o["z1"], o["z2"])
        np.testing.assert_allclose(o["m"], softmax(o["z1"]), rtol=1e-14)


@pytest.mark.parametrize("beta,gamma", [(0.75, 0.0), (0.0, -0.375), (0.5, 0.25)])
def test_mlp_coupling_closed_form(beta, gamma):
    """One layer, E2 := E1, a = 0, b = beta, c = gamma: the paths agree up to
    the MLP, then M2 = (1 + beta) M1 + gamma M1 (Eqs. (13)-(16))."""
    shape = tiny_shape(n_layers=1, vocab=64)
    P = dict(params(shape))
    P["E2"] = P["E1"]
    P["L0.a"] = np.zeros_like(P["L0.a"])
    P["L0.b"] = np.full_like(P["L0.b"], beta)
    P["L0.c"] = np.full_like(P["L0.c"], gamma)
    orc = Oracle(shape, P)
    x = synth.make_tokens(1, 6, (6,), shape.vocab)
    for t, o in enumerate(_decode_all(orc, x)):
        S_in = orc.embed(x[t], 0)
        rec = o["layers"][0]
        np.testing.assert_allclose(o["h1"], S_in + rec["A1"] + rec["M1"], rtol=1e-13)
        np.testing.assert_allclose(o["h2"], S_in + rec["A1"] + (1 + beta + gamma) * rec["M1"],
                                   rtol=1e-12, atol=1e-13)


def test_query_coupling_closed_form():
    """One layer, E2 := E1 (so Q2 = Q1), a random: the branch query is
    (1 + a) * Q1 after RoPE (Eqs. (10)-(11)) and it reads the primary keys and
    values of positions 0..t; at t = 1 the weights follow the two-key closed
    form.  A per-element a distinguishes adding a*Q1 after RoPE from adding
    it before."""
    shape = tiny_shape(n_layers=1, n_q_heads=2, n_kv_heads=2, vocab=64)
    P = dict(params(shape))
    P["E2"] = P["E1"]
    orc = Oracle(shape, P)
    x = synth.make_tokens(1, 7, (2,), shape.vocab)
    out = _decode_all(orc, x)[1]
    q1 = out["layers"][0]["q1"]
    a = np.asarray(P["L0.a"], np.float64).reshape(2, 16)
    K, V = orc.K[0][0], orc.V[0][0]
    heads = []
    for h in range(2):
        qt = (1.0 + a[h]) * q1[h]
        s0, s1 = (qt @ K[0, h]) / 4.0, (qt @ K[1, h]) / 4.0
        w1 = 1.0 / (1.0 + math.exp(s0 - s1))
        heads.append((1 - w1) * V[0, h] + w1 * V[1, h])
    A2 = np.concatenate(heads) @ np.asarray(P["L0.W_O"], np.float64).T
    np.testing.assert_allclose(out["layers"][0]["A2"], A2, rtol=1e-12, atol=1e-14)
    # the same a added before RoPE would give a different query
    pre = rope((1.0 + a) * rope(q1, -1, shape.rope_theta), 1, shape.rope_theta)
    assert np.max(np.abs(pre - (1.0 + a) * q1)) > 1e-3


def test_tolerance_bar_above_fp32_noise():
    """The 1e-5 bar for fp32 sits above fp32 rounding of the whole path:
    the oracle run in float32 stays within it on the tiny fp32 workload."""
    w = synth.workload("tiny_f32")
    shape = w["shape"]
    P = params(shape)
    x = synth.make_tokens(1, 0, (40,), shape.vocab)
    o64 = Oracle(shape, P).prefill([x], run_boundary=True)[0]
    o32 = Oracle(shape, P, ftype=np.float32).prefill([x], run_boundary=True)[0]
    e1, e2 = rel_err(o32["z1"], o64["z1"]), rel_err(o32["z2"], o64["z2"])
    assert 0 < e1 < 3e-6 and 0 < e2 < 3e-6, (e1, e2)


# ----------------------------------------------------------------------------
# MoE (Sec. 3.2, Sec. 4.3, Sec. 5)
# ----------------------------------------------------------------------------

def _moe_as_dense(Pm, shape_m, expert=0):
    """Dense-model parameters whose MLP is expert ``expert`` of an MoE layer."""
    shape_d = with_shape(shape_m, n_experts=0, d_ff=shape_m.d_ff_expert, n_shared_experts=0,
                         d_ff_shared=0, top_k1=0, top_k2=0)
    Pd = {k: v for k, v in Pm.items() if not k.startswith("L0.X_") and not k.startswith("L0.S_")}
    Pd["L0.W_gate"] = Pm["L0.X_gate"][expert]
    Pd["L0.W_up"] = Pm["L0.X_up"][expert]
    Pd["L0.W_down"] = Pm["L0.X_down"][expert]
    Pd["L0.b"] = np.zeros(shape_m.d_ff_expert, np.float32)
    return shape_d, Pd


def _fill(orc, shape, B, L, seed=3):
    for b in range(B):
        (k, _), (v, _) = synth.make_kv(shape, 0, b, L, seed=seed)
        orc.kv_fill(b, L, [k], [v])


def test_moe_single_expert_equals_dense():
    shape = tiny_moe_shape(n_experts=1, top_k1=1, top_k2=1, n_shared_experts=0, d_ff_shared=0)
    P = dict(params(shape))
    shape_d, Pd = _moe_as_dense(P, shape)
    h = synth.make_hidden(shape, 3)
    m_orc, d_orc = Oracle(shape, P), Oracle(shape_d, Pd)
    _fill(m_orc, shape, 3, 21)
    _fill(d_orc, shape_d, 3, 21)
    om = m_orc.decode_step(h1=h[0], h2=h[1])
    od = d_orc.decode_step(h1=h[0], h2=h[1])
    for a, b in zip(om, od):
        assert rel_err(a["h1"], b["h1"]) < 1e-13 and rel_err(a["h2"], b["h2"]) < 1e-13


def test_moe_identical_experts_weights_sum_to_one():
    """All experts equal: any normalized top-k combination equals that one
    expert, so the MoE layer equals the dense layer whatever the routing."""
    shape = tiny_moe_shape(n_experts=6, top_k1=2, top_k2=4, n_shared_experts=0, d_ff_shared=0)
    P = dict(params(shape))
    for nm in ("L0.X_gate", "L0.X_up", "L0.X_down"):
        P[nm] = np.repeat(P[nm][:1], 6, axis=0)
    shape_d, Pd = _moe_as_dense(P, shape)
    h = synth.make_hidden(shape, 2)
    m_orc, d_orc = Oracle(shape, P), Oracle(shape_d, Pd)
    _fill(m_orc, shape, 2, 5)
    _fill(d_orc, shape_d, 2, 5)
    for a, b in zip(m_orc.decode_step(h1=h[0], h2=h[1]), d_orc.decode_step(h1=h[0], h2=h[1])):
        assert rel_err(a["h1"], b["h1"]) < 1e-12 and rel_err(a["h2"], b["h2"]) < 1e-12


def test_moe_replay_equals_independent_when_same_logits():
    """Router replay (Eq. (19)) reduces to independent routing when the
    branch router input equals the primary's and k2 = k1: build that case
    with E2 := E1-like inputs (h2 = h1) and zero couplings."""
    shape = tiny_moe_shape(top_k1=2, top_k2=2)
    P = dict(params(shape))
    P["L0.a"] = np.zeros_like(P["L0.a"])
    P["L0.b"] = np.zeros_like(P["L0.b"])
    P["L0.c"] = np.zeros_like(P["L0.c"])
    h = synth.make_hidden(shape, 3)
    ind = Oracle(shape, P)
    rep = Oracle(with_shape(shape, replay=True), P)
    _fill(ind, shape, 3, 9)
    _fill(rep, shape, 3, 9)
    for a, b in zip(ind.decode_step(h1=h[0], h2=h[0]), rep.decode_step(h1=h[0], h2=h[0])):
        np.testing.assert_array_equal(a["h2"], b["h2"])
        np.testing.assert_array_equal(a["layers"][0]["idx2"], b["layers"][0]["idx2"])
        np.testing.assert_array_equal(a["h1"], a["h2"])


def test_moe_fanouts_independent_and_primary_unaffected():
    """k2 changes only the branch: primary outputs and the primary's expert
    choice are bit-identical for k2 in {2, 4, 8} (Sec. 5, Eq. (22))."""
    h = None
    ref = None
    for k2 in (2, 4, 8):
        shape = tiny_moe_shape(top_k2=k2)
        P = params(shape)
        if h is None:
            h = synth.make_hidden(shape, 4)
        orc = Oracle(shape, P)
        _fill(orc, shape, 4, 17)
        out = orc.decode_step(h1=h[0], h2=h[1])
        for o in out:
            assert len(o["layers"][0]["idx2"]) == k2
            assert abs(o["layers"][0]["w2"].sum() - 1) < 1e-14
        if ref is None:
            ref = out
        else:
            for a, b in zip(ref, out):
                np.testing.assert_array_equal(a["h1"], b["h1"])
                np.testing.assert_array_equal(a["layers"][0]["idx1"], b["layers"][0]["idx1"])


def test_compute_matched_unit_gates_and_replay_reduce_branch_to_primary():
    """App. B.3 with unit gates, the same residual input on both paths and
    router replay: the gated copies hand the branch exactly the primary's
    attention and shared-expert outputs and the routed experts coincide, so
    the branch output equals the primary bit for bit (an extra c * M1 term
    would break this)."""
    shape = tiny_moe_shape(compute_matched=True, replay=True, top_k1=2, top_k2=2)
    P = params(shape)
    h = synth.make_hidden(shape, 3)
    orc = Oracle(shape, P)
    _fill(orc, shape, 3, 13)
    for o in orc.decode_step(h1=h[0], h2=h[0]):
        np.testing.assert_array_equal(o["h1"], o["h2"])


def test_compute_matched_zero_gates_is_routed_experts_of_own_state():
    """App. B.3 with g_A = g_G = 0: the branch layer is its residual plus its
    own routed experts.  That is the primary path of the standard model with
    the attention output and the shared expert switched off (W_O = 0,
    S_down = 0) and the same fan-out."""
    shape = tiny_moe_shape(compute_matched=True, top_k1=3, top_k2=3)
    P = dict(params(shape))
    P["L0.g_A"] = np.zeros_like(P["L0.g_A"])
    P["L0.g_G"] = np.zeros_like(P["L0.g_G"])
    std = with_shape(shape, compute_matched=False)
    Q = dict(params(std))
    Q["L0.W_O"] = np.zeros_like(Q["L0.W_O"])
    Q["L0.S_down"] = np.zeros_like(Q["L0.S_down"])
    h = synth.make_hidden(shape, 3)
    cm, ref = Oracle(shape, P), Oracle(std, Q)
    _fill(cm, shape, 3, 7)
    _fill(ref, std, 3, 7)
    for a, b in zip(cm.decode_step(h1=h[0], h2=h[1]), ref.decode_step(h1=h[1], h2=h[0])):
        assert rel_err(a["h2"], b["h1"]) < 1e-13


def test_compute_matched_branch_never_reads_the_cache():
    """App. B.3: attention is evaluated once, on the primary path.  Replacing
    every cached key/value after the primary pass leaves the branch output
    unchanged."""
    shape = tiny_moe_shape(compute_matched=True)
    P = params(shape)
    h = synth.make_hidden(shape, 2)
    orc = Oracle(shape, P)
    _fill(orc, shape, 2, 11)
    outs = orc.decode_step(h1=h[0], h2=h[1], grouped=False)
    keep = [o["h2"] for o in outs]
    for b in range(2):
        orc.K[0][b] = orc.K[0][b] * 0 + 7.0
        orc.V[0][b] = orc.V[0][b] * 0 - 3.0
    for b, o in enumerate(outs):
        again = orc.branch_layer(0, b, h[1, b].astype(np.float64), len(orc.K[0][b]) - 1, o["layers"][0])[0]
        np.testing.assert_array_equal(again, keep[b])


def test_expert_assignments_brute():
    idx1 = [[0, 3], [3, 1]]
    idx2 = [[3, 2, 0], [1, 0, 2]]
    got = expert_assignments(idx1, idx2, 4)
    assert got == [[(0, 0), (1, 0), (1, 1)], [(0, 1), (1, 1)], [(1, 0), (1, 1)],
                   [(0, 0), (0, 1), (1, 0)]]


def test_more_branches_identical_tables_give_the_one_branch_model():
    """App. C.1: two decode branches whose embeddings are equal (E3 := E2)
    compute the same state; their mean distribution is that branch's own, so
    every output of the one-branch model is reproduced exactly."""
    one = tiny_shape(n_layers=2)
    two = with_shape(one, n_branches=2)
    P1 = params(one)
    P2 = dict(params(two))
    P2["E3"] = P2["E2"]
    x = synth.make_tokens(1, 3, (9,), one.vocab)
    o1, o2 = Oracle(one, P1), Oracle(two, P2)
    b1 = o1.prefill([x])[0]
    b2 = o2.prefill([x])[0]
    for key in ("z1", "z2", "alpha", "next"):
        np.testing.assert_array_equal(b1[key], b2[key])
    tok = b1["next"]
    for _ in range(3):
        s1 = o1.decode_step(tokens=[tok])[0]
        s2 = o2.decode_step(tokens=[tok])[0]
        np.testing.assert_array_equal(s2["hb"][0], s2["hb"][1])
        for key in ("h1", "h2", "z1", "z2", "alpha", "next"):
            np.testing.assert_array_equal(s1[key], s2[key])
        np.testing.assert_allclose(s1["m"], s2["m"], rtol=1e-15, atol=0)
        tok = s1["next"]


def test_more_branches_each_branch_is_the_one_branch_model_with_its_table():
    """App. C.1: branch j has its own embedding and the shared couplings and
    reads only the primary: branch 2 of a three-path model equals the single
    branch of the model whose E2 is that branch's table; the primary is the
    same in all of them."""
    two = tiny_shape(n_layers=2, n_branches=2)
    P2 = params(two)
    one = with_shape(two, n_branches=1)
    P1 = dict(P2)
    P1["E2"] = P2["E3"]
    P1.pop("E3")
    x = synth.make_tokens(1, 4, (7,), two.vocab)
    o1, o2 = Oracle(one, P1), Oracle(two, P2)
    o1.prefill([x], run_boundary=False)
    o2.prefill([x], run_boundary=False)
    for tok in (5, 11):
        s1 = o1.decode_step(tokens=[tok])[0]
        s2 = o2.decode_step(tokens=[tok])[0]
        np.testing.assert_array_equal(s1["h1"], s2["h1"])
        np.testing.assert_array_equal(s1["h2"], s2["hb"][1])
        np.testing.assert_array_equal(s1["z2"], s2["zb"][1])


def test_more_branches_leave_the_primary_and_cache_untouched():
    """Adding decode branches changes nothing on the primary path or in the
    cache (Sec. 4.4 for each branch; App. C.1)."""
    ref = None
    for nb in (1, 2, 3):
        shape = tiny_shape(n_layers=2, n_branches=nb)
        orc = Oracle(shape, params(shape))
        x = synth.make_tokens(1, 5, (6,), shape.vocab)
        orc.prefill([x])
        outs = [orc.decode_step(tokens=[t])[0] for t in (3, 9)]
        got = ([o["h1"] for o in outs], [o["z1"] for o in outs], [np.array(orc.K[l][0]) for l in range(2)])
        if ref is None:
            ref = got
        else:
            for a, b in zip(ref, got):
                for u, v in zip(a, b):
                    np.testing.assert_array_equal(u, v)



# ----------------------------------------------------------------------------
# Pins of the routed combine, the MoE coupling and the branch embeddings
# ----------------------------------------------------------------------------

def _basis_experts(d, gains, ups):
    """E experts of width 1 whose output is a multiple of a basis vector:
    Expert_e(U) = silu(g_e . U) (u_e . U) e_e for U = ones(d), with
    g_e . U = gains[e] and u_e . U = ups[e] (first coordinate carries them)."""
    E = len(gains)
    Xg = np.zeros((E, 1, d), np.float32)
    Xu = np.zeros((E, 1, d), np.float32)
    Xd = np.zeros((E, d, 1), np.float32)
    for e in range(E):
        Xg[e, 0, 0] = gains[e]
        Xu[e, 0, 1] = ups[e]
        Xd[e, e, 0] = 1.0
    return Xg, Xu, Xd


def test_routed_combine_pairs_each_weight_with_its_expert():
    """Sec. 3.2, Eq. (6): the routed output is sum_{e in I} w_e Expert_e(U).
    Three width-1 experts write multiples of distinct basis vectors, so each
    coordinate of the combine shows which weight went with which expert.
    The selection is passed in router order (logit descending), not sorted
    by expert id, with distinct weights."""
    shape = tiny_moe_shape(n_experts=3, d_ff_expert=1, top_k1=2, top_k2=2, n_shared_experts=0,
                           d_ff_shared=0)
    P = dict(params(shape))
    gains, ups = [1.0, 2.0, 0.5], [3.0, -1.5, 4.0]
    P["L0.X_gate"], P["L0.X_up"], P["L0.X_down"] = _basis_experts(shape.d_model, gains, ups)
    orc = Oracle(shape, P)
    U = np.ones(shape.d_model)
    s = [scipy.special.expit(g) * g * u for g, u in zip(gains, ups)]   # silu(g) * u
    for idx, wts in (([2, 0], [0.7, 0.3]), ([1, 2], [0.125, 0.875]), ([0, 1], [0.6, 0.4])):
        out = orc._experts(0, U, np.array(idx), np.array(wts))
        want = np.zeros(shape.d_model)
        for e, w in zip(idx, wts):
            want[e] = w * s[e]
        np.testing.assert_allclose(out, want, rtol=1e-14, atol=1e-15)


def test_moe_coupling_closed_form_on_shared_expert():
    """Reading R10 of the MoE coupling.  With router replay, the same residual
    input on both paths and a = 0, the branch sees the primary's state up to
    the MLP and routes to the same experts with the same weights, so R2 = R1
    and, with b = beta on the shared-expert intermediate and c = gamma on the
    MoE output, M2 = R1 + (1 + beta) G1 + gamma M1 (Eqs. (13)-(16) with the
    shared expert in place of the dense MLP)."""
    beta, gamma = 0.625, -0.25
    shape = tiny_moe_shape(replay=True, top_k1=2, top_k2=2)
    P = dict(params(shape))
    P["L0.a"] = np.zeros_like(P["L0.a"])
    P["L0.b"] = np.full_like(P["L0.b"], beta)
    P["L0.c"] = np.full_like(P["L0.c"], gamma)
    h = synth.make_hidden(shape, 3)
    orc = Oracle(shape, P)
    _fill(orc, shape, 3, 10)
    for b, o in enumerate(orc.decode_step(h1=h[0], h2=h[0])):
        rec = o["layers"][0]
        G1, M1 = rec["G1"], rec["M1"]
        R1 = M1 - G1
        assert np.max(np.abs(G1)) > 1e-2 and np.max(np.abs(R1)) > 1e-2
        Sb = h[0, b].astype(np.float64) + rec["A1"]
        np.testing.assert_allclose(o["h1"], Sb + M1, rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(o["h2"], Sb + R1 + (1 + beta) * G1 + gamma * M1, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("n_branches", [1, 2])
def test_branch_embeddings_are_the_branch_tables(n_branches):
    """Sec. 4, Eq. (7) (and App. C.1 for more branches): path j starts from
    RMSNorm of its own table's row.  With W_O = W_down = 0 and a = b = c = 0
    every layer passes the residual through unchanged, so after the step the
    primary holds RMSNorm(E1[x]) and branch j RMSNorm(E_{j+1}[x]); the tables
    differ, so reading the wrong one shows."""
    shape = tiny_shape(n_layers=2, n_branches=n_branches)
    P = dict(params(shape))
    for l in range(shape.n_layers):
        for nm in ("W_O", "W_down", "a", "b", "c"):
            P[f"L{l}.{nm}"] = np.zeros_like(P[f"L{l}.{nm}"])
    orc = Oracle(shape, P)
    g = np.asarray(P["g_emb"], np.float64)
    for tok in (3, 17, 40):
        o = orc.decode_step(tokens=[tok])[0]
        tabs = [P[f"E{j + 1}"][tok].astype(np.float64) for j in range(n_branches + 1)]
        assert min(np.max(np.abs(tabs[0] - t)) for t in tabs[1:]) > 1e-2
        np.testing.assert_allclose(o["h1"], rmsnorm(tabs[0], g, shape.rms_eps), rtol=1e-13)
        states = o["hb"] if n_branches > 1 else [o["h2"]]
        for j, st in enumerate(states):
            np.testing.assert_allclose(st, rmsnorm(tabs[j + 1], g, shape.rms_eps), rtol=1e-13)
