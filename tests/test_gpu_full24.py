"""The full dense model (24 layers, d 2048, 16q/4kv x 128, SwiGLU 5632, vocab
32000, bf16): prefill through the primary path, the boundary, then grouped
greedy steps (Sec. 4.4).

* At the model's full width and depth with short ragged prompts, every step is
  compared with the oracle (logits per row within 2e-2, alpha, tokens equal or
  a certified near-tie); the GPU is fed the oracle's tokens.
* At the full workload size (batch 64, 8192-token prompts, 256 steps) the
  checks are properties that hold at any size: tokens and alpha in range, the
  cache grows by exactly one position per step, no page is shared, and with
  the same input tokens the branch-off run reproduces the primary logits of
  the branch-on run bit for bit (the branch never feeds the primary).
"""
import numpy as np
import pytest

import synth
from oracle import Oracle
from tests.gpu_util import check_readout, make_session, to_np

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


@pytest.fixture(scope="module")
def full24():
    w = synth.workload("full24_bf16")
    return w, synth.make_weights(w["shape"], seed=0)


def test_full24_model_short_prompts_vs_oracle(full24):
    w, W = full24
    shape = w["shape"]
    lens = [300, 17, 129]
    prompts = [synth.make_tokens(1, 200 + i, (L,), shape.vocab) for i, L in enumerate(lens)]
    orc = Oracle(shape, W.values)
    obs = orc.prefill(prompts, run_boundary=True)
    sess = make_session(shape, W, max_batch=len(lens), max_pos=max(lens) + 16, max_prompt=max(lens))
    t = sess.prefill(prompts, run_boundary=True)
    check_readout(t, obs, BF16_TOL, "boundary")
    toks = [o["next"] for o in obs]
    for step in range(6):
        outs = orc.decode_step(tokens=toks)
        t = sess.decode(tokens=toks)
        check_readout(t, outs, BF16_TOL, f"step {step}")
        toks = [o["next"] for o in outs]
    sess.close()


@pytest.mark.slow
def test_full24_full_size_batch64_prompt8192_256_steps(full24):
    from paper_2608_12385_amd import binding
    w, W = full24
    shape = w["shape"]
    B, T, steps = w["batch"], w["prompt_len"], w["steps"]
    prompts = [synth.make_tokens(1, 1000 + b, (T,), shape.vocab) for b in range(B)]
    sess = make_session(shape, W, max_batch=B, max_pos=T + steps + 16, max_prompt=T)
    t = sess.prefill(prompts, run_boundary=True)
    toks = to_np(t["next_token"]).copy()
    assert np.all((toks >= 0) & (toks < shape.vocab))
    fed, kept = [], []
    for step in range(steps):
        fed.append(toks.copy())
        t = sess.decode(tokens=toks)
        kept.append(t["logits1"])
        a = to_np(t["alpha"])
        assert np.all((a >= 0.5) & (a <= 1.0)), step
        toks = to_np(t["next_token"]).copy()
        assert np.all((toks >= 0) & (toks < shape.vocab)), step
    for b in range(B):
        assert binding.dbt_kv_length(sess.kv, b) == T + steps
    pages = [p for b in range(B) for p in binding.dbt_kv_pages(sess.kv, b)]
    assert len(pages) == len(set(pages)) == B * ((T + steps + 15) // 16)
    # replay the same input tokens with the branch off: identical primary logits
    for b in range(B):
        binding.dbt_kv_truncate(sess.kv, b, T)
    for step in range(steps):
        t = sess.decode(tokens=fed[step], branch_on=False)
        assert bool(torch.equal(t["logits1"], kept[step])), step
        assert np.all(to_np(t["alpha"]) == 1.0)
    sess.close()
