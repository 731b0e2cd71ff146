"""GPU parity of the prefill path (Sec. 4.4: the primary path over the
prompt writes the cache) for every query-group size its attention kernels
tell apart.  G = n_q / n_kv = 1, 2 and 8 run the LDS-shared kernel with 16/G
query blocks per workgroup (G = 4 is covered by test_gpu_parity.py); G = 3,
which does not divide 16, runs the per-position-block fallback.  Prompts of
256 or more positions also run the tiled projections (gate/up with the
SwiGLU epilogue, QKV with the rotary embedding and cache writes in its
epilogue); shorter ones the weight-streaming projections.  Every cache byte
is poisoned with 0xFF (bf16 NaN) first, so slots past each prompt hold NaN.

Bars as elsewhere: bf16 2e-2 max relative error per row for both paths'
logits at the boundary and after one continuation step, alpha within the
same bar, greedy tokens equal except at certified near-ties.
"""
import pytest

import synth
from oracle import Oracle
from tests.gpu_util import check_readout, make_session

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


@pytest.mark.parametrize("n_q,n_kv", [(2, 2), (4, 2), (8, 1), (6, 2)])
def test_prefill_query_group_sizes(n_q, n_kv):
    shape = synth.ModelShape(n_layers=1, d_model=256, n_q_heads=n_q, n_kv_heads=n_kv, head_dim=128, d_ff=512,
                             vocab=512, dtype="bf16", has_embeddings=True, std=0.05, coupling_std=0.5)
    W = synth.make_weights(shape, seed=1)
    # 300 and 529 end inside a page pair (the last pair's value mask), 529
    # one position into its last page; 45 and 17 stay below the tiled
    # projections' 256 rows
    lens = [300, 45, 529, 17]
    prompts = [synth.make_tokens(1, 60 + i, (L,), shape.vocab) for i, L in enumerate(lens)]
    orc = Oracle(shape, W.values)
    obs = orc.prefill(prompts, run_boundary=True)
    sess = make_session(shape, W, max_batch=len(lens), max_pos=540, max_prompt=529)
    sess.k_pages.fill_(0xFF)
    sess.v_pages.fill_(0xFF)
    tag = f"G={n_q // n_kv}"
    t = sess.prefill(prompts, run_boundary=True)
    check_readout(t, obs, BF16_TOL, f"boundary {tag}")
    toks = [o["next"] for o in obs]
    outs = orc.decode_step(tokens=toks)
    t = sess.decode(tokens=toks)
    check_readout(t, outs, BF16_TOL, f"step {tag}")


def test_prefill_tile_threshold_prompts():
    """Prompts of 255, 256 and 257 positions: below, at and one past the
    256-row threshold of the tiled projections (the last also one row into a
    second row tile), against the oracle at the boundary and one step."""
    shape = synth.ModelShape(n_layers=2, d_model=256, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=512,
                             vocab=512, dtype="bf16", has_embeddings=True, std=0.05, coupling_std=0.5)
    W = synth.make_weights(shape, seed=2)
    lens = [255, 256, 257]
    prompts = [synth.make_tokens(1, 80 + i, (L,), shape.vocab) for i, L in enumerate(lens)]
    orc = Oracle(shape, W.values)
    obs = orc.prefill(prompts, run_boundary=True)
    sess = make_session(shape, W, max_batch=len(lens), max_pos=270, max_prompt=257)
    t = sess.prefill(prompts, run_boundary=True)
    check_readout(t, obs, BF16_TOL, "boundary 255/256/257")
    toks = [o["next"] for o in obs]
    outs = orc.decode_step(tokens=toks)
    t = sess.decode(tokens=toks)
    check_readout(t, outs, BF16_TOL, "step 255/256/257")


@pytest.mark.slow
def test_prefill_at_the_shared_kernel_page_limit():
    """A prompt of 16384 positions (1024 pages: the most the LDS-shared
    kernel stages) and one of 16385 (the per-position-block kernel), one
    query head per KV head, against the oracle at the boundary and one step."""
    shape = synth.ModelShape(n_layers=1, d_model=256, n_q_heads=1, n_kv_heads=1, head_dim=128, d_ff=512,
                             vocab=512, dtype="bf16", has_embeddings=True, std=0.05, coupling_std=0.5)
    W = synth.make_weights(shape, seed=3)
    lens = [16384, 16385]
    prompts = [synth.make_tokens(1, 90 + i, (L,), shape.vocab) for i, L in enumerate(lens)]
    orc = Oracle(shape, W.values)
    obs = orc.prefill(prompts, run_boundary=True)
    sess = make_session(shape, W, max_batch=2, max_pos=16400, max_prompt=16385)
    sess.k_pages.fill_(0xFF)
    sess.v_pages.fill_(0xFF)
    t = sess.prefill(prompts, run_boundary=True)
    check_readout(t, obs, BF16_TOL, "boundary 16384/16385")
    toks = [o["next"] for o in obs]
    outs = orc.decode_step(tokens=toks)
    t = sess.decode(tokens=toks)
    check_readout(t, outs, BF16_TOL, "step 16384/16385")
