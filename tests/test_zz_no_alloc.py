"""The allocation-free step (dbt_decode_step_noalloc, step buffers in the
library's static device array) against dbt_decode_step through the C ABI:
outputs and cache bit-identical, on two calls in a row, the second with a
smaller batch."""
import numpy as np
import pytest

import synth
from tests.gpu_util import fill_cache, make_session, to_np

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _shape(moe):
    if moe:
        return synth.ModelShape(n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=0,
                                vocab=512, dtype="bf16", has_embeddings=False, n_experts=16, d_ff_expert=256,
                                n_shared_experts=1, d_ff_shared=256, top_k1=2, top_k2=4, std=0.05,
                                coupling_std=0.5)
    return synth.ModelShape(n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=1024,
                            vocab=1024, dtype="bf16", has_embeddings=False, std=0.05, coupling_std=0.5)


def _call(sess, fn, B, h, branch_on):
    from paper_2608_12385_amd import binding
    h1 = torch.as_tensor(np.ascontiguousarray(h[0, :B])).to(sess.device)
    h2 = torch.as_tensor(np.ascontiguousarray(h[1, :B])).to(sess.device)
    sin = sess.step_in(B, None, h1, h2)
    out, t = sess.outputs(B, routing=True)
    getattr(binding, fn)(sess.model, sess.kv, sin, int(branch_on), out, sess.stream)
    torch.cuda.current_stream().synchronize()
    res = {k: to_np(v).copy() for k, v in t.items()}
    res["k"] = to_np(sess.k_pages).copy()
    res["v"] = to_np(sess.v_pages).copy()
    res["len"] = [binding.dbt_kv_length(sess.kv, b) for b in range(B)]
    return res


@pytest.mark.parametrize("moe", [False, True])
def test_noalloc_step_equals_decode_step_twice_second_smaller(moe):
    from paper_2608_12385_amd import binding
    shape = _shape(moe)
    W = synth.make_weights(shape, seed=0)
    lengths = [3, 40, 530, 16, 77, 1, 250, 64, 129, 15, 300, 31, 2, 17, 99, 512, 47, 8, 160, 33]
    sess = make_session(shape, W, max_batch=len(lengths), max_pos=600)
    sess.k_pages.zero_()
    sess.v_pages.zero_()
    fill_cache(sess, None, shape, lengths)
    for call, (B, branch_on) in enumerate(((20, True), (5, True), (5, False))):
        print(f"no-alloc call {call}: batch {B} branch_on {branch_on} moe {moe}", flush=True)
        h = synth.make_hidden(shape, 20, step=call, seed=2)
        ref = _call(sess, "dbt_decode_step", B, h, branch_on)
        for b in range(B):
            binding.dbt_kv_truncate(sess.kv, b, lengths[b])
        got = _call(sess, "dbt_decode_step_noalloc", B, h, branch_on)
        for b in range(B):
            binding.dbt_kv_truncate(sess.kv, b, lengths[b])
        keys = sorted(ref)
        if not branch_on:
            keys = [k for k in keys if k in ("logits1", "alpha", "next_token", "h1_out", "route_idx1", "route_w1",
                                             "route_logits1", "k", "v", "len")]
        for k in keys:
            np.testing.assert_array_equal(got[k], ref[k], err_msg=f"call {call} {k}")
        assert got["len"] == [L + 1 for L in lengths[:B]]
    sess.close()
