"""Long-context decode at full size: one 8B-shape layer, batch 8, cache
lengths uniform in [16384, 32768], 64 consecutive grouped steps that append
only primary keys/values.  Two sequences are followed by the oracle through
all 64 steps; every sequence's cache length and page table are checked."""
import numpy as np
import pytest

import synth
from oracle import Oracle, PageAllocator
from tests.gpu_util import make_session, row_err

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


@pytest.mark.slow
def test_longctx_64_steps_sampled():
    w = synth.workload("longctx_bf16")
    shape = w["shape"]
    B, steps = w["batch"], w["steps"]
    lengths = synth.make_lengths(4, B, w["len_lo"], w["len_hi"])
    W = synth.make_weights(shape, seed=0)
    max_pos = int(lengths.max()) + steps + 1
    sess = make_session(shape, W, max_batch=B, max_pos=max_pos)
    sample = [0, 5]
    orc = Oracle(shape, W.values)
    alloc = PageAllocator(sess.num_pages, 16)
    for b, L in enumerate(lengths):
        (kv_, kb), (vv_, vb) = synth.make_kv(shape, 0, b, int(L), seed=3)
        sess.reserve_fill(b, [kb], [vb])
        alloc.reserve(b, int(L))
        if b in sample:
            orc.kv_fill(b, int(L), [kv_], [vv_])
    from paper_2608_12385_amd import binding
    for step in range(steps):
        h = synth.make_hidden(shape, B, step=step, seed=2)
        t = sess.decode(h1=h[0], h2=h[1])
        for b in range(B):
            alloc.append_one(b)
        outs = [orc.step_one(b, h1=h[0, b], h2=h[1, b]) for b in sample]
        g1 = t["h1_out"].cpu().numpy()[sample]
        g2 = t["h2_out"].cpu().numpy()[sample]
        assert row_err(g1, np.stack([o["h1"] for o in outs])).max() <= BF16_TOL, step
        assert row_err(g2, np.stack([o["h2"] for o in outs])).max() <= BF16_TOL, step
    for b in range(B):
        assert binding.dbt_kv_length(sess.kv, b) == lengths[b] + steps
        assert binding.dbt_kv_pages(sess.kv, b) == alloc.table[b]
    dev_tab = sess.page_table.cpu().numpy()
    for b in range(B):
        np.testing.assert_array_equal(dev_tab[b, :len(alloc.table[b])], alloc.table[b])
    sess.close()
