"""Long-context decode at full size: one 8B-shape layer, batch 8, cache
lengths uniform in [16384, 32768], 64 consecutive grouped steps that append
only primary keys/values.  Every sequence is followed by the oracle through
all 64 steps (two sequences per test); every sequence's cache length and
page table are checked."""
import numpy as np
import pytest

import synth
from oracle import Oracle, PageAllocator
from tests.gpu_util import make_session, row_err

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


@pytest.fixture(scope="module")
def longctx_run():
    """The 64 GPU steps of the whole batch: per-step final states of every
    sequence, then the cache lengths and page tables against the allocator
    the oracle uses."""
    w = synth.workload("longctx_bf16")
    shape = w["shape"]
    B, steps = w["batch"], w["steps"]
    lengths = synth.make_lengths(4, B, w["len_lo"], w["len_hi"])
    W = synth.make_weights(shape, seed=0)
    max_pos = int(lengths.max()) + steps + 1
    sess = make_session(shape, W, max_batch=B, max_pos=max_pos)
    alloc = PageAllocator(sess.num_pages, 16)
    for b, L in enumerate(lengths):
        (_, kb), (_, vb) = synth.make_kv(shape, 0, b, int(L), seed=3)
        sess.reserve_fill(b, [kb], [vb])
        alloc.reserve(b, int(L))
    from paper_2608_12385_amd import binding
    h1s, h2s = [], []
    for step in range(steps):
        h = synth.make_hidden(shape, B, step=step, seed=2)
        t = sess.decode(h1=h[0], h2=h[1])
        for b in range(B):
            alloc.append_one(b)
        h1s.append(t["h1_out"].cpu().numpy().copy())
        h2s.append(t["h2_out"].cpu().numpy().copy())
    for b in range(B):
        assert binding.dbt_kv_length(sess.kv, b) == lengths[b] + steps
        assert binding.dbt_kv_pages(sess.kv, b) == alloc.table[b]
    dev_tab = sess.page_table.cpu().numpy()
    for b in range(B):
        np.testing.assert_array_equal(dev_tab[b, :len(alloc.table[b])], alloc.table[b])
    sess.close()
    return shape, W, lengths, np.stack(h1s), np.stack(h2s)


@pytest.mark.slow
@pytest.mark.timeout(600)
@pytest.mark.parametrize("rows", [(0, 1), (2, 3), (4, 5), (6, 7)])
def test_longctx_64_steps_every_sequence(longctx_run, rows):
    shape, W, lengths, h1s, h2s = longctx_run
    B = len(lengths)
    orc = Oracle(shape, W.values)
    for b in rows:
        (kv_, _), (vv_, _) = synth.make_kv(shape, 0, b, int(lengths[b]), seed=3)
        orc.kv_fill(b, int(lengths[b]), [kv_], [vv_])
    for step in range(h1s.shape[0]):
        h = synth.make_hidden(shape, B, step=step, seed=2)
        outs = [orc.step_one(b, h1=h[0, b], h2=h[1, b]) for b in rows]
        assert row_err(h1s[step][list(rows)], np.stack([o["h1"] for o in outs])).max() <= BF16_TOL, step
        assert row_err(h2s[step][list(rows)], np.stack([o["h2"] for o in outs])).max() <= BF16_TOL, step
