"""The C-ABI library loads, exports every symbol include/dbt.h declares, and
its host-only calls (config checks, workspace sizing, the page allocator)
behave as documented.  No device memory is touched: host-only calls never
dereference device pointers, so placeholder addresses are passed."""
import json
import os
import re
import subprocess

import pytest

from paper_2608_12385_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dbt.h")
FAKE = 1 << 40   # placeholder device address (256-byte aligned, never dereferenced)


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dbt_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (dbt_\w+)", out))
    declared = _declared()
    assert declared, "no declarations parsed"
    assert set(declared) <= exported, set(declared) - exported
    assert set(declared) == set(B.exported_symbols())
    for name in declared:
        assert getattr(lib, name) is not None


def _cfg(**kw):
    base = dict(n_layers=2, d_model=48, n_q_heads=4, n_kv_heads=2, head_dim=16, d_ff=96, vocab=64,
                dtype=B.DBT_F32, has_embeddings=1, max_batch=4, max_pos=256, max_prompt=64,
                rms_eps=1e-5, rope_theta=1e4)
    base.update(kw)
    return B.dbt_config(**base)


def _fake_weights(cfg):
    layers = (B.dbt_layer_weights * cfg.n_layers)()
    for l in range(cfg.n_layers):
        for f, _ in B.dbt_layer_weights._fields_:
            setattr(layers[l], f, FAKE)
    return B.dbt_weights(emb1=FAKE, emb2=FAKE, emb_norm=FAKE, final_norm=FAKE, lm_head=FAKE, h_layers=layers), layers


def test_config_checks():
    assert B.dbt_workspace_bytes(_cfg()) > 0
    for bad, status in [(dict(n_q_heads=3), 2), (dict(dtype=7), 1), (dict(max_batch=0), 1),
                        (dict(n_experts=4, d_ff_expert=32, top_k1=2, top_k2=2), 5),
                        (dict(dtype=B.DBT_BF16), 5), (dict(n_q_heads=36, n_kv_heads=2), 5),
                        (dict(max_prompt=300), 2)]:
        assert B.dbt_workspace_bytes(_cfg(**bad)) == 0, bad
        w, _keep = _fake_weights(_cfg())
        with pytest.raises(B.DbtError) as e:
            B.dbt_create(_cfg(**bad), w, FAKE)
        assert e.value.status == status, (bad, e.value)
    # bf16 shapes the kernels support
    ok = _cfg(dtype=B.DBT_BF16, d_model=512, n_q_heads=4, n_kv_heads=2, head_dim=128, d_ff=1024, vocab=512)
    assert B.dbt_workspace_bytes(ok) > 0
    # a layer stack without output matrix or embeddings (hidden states in and
    # out), at several batch caps: sizing must not depend on a nonzero vocab
    for mb in (1, 3, 64):
        hid = _cfg(dtype=B.DBT_BF16, d_model=512, n_q_heads=4, n_kv_heads=2, head_dim=128, d_ff=1024,
                   vocab=0, has_embeddings=0, max_prompt=0, max_batch=mb)
        assert B.dbt_workspace_bytes(hid) > 0, mb


def test_branch_count_checks():
    """More decode branches (App. C.1): 0..3 (0 reads as one), dense MLPs only,
    and every branch's query heads of a KV group must fit the attention tile
    ((1 + n_branches) * n_q / n_kv <= 16)."""
    bf = dict(dtype=B.DBT_BF16, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=1024, vocab=512)
    one = B.dbt_workspace_bytes(_cfg(**bf, n_branches=1))
    assert one > 0 and B.dbt_workspace_bytes(_cfg(**bf, n_branches=0)) == one
    # three branches: 4 paths x 4 query heads per KV head = 16 rows; more rows need more workspace
    assert B.dbt_workspace_bytes(_cfg(**bf, n_branches=3)) > one
    w, _keep = _fake_weights(_cfg())
    for bad, status in [(dict(bf, n_branches=4), 1), (dict(bf, n_branches=-1), 1),
                        (dict(bf, n_branches=3, n_q_heads=16, n_kv_heads=2), 5),
                        (dict(bf, n_branches=2, n_experts=4, d_ff_expert=128, top_k1=2, top_k2=2,
                              d_model=512, d_ff=0), 5)]:
        assert B.dbt_workspace_bytes(_cfg(**bad)) == 0, bad
        with pytest.raises(B.DbtError) as e:
            B.dbt_create(_cfg(**bad), w, FAKE)
        assert e.value.status == status, (bad, e.value)


def test_create_rejects_null_and_misaligned():
    cfg = _cfg()
    w, _keep = _fake_weights(cfg)
    with pytest.raises(B.DbtError) as e:
        B.dbt_create(cfg, w, FAKE + 4)
    assert e.value.status == 1
    w.lm_head = 0
    with pytest.raises(B.DbtError):
        B.dbt_create(cfg, w, FAKE)


def test_page_allocator_script_through_abi():
    """Same hand-written script as the oracle's allocator pin."""
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "page_script.json")))
    cfg = _cfg()
    w, _keep = _fake_weights(cfg)
    m = B.dbt_create(cfg, w, FAKE)
    kv = B.dbt_kv_create(m, FAKE, FAKE, g["num_pages"], FAKE, 16)
    length = {}
    try:
        for op in g["ops"]:
            b = op["b"]
            if op["op"] == "reserve":
                B.dbt_kv_reserve(kv, b, op["len"])
            elif op["op"] == "append":   # one continuation position, as a decode step takes it
                n = B.dbt_kv_length(kv, b)
                assert n == op["pos"]
                B.dbt_kv_reserve(kv, b, n + 1)
            else:
                B.dbt_kv_truncate(kv, b, op["len"])
            for bb, tab in op["expect"].items():
                assert B.dbt_kv_pages(kv, int(bb)) == tab, (op, bb)
        # errors leave state unchanged
        before = [B.dbt_kv_pages(kv, b) for b in range(4)]
        with pytest.raises(B.DbtError) as e:
            B.dbt_kv_reserve(kv, 0, 16 * 12)
        assert e.value.status == 3
        with pytest.raises(B.DbtError):
            B.dbt_kv_truncate(kv, 0, 10 ** 6)
        with pytest.raises(B.DbtError):
            B.dbt_kv_reserve(kv, 9, 1)
        assert [B.dbt_kv_pages(kv, b) for b in range(4)] == before
    finally:
        B.dbt_kv_destroy(kv)
        B.dbt_destroy(m)
    del length


def test_boundary_without_prefill_is_state_error():
    cfg = _cfg()
    w, _keep = _fake_weights(cfg)
    m = B.dbt_create(cfg, w, FAKE)
    kv = B.dbt_kv_create(m, FAKE, FAKE, 64, FAKE, 16)
    try:
        out = B.dbt_step_out()
        with pytest.raises(B.DbtError) as e:
            B.dbt_boundary(m, kv, 1, out, 0)
        assert e.value.status == 4
        # decode with a batch beyond max_batch: argument error before any device work
        sin = B.dbt_step_in(tokens=FAKE, batch=9)
        with pytest.raises(B.DbtError) as e:
            B.dbt_decode_step(m, kv, sin, 1, out, 0)
        assert e.value.status == 1
    finally:
        B.dbt_kv_destroy(kv)
        B.dbt_destroy(m)


def test_degenerate_calls_rejected_without_state_change():
    """Empty batches and prompts, a batch above max_batch, a prompt above
    max_prompt, a step past max_pos, a non-empty sequence given to prefill and
    an exhausted page pool are rejected with their documented status before
    any device work, and leave every length and page table as it was."""
    cfg = _cfg(max_pos=64)
    w, _keep = _fake_weights(cfg)
    m = B.dbt_create(cfg, w, FAKE)
    kv = B.dbt_kv_create(m, FAKE, FAKE, 9, FAKE, 16)   # 9 pages of 16 positions
    try:
        B.dbt_kv_reserve(kv, 0, 64)     # at max_pos: 4 pages
        B.dbt_kv_reserve(kv, 1, 32)     # 2 pages, a step needs a new page
        B.dbt_kv_reserve(kv, 2, 48)     # 3 pages: the pool is empty
        state = lambda: [(B.dbt_kv_length(kv, b), B.dbt_kv_pages(kv, b)) for b in range(4)]
        before = state()
        out = B.dbt_step_out()

        def status(fn, *a):
            with pytest.raises(B.DbtError) as e:
                fn(*a)
            assert state() == before, fn.__name__
            return e.value.status

        for batch in (0, -1, 5):
            sin = B.dbt_step_in(tokens=FAKE, batch=batch)
            assert status(B.dbt_decode_step, m, kv, sin, 1, out, 0) == 1
            assert status(B.dbt_decode_step_ungrouped, m, kv, sin, out, 0) == 1
        assert status(B.dbt_prefill, m, kv, FAKE, [], 0, 1, out, 0) == 1
        # sequence 0 is at max_pos: no room for another position
        assert status(B.dbt_decode_step, m, kv, B.dbt_step_in(tokens=FAKE, batch=1), 1, out, 0) == 2
        # prompts: empty, longer than max_prompt, into a non-empty sequence
        B.dbt_kv_truncate(kv, 0, 0)
        before = state()
        assert status(B.dbt_prefill, m, kv, FAKE, [0], 1, 1, out, 0) == 2
        assert status(B.dbt_prefill, m, kv, FAKE, [cfg.max_prompt + 1], 1, 1, out, 0) == 2
        assert status(B.dbt_prefill, m, kv, FAKE, [5, 5], 2, 1, out, 0) == 4
        # the truncation freed four pages; two more taken leave two free,
        # while sequences at 16, 32, 48 and 16 positions need four
        B.dbt_kv_reserve(kv, 3, 16)
        B.dbt_kv_reserve(kv, 0, 16)
        before = state()
        sin = B.dbt_step_in(tokens=FAKE, batch=4)
        assert status(B.dbt_decode_step, m, kv, sin, 1, out, 0) == 3
        assert status(B.dbt_decode_step_ungrouped, m, kv, sin, out, 0) == 3
    finally:
        B.dbt_kv_destroy(kv)
        B.dbt_destroy(m)


def test_noalloc_step_rejects_models_whose_step_buffers_exceed_the_static_scratch():
    """The allocation-free step refuses, before touching the GPU or any
    state, a model whose step buffers exceed the library's static array:
    64 sequences of a 128256-entry vocabulary need 128 rows of logits
    alone (62.6 MiB)."""
    big = _cfg(dtype=B.DBT_BF16, n_layers=1, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
               d_ff=14336, vocab=128256, has_embeddings=0, max_batch=64, max_pos=4112, max_prompt=0)
    assert B.dbt_workspace_bytes(big) > 0
    w, _keep = _fake_weights(big)
    m = B.dbt_create(big, w, FAKE)
    kv = B.dbt_kv_create(m, FAKE, FAKE, 64 * 257, FAKE, 257)
    sin = B.dbt_step_in(tokens=0, h1_in=FAKE, h2_in=FAKE, batch=4)
    out = B.dbt_step_out()
    with pytest.raises(B.DbtError) as e:
        B.dbt_decode_step_noalloc(m, kv, sin, 1, out, 0)
    assert e.value.status == 5 and "static scratch" in str(e.value), e.value
    assert B.dbt_kv_length(kv, 0) == 0
    B.dbt_kv_destroy(kv)
    B.dbt_destroy(m)
