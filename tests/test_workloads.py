"""The synthetic workloads have the sizes the measurement plan states, and the
KV content formula agrees between its device (torch) and host (numpy) forms."""
import numpy as np
import pytest
import torch

import workloads as W


def test_shapes():
    assert W.SHAPE_32L.bytes_per_token == 128 * 1024          # 8 GiB for a 64k-token prefix
    assert W.SHAPE_80L.bytes_per_token == 320 * 1024
    assert W.SHAPE_TINY.bytes_per_token == 1024
    assert W.SHAPE_32L.seg_bytes == 32 * 1024
    assert W.SHAPE_32L.slot_bytes == 32 * 1024 * 1024
    assert W.SHAPE_80L.slot_bytes == 80 * 1024 * 1024


def test_tiny():
    w = W.tiny()
    assert w.num_reqs == 8 and np.all(w.lengths == 256)
    assert w.num_blocks == 128
    for r in range(8):
        assert np.array_equal(w.tokens[w.tok_off[r]:w.tok_off[r] + 128], w.prefix_streams[0][:128])
    assert sorted(w.block_tables.ravel().tolist()) == list(range(128))
    assert w.tokens.min() >= 0 and w.tokens.max() < 32000


def test_l32_uniform():
    w = W.l32_uniform()
    assert w.num_reqs == 64 and w.tokens.size == 262144
    assert w.num_blocks == 20480
    assert len(w.prestage_chunks) == 64 and w.num_slots == 576
    assert w.pool_bytes() == 40 * 2**30 and w.staged_bytes() == 18 * 2**30
    bt = w.block_tables
    assert bt.shape == (64, 256) and len(set(bt.ravel().tolist())) == 64 * 256


def test_single_prefix_64k():
    # a 64k-token prefix: 8 GiB of KV at 128 KiB/token, 12 GiB at 192 KiB/token
    assert W.SHAPE_48L.bytes_per_token == 192 * 1024
    for name, gib in (("l32-1x65536", 8), ("l48-1x65536", 12), ("l32-1x65536-host", 8)):
        w = W.make(name)
        assert w.num_reqs == 1 and w.tokens.size == 65536
        assert len(w.prestage_chunks) == 256 == w.num_slots
        assert w.staged_bytes() == gib * 2**30
        assert np.array_equal(w.tokens, w.prefix_streams[0])
        assert w.staging_in_host == name.endswith("-host")
        assert w.num_blocks == 5120 and len(set(w.block_tables.ravel().tolist())) == 4096


def test_layout_variants_of_the_64x4096_batch():
    base = W.make("l32-64x4096")
    for name, layout, pad in (("l32-64x4096-block_first", "block_first", 0), ("l32-64x4096-pad4096", "kv_first", 4096),
                              ("l48-64x4096", "kv_first", 0)):
        w = W.make(name)
        assert w.paged_layout == layout and w.block_pad == pad
        assert np.array_equal(w.tokens, base.tokens) and np.array_equal(w.block_tables, base.block_tables)
        seg = w.shape.seg_bytes + pad
        kvs, bs = w.strides()
        assert (kvs, bs) == ((w.num_blocks * seg, seg) if layout == "kv_first" else (seg, 2 * seg))
        assert w.layer_bytes() == 2 * w.num_blocks * seg
    assert W.make("l48-64x4096").staged_bytes() == 576 * 48 * 2**20
    assert W.make("l32-64x4096-pad4096").pool_bytes() == 40 * 2**30 * 36 // 32


def test_l80_long():
    w = W.l80_long()
    assert w.num_blocks == 18023 and w.num_slots == 1024
    assert len(w.prestage_chunks) == 768


def test_lognormal():
    for ratio in (0.25, 0.5, 0.75):
        w = W.l32_lognormal(ratio)
        assert w.num_reqs == 256
        assert w.lengths.min() >= 256 and w.lengths.max() <= 8192
        assert 1700 < w.lengths.mean() < 2300
        assert np.all(w.prefix_tokens % 256 == 0)


def test_capacity():
    full = W.l32_capacity(1.0, False)
    assert full.num_blocks == 72090
    assert np.all(full.prefix_tokens == 768)
    u = full.notes["unique_prefixes"]
    assert len(full.prestage_chunks) == 3 * u
    half = W.l32_capacity(0.5, False)
    quarter = W.l32_capacity(0.25, True)
    assert len(half.prestage_chunks) <= round(1.5 * u) and len(half.prestage_chunks) % 3 == 0
    assert len(quarter.prestage_chunks) <= round(0.75 * u) and quarter.staging_in_host


@pytest.mark.parametrize("finite", [True, False])
def test_fill_formula_device_form_matches_host_form(finite):
    buf = torch.empty(1 << 16, dtype=torch.uint8)
    W.fill_kv_(buf, 7, 3, finite=finite, chunk_words=1000)
    ref = W.kv_bytes_np(7, 3, 0, buf.numel(), finite=finite)
    assert np.array_equal(buf.numpy(), ref)
    # an offset window recomputes the same bytes
    assert np.array_equal(W.kv_bytes_np(7, 3, 4096, 512, finite), ref[4096:4096 + 512])
    if finite:
        halves = ref.view(np.uint16)
        assert np.all((halves & 0x4000) == 0)


def test_fill_formula_high_words():
    # Words past 2^32 (buffers over 16 GiB) use the high half of the index.
    a = W.kv_words_np(1, 1, (1 << 32) + 5, 4)
    b = W.kv_words_np(1, 1, 5, 4)
    assert not np.array_equal(a, b)


def test_random_shapes_respect_the_layout_rules():
    shapes = W.random_shapes(2026, 40)
    assert len(shapes) == 40 and len(set(shapes)) > 30
    for sh in shapes:
        assert sh.chunk_tokens % 16 == 0 and sh.chunk_tokens % sh.block_size == 0
        assert sh.seg_bytes % 16 == 0
    assert W.random_shapes(2026, 40) == shapes                      # seeded
    assert {sh.elem_bytes for sh in shapes} == {1, 2, 4}


def test_pool_holds_the_live_blocks_of_many_short_requests():
    # eight one-token requests with 32-token blocks: 8 live blocks, though 1.5 x 8 tokens fit in one block
    shape = W.KVShape(1, 1, 16, 2, 32, 32)
    w = W._assemble("short", shape, 1, [1] * 8, [-1] * 8, [0] * 8, 0, prestage=[], num_slots=4, pool_factor=1.5)
    assert w.num_blocks == 8
    assert sorted(w.block_tables[:, 0].tolist()) == list(range(8))
    # the configurations' pools are sized by their tokens as before
    assert W.make("l32-64x4096").num_blocks == 20480 and W.make("l80-32x8192").num_blocks == 18023
