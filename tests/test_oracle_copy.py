"""Pins for the oracle's retrieve scatter and store gather.

The oracle walks every byte with its own index arithmetic.  It is checked
against independent routes to the same result:
  * numpy advanced indexing on the reshaped layouts
    (paged.view(2, NB, B, H, D)[kv, ids] = slot.view(L, 2, C/B, B, H, D)[l, kv]);
  * with B == C, a single chunk and an identity table, a contiguous copy;
  * store followed by retrieve into fresh blocks is the identity;
  * blocks no job targets keep their sentinel bytes;
  * jobs or block ids out of range touch nothing;
  * the one-by-one source functions agree with the full copies.
"""
import itertools

import numpy as np
import pytest

import oracle
from workloads import KVShape


def _split(layout):
    """'kv_first', 'block_first', or either with '+<pad>' bytes after every segment."""
    name, _, pad = layout.partition("+")
    return name, int(pad or 0)


def _setup(seed, L, H, D, e, B, C, layout, num_reqs=3, chunks_per_req=3, spare=5, nslots=6):
    rng = np.random.default_rng(seed)
    shape = KVShape(L, H, D, e, B, C)
    nseg = C // B
    nb = num_reqs * chunks_per_req * nseg + spare
    name, pad = _split(layout)
    seg = shape.seg_bytes + pad
    if name == "kv_first":
        kv_stride, block_stride = nb * seg, seg
    else:
        kv_stride, block_stride = seg, 2 * seg
    lo = oracle.make_layout(shape, nb, nslots, kv_stride, block_stride)
    perm = rng.permutation(nb).astype(np.int32)
    bt = perm[:num_reqs * chunks_per_req * nseg].reshape(num_reqs, chunks_per_req * nseg).copy()
    staging = rng.integers(0, 256, nslots * shape.slot_bytes, dtype=np.uint8)
    layers = [rng.integers(0, 256, 2 * nb * seg, dtype=np.uint8) for _ in range(L)]
    return shape, lo, bt, staging, layers, nb


def _paged_view(layer, shape, nb, layout):
    """[2, NB, B, H, D, e] view (writes go through to ``layer``); padding
    bytes are outside the view."""
    B, H, D, e = shape.block_size, shape.kv_heads, shape.head_dim, shape.elem_bytes
    name, pad = _split(layout)
    seg = shape.seg_bytes
    if name == "kv_first":
        v = layer.reshape(2, nb, seg + pad)[:, :, :seg]
    else:
        v = layer.reshape(nb, 2, seg + pad)[:, :, :seg].transpose(1, 0, 2)
    v = v.reshape(2, nb, B, H, D, e) if pad == 0 and name == "kv_first" else \
        np.lib.stride_tricks.as_strided(v, (2, nb, B, H, D, e), v.strides[:2] + (H * D * e, D * e, e, 1))
    assert np.shares_memory(v, layer)
    return v


SHAPES = [(1, 1, 64, 2, 16, 16), (2, 2, 64, 2, 16, 64), (3, 8, 128, 2, 16, 32),
          (2, 1, 128, 4, 32, 128), (1, 2, 64, 1, 32, 32), (2, 8, 64, 2, 16, 256)]
LAYOUTS = ["kv_first", "block_first", "kv_first+4096", "block_first+48"]


@pytest.mark.parametrize("shape_args,layout", list(itertools.product(SHAPES, LAYOUTS)))
def test_scatter_matches_numpy_indexing(shape_args, layout):
    shape, lo, bt, staging, layers, nb = _setup(11, *shape_args, layout)
    L, C, B = shape.num_layers, shape.chunk_tokens, shape.block_size
    nseg = C // B
    jobs = np.array([[4, 0, 0, 0], [1, 2, 1, 0], [4, 1, 2, 0], [0, 2, 0, 0]], np.int32)
    ref = [a.copy() for a in layers]
    for slot, r, j, _ in jobs:
        chunk = staging[slot * shape.slot_bytes:(slot + 1) * shape.slot_bytes].reshape(
            L, 2, nseg, B, shape.kv_heads, shape.head_dim, shape.elem_bytes)
        ids = bt[r, j * nseg:(j + 1) * nseg]
        for l in range(L):
            pv = _paged_view(ref[l], shape, nb, layout)
            for kv in range(2):
                pv[kv, ids] = chunk[l, kv]
    out = [a.copy() for a in layers]
    oracle.retrieve_scatter(lo, staging, out, bt, jobs)
    for a, b in zip(out, ref):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("shape_args,layout", list(itertools.product(SHAPES, LAYOUTS)))
def test_gather_matches_numpy_indexing(shape_args, layout):
    shape, lo, bt, staging, layers, nb = _setup(12, *shape_args, layout)
    L, C, B = shape.num_layers, shape.chunk_tokens, shape.block_size
    nseg = C // B
    jobs = np.array([[5, 0, 1, 0], [2, 2, 2, 0], [3, 1, 0, 0]], np.int32)
    ref = staging.copy()
    for slot, r, j, _ in jobs:
        chunk = ref[slot * shape.slot_bytes:(slot + 1) * shape.slot_bytes].reshape(
            L, 2, nseg, B, shape.kv_heads, shape.head_dim, shape.elem_bytes)
        ids = bt[r, j * nseg:(j + 1) * nseg]
        for l in range(L):
            pv = _paged_view(layers[l], shape, nb, layout)
            for kv in range(2):
                chunk[l, kv] = pv[kv, ids]
    out = staging.copy()
    oracle.store_gather(lo, out, layers, bt, jobs)
    assert np.array_equal(out, ref)


def test_block_equals_chunk_identity_table_is_memcpy():
    # B == C, one layer, block_first layout with one block: the paged block
    # [2][B][H][D] and the slot [1][2][C][H][D] are the same bytes.
    rng = np.random.default_rng(3)
    shape = KVShape(1, 2, 64, 2, 64, 64)
    seg = shape.seg_bytes
    lo = oracle.make_layout(shape, 1, 1, seg, 2 * seg)
    staging = rng.integers(0, 256, shape.slot_bytes, dtype=np.uint8)
    layer = np.zeros(2 * seg, np.uint8)
    oracle.retrieve_scatter(lo, staging, [layer], np.array([[0]], np.int32), np.array([[0, 0, 0, 0]], np.int32))
    assert np.array_equal(layer, staging)
    back = np.zeros_like(staging)
    oracle.store_gather(lo, back, [layer], np.array([[0]], np.int32), np.array([[0, 0, 0, 0]], np.int32))
    assert np.array_equal(back, staging)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_store_then_retrieve_roundtrip_and_sentinels(layout):
    shape, lo, bt, staging, layers, nb = _setup(21, 2, 2, 64, 2, 16, 64, layout, num_reqs=4,
                                                 chunks_per_req=2, spare=7, nslots=8)
    nseg = shape.blocks_per_chunk
    store_jobs = np.array([[s, s // 2, s % 2, 0] for s in range(8)], np.int32)
    st = np.zeros_like(staging)
    oracle.store_gather(lo, st, layers, bt, store_jobs)
    # fresh pool with a sentinel and fresh (re-permuted) tables
    rng = np.random.default_rng(99)
    perm = rng.permutation(nb).astype(np.int32)
    bt2 = perm[:bt.size].reshape(bt.shape).copy()
    sentinel = [np.full_like(a, 0xA5) for a in layers]
    oracle.retrieve_scatter(lo, st, sentinel, bt2, store_jobs)
    touched = set(int(x) for x in bt2.ravel())
    for l in range(shape.num_layers):
        got = _paged_view(sentinel[l], shape, nb, layout)
        orig = _paged_view(layers[l], shape, nb, layout)
        for r in range(bt.shape[0]):
            for c in range(bt.shape[1]):
                for kv in range(2):
                    assert np.array_equal(got[kv, bt2[r, c]], orig[kv, bt[r, c]])
        for blk in range(nb):
            if blk not in touched:
                assert np.all(got[:, blk] == 0xA5)
        # padding between segments is never written
        name, pad = _split(layout)
        if pad:
            seg = shape.seg_bytes
            rows = sentinel[l].reshape(-1, seg + pad)
            assert np.all(rows[:, seg:] == 0xA5)


def test_out_of_range_jobs_and_blocks_touch_nothing():
    shape, lo, bt, staging, layers, nb = _setup(31, 2, 2, 64, 2, 16, 64, "kv_first")
    bt = bt.copy()
    bt[0, 1] = -1            # unassigned block
    bt[0, 2] = nb            # past the pool
    # chunk = INT32_MAX: its end (chunk + 1) * C/B lies far past the table, however it is formed
    bad = np.array([[-1, 0, 0, 0], [6, 0, 0, 0], [0, -1, 0, 0], [0, 3, 0, 0],
                    [0, 0, -1, 0], [0, 0, 3, 0], [0, 0, 0x7FFFFFFF, 0], [0, 1, 0x3FFFFFFF, 0]], np.int32)
    out = [a.copy() for a in layers]
    oracle.retrieve_scatter(lo, staging, out, bt, bad)
    assert all(np.array_equal(a, b) for a, b in zip(out, layers))
    st = staging.copy()
    oracle.store_gather(lo, st, layers, bt, bad)
    assert np.array_equal(st, staging)
    # a valid job whose table has two bad entries copies the other segments only
    good = np.array([[2, 0, 0, 0]], np.int32)
    out = [a.copy() for a in layers]
    oracle.retrieve_scatter(lo, staging, out, bt, good)
    seg = shape.seg_bytes
    for l in range(2):
        v = out[l].reshape(2, nb, seg)
        base = layers[l].reshape(2, nb, seg)
        s = staging[2 * shape.slot_bytes:3 * shape.slot_bytes].reshape(2, 2, 4, seg)
        for i in range(4):
            blk = bt[0, i]
            if 0 <= blk < nb:
                assert np.array_equal(v[:, blk], s[l, :, i])
        changed = [b for b in range(nb) if not np.array_equal(v[:, b], base[:, b])]
        assert set(changed) <= {int(bt[0, 0]), int(bt[0, 3])}


@pytest.mark.parametrize("repeat", [False, True])
def test_one_by_one_sources_agree_with_full_copies(repeat):
    # repeat: a later job names the destination of an earlier one (the same blocks for the scatter, the same
    # slot for the gather); in the full copies the later job's bytes land last, and the one-by-one forms must
    # name the later job too
    shape, lo, bt, staging, layers, nb = _setup(41, 2, 2, 64, 2, 16, 64, "block_first")
    nseg = shape.blocks_per_chunk
    jobs = np.array([[3, 0, 2, 0], [1, 1, 0, 0], [3, 2, 1, 0]] + ([[4, 1, 0, 0]] if repeat else []), np.int32)
    out = [np.zeros_like(a) for a in layers]
    oracle.retrieve_scatter(lo, staging, out, bt, jobs)
    seg = shape.seg_bytes
    for l in range(2):
        pv = _paged_view(out[l], shape, nb, "block_first").reshape(2, nb, seg)
        for kv in range(2):
            for blk in range(nb):
                src = oracle.scatter_source(lo, bt, jobs, l, kv, blk)
                if src is None:
                    assert np.all(pv[kv, blk] == 0)
                else:
                    assert np.array_equal(pv[kv, blk], staging[src:src + seg])
    sj = np.array([[5, 2, 2, 0], [0, 0, 1, 0]] + ([[5, 1, 1, 0]] if repeat else []), np.int32)
    st = np.zeros_like(staging)
    oracle.store_gather(lo, st, layers, bt, sj)
    for slot in range(6):
        s = st[slot * shape.slot_bytes:(slot + 1) * shape.slot_bytes].reshape(2, 2, nseg, seg)
        for i in range(nseg):
            blk = oracle.gather_source(lo, bt, sj, slot, i)
            for l in range(2):
                pv = _paged_view(layers[l], shape, nb, "block_first").reshape(2, nb, seg)
                for kv in range(2):
                    if blk is None:
                        assert np.all(s[l, kv, i] == 0)
                    else:
                        assert np.array_equal(s[l, kv, i], pv[kv, blk])


def test_bit_patterns_are_opaque():
    # Every 16-bit pattern, NaN payloads and denormals included, survives.
    shape = KVShape(1, 2, 64, 2, 16, 16)
    seg = shape.seg_bytes
    n_slots = (65536 * 2) // shape.slot_bytes
    lo = oracle.make_layout(shape, n_slots, n_slots, n_slots * seg, seg)
    staging = np.arange(65536, dtype=np.uint16).view(np.uint8).copy()
    bt = np.arange(n_slots, dtype=np.int32)[::-1].reshape(n_slots, 1).copy()
    jobs = np.array([[s, s, 0, 0] for s in range(n_slots)], np.int32)
    layer = np.zeros(2 * n_slots * seg, np.uint8)
    oracle.retrieve_scatter(lo, staging, [layer], bt, jobs)
    back = np.zeros_like(staging)
    oracle.store_gather(lo, back, [layer], bt, jobs)
    assert np.array_equal(back, staging)


@pytest.mark.parametrize("shape_args,layout", list(itertools.product(SHAPES, LAYOUTS)))
def test_one_layer_walks_agree_with_full_walks(shape_args, layout):
    # the one-layer forms (used for complete checks at full size, one layer at a time) give, layer by layer,
    # what the full walks give, including skipped jobs and blocks and a slot read by several jobs
    shape, lo, bt, staging, layers, nb = _setup(61, *shape_args, layout)
    bt = bt.copy()
    bt[1, 0] = -1
    bt[2, 1] = nb
    L, S = shape.num_layers, lo.num_slots
    part = oracle.layer_part_bytes(lo)
    assert part * L == shape.slot_bytes
    retr = np.array([[4, 0, 0, 0], [1, 2, 1, 0], [4, 1, 2, 0], [0, 1, 0, 0], [9, 0, 1, 0], [2, 0, 7, 0]], np.int32)
    store = np.array([[5, 2, 2, 0], [3, 1, 1, 0], [0, 0, 2, 0], [1, 5, 0, 0]], np.int32)
    full = [a.copy() for a in layers]
    oracle.retrieve_scatter(lo, staging, full, bt, retr)
    st_full = staging.copy()
    oracle.store_gather(lo, st_full, full, bt, store)
    by_layer = staging.reshape(S, L, part)
    out_by_layer = st_full.reshape(S, L, part)
    for l in range(L):
        stg_l = np.ascontiguousarray(by_layer[:, l, :])
        paged = layers[l].copy()
        oracle.retrieve_scatter_layer(lo, stg_l, paged, bt, retr)
        assert np.array_equal(paged, full[l]), l
        oracle.store_gather_layer(lo, stg_l, paged, bt, store)
        assert np.array_equal(stg_l, out_by_layer[:, l, :]), l
