"""GPU parity: the HIP path against the CPU oracle, bit for bit.

Every test runs the library through its C ABI (via the Python binding) and
the oracle on the same seeded inputs, and compares outputs exactly: block
hashes, lookup results, job lists, and every byte of the staging buffer and
the paged pool.  Inputs come from the workload generator only."""
import copy
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2609_35065_amd as kv
import workloads as W
from oracle.pipeline import OraclePath
from paper_2609_35065_amd.pipeline import StagingPath

pytestmark = pytest.mark.gpu

STG_TAG, POOL_TAG = 1, 1000


def _pair(w, kv_seed=None, finite=True, hash_seed=0):
    kv_seed = w.seed if kv_seed is None else kv_seed
    g = StagingPath(w, hash_seed=hash_seed)
    g.fill(STG_TAG, POOL_TAG, kv_seed, finite)
    g.prestage()
    o = OraclePath(w, hash_seed=hash_seed, kv_seed=kv_seed, finite=finite, staging_tag=STG_TAG,
                   pool_tag_base=POOL_TAG)
    o.prestage()
    return g, o


def _compare_pass(g, o, sg, so, check_kv=True):
    torch.cuda.synchronize()
    nblk = int(g.blk_off_h[-1])
    nch = int(g.chunk_off_h[-1])
    R = g.batch.num_reqs
    assert np.array_equal(g.h_block_hash.numpy()[:nblk].view(np.uint64), so["block_hash"])
    assert np.array_equal(g.h_chunk_slot.numpy()[:nch], so["chunk_slot"])
    assert np.array_equal(g.h_hit.numpy()[:R], so["hit"])
    assert np.array_equal(g.last_retrieve, so["retrieve"])
    assert np.array_equal(g.last_ordinary, so["ordinary"])
    assert np.array_equal(g.last_decisions, so["decisions"])
    assert np.array_equal(g.last_store, so["store"])
    assert sg.dropped == so["dropped"]
    if check_kv:
        assert np.array_equal(g.staging_view().cpu().numpy(), o.staging), "staging differs"
        for l in range(len(g.layers)):
            assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l]), f"layer {l} differs"


def _free(*objs):
    for x in objs:
        del x
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# tiny workload: store every chunk, then retrieve the hits
# ---------------------------------------------------------------------------

def test_tiny_store_all_then_retrieve_all():
    w = W.tiny()
    g, o = _pair(w)
    sg, so = g.run_pass(validate=True), o.run_pass()
    _compare_pass(g, o, sg, so)
    assert sg.num_retrieve == 0 and sg.num_store == 18      # 4 chunks of request 0, 2 private x 7
    # sentinel pool, fresh block tables, retrieve everything back
    for t in g.layers:
        t.fill_(0xA5)
    for a in o.layers:
        a[:] = 0xA5
    w2 = copy.deepcopy(w)
    W.repermute_block_tables(w2, 1)
    g.set_batch(w2)
    o.set_batch(w2)
    sg, so = g.run_pass(validate=True), o.run_pass()
    _compare_pass(g, o, sg, so)
    assert sg.num_retrieve == 32 and sg.num_store == 0
    assert all(np.all(so["hit"] == 4) for _ in [0])
    # the pool is exactly the live blocks, so no sentinel block remains
    for l in range(w.shape.num_layers):
        segs = g.layers[l].cpu().numpy().reshape(2, w.num_blocks, -1)
        assert not np.any(np.all(segs == 0xA5, axis=-1))


def test_tiny_store_one_request_then_partial_hits():
    w = W.tiny()
    w0 = copy.deepcopy(w)
    w0.tokens = w.tokens[:256].copy()
    w0.tok_off = np.array([0, 256], np.int64)
    w0.block_tables = w.block_tables[:1].copy()
    g, o = _pair(w)
    g.set_batch(w0)
    o.set_batch(w0)
    sg, so = g.run_pass(validate=True), o.run_pass()
    _compare_pass(g, o, sg, so)
    assert sg.num_store == 4
    for t in g.layers:
        t.fill_(0x5A)
    for a in o.layers:
        a[:] = 0x5A
    g.set_batch(w)
    o.set_batch(w)
    sg, so = g.run_pass(validate=True), o.run_pass()
    _compare_pass(g, o, sg, so)
    assert list(so["hit"]) == [4] + [2] * 7
    assert sg.num_retrieve == 18 and sg.num_store == 14
    # blocks no retrieve job wrote keep the sentinel
    written = set(int(b) for q in so["retrieve"] for b in
                  w.block_tables[q[1], q[2] * 4:(q[2] + 1) * 4])
    for l in range(w.shape.num_layers):
        segs = g.layers[l].cpu().numpy().reshape(2, w.num_blocks, -1)
        for blk in range(w.num_blocks):
            assert np.all(segs[:, blk] == 0x5A) == (blk not in written)


# ---------------------------------------------------------------------------
# random small workloads over shapes and layouts
# ---------------------------------------------------------------------------

# Segment sizes B*H*D*e cover every copy path: 4 KiB rows x 1, 2, 4, 8, 16 (retrieve) and 16/8/4 KiB rows
# (store), and sizes that are none of these (generic path); also fp8 and fp32 elements, a head size that is
# not a power of two, and the largest layer count a layout may name.
SHAPES = [W.KVShape(2, 2, 64, 2, 16, 64), W.KVShape(3, 1, 64, 2, 16, 16), W.KVShape(1, 8, 128, 2, 16, 256),
          W.KVShape(2, 2, 128, 2, 32, 128), W.KVShape(2, 1, 64, 1, 32, 32), W.KVShape(1, 2, 64, 4, 16, 64),
          W.KVShape(4, 8, 64, 2, 32, 512), W.KVShape(2, 1, 128, 2, 16, 16),
          W.KVShape(2, 8, 128, 2, 32, 64),        # 64 KiB segments
          W.KVShape(1, 3, 80, 4, 16, 32),         # 15 KiB segments, fp32, head size 80
          W.KVShape(2, 4, 128, 1, 16, 64),        # fp8 elements, 8 KiB segments
          W.KVShape(128, 1, 16, 2, 16, 16)]       # 128 layers of 512-byte segments


@pytest.mark.parametrize("layout,pad", [("kv_first", 0), ("block_first", 0), ("kv_first", 4096), ("block_first", 48)])
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_random_workloads(si, layout, pad):
    # pad: bytes between consecutive paged segments (padded block strides)
    shape = SHAPES[si]
    w = W.small_random(100 + si, shape, num_reqs=9, max_len=5 * shape.chunk_tokens + 37, paged_layout=layout,
                       block_pad=pad)
    g, o = _pair(w)
    for p in range(3):       # stores, then hits on what was stored, then an evicting pass
        evict = p == 2
        sg, so = g.run_pass(validate=True, evict_stored=evict), o.run_pass(evict_stored=evict)
        _compare_pass(g, o, sg, so)
    _free(g, o)


@pytest.mark.parametrize("k", range(40))
def test_random_shape_sweep(k):
    # Forty seeded shapes (layers, heads, head size, element size, block and chunk sizes drawn at random),
    # random paged layout and padding; two passes each, every byte compared.
    shape = W.random_shapes(2026, 40)[k]
    layout = "kv_first" if k % 2 == 0 else "block_first"
    pad = [0, 16, 4096, 48][k % 4]
    w = W.small_random(700 + k, shape, num_reqs=6, max_len=4 * shape.chunk_tokens + 23, paged_layout=layout,
                       block_pad=pad)
    g, o = _pair(w)
    for p in range(2):
        sg, so = g.run_pass(validate=True), o.run_pass()
        _compare_pass(g, o, sg, so)
    _free(g, o)


def test_raw_bit_patterns_nan_payloads():
    shape = W.KVShape(2, 2, 64, 2, 16, 64)
    w = W.small_random(7, shape, num_reqs=6, max_len=300)
    g, o = _pair(w, finite=False)
    sg, so = g.run_pass(validate=True), o.run_pass()
    _compare_pass(g, o, sg, so)
    sg, so = g.run_pass(validate=True), o.run_pass()
    _compare_pass(g, o, sg, so)
    halves = g.staging_view().cpu().numpy().view(np.uint16)
    assert np.any((halves & 0x7C00) == 0x7C00)              # fp16 Inf/NaN patterns were moved too


def test_slot_exhaustion_drops_misses():
    shape = W.KVShape(1, 2, 64, 2, 16, 32)
    w = W.small_random(9, shape, num_reqs=8, max_len=200, extra_slots=0)
    w.num_slots = len(w.prestage_chunks) + 3                  # only three free slots
    g, o = _pair(w)
    sg, so = g.run_pass(validate=True), o.run_pass()
    _compare_pass(g, o, sg, so)
    assert sg.num_store == 3 and sg.dropped > 0


# ---------------------------------------------------------------------------
# kernels one by one, edge cases
# ---------------------------------------------------------------------------

def _hash_gpu(toks, tok_off, seed):
    blk_off = oracle.block_offsets(tok_off)
    d_t = torch.from_numpy(toks if toks.size else np.zeros(1, np.int32)).cuda()
    d_o = torch.from_numpy(tok_off).cuda()
    d_b = torch.from_numpy(blk_off).cuda()
    out = torch.zeros(max(int(blk_off[-1]), 1), dtype=torch.int64, device="cuda")
    kv.kv_hash_prefix(d_t, d_o, tok_off.size - 1, seed, d_b, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()[:int(blk_off[-1])].view(np.uint64)


@pytest.mark.parametrize("seed", [0, 1, 0xFFFFFFFFFFFFFFFF, 0x0123456789ABCDEF])
def test_hash_ragged_lengths(seed):
    rng = np.random.default_rng(seed & 0xFFFF)
    lengths = list(range(0, 70)) + [255, 256, 257, 4095, 4096, 4097, 4112, 20000, 16 * 513]
    toks = rng.integers(-2**31, 2**31, sum(lengths), dtype=np.int64).astype(np.int32)
    tok_off = np.zeros(len(lengths) + 1, np.int64)
    np.cumsum(lengths, out=tok_off[1:])
    assert np.array_equal(_hash_gpu(toks, tok_off, seed), oracle.hash_prefix(toks, tok_off, seed))


def test_hash_many_requests():
    rng = np.random.default_rng(5)
    lengths = rng.integers(0, 700, 3000)
    toks = rng.integers(0, 32000, int(lengths.sum())).astype(np.int32)
    tok_off = np.zeros(lengths.size + 1, np.int64)
    np.cumsum(lengths, out=tok_off[1:])
    assert np.array_equal(_hash_gpu(toks, tok_off, 3), oracle.hash_prefix(toks, tok_off, 3))


def test_hash_empty_batch():
    kv.kv_hash_prefix(torch.zeros(1, dtype=torch.int32, device="cuda"), torch.zeros(1, dtype=torch.int64, device="cuda"),
                      0, 0, torch.zeros(1, dtype=torch.int64, device="cuda"),
                      torch.zeros(1, dtype=torch.int64, device="cuda"))
    torch.cuda.synchronize()


def _lookup_gpu(idx, bh, blk_off, bpc):
    chunk_off = oracle.chunk_offsets(blk_off, bpc)
    R = blk_off.size - 1
    d_bh = torch.from_numpy(bh.view(np.int64) if bh.size else np.zeros(1, np.int64)).cuda()
    cs = torch.full((max(int(chunk_off[-1]), 1),), -7, dtype=torch.int32, device="cuda")
    hit = torch.full((max(R, 1),), -7, dtype=torch.int32, device="cuda")
    kv.kv_lookup(idx, d_bh, torch.from_numpy(blk_off).cuda(), R, bpc, torch.from_numpy(chunk_off).cuda(), cs, hit)
    torch.cuda.synchronize()
    return cs.cpu().numpy()[:int(chunk_off[-1])], hit.cpu().numpy()[:R]


def test_lookup_long_runs_cross_wave_width():
    rng = np.random.default_rng(11)
    base = rng.integers(0, 32000, 16 * 200).astype(np.int32)
    reqs = [base, base[:16 * 64], base[:16 * 65], base[:16 * 63 + 5], base[:16 * 130], np.zeros(0, np.int32)]
    tok_off = np.zeros(len(reqs) + 1, np.int64)
    np.cumsum([r.size for r in reqs], out=tok_off[1:])
    toks = np.concatenate(reqs)
    bh = oracle.hash_prefix(toks, tok_off)
    blk_off = oracle.block_offsets(tok_off)
    keys = bh[blk_off[0]:blk_off[1]]
    idx = kv.KvIndex(400)
    ref = {}
    for n_idx in [0, 63, 64, 65, 128, 129, 200]:
        present = {int(k): i for i, k in enumerate(keys[:n_idx])}
        present[int(keys[150])] = 150                       # present after a miss for some requests
        add = {k: v for k, v in present.items() if k not in ref}
        if add:
            idx.insert(np.array(list(add.keys()), np.uint64), np.array(list(add.values()), np.int32))
            ref.update(add)
        cs, hit = _lookup_gpu(idx, bh, blk_off, 1)
        ocs, ohit = oracle.lookup(ref, bh, blk_off, 1)
        assert np.array_equal(cs, ocs) and np.array_equal(hit, ohit)
    idx.destroy()


def test_index_insert_erase_churn():
    rng = np.random.default_rng(12)
    toks = rng.integers(0, 32000, 16 * 3000).astype(np.int32)
    tok_off = np.array([0, toks.size], np.int64)
    bh = oracle.hash_prefix(toks, tok_off)
    blk_off = oracle.block_offsets(tok_off)
    keys = bh.copy()
    idx = kv.KvIndex(300)
    ref = {}
    for it in range(60):
        add = rng.choice(keys.size, 40, replace=False)
        cand = {int(keys[i]): int(rng.integers(0, 1000)) for i in add}
        room = 300 - len(ref)
        items = [(k, v) for k, v in cand.items() if k in ref] + \
                [(k, v) for k, v in cand.items() if k not in ref][:max(room, 0)]
        if items:
            idx.insert(np.array([k for k, _ in items], np.uint64), np.array([v for _, v in items], np.int32))
            ref.update(items)
        if ref:
            live = list(ref.keys())
            gone = [live[i] for i in rng.choice(len(live), min(len(live), 30), replace=False)]
            idx.erase(np.array(gone, np.uint64))
            for k in gone:
                ref.pop(k)
        assert idx.size() == len(ref)
        cs, hit = _lookup_gpu(idx, bh, blk_off, 1)
        ocs, ohit = oracle.lookup(ref, bh, blk_off, 1)
        assert np.array_equal(cs, ocs) and np.array_equal(hit, ohit)
    with pytest.raises(kv.KvError) as e:
        fresh = [int(k) for k in keys if int(k) not in ref][:400]
        idx.insert(np.array(fresh, np.uint64), np.zeros(len(fresh), np.int32))
    assert e.value.status == kv.KV_ENOSPC
    idx.destroy()


def test_index_updates_small_and_large_batches():
    # The device table follows the host table through incremental updates (few
    # changed entries) and whole-table uploads (many changes, rehash); batch
    # sizes straddle the incremental limit (an eighth of the table).
    rng = np.random.default_rng(21)
    toks = rng.integers(0, 32000, 16 * 9000).astype(np.int32)
    tok_off = np.array([0, toks.size], np.int64)
    bh = oracle.hash_prefix(toks, tok_off)
    blk_off = oracle.block_offsets(tok_off)
    keys = bh.copy()
    cap_entries = 4096                      # table of 8192 positions: incremental up to 1024 changes
    idx = kv.KvIndex(cap_entries)
    ref = {}
    for it, n in enumerate([1, 10, 1023, 1024, 1025, 3000, 5, 2000, 700, 1, 4096]):
        cand = {int(keys[i]): int(rng.integers(0, 1 << 20)) for i in rng.choice(keys.size, n, replace=False)}
        room = cap_entries - len(ref)
        items = [(k, v) for k, v in cand.items() if k in ref] + \
                [(k, v) for k, v in cand.items() if k not in ref][:max(room, 0)]
        if items:
            idx.insert(np.array([k for k, _ in items], np.uint64), np.array([v for _, v in items], np.int32))
            ref.update(items)
        cs, hit = _lookup_gpu(idx, bh, blk_off, 1)
        ocs, ohit = oracle.lookup(ref, bh, blk_off, 1)
        assert np.array_equal(cs, ocs) and np.array_equal(hit, ohit), ("insert", it, n)
        live = list(ref.keys())
        m = min(len(live), [0, 3, 500, 1024, 1100, 2500][it % 6])
        gone = [live[i] for i in rng.choice(len(live), m, replace=False)] if m else []
        if gone:
            idx.erase(np.array(gone, np.uint64))
            for k in gone:
                ref.pop(k)
        cs, hit = _lookup_gpu(idx, bh, blk_off, 1)
        ocs, ohit = oracle.lookup(ref, bh, blk_off, 1)
        assert np.array_equal(cs, ocs) and np.array_equal(hit, ohit), ("erase", it, m)
        assert idx.size() == len(ref)
    idx.destroy()


def test_index_large_table_update_limits():
    # A table of 2^21 positions (a million staged chunks): incremental uploads are capped at 65,536 changed
    # entries rather than an eighth of the table.  Inserts and erases at, just over and well under that cap
    # (incremental, whole image, incremental), each followed by a device lookup of every key.
    rng = np.random.default_rng(33)
    keys = np.unique(rng.integers(1, 2**63, 200000, dtype=np.int64)).astype(np.uint64)
    rng.shuffle(keys)
    idx = kv.KvIndex(1 << 20)
    ref = {}

    def check(tag):
        # one-block chunks in requests of 64 keys: every key's slot in chunk_slot, absent keys -1
        n = keys.size
        blk_off = np.arange(0, n + 64, 64, dtype=np.int64)
        blk_off[-1] = n
        cs, _ = _lookup_gpu(idx, keys, blk_off, 1)
        want = np.array([ref.get(int(k), -1) for k in keys], np.int32)
        assert np.array_equal(cs, want), tag
        assert idx.size() == len(ref), tag

    pos = 0
    for n in (16, 65536, 65537, 1000):     # the first upload of an index sends its whole table
        batch = keys[pos:pos + n]
        pos += n
        slots = rng.integers(0, 1 << 20, n).astype(np.int32)
        idx.insert(batch, slots)
        ref.update(zip((int(k) for k in batch), (int(s) for s in slots)))
        check(("insert", n))
    live = np.array(list(ref.keys()), np.uint64)
    for n in (65536, 65537, 10):
        gone = live[:n]
        live = live[n:]
        idx.erase(gone)
        for k in gone:
            ref.pop(int(k))
        check(("erase", n))
    idx.destroy()


def test_out_of_range_jobs_are_skipped_on_device():
    shape = W.KVShape(2, 2, 64, 2, 16, 64)
    w = W.small_random(21, shape, num_reqs=4, max_len=256)
    g, o = _pair(w)
    bt = w.block_tables.copy()
    bt[0, 1] = -1
    bt[0, 2] = w.num_blocks + 5
    d_bt = torch.from_numpy(bt).cuda()
    # chunk = INT32_MAX (and 2^30 - 1): the kernels form (chunk + 1) * C/B in 64 bits and skip the job
    jobs = np.array([[-1, 0, 0, 0], [w.num_slots, 0, 0, 0], [0, -1, 0, 0], [0, w.num_reqs, 0, 0],
                     [0, 0, -1, 0], [0, 0, bt.shape[1], 0], [0, 0, 0x7FFFFFFF, 0], [0, 1, 0x3FFFFFFF, 0],
                     [1, 0, 0, 0]], np.int32)
    d_jobs = torch.from_numpy(jobs).cuda()
    kv.kv_retrieve_scatter(g.layout, g.staging, g.layers, d_bt, bt.shape[1], w.num_reqs, d_jobs, len(jobs))
    oracle.retrieve_scatter(o.layout, o.staging, o.layers, bt, jobs)
    kv.kv_store_gather(g.layout, g.staging, g.layers, d_bt, bt.shape[1], w.num_reqs, d_jobs, len(jobs))
    oracle.store_gather(o.layout, o.staging, o.layers, bt, jobs)
    for kind in (kv.KV_RETRIEVE_PAIR, kv.KV_RETRIEVE_STREAM, kv.KV_RETRIEVE_QUAD):
        jobs2 = jobs.copy()
        jobs2[-1, 0] = (2 + kind) % w.num_slots
        kv.kv_retrieve_scatter_as(kind, g.layout, g.staging, g.layers, d_bt, bt.shape[1], w.num_reqs,
                                  torch.from_numpy(jobs2).cuda(), len(jobs2))
        oracle.retrieve_scatter(o.layout, o.staging, o.layers, bt, jobs2)
    torch.cuda.synchronize()
    assert np.array_equal(g.staging.cpu().numpy(), o.staging)
    for l in range(2):
        assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l])


@pytest.mark.parametrize("layout,pad", [("kv_first", 0), ("block_first", 48)])
@pytest.mark.parametrize("si", range(len(SHAPES)))
@pytest.mark.parametrize("sharing", ["distinct", "pairs", "groups", "mixed"])
@pytest.mark.parametrize("kind", [1, 2, 3])
def test_retrieve_variants_match_oracle(kind, sharing, si, layout, pad):
    # Every variant must give the oracle's bytes for any job list: distinct slots, slots shared by aligned
    # pairs, and a mixed list (odd length, pairs that straddle two slots, out-of-range jobs in between).
    shape = SHAPES[si]
    w = W.small_random(300 + si, shape, num_reqs=9, max_len=5 * shape.chunk_tokens + 37, paged_layout=layout,
                       block_pad=pad)
    g, o = _pair(w)
    jobs = W.random_retrieve_jobs(w, 300 + si, slots_used=w.num_slots)
    n = len(jobs)
    if sharing == "distinct":
        jobs[:, 0] = np.arange(n) % w.num_slots
    elif sharing == "pairs":
        jobs[:, 0] = (np.arange(n) // 2) % w.num_slots
    elif sharing == "groups":
        jobs[:, 0] = (np.arange(n) // 8) % w.num_slots
    else:
        jobs[:, 0] = (np.arange(n) // 3) % w.num_slots
        jobs = np.concatenate([jobs[: n - 1 + (n % 2)], [[w.num_slots, 0, 0, 0], [0, w.num_reqs, 0, 0]]])
        jobs[1::5, 2] = -1                                          # invalid chunk: skipped
        assert len(jobs) % 2 == 1
    jobs = np.ascontiguousarray(jobs, np.int32)
    d_jobs = torch.from_numpy(jobs).cuda()
    kv.kv_retrieve_scatter_as(kind, g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs, d_jobs, len(jobs))
    oracle.retrieve_scatter(o.layout, o.staging, o.layers, w.block_tables, jobs)
    torch.cuda.synchronize()
    for l in range(len(g.layers)):
        assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l]), f"layer {l} differs"
    _free(g, o)


def test_zero_jobs_enqueue_nothing():
    shape = W.KVShape(1, 2, 64, 2, 16, 64)
    w = W.small_random(22, shape, num_reqs=2, max_len=128)
    g, _ = _pair(w)
    before = [t.clone() for t in g.layers]
    kv.kv_retrieve_scatter(g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs, None, 0)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(before, g.layers))


@pytest.mark.parametrize("layout", ["kv_first", "block_first"])
def test_host_staging_zero_copy(layout):
    # Staging buffer in mapped pinned host memory, read and written by the
    # kernels over the host link; every byte compared.
    shape = W.KVShape(2, 8, 128, 2, 16, 64)
    w = W.small_random(31, shape, num_reqs=6, max_len=400, paged_layout=layout)
    w.staging_in_host = True
    g, o = _pair(w)
    assert g.staging is None and g.staging_host is not None
    for p in range(2):
        sg, so = g.run_pass(validate=True), o.run_pass()
        _compare_pass(g, o, sg, so)


@pytest.mark.parametrize("evict", [False, True])
def test_overlapped_passes_match_sequential_oracle(evict):
    # Hash and lookup of pass i+1 are enqueued on their own stream right after
    # pass i's copies and index update; the jobs and every byte must be those
    # of the oracle's passes run one after another.
    shape = W.KVShape(2, 2, 64, 2, 16, 64)
    w = W.small_random(77, shape, num_reqs=9, max_len=5 * 64 + 21)
    g = StagingPath(w, overlap=True)
    g.fill(STG_TAG, POOL_TAG, w.seed, True)
    g.prestage()
    o = OraclePath(w, kv_seed=w.seed, finite=True, staging_tag=STG_TAG, pool_tag_base=POOL_TAG)
    o.prestage()
    assert g.lookup_stream is not g.stream
    n = 4
    g.launch_lookup()
    for i in range(n):
        sg = g.complete_pass(evict_stored=evict, validate=True)
        so = o.run_pass(evict_stored=evict)
        assert np.array_equal(g.last_retrieve, so["retrieve"]), i
        assert np.array_equal(g.last_store, so["store"]), i
        assert sg.dropped == so["dropped"]
        if i + 1 < n:
            g.launch_lookup()
    torch.cuda.synchronize()
    assert np.array_equal(g.staging_view().cpu().numpy(), o.staging)
    for l in range(len(g.layers)):
        assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l])
    _free(g, o)


@pytest.mark.parametrize("workload_seed", [78, 79])
def test_tuned_retrieve_passes_match_oracle(workload_seed):
    # tune_retrieve times the planned retrieve against the four-job-window one on the live pool (re-running
    # the last pass's retrieve, which is idempotent) and keeps the faster; later passes must still give the
    # oracle's bytes, whichever was chosen.
    shape = W.KVShape(2, 2, 64, 2, 16, 64)
    w = W.small_random(workload_seed, shape, num_reqs=12, max_len=6 * 64 + 5)
    g = StagingPath(w)
    g.fill(STG_TAG, POOL_TAG, w.seed, True)
    g.prestage()
    o = OraclePath(w, kv_seed=w.seed, finite=True, staging_tag=STG_TAG, pool_tag_base=POOL_TAG)
    o.prestage()
    g.run_pass(evict_stored=False)
    o.run_pass(evict_stored=False)
    tuned = g.tune_retrieve(reps=3)
    if len(g.last_retrieve):
        assert "quad" in tuned and len(tuned) == 2 and all(v > 0 for v in tuned.values())
        assert set(g.retrieve_choice.values()) <= {kv.KV_RETRIEVE_QUAD, kv.KV_RETRIEVE_UNIT, kv.KV_RETRIEVE_PAIR}
    torch.cuda.synchronize()
    assert np.array_equal(g.staging_view().cpu().numpy(), o.staging)
    for l in range(len(g.layers)):
        assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l])
    for i in range(3):
        g.run_pass(evict_stored=True)
        so = o.run_pass(evict_stored=True)
        assert np.array_equal(g.last_retrieve, so["retrieve"]), i
    torch.cuda.synchronize()
    assert np.array_equal(g.staging_view().cpu().numpy(), o.staging)
    for l in range(len(g.layers)):
        assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l])
    _free(g, o)


@pytest.mark.parametrize("kind", ["store", 0, 1, 2, 3])
def test_million_job_lists_match_oracle(kind):
    # 2^20 jobs (grids of 2^20-2^22 workgroups) cycling over a few (slot, request, chunk) triples: every
    # repeat of a triple copies the same bytes to the same place, so the result is the oracle's over the
    # distinct triples, whatever order the repeats land in
    shape = W.KVShape(1, 2, 64, 2, 16, 64)                  # 4 KiB segments, 4 per chunk
    w = W.small_random(501, shape, num_reqs=6, max_len=4 * 64)
    g, o = _pair(w)
    base = W.random_retrieve_jobs(w, 501, slots_used=w.num_slots)[:5]
    assert len(base) == 5 and w.num_slots >= 5
    if kind == "store":
        base[:, 0] = np.arange(len(base))                   # one slot per distinct triple
    n = 1 << 20
    jobs = np.ascontiguousarray(base[np.arange(n) % len(base)], np.int32)
    d_jobs = torch.from_numpy(jobs).cuda()
    print(f"[million] kind {kind}: {n} jobs over {len(base)} triples, shape {shape}", flush=True)
    if kind == "store":
        kv.kv_store_gather(g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs, d_jobs, n)
        oracle.store_gather(o.layout, o.staging, o.layers, w.block_tables, base)
    else:
        kv.kv_retrieve_scatter_as(kind, g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs, d_jobs, n)
        oracle.retrieve_scatter(o.layout, o.staging, o.layers, w.block_tables, base)
    torch.cuda.synchronize()
    assert np.array_equal(g.staging.cpu().numpy(), o.staging)
    for l in range(len(g.layers)):
        assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l])
    _free(g, o)


def test_many_random_shapes_every_variant():
    # A wider sweep than the forty above: TEMPOKV_SOAK_SHAPES random shapes (300 by default) drawn from
    # TEMPOKV_SOAK_SEED (3030 by default), each with two whole passes and then every retrieve variant on a
    # random job list (grouped or not), every byte compared with the oracle.
    n = int(os.environ.get("TEMPOKV_SOAK_SHAPES", "300"))
    seed = os.environ.get("TEMPOKV_SOAK_SEED")
    shape_seed, wl_seed = (3030, 5000) if seed is None else (int(seed), 7 * int(seed))
    for k, shape in enumerate(W.random_shapes(shape_seed, n)):
        layout = ["kv_first", "block_first"][k % 2]
        pad = [0, 16, 4096, 48, 32][k % 5]
        w = W.small_random(wl_seed + k, shape, num_reqs=5 + k % 4, max_len=3 * shape.chunk_tokens + 7 * (k % 5),
                           paged_layout=layout, block_pad=pad)
        g, o = _pair(w)
        for p in range(2):
            sg, so = g.run_pass(validate=True), o.run_pass()
            _compare_pass(g, o, sg, so)
        jobs = W.random_retrieve_jobs(w, wl_seed + k, slots_used=max(1, w.num_slots // 3))
        if len(jobs):
            jobs = np.ascontiguousarray(kv.kv_group_jobs_by_slot(jobs) if k % 2 else jobs, np.int32)
            d_jobs = torch.from_numpy(jobs).cuda()
            for kind in (kv.KV_RETRIEVE_UNIT, kv.KV_RETRIEVE_PAIR, kv.KV_RETRIEVE_STREAM, kv.KV_RETRIEVE_QUAD):
                kv.kv_retrieve_scatter_as(kind, g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs,
                                          d_jobs, len(jobs))
            oracle.retrieve_scatter(o.layout, o.staging, o.layers, w.block_tables, jobs)
            torch.cuda.synchronize()
            for l in range(len(g.layers)):
                assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l]), (k, shape, l)
        _free(g, o)
        if k % 100 == 99:
            print(f"[shapes] {k + 1}/{n} ok", flush=True)
