"""GPU parity of the staging copies and the stage-ready-gated retrieve.

The lower tier is pinned host memory, the fast tier an HBM staging buffer.
kv_stage_in / kv_stage_out must move exactly the named slots, and
kv_retrieve_pipelined must leave the paged pool byte-identical to the
oracle's retrieve scatter over the same jobs, for every batch size, with
copies and scatters on two streams or one, grouped or ungrouped jobs, and a
pipeline too small for one batch per slot (the batch size is then raised).
Every byte of the pool and of the staging buffer is compared."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_35065_amd as kv
import workloads as W
from oracle.pipeline import OraclePath
from paper_2609_35065_amd.pipeline import StagingPath

pytestmark = pytest.mark.gpu

SENT_STG, SENT_POOL = 0x11, 0x22


def _pinned_kv(nbytes, tag, seed):
    t = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    t.numpy()[:] = W.kv_bytes_np(tag, seed, 0, nbytes)
    return t


def _setup(seed, shape=W.KVShape(3, 2, 64, 2, 16, 64), num_reqs=6, max_len=300, layout="kv_first"):
    w = W.small_random(seed, shape, num_reqs=num_reqs, max_len=max_len, paged_layout=layout)
    kv_stride, block_stride = w.strides()
    lo = kv.make_layout(shape.num_layers, shape.kv_heads, shape.head_dim, shape.elem_bytes, shape.block_size,
                        shape.chunk_tokens, w.num_blocks, w.num_slots, kv_stride, block_stride)
    olo = oracle.make_layout(shape, w.num_blocks, w.num_slots, kv_stride, block_stride)
    return w, lo, olo


def test_stage_in_and_out_move_exactly_the_named_slots():
    w, lo, _ = _setup(61)
    sb, S = w.shape.slot_bytes, w.num_slots
    host = _pinned_kv(S * sb, 7, 61)
    dev = torch.full((S * sb,), SENT_STG, dtype=torch.uint8, device="cuda")
    slots = np.array([3, 4, 5, 0, 9, S - 1], np.int32)[: min(6, S)]
    slots = slots[slots < S]
    kv.kv_stage_in(lo, host, dev, slots)
    torch.cuda.synchronize()
    d = dev.cpu().numpy().reshape(S, sb)
    h = host.numpy().reshape(S, sb)
    for s in range(S):
        if s in set(slots.tolist()):
            assert np.array_equal(d[s], h[s]), f"slot {s} not staged"
        else:
            assert np.all(d[s] == SENT_STG), f"slot {s} written"
    # the reverse direction: device content of other slots back into the host
    dev.copy_(torch.from_numpy(W.kv_bytes_np(8, 61, 0, S * sb)).cuda())
    back = np.array([1, 2, 7], np.int32)
    back = back[back < S]
    before = host.numpy().copy().reshape(S, sb)
    kv.kv_stage_out(lo, dev, host, back)
    torch.cuda.synchronize()
    d = dev.cpu().numpy().reshape(S, sb)
    h = host.numpy().reshape(S, sb)
    for s in range(S):
        assert np.array_equal(h[s], d[s] if s in set(back.tolist()) else before[s])
    # empty lists enqueue nothing
    kv.kv_stage_in(lo, host, dev, np.zeros(0, np.int32))
    kv.kv_stage_out(lo, dev, host, np.zeros(0, np.int32))


@pytest.mark.parametrize("max_batches,spb,same_stream,grouped,layout", [
    (64, 1, False, True, "kv_first"),
    (64, 3, False, True, "block_first"),
    (64, 1000, False, True, "kv_first"),
    (64, 2, True, True, "kv_first"),
    (64, 1, False, False, "kv_first"),
    (2, 1, False, True, "block_first"),
    (2, 1, True, False, "kv_first"),
])
def test_retrieve_pipelined_matches_oracle(max_batches, spb, same_stream, grouped, layout):
    w, lo, olo = _setup(67, layout=layout)
    sb, S = w.shape.slot_bytes, w.num_slots
    jobs = W.random_retrieve_jobs(w, 67, slots_used=min(S, 9))
    assert len(jobs) > 4 and not np.all(np.diff(jobs[:, 0]) >= 0)
    if grouped:
        jobs = kv.kv_group_jobs_by_slot(jobs)
    host = _pinned_kv(S * sb, 1, 67)
    stg = torch.full((S * sb,), SENT_STG, dtype=torch.uint8, device="cuda")
    layers = [torch.full((w.layer_bytes(),), SENT_POOL, dtype=torch.uint8, device="cuda")
              for _ in range(w.shape.num_layers)]
    bt = torch.from_numpy(np.ascontiguousarray(w.block_tables)).cuda()
    d_jobs = torch.from_numpy(jobs).cuda()
    stream = torch.cuda.current_stream()
    copy_stream = stream if same_stream else torch.cuda.Stream()
    with kv.KvPipeline(max_batches) as pl:
        copy_stream.wait_stream(stream)
        kv.kv_retrieve_pipelined(pl, lo, host, stg, layers, bt, w.bt_stride, w.num_reqs, jobs, d_jobs, spb,
                                 copy_stream, stream)
        torch.cuda.synchronize()
    # oracle: the plain scatter from the lower tier's bytes
    o_layers = [np.full(w.layer_bytes(), SENT_POOL, np.uint8) for _ in range(w.shape.num_layers)]
    oracle.retrieve_scatter(olo, host.numpy().copy(), o_layers, w.block_tables, jobs)
    for l in range(w.shape.num_layers):
        assert np.array_equal(layers[l].cpu().numpy(), o_layers[l]), f"layer {l} differs"
    named = set(int(s) for s in jobs[:, 0])
    d = stg.cpu().numpy().reshape(S, sb)
    h = host.numpy().reshape(S, sb)
    for s in range(S):
        assert np.array_equal(d[s], h[s]) if s in named else np.all(d[s] == SENT_STG)


def test_retrieve_pipelined_random_sweep():
    # 60 random shapes and layouts, each with a random batch size (1-5 slots, or everything), pipeline size
    # (2-64 events), one or two streams, grouped or ungrouped jobs: pool and staging bytes against the oracle
    rng = np.random.default_rng(4242)
    shapes = W.random_shapes(4242, 60)
    for k, shape in enumerate(shapes):
        w = W.small_random(900 + k, shape, num_reqs=4 + k % 4, max_len=4 * shape.chunk_tokens + 11,
                           paged_layout=["kv_first", "block_first"][k % 2], block_pad=[0, 16, 48][k % 3])
        kv_stride, block_stride = w.strides()
        lo = kv.make_layout(shape.num_layers, shape.kv_heads, shape.head_dim, shape.elem_bytes, shape.block_size,
                            shape.chunk_tokens, w.num_blocks, w.num_slots, kv_stride, block_stride)
        olo = oracle.make_layout(shape, w.num_blocks, w.num_slots, kv_stride, block_stride)
        sb, S = shape.slot_bytes, w.num_slots
        jobs = W.random_retrieve_jobs(w, 900 + k, slots_used=max(1, int(rng.integers(1, S + 1))))
        if len(jobs) == 0:
            continue
        if rng.integers(0, 2):
            jobs = kv.kv_group_jobs_by_slot(jobs)
        jobs = np.ascontiguousarray(jobs, np.int32)
        spb = int(rng.choice([1, 2, 3, 5, 1000]))
        max_batches = int(rng.choice([2, 3, 8, 64]))
        host = _pinned_kv(S * sb, 1, 900 + k)
        stg = torch.full((S * sb,), SENT_STG, dtype=torch.uint8, device="cuda")
        layers = [torch.full((w.layer_bytes(),), SENT_POOL, dtype=torch.uint8, device="cuda")
                  for _ in range(shape.num_layers)]
        bt = torch.from_numpy(np.ascontiguousarray(w.block_tables)).cuda()
        d_jobs = torch.from_numpy(jobs).cuda()
        stream = torch.cuda.current_stream()
        copy_stream = stream if k % 3 == 0 else torch.cuda.Stream()
        with kv.KvPipeline(max_batches) as pl:
            copy_stream.wait_stream(stream)
            kv.kv_retrieve_pipelined(pl, lo, host, stg, layers, bt, w.bt_stride, w.num_reqs, jobs, d_jobs, spb,
                                     copy_stream, stream)
            torch.cuda.synchronize()
        o_layers = [np.full(w.layer_bytes(), SENT_POOL, np.uint8) for _ in range(shape.num_layers)]
        oracle.retrieve_scatter(olo, host.numpy().copy(), o_layers, w.block_tables, jobs)
        for l in range(shape.num_layers):
            assert np.array_equal(layers[l].cpu().numpy(), o_layers[l]), (k, shape, spb, max_batches, l)
        named = set(int(x) for x in jobs[:, 0])
        d, h = stg.cpu().numpy().reshape(S, sb), host.numpy().reshape(S, sb)
        for x in range(S):
            assert np.array_equal(d[x], h[x]) if x in named else np.all(d[x] == SENT_STG), (k, x)


def test_retrieve_pipelined_empty_and_errors():
    w, lo, _ = _setup(71)
    sb, S = w.shape.slot_bytes, w.num_slots
    host = _pinned_kv(S * sb, 1, 71)
    stg = torch.zeros(S * sb, dtype=torch.uint8, device="cuda")
    layers = [torch.zeros(w.layer_bytes(), dtype=torch.uint8, device="cuda") for _ in range(w.shape.num_layers)]
    bt = torch.from_numpy(np.ascontiguousarray(w.block_tables)).cuda()
    with kv.KvPipeline(4) as pl:
        kv.kv_retrieve_pipelined(pl, lo, host, stg, layers, bt, w.bt_stride, w.num_reqs, np.zeros((0, 4), np.int32),
                                 None, 1, torch.cuda.Stream())
        bad = np.array([[S, 0, 0, 0]], np.int32)
        with pytest.raises(kv.KvError) as e:
            kv.kv_retrieve_pipelined(pl, lo, host, stg, layers, bt, w.bt_stride, w.num_reqs, bad,
                                     torch.from_numpy(bad).cuda(), 1, torch.cuda.Stream())
        assert e.value.status == kv.KV_ERANGE
        with pytest.raises(ValueError):      # the lower tier must be pinned host memory
            kv.kv_retrieve_pipelined(pl, lo, torch.zeros(S * sb, dtype=torch.uint8), stg, layers, bt, w.bt_stride,
                                     w.num_reqs, bad, torch.from_numpy(bad).cuda(), 1, torch.cuda.Stream())
    torch.cuda.synchronize()
    assert not torch.any(torch.stack([t.sum(dtype=torch.int64) for t in layers]))


@pytest.mark.parametrize("mode,spb", [("pipelined", 1), ("pipelined", 3), ("pipelined", 1000), ("serialized", 2)])
def test_staged_lower_tier_pass_matches_oracle(mode, spb):
    # Whole passes (hash, lookup, job build, pipelined retrieve, store with
    # write-back) with the staged chunks in host memory: cold fast tier, warm
    # fast tier, then cold again.
    shape = W.KVShape(2, 8, 128, 2, 16, 64)
    w = W.small_random(43, shape, num_reqs=8, max_len=520)
    w.staging_in_host = True
    g = StagingPath(w, lower_tier=mode, slots_per_batch=spb)
    g.fill(1, 1000, w.seed)
    g.prestage()
    o = OraclePath(w, kv_seed=w.seed, staging_tag=1, pool_tag_base=1000)
    o.prestage()
    staged = []
    for p in range(3):
        if p == 2:
            g.drop_fast_tier()
        sg, so = g.run_pass(validate=True), o.run_pass()
        torch.cuda.synchronize()
        assert np.array_equal(g.last_retrieve, so["retrieve"])
        assert np.array_equal(g.last_store, so["store"])
        assert np.array_equal(g.staging_host.numpy(), o.staging), f"lower tier differs after pass {p}"
        for l in range(len(g.layers)):
            assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l]), f"layer {l} differs after pass {p}"
        hb = g.staging.cpu().numpy().reshape(w.num_slots, -1)
        hh = g.staging_host.numpy().reshape(w.num_slots, -1)
        assert np.array_equal(hb[g.resident], hh[g.resident]), "a resident HBM slot differs from host"
        staged.append(sg.staged_bytes)
        assert sg.num_retrieve > 0
    assert staged[0] > 0 and staged[1] == 0 and staged[2] > 0
