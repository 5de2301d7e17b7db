"""The measurement reference kv_probe_mixed_traffic, on the GPU: it must write
its filler into exactly the blocks the retrieve of the same jobs would write,
skip what the copies skip, and leave every other byte of the pool and the
whole staging buffer as they were.  The expected bytes are the snapshot taken
before the call with the destination segments (from the block tables and the
layout's strides) set to the filler."""
import numpy as np
import pytest
import torch

import paper_2609_35065_amd as kv
import workloads as W
from paper_2609_35065_amd.pipeline import StagingPath

pytestmark = pytest.mark.gpu

FILL = 0xA5C3E1F7


def _expected_layers(w, g, before, jobs):
    lo = g.layout
    seg = w.shape.seg_bytes
    nseg = w.shape.chunk_tokens // w.shape.block_size
    fill = np.frombuffer(np.array([FILL], "<u4").tobytes() * (seg // 4), np.uint8)
    out = [a.copy() for a in before]
    for slot, req, chunk, _ in jobs:
        if not (0 <= slot < w.num_slots and 0 <= req < w.num_reqs and chunk >= 0 and
                (chunk + 1) * nseg <= w.bt_stride):
            continue
        for i in range(nseg):
            blk = int(w.block_tables[req, chunk * nseg + i])
            if not 0 <= blk < w.num_blocks:
                continue
            for l in range(w.shape.num_layers):
                for p in range(2):
                    o = p * lo.paged_kv_stride + blk * lo.paged_block_stride
                    out[l][o:o + seg] = fill
    return out


@pytest.mark.parametrize("case", ["32k_kv_first", "random_shape", "block_first_padded"])
def test_probe_writes_exactly_the_retrieve_destinations(case):
    if case == "32k_kv_first":
        shape, kw = W.KVShape(2, 8, 128, 2, 16, 64), {}
    elif case == "random_shape":
        shape, kw = W.random_shapes(911, 1)[0], {}
    else:
        shape, kw = W.KVShape(3, 2, 64, 2, 16, 64), {"paged_layout": "block_first", "block_pad": 4096}
    w = W.small_random(712, shape, num_reqs=9, max_len=5 * shape.chunk_tokens + 3, **kw)
    g = StagingPath(w)
    g.fill(1, 1000, w.seed, True)
    jobs = W.random_retrieve_jobs(w, 712, slots_used=w.num_slots)
    assert len(jobs) > 0
    # jobs the copies skip: slot, request or chunk out of range
    bad = np.array([[w.num_slots, 0, 0, 0], [-1, 0, 0, 0], [0, w.num_reqs, 0, 0], [0, 0, w.bt_stride, 0]], np.int32)
    all_jobs = np.ascontiguousarray(np.concatenate([jobs, bad]), np.int32)
    slots = np.unique(jobs[:, 0]).astype(np.int32)
    read_slots = np.ascontiguousarray(np.concatenate([slots, [-1, w.num_slots]]), np.int32)   # two skipped
    torch.cuda.synchronize()
    before = [t.cpu().numpy().copy() for t in g.layers]
    stg_before = g.staging_view().cpu().numpy().copy()
    print(f"[probe] {case}: shape {shape}, {len(all_jobs)} jobs, {len(read_slots)} read slots", flush=True)
    d_jobs = torch.from_numpy(all_jobs).cuda()
    d_slots = torch.from_numpy(read_slots).cuda()
    kv.kv_probe_mixed_traffic(g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs, d_jobs, len(all_jobs),
                              d_slots, len(read_slots), FILL)
    torch.cuda.synchronize()
    assert np.array_equal(g.staging_view().cpu().numpy(), stg_before), "staging changed"
    exp = _expected_layers(w, g, before, all_jobs)
    for l in range(w.shape.num_layers):
        assert np.array_equal(g.layers[l].cpu().numpy(), exp[l]), f"layer {l}"
    # the retrieve of the same jobs afterwards restores real data into those blocks
    kv.kv_retrieve_scatter(g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs, d_jobs, len(all_jobs))
    torch.cuda.synchronize()
    assert not any(np.array_equal(g.layers[l].cpu().numpy(), exp[l]) for l in range(w.shape.num_layers))


def test_probe_rejects_bad_arguments():
    shape = W.KVShape(1, 2, 64, 2, 16, 64)
    w = W.small_random(713, shape, num_reqs=3, max_len=2 * 64)
    g = StagingPath(w)
    d_jobs = torch.zeros((1, 4), dtype=torch.int32, device="cuda")
    d_slots = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(kv.KvError):
        kv.kv_probe_mixed_traffic(g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs, d_jobs, 1,
                                  d_slots, -1, FILL)
    # nothing to do: no launch, no error
    kv.kv_probe_mixed_traffic(g.layout, g.staging, g.layers, g.bt, w.bt_stride, w.num_reqs, d_jobs, 0, None, 0, FILL)
    torch.cuda.synchronize()
