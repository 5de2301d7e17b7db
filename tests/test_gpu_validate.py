"""GPU parity of the device job-batch check (kv_validate_jobs_device) with the
oracle's check: closed-form cases (each out-of-range field and block id, each
kind of duplicate destination, shared reads), random batches, the benchmark's
own job lists, scratch reuse across calls and a non-default stream.  The host
form (kv_validate_jobs) is compared on the same batches."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_35065_amd as kv
import workloads as W
from oracle.pipeline import OraclePath
from workloads import KVShape

pytestmark = pytest.mark.gpu

CODE = {oracle.VOK: kv.KV_OK, oracle.VERANGE: kv.KV_ERANGE, oracle.VEDUP: kv.KV_EDUP}


def _layouts(shape, nb, ns):
    seg = shape.seg_bytes
    args = (shape.num_layers, shape.kv_heads, shape.head_dim, shape.elem_bytes, shape.block_size,
            shape.chunk_tokens, nb, ns, nb * seg, seg)
    return kv.make_layout(*args), oracle.make_layout(shape, nb, ns, nb * seg, seg)


class _Device:
    """Device buffers for one layout; the scratch is reused by every call."""

    def __init__(self, lo, stream=None):
        self.lo = lo
        self.marks = torch.full((2 + max(lo.num_blocks, lo.num_slots),), 7, dtype=torch.int32, device="cuda")
        self.status = torch.zeros(1, dtype=torch.int32, device="cuda")
        self.stream = stream

    def check(self, bt, jobs, is_store):
        d_bt = torch.from_numpy(np.ascontiguousarray(bt, np.int32)).cuda()
        d_jobs = torch.from_numpy(np.ascontiguousarray(jobs, np.int32).reshape(-1, 4) if len(jobs)
                                  else np.zeros((1, 4), np.int32)).cuda()
        self.status.fill_(12345)                        # not a status: the call must overwrite it
        torch.cuda.synchronize()
        kv.kv_validate_jobs_device(self.lo, d_bt, bt.shape[1], bt.shape[0], d_jobs, len(jobs), is_store,
                                   self.marks, self.status, self.stream)
        (self.stream or torch.cuda.current_stream()).synchronize()
        return int(self.status.item())


def _compare(dev, olo, bt, jobs, is_store):
    want = CODE[oracle.validate_jobs(olo, bt, jobs, is_store)]
    got = dev.check(bt, jobs, is_store)
    assert got == want, (got, want, is_store)
    assert kv.kv_validate_jobs(dev.lo, bt, jobs if len(jobs) else np.zeros((0, 4), np.int32), is_store) == want
    return want


SHAPE = KVShape(2, 2, 64, 2, 16, 64)        # 4 blocks per chunk
NSEG, R, CPR = 4, 4, 2
NB, NS = R * CPR * NSEG + 6, R * CPR


def _small(seed=0):
    rng = np.random.default_rng(seed)
    bt = rng.permutation(NB)[:R * CPR * NSEG].astype(np.int32).reshape(R, CPR * NSEG)
    jobs = np.array([[r * CPR + c, r, c, 0] for r in range(R) for c in range(CPR)], np.int32)
    return bt, jobs


def _cases():
    bt, jobs = _small()
    yield "valid", bt, jobs
    yield "empty", bt, jobs[:0]
    for f, v in [(0, -1), (0, NS), (1, -1), (1, R), (2, -1), (2, CPR), (2, 2**31 - 1), (3, 1)]:
        j = jobs.copy()
        j[3, f] = v
        yield f"field{f}={v}", bt, j
    for blk in (-1, NB, 2**31 - 1):
        b = bt.copy()
        b[1, NSEG + 2] = blk
        yield f"block={blk}", b, jobs
    yield "same chunk twice", bt, np.concatenate([jobs, [[0, 2, 1, 0]]]).astype(np.int32)
    j = jobs.copy()
    j[5, 0] = j[2, 0]
    yield "same slot twice", bt, j
    b = bt.copy()
    b[2, NSEG + 3] = b[0, 1]
    yield "tables share a block", b, jobs
    b = bt.copy()
    b[1, 1] = b[1, 0]
    yield "chunk names a block twice", b, jobs
    j = np.concatenate([jobs, jobs[:2]]).astype(np.int32)
    j[-1, 2] = CPR
    yield "range and duplicate", bt, j


@pytest.mark.parametrize("is_store", [False, True])
def test_closed_form_cases(is_store):
    lo, olo = _layouts(SHAPE, NB, NS)
    dev = _Device(lo)
    seen = set()
    for name, bt, jobs in _cases():
        seen.add(_compare(dev, olo, bt, jobs, is_store))
    assert seen == {kv.KV_OK, kv.KV_ERANGE, kv.KV_EDUP}


def test_random_batches_and_scratch_reuse():
    # one scratch buffer for every call: marks left by one call must not leak into the next
    lo, olo = _layouts(SHAPE, NB, NS)
    dev = _Device(lo)
    seen = set()
    for seed in range(300):
        rng = np.random.default_rng(1000 + seed)
        bt, _ = _small(seed)
        if seed % 3 == 0:
            bt[rng.integers(R), rng.integers(CPR * NSEG)] = bt[rng.integers(R), rng.integers(CPR * NSEG)]
        n = int(rng.integers(0, 14))
        jobs = np.stack([rng.integers(-1, NS + 1, n), rng.integers(0, R, n), rng.integers(0, CPR, n),
                         (rng.random(n) < 0.05).astype(np.int64)], axis=1).astype(np.int32)
        if seed % 2:
            jobs[:, 0] = np.clip(jobs[:, 0], 0, NS - 1)
        for is_store in (False, True):
            seen.add(_compare(dev, olo, bt, jobs, is_store))
    assert seen == {kv.KV_OK, kv.KV_ERANGE, kv.KV_EDUP}


@pytest.mark.parametrize("shape", [KVShape(2, 8, 128, 2, 16, 256), KVShape(3, 1, 64, 2, 16, 16),
                                   KVShape(2, 2, 128, 2, 32, 128)])
def test_workload_job_lists(shape):
    # the retrieve and store jobs of real passes, then with one planted duplicate and one planted range error
    w = W.small_random(31, shape, num_reqs=12, max_len=2048)
    o = OraclePath(w, with_kv=False)
    o.prestage()
    so = o.run_pass()
    lo, olo = _layouts(shape, w.num_blocks, w.num_slots)
    dev = _Device(lo, torch.cuda.Stream())
    bt = np.ascontiguousarray(w.block_tables, np.int32)
    assert len(so["retrieve"]) >= 2 and len(so["store"]) >= 2
    for jobs, is_store in ((so["retrieve"], False), (so["store"], True)):
        assert _compare(dev, olo, bt, jobs, is_store) == kv.KV_OK
        dup = jobs.copy()
        dup[-1] = dup[0] if not is_store else [dup[0, 0], *dup[-1, 1:]]
        assert _compare(dev, olo, bt, dup, is_store) == kv.KV_EDUP
        bad = jobs.copy()
        bad[len(bad) // 2, 1] = w.num_reqs
        assert _compare(dev, olo, bt, bad, is_store) == kv.KV_ERANGE


def test_benchmark_batch_job_lists():
    # the 32-layer benchmark's 512 retrieve and 512 store jobs (8,192 destination blocks each way)
    w = W.make("l32-64x4096")
    o = OraclePath(w, with_kv=False)
    o.prestage()
    so = o.run_pass()
    lo, olo = _layouts(w.shape, w.num_blocks, w.num_slots)
    dev = _Device(lo)
    bt = np.ascontiguousarray(w.block_tables, np.int32)
    assert len(so["retrieve"]) == 512 and len(so["store"]) == 512
    for jobs, is_store in ((so["retrieve"], False), (so["store"], True)):
        assert _compare(dev, olo, bt, jobs, is_store) == kv.KV_OK
        dup = np.concatenate([jobs, jobs[[100]]]).astype(np.int32)
        if is_store:
            dup[-1, 1:3] = jobs[200, 1:3]           # another chunk into slot jobs[100]
        assert _compare(dev, olo, bt, dup, is_store) == kv.KV_EDUP
