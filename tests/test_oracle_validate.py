"""Pins for the oracle's job-batch check (``oracle.validate_jobs``).

Within one copy launch the only writes that can race are two jobs naming one
destination: a paged block in the scatter, a staging slot in the gather.  The
check is pinned by closed-form cases (each out-of-range field, each kind of
duplicate destination, the reads that may be shared) and by a second route to
the same answer on random batches: destinations collected into a Python set.
"""
import numpy as np
import pytest

import oracle
from workloads import KVShape

SHAPE = KVShape(2, 2, 64, 2, 16, 64)     # 4 blocks per chunk
NSEG = SHAPE.chunk_tokens // SHAPE.block_size
R, CPR = 4, 2                            # requests, chunks per request
NB = R * CPR * NSEG + 6                  # spare blocks no table names
NSLOTS = R * CPR
INT32_MAX = 2**31 - 1


def _setup(seed=0):
    rng = np.random.default_rng(seed)
    lo = oracle.make_layout(SHAPE, NB, NSLOTS, NB * SHAPE.seg_bytes, SHAPE.seg_bytes)
    bt = rng.permutation(NB)[:R * CPR * NSEG].astype(np.int32).reshape(R, CPR * NSEG)
    return lo, bt


def _valid():
    # every (request, chunk) once, each with a slot of its own
    return np.array([[r * CPR + c, r, c, 0] for r in range(R) for c in range(CPR)], np.int32)


@pytest.mark.parametrize("is_store", [False, True])
def test_valid_and_empty_batches_are_ok(is_store):
    lo, bt = _setup()
    assert oracle.validate_jobs(lo, bt, _valid(), is_store) == oracle.VOK
    assert oracle.validate_jobs(lo, bt, np.zeros((0, 4), np.int32), is_store) == oracle.VOK


@pytest.mark.parametrize("is_store", [False, True])
@pytest.mark.parametrize("field,value", [(0, -1), (0, NSLOTS), (1, -1), (1, R), (2, -1), (2, CPR), (2, INT32_MAX),
                                         (3, 1), (3, -1)])
def test_each_out_of_range_field(is_store, field, value):
    lo, bt = _setup()
    jobs = _valid()
    jobs[3, field] = value
    assert oracle.validate_jobs(lo, bt, jobs, is_store) == oracle.VERANGE


@pytest.mark.parametrize("is_store", [False, True])
@pytest.mark.parametrize("blk", [-1, NB, INT32_MAX])
def test_out_of_range_block_of_a_named_chunk(is_store, blk):
    lo, bt = _setup()
    bt[1, NSEG + 2] = blk                         # request 1, chunk 1, segment 2
    assert oracle.validate_jobs(lo, bt, _valid(), is_store) == oracle.VERANGE
    # the same bad id in a chunk that no job names is not looked at
    jobs = _valid()
    jobs = jobs[~((jobs[:, 1] == 1) & (jobs[:, 2] == 1))]
    assert oracle.validate_jobs(lo, bt, jobs, is_store) == oracle.VOK


def test_two_jobs_writing_one_chunks_blocks():
    lo, bt = _setup()
    jobs = np.concatenate([_valid(), [[0, 2, 1, 0]]]).astype(np.int32)   # (2, 1) again, from another slot
    assert oracle.validate_jobs(lo, bt, jobs, False) == oracle.VEDUP
    jobs[-1, 0] = 7
    assert oracle.validate_jobs(lo, bt, jobs[[0, -1]], True) == oracle.VOK   # gathering one chunk twice: no race


def test_two_jobs_naming_one_slot():
    lo, bt = _setup()
    jobs = _valid()
    jobs[5, 0] = jobs[2, 0]
    assert oracle.validate_jobs(lo, bt, jobs, True) == oracle.VEDUP
    assert oracle.validate_jobs(lo, bt, jobs, False) == oracle.VOK           # many scatters may read one slot


def test_tables_of_two_requests_sharing_a_block():
    lo, bt = _setup()
    bt[2, NSEG + 3] = bt[0, 1]
    assert oracle.validate_jobs(lo, bt, _valid(), False) == oracle.VEDUP
    assert oracle.validate_jobs(lo, bt, _valid(), True) == oracle.VOK


def test_one_chunk_naming_a_block_twice():
    lo, bt = _setup()
    bt[1, 1] = bt[1, 0]
    assert oracle.validate_jobs(lo, bt, _valid(), False) == oracle.VEDUP
    assert oracle.validate_jobs(lo, bt, _valid()[[1]], False) == oracle.VOK   # request 0, chunk 1: untouched
    assert oracle.validate_jobs(lo, bt, _valid()[[2]], False) == oracle.VEDUP  # request 1, chunk 0 alone


@pytest.mark.parametrize("is_store", [False, True])
def test_range_error_decides_over_a_duplicate(is_store):
    lo, bt = _setup()
    jobs = np.concatenate([_valid(), _valid()[:2]]).astype(np.int32)
    assert oracle.validate_jobs(lo, bt, jobs, is_store) == oracle.VEDUP
    jobs[-1, 2] = CPR
    assert oracle.validate_jobs(lo, bt, jobs, is_store) == oracle.VERANGE


def _by_sets(bt, jobs, is_store):
    """The same outcome by another route: range checks, then destinations in a set."""
    for s, r, c, z in jobs.tolist():
        if z != 0 or not (0 <= s < NSLOTS) or not (0 <= r < R) or not (0 <= c and (c + 1) * NSEG <= bt.shape[1]):
            return oracle.VERANGE
        if any(not (0 <= b < NB) for b in bt[r, c * NSEG:(c + 1) * NSEG].tolist()):
            return oracle.VERANGE
    dests = [s for s, _, _, _ in jobs.tolist()] if is_store else \
        [b for _, r, c, _ in jobs.tolist() for b in bt[r, c * NSEG:(c + 1) * NSEG].tolist()]
    return oracle.VOK if len(set(dests)) == len(dests) else oracle.VEDUP


@pytest.mark.parametrize("seed", range(60))
def test_random_batches_against_sets(seed):
    rng = np.random.default_rng(seed)
    lo, bt = _setup(seed)
    if seed % 3 == 0:                                   # tables that collide somewhere
        bt[rng.integers(R), rng.integers(CPR * NSEG)] = bt[rng.integers(R), rng.integers(CPR * NSEG)]
    n = int(rng.integers(0, 12))
    jobs = np.stack([rng.integers(-1, NSLOTS + 1, n), rng.integers(0, R, n), rng.integers(0, CPR, n),
                     (rng.random(n) < 0.05).astype(np.int64)], axis=1).astype(np.int32) if n else np.zeros((0, 4), np.int32)
    if n and seed % 2:
        jobs[:, 0] = np.clip(jobs[:, 0], 0, NSLOTS - 1)  # keep slots in range half the time
    for is_store in (False, True):
        want = _by_sets(bt, jobs, is_store)
        assert oracle.validate_jobs(lo, bt, jobs, is_store) == want
        # the outcome does not depend on the order of the jobs
        assert oracle.validate_jobs(lo, bt, jobs[rng.permutation(n)] if n else jobs, is_store) == want
