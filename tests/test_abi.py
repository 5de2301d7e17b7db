"""The C-ABI library without a GPU: it loads, exports every symbol the header
declares, and its host-side logic (job build, job validation, commitment
rule, argument checks) agrees with the oracle.  No call here reaches a
kernel launch or a HIP allocation."""
import ctypes as ct
import math
import os
import re

import numpy as np
import pytest

import oracle
import paper_2609_35065_amd as kv

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "tempokv.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    declared = _declared()
    assert len(declared) >= 15
    assert sorted(kv.EXPORTS) == declared
    L = ct.CDLL(kv.LIB_PATH)
    for name in declared:
        assert hasattr(L, name), name


def test_version_and_strerror():
    assert "gfx950" in kv.kv_version()
    for code in [0, -1, -2, -3, -4, -5, -6, -7]:
        assert kv.strerror(code) and kv.strerror(code) != "unknown status"
    assert kv.strerror(-99) == "unknown status"


@pytest.mark.parametrize("seed", range(8))
def test_commit_rule_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    vals = [-math.inf, -1.0, 0.0, 0.5, 1.0, 2.0, math.inf, math.nan]
    for _ in range(300):
        ttu, ttr = rng.choice(vals), rng.choice(vals)
        free, new, total, budget = (int(x) for x in rng.integers(0, 10, 4))
        req = bool(rng.integers(0, 2))
        assert kv.kv_commit_should_stage(ttu, ttr, free, new, total, budget, req) == \
            oracle.commit_should_stage(ttu, ttr, free, new, total, budget, req)


@pytest.mark.parametrize("seed", range(6))
def test_batched_commit_rule_matches_oracle_elementwise(seed):
    rng = np.random.default_rng(50 + seed)
    vals = np.array([-math.inf, -1.0, 0.0, 0.5, 1.0, 2.0, math.inf, math.nan])
    n = 400
    ttu, ttr = rng.choice(vals, n), rng.choice(vals, n)
    new = rng.integers(0, 12, n).astype(np.uint64)
    total = rng.integers(0, 12, n).astype(np.uint64)
    req = rng.integers(0, 2, n).astype(bool)
    free, budget = (int(x) for x in rng.integers(0, 12, 2))
    got = kv.kv_commit_should_stage_n(ttu, ttr, free, new, total, budget, req)
    exp = [oracle.commit_should_stage(float(ttu[i]), float(ttr[i]), free, int(new[i]), int(total[i]), budget,
                                      bool(req[i])) for i in range(n)]
    assert got.tolist() == exp
    assert kv.KV_EINVAL in exp and kv.KV_COMMIT in exp           # invalid elements do not stop the batch
    assert kv.kv_commit_should_stage_n([], [], 0, [], [], 0, []).size == 0
    L = kv.host_lib()
    assert L.kv_commit_should_stage_n(-1, None, None, 0, None, None, 0, None, None) == kv.KV_EINVAL
    assert L.kv_commit_should_stage_n(3, None, None, 0, None, None, 0, None, None) == kv.KV_EINVAL
    assert L.kv_commit_should_stage_n(0, None, None, 0, None, None, 0, None, None) == kv.KV_OK


def _lookup_case(seed):
    rng = np.random.default_rng(seed)
    C = int(rng.choice([16, 32, 64]))
    bpc = C // 16
    shared = rng.integers(0, 32000, 6 * C)
    reqs = []
    for _ in range(int(rng.integers(0, 9))):
        k = int(rng.integers(0, 6)) * C
        reqs.append(np.concatenate([shared[:k], rng.integers(0, 32000, int(rng.integers(0, 4 * C)))]).astype(np.int32))
    if rng.random() < 0.3:
        reqs += [r.copy() for r in reqs[:2]]
    tok_off = np.zeros(len(reqs) + 1, np.int64)
    np.cumsum([r.size for r in reqs], out=tok_off[1:])
    toks = np.concatenate(reqs).astype(np.int32) if reqs else np.zeros(0, np.int32)
    bh = oracle.hash_prefix(toks, tok_off)
    blk_off = oracle.block_offsets(tok_off)
    chunk_off = oracle.chunk_offsets(blk_off, bpc)
    keys = oracle.chunk_keys(bh, blk_off, bpc)
    st = shared.astype(np.int32)
    sh = oracle.hash_prefix(st, np.array([0, st.size], np.int64))
    index = {int(sh[(j + 1) * bpc - 1]): 50 + j for j in range(int(rng.integers(0, 6)))}
    for k in keys[rng.random(keys.size) < 0.1]:
        index.setdefault(int(k), 90)
    cs, hit = oracle.lookup(index, bh, blk_off, bpc, chunk_off)
    return bh, blk_off, chunk_off, bpc, cs, hit


@pytest.mark.parametrize("seed", range(30))
def test_build_jobs_matches_oracle(seed):
    bh, blk_off, chunk_off, bpc, cs, hit = _lookup_case(seed)
    rng = np.random.default_rng(seed + 100)
    free = rng.permutation(200).astype(np.int32)[:int(rng.integers(0, 40))]
    r1, s1, k1, d1 = oracle.build_jobs(hit, cs, bh, blk_off, chunk_off, bpc, free)
    r2, s2, k2, d2, rc = kv.kv_build_jobs(hit, cs, bh, blk_off, chunk_off, bpc, free)
    assert np.array_equal(r1, r2) and np.array_equal(s1, s2) and np.array_equal(k1, k2) and d1 == d2
    assert rc == (kv.KV_ENOSPC if d2 else kv.KV_OK)


def test_build_jobs_rejects_bad_offsets():
    with pytest.raises(kv.KvError):
        kv.kv_build_jobs(np.array([5], np.int32), np.zeros(1, np.int32), np.zeros(2, np.uint64),
                         np.array([0, 2], np.int64), np.array([0, 1], np.int64), 2, np.zeros(0, np.int32))


def _layout(**over):
    d = dict(num_layers=2, kv_heads=2, head_dim=64, elem_bytes=2, block_size=16, chunk_tokens=64,
             num_blocks=20, num_slots=4, paged_kv_stride=20 * 4096, paged_block_stride=4096)
    d.update(over)
    return kv.make_layout(**d)


def test_validate_jobs():
    lo = _layout()
    bt = np.arange(20, dtype=np.int32)[::-1].reshape(2, 10).copy()
    ok = np.array([[0, 0, 0, 0], [1, 1, 1, 0]], np.int32)
    assert kv.kv_validate_jobs(lo, bt, ok, False) == kv.KV_OK
    assert kv.kv_validate_jobs(lo, bt, ok, True) == kv.KV_OK
    assert kv.kv_validate_jobs(lo, bt, np.array([[0, 0, 0, 0], [1, 0, 0, 0]], np.int32), False) == kv.KV_EDUP
    assert kv.kv_validate_jobs(lo, bt, np.array([[2, 0, 0, 0], [2, 1, 0, 0]], np.int32), True) == kv.KV_EDUP
    # chunk = INT32_MAX: (chunk + 1) * C/B must be formed in 64 bits, or the bound check wraps and passes
    for bad in ([4, 0, 0, 0], [-1, 0, 0, 0], [0, 2, 0, 0], [0, 0, 2, 0], [0, 0, -1, 0], [0, 0, 0, 1],
                [0, 0, 0x7FFFFFFF, 0], [0, 1, 0x3FFFFFFF, 0]):
        assert kv.kv_validate_jobs(lo, bt, np.array([bad], np.int32), False) == kv.KV_ERANGE
    bt2 = bt.copy()
    bt2[0, 2] = 20
    assert kv.kv_validate_jobs(lo, bt2, ok, False) == kv.KV_ERANGE
    bt2[0, 2] = -1
    assert kv.kv_validate_jobs(lo, bt2, ok, True) == kv.KV_ERANGE


def _as(L, kind):
    return lambda *args: L.kv_retrieve_scatter_as(kind, *args)


@pytest.mark.parametrize("over,code", [
    (dict(num_layers=0), kv.KV_EINVAL), (dict(num_layers=129), kv.KV_EINVAL), (dict(elem_bytes=3), kv.KV_EINVAL),
    (dict(chunk_tokens=24), kv.KV_EINVAL), (dict(num_blocks=0), kv.KV_EINVAL), (dict(num_slots=0), kv.KV_EINVAL),
    (dict(paged_block_stride=4096 + 8), kv.KV_EALIGN), (dict(paged_kv_stride=4104), kv.KV_EALIGN),
    (dict(paged_block_stride=2048), kv.KV_EINVAL), (dict(kv_heads=1, head_dim=4, elem_bytes=1, block_size=2,
                                                         chunk_tokens=4), kv.KV_EALIGN)])
def test_copy_calls_reject_bad_layouts_before_any_launch(over, code):
    lo = _layout(**over)
    L = kv.lib()
    layers = (ct.c_void_p * 128)(*([0x10000] * 128))
    for f in (L.kv_retrieve_scatter, _as(L, kv.KV_RETRIEVE_PAIR), _as(L, kv.KV_RETRIEVE_STREAM),
              _as(L, kv.KV_RETRIEVE_QUAD), L.kv_store_gather):
        assert f(ct.byref(lo), 0x10000, layers, 0x10000, 10, 2, 0x10000, 1, None) == code


def test_device_validate_rejects_bad_arguments_before_any_launch():
    L = kv.lib()
    f = L.kv_validate_jobs_device
    A, J, M, S = 0x10000, 0x20000, 0x30000, 0x40000      # block tables, jobs, marks, status (never dereferenced)
    for over in (dict(num_layers=0), dict(chunk_tokens=24), dict(num_blocks=0), dict(num_slots=0)):
        assert f(ct.byref(_layout(**over)), A, 10, 2, J, 1, 0, M, S, None) == kv.KV_EINVAL
    lo = _layout()
    for args in ((A, 10, 2, J, -1, 0, M, S), (A, 10, -1, J, 1, 0, M, S), (A, 0, 2, J, 1, 0, M, S),
                 (A, 10, 2, J, 1, 0, None, S), (A, 10, 2, J, 1, 0, M, None), (None, 10, 2, J, 1, 1, M, S),
                 (A, 10, 2, None, 1, 1, M, S)):
        assert f(ct.byref(lo), *args, None) == kv.KV_EINVAL, args
    for args in ((A, 10, 2, J + 8, 1, 0, M, S), (A, 10, 2, J, 1, 0, M + 2, S), (A, 10, 2, J, 1, 0, M, S + 1),
                 (A + 2, 10, 2, J, 1, 0, M, S)):
        assert f(ct.byref(lo), *args, None) == kv.KV_EALIGN, args


def test_copy_calls_reject_bad_pointers_before_any_launch():
    lo = _layout()
    L = kv.lib()
    good = (ct.c_void_p * 2)(0x10000, 0x20000)
    for f in (L.kv_retrieve_scatter, _as(L, kv.KV_RETRIEVE_UNIT), _as(L, kv.KV_RETRIEVE_PAIR),
              _as(L, kv.KV_RETRIEVE_STREAM), _as(L, kv.KV_RETRIEVE_QUAD), L.kv_store_gather):
        assert f(ct.byref(lo), None, good, 0x10000, 10, 2, 0x10000, 1, None) == kv.KV_EINVAL
        assert f(ct.byref(lo), 0x10008, good, 0x10000, 10, 2, 0x10000, 1, None) == kv.KV_EALIGN
        assert f(ct.byref(lo), 0x10000, (ct.c_void_p * 2)(0x10000, 0x20004), 0x10000, 10, 2, 0x10000, 1,
                 None) == kv.KV_EALIGN
        assert f(ct.byref(lo), 0x10000, (ct.c_void_p * 2)(0x10000, None), 0x10000, 10, 2, 0x10000, 1,
                 None) == kv.KV_EINVAL
        assert f(ct.byref(lo), 0x10000, good, None, 10, 2, 0x10000, 1, None) == kv.KV_EINVAL
        assert f(ct.byref(lo), 0x10000, good, 0x10000, 10, 2, None, 1, None) == kv.KV_EINVAL
        assert f(ct.byref(lo), 0x10000, good, 0x10000, 0, 2, 0x10000, 1, None) == kv.KV_EINVAL
        assert f(ct.byref(lo), 0x10000, good, 0x10000, 10, -1, 0x10000, 1, None) == kv.KV_EINVAL
        assert f(ct.byref(lo), 0x10000, good, 0x10000, 10, 2, 0x10000, -1, None) == kv.KV_EINVAL
        assert f(None, 0x10000, good, 0x10000, 10, 2, 0x10000, 1, None) == kv.KV_EINVAL
        # zero jobs: valid, enqueues nothing
        assert f(ct.byref(lo), 0x10000, good, 0x10000, 10, 2, None, 0, None) == kv.KV_OK


def test_hash_and_lookup_argument_checks():
    L = kv.lib()
    assert L.kv_hash_prefix(None, None, 0, 0, None, None, None) == kv.KV_OK           # empty batch
    assert L.kv_hash_prefix(None, 0x1000, 3, 0, 0x1000, 0x1000, None) == kv.KV_EINVAL
    assert L.kv_hash_prefix(0x1000, 0x1000, -1, 0, 0x1000, 0x1000, None) == kv.KV_EINVAL
    assert L.kv_lookup(None, 0x1000, 0x1000, 1, 1, 0x1000, 0x1000, 0x1000, None) == kv.KV_EINVAL
    assert L.kv_index_create(0, ct.byref(ct.c_void_p())) == kv.KV_EINVAL
    assert L.kv_index_create(10, None) == kv.KV_EINVAL
    assert L.kv_index_destroy(None) == kv.KV_EINVAL
    assert L.kv_index_insert(None, None, None, 0, None) == kv.KV_EINVAL
    assert L.kv_host_device_pointer(None, ct.byref(ct.c_void_p())) == kv.KV_EINVAL


@pytest.mark.parametrize("seed", range(5))
def test_group_jobs_by_slot_is_a_stable_sort(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 300))
    jobs = np.stack([rng.integers(0, 20, n), np.arange(n), rng.integers(0, 4, n), np.zeros(n, np.int64)], 1).astype(np.int32)
    got = kv.kv_group_jobs_by_slot(jobs)
    want = jobs[np.argsort(jobs[:, 0], kind="stable")]
    assert np.array_equal(got, want)
    assert kv.host_lib().kv_group_jobs_by_slot(None, -1) == kv.KV_EINVAL


def test_stage_calls_check_arguments_before_any_copy():
    lo = _layout()
    L = kv.lib()
    sl = np.array([0, 1, 3], np.int32)
    for f in (L.kv_stage_in, L.kv_stage_out):
        assert f(ct.byref(lo), 0x10000, 0x20000, None, 0, None) == kv.KV_OK            # nothing to copy
        assert f(ct.byref(lo), 0x10000, 0x20000, sl.ctypes.data, -1, None) == kv.KV_EINVAL
        assert f(ct.byref(lo), None, 0x20000, sl.ctypes.data, 3, None) == kv.KV_EINVAL
        assert f(ct.byref(lo), 0x10000, None, sl.ctypes.data, 3, None) == kv.KV_EINVAL
        assert f(ct.byref(lo), 0x10000, 0x20000, None, 3, None) == kv.KV_EINVAL
        assert f(None, 0x10000, 0x20000, sl.ctypes.data, 3, None) == kv.KV_EINVAL
        bad = _layout(num_layers=0)
        assert f(ct.byref(bad), 0x10000, 0x20000, sl.ctypes.data, 3, None) == kv.KV_EINVAL
        for s in (-1, lo.num_slots):
            b = np.array([0, s], np.int32)
            assert f(ct.byref(lo), 0x10000, 0x20000, b.ctypes.data, 2, None) == kv.KV_ERANGE


def test_pipeline_calls_check_arguments():
    L = kv.lib()
    h = ct.c_void_p()
    assert L.kv_pipeline_create(0, ct.byref(h)) == kv.KV_EINVAL
    assert L.kv_pipeline_create(-3, ct.byref(h)) == kv.KV_EINVAL
    assert L.kv_pipeline_create(4, None) == kv.KV_EINVAL
    assert L.kv_pipeline_destroy(None) == kv.KV_EINVAL
    lo = _layout()
    layers = (ct.c_void_p * 2)(0x10000, 0x20000)
    jobs = np.zeros((1, 4), np.int32)
    assert L.kv_retrieve_pipelined(None, ct.byref(lo), 0x10000, 0x10000, layers, 0x10000, 10, 2, jobs.ctypes.data,
                                   0x10000, 1, 1, None, None) == kv.KV_EINVAL
    assert L.kv_retrieve_pipelined(0x1000, ct.byref(lo), 0x10000, 0x10000, layers, 0x10000, 10, 2,
                                   jobs.ctypes.data, 0x10000, 1, 0, None, None) == kv.KV_EINVAL


def _jobs(slots):
    j = np.zeros((len(slots), 4), np.int32)
    j[:, 0] = slots
    j[:, 1] = np.arange(len(slots))
    return j


def test_retrieve_plan_rules():
    lo32 = kv.make_layout(2, 8, 128, 2, 16, 256, 1000, 700, 1000 * 32768, 32768)     # 32 KiB segments
    lo4 = kv.make_layout(2, 2, 64, 2, 16, 64, 1000, 700, 1000 * 4096, 4096)          # 4 KiB segments
    P = kv.kv_retrieve_plan
    assert P(lo32, np.zeros((0, 4), np.int32)) == kv.KV_RETRIEVE_UNIT
    assert P(lo32, _jobs(np.arange(100))) == kv.KV_RETRIEVE_STREAM                   # every slot once
    assert P(lo32, _jobs(np.arange(100)[::-1])) == kv.KV_RETRIEVE_STREAM
    assert P(lo32, _jobs([0, 1, 0, 1])) == kv.KV_RETRIEVE_UNIT                        # no run, but not distinct
    groups8 = np.repeat(np.arange(64), 8)                                             # 64 chunks x 8 requests
    assert P(lo32, _jobs(groups8)) == kv.KV_RETRIEVE_PAIR
    assert P(lo4, _jobs(groups8)) == kv.KV_RETRIEVE_UNIT                              # pairs only at 32 KiB
    assert P(lo32, _jobs(np.repeat(np.arange(4), 64))) == kv.KV_RETRIEVE_UNIT         # groups of 64
    assert P(lo32, _jobs(np.repeat(np.arange(40), 16))) == kv.KV_RETRIEVE_PAIR        # groups of 16
    odd = np.concatenate([np.repeat(np.arange(50), 3), np.repeat(np.arange(50, 60), 2)])
    assert P(lo32, _jobs(odd)) == kv.KV_RETRIEVE_UNIT                                 # groups of 3: pairs misalign
    rng = np.random.default_rng(3)
    sizes = rng.integers(1, 9, 200)
    assert P(lo32, _jobs(np.repeat(np.arange(200), sizes))) == kv.KV_RETRIEVE_UNIT    # irregular groups
    L = kv.host_lib()
    assert L.kv_retrieve_plan(None, None, 0) == kv.KV_EINVAL
    assert L.kv_retrieve_plan(ct.byref(lo32), None, 3) == kv.KV_EINVAL
    assert L.kv_retrieve_plan(ct.byref(lo32), None, -1) == kv.KV_EINVAL


def test_retrieve_as_rejects_unknown_kinds():
    lo = _layout()
    L = kv.lib()
    layers = (ct.c_void_p * 2)(0x10000, 0x20000)
    for kind in (-1, 4, 99):
        assert L.kv_retrieve_scatter_as(kind, ct.byref(lo), 0x10000, layers, 0x10000, 10, 2, 0x10000, 1,
                                        None) == kv.KV_EINVAL


def test_probe_checks_arguments_before_any_launch():
    # the measurement reference takes the retrieve's arguments plus the slots it reads
    lo = _layout()
    L = kv.lib()
    f = L.kv_probe_mixed_traffic
    good = (ct.c_void_p * 2)(0x10000, 0x20000)
    A, J, S = 0x10000, 0x20000, 0x30000                  # block tables, jobs, slots (never dereferenced)
    assert f(ct.byref(_layout(num_layers=0)), A, good, A, 10, 2, J, 1, S, 1, 7, None) == kv.KV_EINVAL
    assert f(ct.byref(lo), 0x10008, good, A, 10, 2, J, 1, S, 1, 7, None) == kv.KV_EALIGN
    assert f(ct.byref(lo), A, good, A, 10, 2, None, 1, S, 1, 7, None) == kv.KV_EINVAL
    assert f(ct.byref(lo), A, good, A, 10, 2, J, 1, S, -1, 7, None) == kv.KV_EINVAL
    assert f(ct.byref(lo), A, good, A, 10, 2, J, 1, None, 1, 7, None) == kv.KV_EINVAL
    # 2^31 or more segments in one launch: refused (keeps the kernel's index arithmetic in 64 bits)
    assert f(ct.byref(lo), A, good, A, 10, 2, J, 2**31 - 1, S, 0, 7, None) == kv.KV_EINVAL
    # nothing to move: valid, enqueues nothing
    assert f(ct.byref(lo), A, good, A, 10, 2, None, 0, None, 0, 7, None) == kv.KV_OK


@pytest.mark.parametrize("seed", range(10))
def test_chunk_keys_match_oracle(seed):
    bh, blk_off, chunk_off, bpc, cs, hit = _lookup_case(seed)
    got = kv.kv_chunk_keys(bh, blk_off, bpc, chunk_off)
    assert np.array_equal(got, oracle.chunk_keys(bh, blk_off, bpc))
    if blk_off.size > 1:
        with pytest.raises(kv.KvError):      # offsets that do not match blocks_per_chunk
            bad = chunk_off.copy()
            bad[-1] += 1
            kv.kv_chunk_keys(bh, blk_off, bpc, bad)
