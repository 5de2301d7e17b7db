"""kv_index_insert_static, the allocation-free insert, against kv_index_insert.

Both entry points are called through the C ABI on two indexes fed the same
keys: a set-up insert (the first upload of an index sends its whole table),
then two incremental inserts in a row, the second smaller and partly
re-assigning slots of keys already present.  After each call every key's slot
as seen by kv_lookup on the device must be identical through both indexes,
and equal to the oracle's lookup against a plain dict.  Sizes beyond the
fixed capacity are rejected without inserting anything."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_35065_amd as kv

pytestmark = pytest.mark.gpu


def _insert(fn, idx, keys, slots, stream):
    keys = np.ascontiguousarray(keys, np.uint64)
    slots = np.ascontiguousarray(slots, np.int32)
    return fn(idx.handle, keys.ctypes.data, slots.ctypes.data, keys.size, stream.cuda_stream)


def _device_slots(idx, keys, stream):
    """kv_lookup with one-block chunks: chunk_slot holds every key's slot (-1 if absent)."""
    per = 64
    n = keys.size
    R = (n + per - 1) // per
    lens = np.full(R, per, np.int64)
    lens[-1] = n - per * (R - 1)
    off = np.zeros(R + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    d_bh = torch.from_numpy(keys.view(np.int64).copy()).cuda()
    d_off = torch.from_numpy(off).cuda()
    d_slot = torch.empty(n, dtype=torch.int32, device="cuda")
    d_hit = torch.empty(R, dtype=torch.int32, device="cuda")
    kv.kv_lookup(idx, d_bh, d_off, R, 1, d_off, d_slot, d_hit, stream)
    stream.synchronize()
    return d_slot.cpu().numpy(), d_hit.cpu().numpy(), off


def test_static_insert_matches_insert_on_two_calls():
    L = kv.lib()
    rng = np.random.default_rng(77)
    stream = torch.cuda.current_stream()
    a, b = kv.KvIndex(40000), kv.KvIndex(40000)   # 2^17 positions; incremental uploads up to 16,384 pairs
    ref = {}
    universe = rng.integers(1, 2**63, 30000, dtype=np.int64).astype(np.uint64)
    setup = universe[:16]
    calls = [(universe[16:12016], rng.integers(0, 1 << 20, 12000)),          # 12,000 new keys
             (np.concatenate([universe[12016:14016], universe[100:1100]]),  # 2,000 new, 1,000 re-assigned
              rng.integers(0, 1 << 20, 3000))]
    for keys, slots in [(setup, np.arange(16))] + calls:
        print(f"[no-alloc] insert of {keys.size} keys", flush=True)
        assert _insert(L.kv_index_insert, a, keys, slots, stream) == kv.KV_OK
        assert _insert(L.kv_index_insert_static, b, keys, slots, stream) == kv.KV_OK
        for k, s in zip(keys, slots):
            ref[int(k)] = int(s)
        probe = np.concatenate([universe, rng.integers(1, 2**63, 500, dtype=np.int64).astype(np.uint64)])
        sa, ha, off = _device_slots(a, probe, stream)
        sb, hb, _ = _device_slots(b, probe, stream)
        assert np.array_equal(sa, sb) and np.array_equal(ha, hb)
        so, ho = oracle.lookup(ref, probe, off, 1, off)
        assert np.array_equal(sb, so) and np.array_equal(hb, ho)
        assert a.size() == b.size() == len(ref)
    # beyond the fixed capacity: rejected before anything is inserted
    big = rng.integers(1, 2**63, kv.KV_INDEX_STATIC_MAX_PAIRS + 1, dtype=np.int64).astype(np.uint64)
    before = b.size()
    assert _insert(L.kv_index_insert_static, b, big, np.zeros(big.size, np.int32), stream) == kv.KV_ELIMIT
    assert b.size() == before
    assert b"fixed capacity" in L.kv_strerror(kv.KV_ELIMIT)
    a.destroy()
    b.destroy()
