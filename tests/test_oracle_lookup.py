"""Pins for the oracle's lookup and host job build.

Lookup is checked against a brute-force prefix match on tokens that uses no
hashing at all: chunk j of request r is a hit iff some stored chunk's full
token prefix equals the request's first (j+1)*C tokens, and the hit count is
the longest such run from chunk 0 (prefix semantics: the matched prefix
fixes which objects a request reads and in what order, Section 2.1).

Job build is checked against its invariants: retrieve jobs are exactly the
hit prefix; every distinct missing key gets at most one store job, the first
(request, chunk) in order; slots come from the free list in order; and
misses beyond the free slots are counted as dropped.
"""
import numpy as np
import pytest

import oracle


def _batch(reqs):
    tok_off = np.zeros(len(reqs) + 1, np.int64)
    np.cumsum([len(r) for r in reqs], out=tok_off[1:])
    toks = np.concatenate(reqs).astype(np.int32) if reqs else np.zeros(0, np.int32)
    return toks, tok_off


def _brute_force(stored_prefixes, reqs, C):
    """stored_prefixes: list of (token tuple of length (j+1)*C, slot)."""
    table = {tuple(p): s for p, s in stored_prefixes}
    slots, hits = [], []
    for r in reqs:
        nc = len(r) // C
        cs = [table.get(tuple(int(t) for t in r[:(j + 1) * C]), -1) for j in range(nc)]
        h = 0
        while h < nc and cs[h] >= 0:
            h += 1
        slots += cs
        hits.append(h)
    return np.array(slots, np.int32), np.array(hits, np.int32)


@pytest.mark.parametrize("trial", range(25))
@pytest.mark.parametrize("C", [16, 32, 64])
def test_lookup_equals_brute_force_prefix_match(trial, C):
    rng = np.random.default_rng(1000 * C + trial)
    vocab = int(rng.choice([2, 3, 32000]))      # tiny vocabularies force many equal prefixes
    bases = [rng.integers(0, vocab, 6 * C) for _ in range(3)]
    reqs = []
    for _ in range(int(rng.integers(1, 8))):
        b = bases[int(rng.integers(0, 3))]
        k = int(rng.integers(0, 6 * C + 1))
        tail = rng.integers(0, vocab, int(rng.integers(0, 3 * C)))
        reqs.append(np.concatenate([b[:k], tail]).astype(np.int32))
    # stored chunks: random chunk prefixes of the bases and of the requests
    stored, seen = [], set()
    slot = 0
    for src in bases + reqs:
        for j in range(len(src) // C):
            if rng.random() < 0.5:
                p = tuple(int(t) for t in src[:(j + 1) * C])
                if p not in seen:
                    seen.add(p)
                    stored.append((p, slot))
                    slot += 1
    toks, tok_off = _batch(reqs)
    bh = oracle.hash_prefix(toks, tok_off, seed=0)
    blk_off = oracle.block_offsets(tok_off)
    bpc = C // 16
    index = {}
    for p, s in stored:
        pt = np.array(p, np.int32)
        h = oracle.hash_prefix(pt, np.array([0, pt.size], np.int64), seed=0)
        index[int(h[-1])] = s
    assert len(index) == len(stored)            # no key collisions among distinct prefixes
    cs, hits = oracle.lookup(index, bh, blk_off, bpc)
    bcs, bhits = _brute_force(stored, reqs, C)
    assert np.array_equal(cs, bcs)
    assert np.array_equal(hits, bhits)


def test_lookup_empty_batch_and_empty_index():
    toks, tok_off = _batch([np.zeros(0, np.int32), np.arange(40, dtype=np.int32)])
    bh = oracle.hash_prefix(toks, tok_off)
    blk_off = oracle.block_offsets(tok_off)
    cs, hits = oracle.lookup({}, bh, blk_off, 1)
    assert list(hits) == [0, 0] and list(cs) == [-1, -1]


def _jobs_case(seed, free):
    rng = np.random.default_rng(seed)
    C = 32
    shared = rng.integers(0, 32000, 4 * C)
    reqs = [np.concatenate([shared[:int(rng.integers(0, 4)) * C], rng.integers(0, 32000, int(rng.integers(0, 5 * C)))]).astype(np.int32)
            for _ in range(6)]
    reqs.append(reqs[0].copy())                 # an exact duplicate request
    toks, tok_off = _batch(reqs)
    bh = oracle.hash_prefix(toks, tok_off)
    blk_off = oracle.block_offsets(tok_off)
    bpc = C // 16
    chunk_off = oracle.chunk_offsets(blk_off, bpc)
    keys = oracle.chunk_keys(bh, blk_off, bpc)
    # index: the first two chunks of the shared stream, plus one chunk that
    # sits after a miss in some request (present but not a hit)
    st = np.array(shared, np.int32)
    sh = oracle.hash_prefix(st, np.array([0, st.size], np.int64))
    index = {int(sh[bpc - 1]): 100, int(sh[2 * bpc - 1]): 101}
    if keys.size > 3:
        index.setdefault(int(keys[3]), 102)
    cs, hits = oracle.lookup(index, bh, blk_off, bpc, chunk_off)
    retr, store, skeys, dropped = oracle.build_jobs(hits, cs, bh, blk_off, chunk_off, bpc, free)
    return dict(reqs=reqs, chunk_off=chunk_off, keys=keys, index=index, cs=cs, hits=hits,
                retr=retr, store=store, skeys=skeys, dropped=dropped)


@pytest.mark.parametrize("seed", range(10))
def test_job_build_invariants(seed):
    free = np.arange(200, 260, dtype=np.int32)
    d = _jobs_case(seed, free)
    co, cs, hits, keys = d["chunk_off"], d["cs"], d["hits"], d["keys"]
    R = len(d["reqs"])
    exp_retr = [[int(cs[co[r] + j]), r, j, 0] for r in range(R) for j in range(int(hits[r]))]
    assert d["retr"].tolist() == exp_retr
    # misses in (r, j) order, first occurrence of each key wins
    want, seen = [], set()
    for r in range(R):
        for j in range(int(hits[r]), int(co[r + 1] - co[r])):
            if cs[co[r] + j] >= 0:
                continue
            k = int(keys[co[r] + j])
            if k in seen:
                continue
            seen.add(k)
            want.append((r, j, k))
    assert [(int(a[1]), int(a[2])) for a in d["store"]] == [(r, j) for r, j, _ in want]
    assert [int(k) for k in d["skeys"]] == [k for _, _, k in want]
    assert d["store"][:, 0].tolist() == free[:len(want)].tolist()
    assert d["dropped"] == 0
    assert not set(int(k) for k in d["skeys"]) & set(d["index"].keys())


def test_job_build_drops_when_slots_run_out():
    full = _jobs_case(3, np.arange(0, 1000, dtype=np.int32))
    n = len(full["store"])
    assert n >= 3
    part = _jobs_case(3, np.arange(0, 2, dtype=np.int32))
    assert len(part["store"]) == 2
    assert part["dropped"] == n - 2
    assert part["store"][:, 1:3].tolist() == full["store"][:2, 1:3].tolist()
