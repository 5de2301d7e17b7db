"""Property-based checks of the oracle (hypothesis): the invariants of the
chained hash, the prefix lookup and the copies hold for arbitrary inputs,
not just the seeded trials of the other tests."""
import math

import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
from workloads import KVShape

tokens = st.lists(st.integers(-2**31, 2**31 - 1), min_size=0, max_size=200)


def _h(toks, seed=0):
    t = np.array(toks, np.int64).astype(np.int32)
    return oracle.hash_prefix(t, np.array([0, t.size], np.int64), seed)


@settings(max_examples=200, deadline=None)
@given(tokens, st.integers(0, 200), st.integers(0, 2**64 - 1))
def test_prefix_property(toks, cut, seed):
    full = _h(toks, seed)
    part = _h(toks[:cut], seed)
    assert part.size == min(cut, len(toks)) // 16
    assert np.array_equal(part, full[:part.size])


@settings(max_examples=200, deadline=None)
@given(tokens.filter(lambda t: len(t) >= 16), st.data())
def test_change_moves_exactly_the_later_blocks(toks, data):
    p = data.draw(st.integers(0, len(toks) - 1))
    v = data.draw(st.integers(-2**31, 2**31 - 1).filter(lambda x: x != toks[p]))
    t2 = list(toks)
    t2[p] = v
    a, b = _h(toks), _h(t2)
    blk = p // 16
    assert np.array_equal(a[:blk], b[:blk])
    assert np.all(a[blk:] != b[blk:])


@settings(max_examples=100, deadline=None)
@given(st.integers(1, 3), st.sampled_from([1, 2, 8]), st.sampled_from([64, 128]), st.sampled_from([1, 2, 4]),
       st.sampled_from([16, 32]), st.integers(1, 4), st.integers(0, 2**32 - 1))
def test_store_then_retrieve_is_identity(L, H, D, e, B, cpb, seed):
    rng = np.random.default_rng(seed)
    C = B * cpb
    shape = KVShape(L, H, D, e, B, C)
    R, chunks = 3, 2
    nb = R * chunks * cpb + 3
    seg = shape.seg_bytes
    lo = oracle.make_layout(shape, nb, R * chunks, nb * seg, seg)
    bt = rng.permutation(nb)[:R * chunks * cpb].astype(np.int32).reshape(R, chunks * cpb)
    layers = [rng.integers(0, 256, 2 * nb * seg, dtype=np.uint8) for _ in range(L)]
    jobs = np.array([[r * chunks + j, r, j, 0] for r in range(R) for j in range(chunks)], np.int32)
    staged = np.zeros(R * chunks * shape.slot_bytes, np.uint8)
    oracle.store_gather(lo, staged, layers, bt, jobs)
    bt2 = rng.permutation(nb)[:bt.size].astype(np.int32).reshape(bt.shape)
    fresh = [np.zeros_like(a) for a in layers]
    oracle.retrieve_scatter(lo, staged, fresh, bt2, jobs)
    for l in range(L):
        a = layers[l].reshape(2, nb, seg)
        b = fresh[l].reshape(2, nb, seg)
        assert np.array_equal(b[:, bt2.ravel()], a[:, bt.ravel()])


finite = st.floats(allow_nan=False)


@settings(max_examples=500, deadline=None)
@given(finite, finite, st.integers(0, 2**64 - 1), st.integers(0, 2**64 - 1), st.integers(0, 2**64 - 1),
       st.integers(0, 2**64 - 1), st.booleans())
def test_commit_rule_properties(ttu, ttr, free, new, total, budget, req):
    d = oracle.commit_should_stage(ttu, ttr, free, new, total, budget, req)
    if new > total:
        assert d == oracle.EINVAL
        return
    eligible = ttu <= ttr or req
    fits = total <= budget and new <= free
    assert (d == oracle.DEFER) == (not eligible)
    assert (d == oracle.COMMIT) == (eligible and fits)
    assert (d == oracle.ORDINARY) == (eligible and not fits and req)
    assert (d == oracle.BLOCKED) == (eligible and not fits and not req)
