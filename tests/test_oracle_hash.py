"""Pins for the oracle's chained prefix hash.

The paper does not define the hash (it takes its prefix matching from LMCache,
Section 4), so the oracle's hash is this library's own definition: a 64-bit
chain over 16-token blocks built on the SplitMix64 finalizer M.  These tests
pin it to things outside the oracle:
  * M against SplitMix64's published output sequences;
  * M is a bijection (inverted here from the xor-shift / odd-multiply algebra);
  * structural invariants of a chained prefix hash over 16-token blocks
    (prefix property, locality of a token change, restartability of the
    chain from an intermediate hash, additivity of the block digest over
    positions, position dependence, partial blocks ignored);
  * frozen golden vectors (regression guard, written by tests/golden/make_golden.py
    from the oracle alone).
"""
import os

import numpy as np
import pytest

import oracle

MASK = (1 << 64) - 1
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hash_vectors.txt")


def test_splitmix64_published_sequence_seed_1234567():
    # SplitMix64 (state += 0x9E3779B97F4A7C15; output M(state)) from seed
    # 1234567: the first five outputs as published with the generator's
    # reference description (e.g. the Rosetta Code "Splitmix64" task).
    assert oracle.splitmix64_sequence(1234567, 5) == [
        6457827717110365317, 3203168211198807973, 9817491932198370423,
        4593380528125082431, 16408922859458223821]


def test_splitmix64_published_sequence_seed_0():
    # First outputs of splitmix64.c (Vigna, public domain) seeded with 0.
    assert oracle.splitmix64_sequence(0, 3) == [
        0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def _unxorshift(y, s):
    x = y
    for _ in range(64 // s + 1):
        x = y ^ (x >> s)
    return x & MASK


def test_mix64_is_a_bijection():
    c1 = pow(0xBF58476D1CE4E5B9, -1, 1 << 64)
    c2 = pow(0x94D049BB133111EB, -1, 1 << 64)
    rng = np.random.default_rng(7)
    xs = [0, 1, MASK, 1 << 63] + [int(v) for v in rng.integers(0, 2**63, 200, dtype=np.int64)] \
        + [int(v) | (1 << 63) for v in rng.integers(0, 2**63, 50, dtype=np.int64)]
    for x in xs:
        y = oracle.mix64(x)
        z = _unxorshift(y, 31)
        z = (z * c2) & MASK
        z = _unxorshift(z, 27)
        z = (z * c1) & MASK
        z = _unxorshift(z, 30)
        assert z == x


def _hash_one(toks, seed=0):
    toks = np.asarray(toks, np.int32)
    return oracle.hash_prefix(toks, np.array([0, toks.size], np.int64), seed)


@pytest.mark.parametrize("n", [0, 1, 15, 16, 17, 31, 32, 33, 255, 256, 257])
def test_partial_trailing_block_gives_no_hash(n):
    rng = np.random.default_rng(n)
    h = _hash_one(rng.integers(0, 32000, n))
    assert h.size == n // 16


def test_prefix_property():
    rng = np.random.default_rng(1)
    toks = rng.integers(0, 32000, 16 * 40 + 5).astype(np.int32)
    full = _hash_one(toks)
    for n in [16, 17, 64, 100, 320, 640]:
        part = _hash_one(toks[:n])
        assert np.array_equal(part, full[:n // 16])


def test_token_change_is_local_to_later_blocks():
    rng = np.random.default_rng(2)
    toks = rng.integers(0, 32000, 16 * 24).astype(np.int32)
    base = _hash_one(toks)
    for p in rng.integers(0, toks.size, 40):
        t2 = toks.copy()
        t2[p] = (t2[p] + 1 + rng.integers(0, 31999)) % 32000
        h2 = _hash_one(t2)
        b = p // 16
        assert np.array_equal(h2[:b], base[:b])
        assert np.all(h2[b:] != base[b:])


def test_chain_restarts_from_intermediate_hash():
    # h_b depends on earlier blocks only through h_{b-1}: hashing the tail with
    # seed = h_{b-1} reproduces h_b, h_{b+1}, ...
    rng = np.random.default_rng(3)
    toks = rng.integers(0, 32000, 16 * 12).astype(np.int32)
    for seed in [0, 12345, MASK]:
        full = _hash_one(toks, seed)
        for b in range(1, 12):
            tail = _hash_one(toks[16 * b:], int(full[b - 1]))
            assert np.array_equal(tail, full[b:])


def test_seed_changes_every_hash():
    rng = np.random.default_rng(4)
    toks = rng.integers(0, 32000, 16 * 10).astype(np.int32)
    assert np.all(_hash_one(toks, 0) != _hash_one(toks, 1))


def test_block_digest_is_additive_over_positions():
    # Changing token j from a to b shifts the digest by an amount that does
    # not depend on the other 15 tokens (the digest is a sum of per-position
    # words), and swapping two unequal tokens changes it (position matters).
    rng = np.random.default_rng(5)
    for _ in range(50):
        x = rng.integers(0, 32000, 16).astype(np.int32)
        y = rng.integers(0, 32000, 16).astype(np.int32)
        j = int(rng.integers(0, 16))
        a, b = int(rng.integers(0, 32000)), int(rng.integers(0, 32000))
        x[j] = y[j] = a
        xb, yb = x.copy(), y.copy()
        xb[j] = yb[j] = b
        dx = (oracle.block_digest(xb) - oracle.block_digest(x)) & MASK
        dy = (oracle.block_digest(yb) - oracle.block_digest(y)) & MASK
        assert dx == dy
        i, k = 0, 15
        if x[i] != x[k]:
            s = x.copy()
            s[i], s[k] = x[k], x[i]
            assert oracle.block_digest(s) != oracle.block_digest(x)


def test_batch_equals_single_and_equal_prefixes_share_keys():
    rng = np.random.default_rng(6)
    shared = rng.integers(0, 32000, 200).astype(np.int32)
    reqs = [np.concatenate([shared[:k], rng.integers(0, 32000, n).astype(np.int32)])
            for k, n in [(200, 57), (128, 300), (0, 33), (160, 0), (5, 10)]]
    tok_off = np.zeros(len(reqs) + 1, np.int64)
    np.cumsum([r.size for r in reqs], out=tok_off[1:])
    batch = oracle.hash_prefix(np.concatenate(reqs), tok_off)
    blk_off = oracle.block_offsets(tok_off)
    for i, r in enumerate(reqs):
        assert np.array_equal(batch[blk_off[i]:blk_off[i + 1]], _hash_one(r))
    h0, h1 = _hash_one(reqs[0]), _hash_one(reqs[1])
    assert np.array_equal(h0[:8], h1[:8])      # 128 shared tokens = 8 blocks
    assert h0[8] != h1[8] or np.array_equal(reqs[0][:144], reqs[1][:144])


def test_negative_and_large_token_ids_are_words():
    # Token ids are taken as unsigned 32-bit words: -1 and 0xFFFFFFFF agree.
    a = _hash_one(np.full(16, -1, np.int32))
    b = _hash_one(np.array([0xFFFFFFFF] * 16, np.uint32).view(np.int32))
    assert np.array_equal(a, b)
    assert not np.array_equal(a, _hash_one(np.full(16, 0x7FFFFFFF, np.int32)))


def test_rejects_inconsistent_offsets():
    toks = np.zeros(32, np.int32)
    with pytest.raises(ValueError):
        oracle.hash_prefix(toks, np.array([0, 32], np.int64), 0, np.array([0, 3], np.int64))


def _read_golden():
    cases = []
    with open(GOLDEN) as f:
        cur = None
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, v = line.split("=", 1)
            if k == "case":
                cur = {"name": v}
                cases.append(cur)
            elif k in ("tokens",):
                cur[k] = np.array([int(t) for t in v.split()] if v.strip() else [], np.int64).astype(np.int32)
            elif k in ("seed",):
                cur[k] = int(v, 0)
            elif k == "hashes":
                cur[k] = [int(t, 16) for t in v.split()]
    return cases


def test_golden_vectors():
    cases = _read_golden()
    assert len(cases) >= 5
    for c in cases:
        got = _hash_one(c["tokens"], c["seed"])
        assert [int(x) for x in got] == c["hashes"], c["name"]
