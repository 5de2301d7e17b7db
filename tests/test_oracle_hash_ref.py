"""The oracle's prefix hash against ``tests/ref_hash.py``, an independent
Python implementation written from the documented definition.

This is what pins the composition of the hash that the invariants cannot
see: the position word (j+1) << 32, the xor with G in the chain, and token
ids read as unsigned 32-bit words.  The reference is itself pinned to
SplitMix64's published outputs, and the frozen golden vectors (written by the
oracle) must agree with it too."""
import os

import numpy as np
import pytest

import oracle
import ref_hash as R

MASK = (1 << 64) - 1
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hash_vectors.txt")


def test_reference_finalizer_matches_published_splitmix64():
    # the same published sequences the oracle's M is checked against
    assert R.splitmix64(1234567, 5) == [6457827717110365317, 3203168211198807973, 9817491932198370423,
                                        4593380528125082431, 16408922859458223821]
    assert R.splitmix64(0, 3) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_reference_token_word_reads_ids_unsigned():
    assert R.token_word(0, -1) == 0xFFFFFFFF + (1 << 32)
    assert R.token_word(15, -0x80000000) == 0x80000000 + (16 << 32)
    assert R.token_word(3, 0x7FFFFFFF) == 0x7FFFFFFF + (4 << 32)


def _oracle_chain(toks, seed):
    t = np.asarray(toks, np.int64).astype(np.int32)
    return [int(x) for x in oracle.hash_prefix(t, np.array([0, t.size], np.int64), seed)]


def _edge_inputs():
    rng = np.random.default_rng(515)
    ids = [0, 1, -1, 0x7FFFFFFF, -0x80000000, 31999, -12345]
    yield "empty", [], 0
    for n in (15, 16, 17):
        yield f"ramp_{n}", list(range(n)), 0
        yield f"ramp_{n}_seed_max", list(range(n)), MASK
    yield "negative_ids", [-1, -2, -3, -0x80000000] * 4, 0
    yield "max_positive_ids", [0x7FFFFFFF] * 32, 0
    yield "mixed_extremes", [ids[k % len(ids)] for k in range(48)], MASK
    yield "full_range_random_64", [int(v) for v in rng.integers(-2**31, 2**31, 64)], 0
    for seed in (0, MASK, 0x5EED, 1 << 63):
        yield f"random_256_seed_{seed:x}", [int(v) for v in rng.integers(0, 32000, 256)], seed
        yield f"random_300_seed_{seed:x}", [int(v) for v in rng.integers(0, 32000, 300)], seed


@pytest.mark.parametrize("name,toks,seed", list(_edge_inputs()), ids=[c[0] for c in _edge_inputs()])
def test_oracle_chain_equals_reference(name, toks, seed):
    assert _oracle_chain(toks, seed) == R.chain(toks, seed), name


def test_oracle_digest_equals_reference():
    rng = np.random.default_rng(9)
    for _ in range(200):
        blk = rng.integers(-2**31, 2**31, 16).astype(np.int32)
        assert oracle.block_digest(blk) == R.digest(blk.tolist())


def test_oracle_batch_and_chunk_keys_equal_reference():
    # a ragged batch through the oracle's batch interface, and chunk keys as the lookup forms them
    rng = np.random.default_rng(10)
    reqs = [rng.integers(-2**31, 2**31, n).astype(np.int32) for n in (0, 15, 16, 17, 256, 300, 1024, 1031)]
    tok_off = np.zeros(len(reqs) + 1, np.int64)
    np.cumsum([r.size for r in reqs], out=tok_off[1:])
    seed = 0xDEADBEEFCAFEF00D
    bh = oracle.hash_prefix(np.concatenate(reqs), tok_off, seed)
    blk_off = oracle.block_offsets(tok_off)
    for i, r in enumerate(reqs):
        assert [int(x) for x in bh[blk_off[i]:blk_off[i + 1]]] == R.chain(r.tolist(), seed)
    keys = oracle.chunk_keys(bh, blk_off, 256 // 16)
    want = [k for r in reqs for k in R.chunk_keys(r.tolist(), 256, seed)]
    assert [int(k) for k in keys] == want


def test_golden_vectors_equal_reference():
    # the golden file was written by the oracle; it must also be what the definition gives
    from test_oracle_hash import _read_golden
    cases = _read_golden()
    assert len(cases) >= 5
    for c in cases:
        assert c["hashes"] == R.chain(c["tokens"].tolist(), c["seed"]), c["name"]
