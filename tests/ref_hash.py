"""A second, independent implementation of the library's chained prefix hash.

Written in plain Python integers from the documented definition of
``kv_hash_prefix`` (the paper takes its prefix matching from LMCache without defining
a hash, Section 4, so the definition is this library's own):

    M      SplitMix64's output finalizer: xor-shift right 30, multiply by
           0xBF58476D1CE4E5B9, xor-shift right 27, multiply by
           0x94D049BB133111EB, xor-shift right 31 (all mod 2^64)
    G      0x9E3779B97F4A7C15, SplitMix64's golden-ratio increment
    word   for position j in 0..15 of a block and token id t (an int32 read
           as an unsigned 32-bit word):  w(j, t) = (t mod 2^32) + (j+1) * 2^32
    d_b    = sum over j of M(w(j, tok[16b + j]))               (mod 2^64)
    h_b    = M(h_{b-1} xor d_b xor G), with h_{-1} = seed
    key    of chunk c (C tokens, C a multiple of 16): h at the chunk's last
           block, h_{(c+1)*C/16 - 1}

Only complete 16-token blocks are hashed.  This module imports nothing from
the oracle or the library: the tests compare the three against it.
"""
from __future__ import annotations

from typing import Iterable, List

MOD = 1 << 64
MASK = MOD - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15
_MUL1 = 0xBF58476D1CE4E5B9
_MUL2 = 0x94D049BB133111EB


def finalize(z: int) -> int:
    """SplitMix64's finalizer M on a 64-bit word."""
    z &= MASK
    for shift, mul in ((30, _MUL1), (27, _MUL2)):
        z ^= z >> shift
        z = (z * mul) % MOD
    return z ^ (z >> 31)


def splitmix64(seed: int, count: int) -> List[int]:
    """The first ``count`` outputs of the SplitMix64 generator: the state
    advances by G and each output is M(state)."""
    state, out = seed & MASK, []
    for _ in range(count):
        state = (state + GOLDEN_GAMMA) % MOD
        out.append(finalize(state))
    return out


def token_word(position: int, token: int) -> int:
    """w(j, t): the id as an unsigned 32-bit word in the low half, j+1 in the high half."""
    return (token % (1 << 32)) + (position + 1) * (1 << 32)


def digest(block: Iterable[int]) -> int:
    """d_b of one 16-token block."""
    toks = list(block)
    assert len(toks) == 16
    total = 0
    for j, t in enumerate(toks):
        total += finalize(token_word(j, int(t)))
    return total % MOD


def chain(tokens: Iterable[int], seed: int = 0) -> List[int]:
    """Block hashes h_0 .. h_{n//16 - 1} of one token sequence."""
    toks = [int(t) for t in tokens]
    h, out = seed & MASK, []
    for b in range(len(toks) // 16):
        h = finalize(h ^ digest(toks[16 * b:16 * b + 16]) ^ GOLDEN_GAMMA)
        out.append(h)
    return out


def chunk_keys(tokens: Iterable[int], chunk_tokens: int, seed: int = 0) -> List[int]:
    """Keys of the complete chunks of one sequence."""
    hs = chain(tokens, seed)
    per = chunk_tokens // 16
    return [hs[(c + 1) * per - 1] for c in range(len(hs) // per)]
