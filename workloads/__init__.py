"""Seeded synthetic workloads for the KV staging path.

This module only *generates inputs*: token ids, prompt lengths, shared-prefix
assignment, block tables, staging placement and KV byte contents.  It holds
none of the method's arithmetic (no prefix hash, no lookup, no copy), so both
the CPU oracle and the GPU library can be fed from it without sharing any of
the computation under test.

Workload shapes follow the paper's evaluation (Section 5): BF16 KV, reusable
prefixes retained as complete 256-token chunks of a per-request prefix cache
ratio, the final incomplete chunk left uncached; and the 32-layer / 8-KV-head /
head_dim-128 model shape whose 64k-token prefix is 8 GiB (Section 2.3,
"Early staging trades latency for capacity").  The paper's datasets are not
used: token ids are uniform random in [0, 32000).

Randomness:
  * structure (tokens, lengths, Zipf prefix draws, block permutations) comes
    from numpy's PCG64 generator, seeded per (config seed, purpose);
  * KV contents are a counter-based formula, ``kv_word(tag, seed, index)``,
    built on the 32-bit MurmurHash3 finalizer (Appleby, public domain).  It
    has a torch form that fills device memory and a numpy form that recomputes
    any sampled word on the host, so full-size buffers never need to exist on
    the host.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

M32 = 0xFFFFFFFF
FINITE_MASK = 0xBFFFBFFF   # clears bit 14 of each 16-bit half: no Inf/NaN in fp16 or bf16

# purposes for numpy sub-seeds
_P_TOK, _P_LEN, _P_ZIPF, _P_PERM, _P_PERM2, _P_SMALL, _P_JOBS, _P_SHAPES = range(8)


# --------------------------------------------------------------------------
# KV content formula
# --------------------------------------------------------------------------

def _fmix32_int(x: int) -> int:
    x &= M32
    x ^= x >> 16
    x = (x * 0x85EBCA6B) & M32
    x ^= x >> 13
    x = (x * 0xC2B2AE35) & M32
    x ^= x >> 16
    return x


def _fmix32_np(x: np.ndarray) -> np.ndarray:
    x = x.astype(np.uint32, copy=True)
    x ^= x >> np.uint32(16)
    x *= np.uint32(0x85EBCA6B)
    x ^= x >> np.uint32(13)
    x *= np.uint32(0xC2B2AE35)
    x ^= x >> np.uint32(16)
    return x


def _keys(tag: int, seed: int) -> Tuple[int, int]:
    k1 = _fmix32_int(_fmix32_int(seed * 0x9E3779B1 + 0x632BE5AB) ^ (tag * 0x85EBCA77 + 1))
    k2 = _fmix32_int(k1 ^ 0x27D4EB2F)
    return k1, k2


_HERE = os.path.dirname(os.path.abspath(__file__))
_FILL_SRC = os.path.join(_HERE, "kvfill.c")
_FILL_LIB = os.path.join(_HERE, "libkvfill.so")
_fill_lib = None


def build_fill_lib() -> str:
    """Compile the host form of the KV formula (always recompiles)."""
    tmp = _FILL_LIB + ".tmp"
    subprocess.check_call(["gcc", "-O3", "-std=c11", "-fPIC", "-shared", "-o", tmp, _FILL_SRC])
    os.replace(tmp, _FILL_LIB)
    return _FILL_LIB


def _fill():
    global _fill_lib
    if _fill_lib is None:
        if not os.path.exists(_FILL_LIB) or os.path.getmtime(_FILL_LIB) < os.path.getmtime(_FILL_SRC):
            build_fill_lib()
        lib = ctypes.CDLL(_FILL_LIB)
        lib.kvfill_words.restype = None
        lib.kvfill_words.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64,
                                     ctypes.c_int, ctypes.c_void_p]
        _fill_lib = lib
    return _fill_lib


def kv_words_np(tag: int, seed: int, start: int, count: int, finite: bool = True,
                out: Optional[np.ndarray] = None) -> np.ndarray:
    """uint32 words [start, start+count) of buffer ``tag`` (host form)."""
    k1, k2 = _keys(tag, seed)
    if out is None:
        out = np.empty(count, np.uint32)
    assert out.dtype == np.uint32 and out.flags.c_contiguous and out.size >= count
    if count:
        _fill().kvfill_words(k1, k2, start, count, 1 if finite else 0, out.ctypes.data)
    return out


def kv_words_np_reference(tag: int, seed: int, start: int, count: int, finite: bool = True) -> np.ndarray:
    """The same words computed with numpy alone (slow; cross-checks the C form)."""
    k1, k2 = _keys(tag, seed)
    out = np.empty(count, np.uint32)
    step = 1 << 16
    tmp = np.empty(min(step, max(count, 1)), np.uint32)
    pos = 0
    while pos < count:
        idx0 = start + pos
        hi = idx0 >> 32
        n = min(step, count - pos, (1 << 32) - (idx0 & M32))
        chi = _fmix32_int((hi + k2) & M32)
        v = out[pos:pos + n]
        t = tmp[:n]
        np.add(_RAMP[:n], np.uint32(idx0 & M32), out=v, casting="unsafe")
        v ^= np.uint32(k1)
        _fmix32_inplace(v, t)
        v ^= np.uint32(chi)
        _fmix32_inplace(v, t)
        if finite:
            v &= np.uint32(FINITE_MASK)
        pos += n
    return out


_RAMP = np.arange(1 << 16, dtype=np.uint32)


def _fmix32_inplace(x: np.ndarray, t: np.ndarray) -> None:
    np.right_shift(x, 16, out=t)
    x ^= t
    x *= np.uint32(0x85EBCA6B)
    np.right_shift(x, 13, out=t)
    x ^= t
    x *= np.uint32(0xC2B2AE35)
    np.right_shift(x, 16, out=t)
    x ^= t


def kv_bytes_np(tag: int, seed: int, byte_start: int, nbytes: int, finite: bool = True) -> np.ndarray:
    """Bytes [byte_start, byte_start+nbytes) of buffer ``tag``; 4-aligned ranges."""
    assert byte_start % 4 == 0 and nbytes % 4 == 0
    return kv_words_np(tag, seed, byte_start // 4, nbytes // 4, finite).view(np.uint8)


def _mul32_t(x, c: int):
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & M32


def _fmix32_t(x):
    x = x ^ (x >> 16)
    x = _mul32_t(x, 0x85EBCA6B)
    x = x ^ (x >> 13)
    x = _mul32_t(x, 0xC2B2AE35)
    return x ^ (x >> 16)


def fill_kv_(buf, tag: int, seed: int, finite: bool = True, chunk_words: int = 1 << 25,
             byte_start: int = 0) -> None:
    """Fill a torch uint8 tensor (any device, numel % 4 == 0) with the formula.

    ``buf`` receives bytes [byte_start, byte_start + numel) of buffer ``tag``:
    the result equals ``kv_bytes_np(tag, seed, byte_start, buf.numel())``."""
    import torch
    assert buf.dtype == torch.uint8 and buf.numel() % 4 == 0 and buf.is_contiguous()
    assert byte_start % 4 == 0
    words = buf.view(torch.int32)
    n = words.numel()
    w0 = byte_start // 4
    k1, k2 = _keys(tag, seed)
    for s in range(0, n, chunk_words):
        e = min(n, s + chunk_words)
        idx = torch.arange(w0 + s, w0 + e, device=buf.device, dtype=torch.int64)
        lo = idx & M32
        hi = idx >> 32
        chi = _fmix32_t((hi + k2) & M32)
        v = _fmix32_t(_fmix32_t(lo ^ k1) ^ chi)
        if finite:
            v = v & FINITE_MASK
        v = v - ((v >> 31) << 32)          # to the int32 bit pattern
        words[s:e] = v.to(torch.int32)
        del idx, lo, hi, chi, v


# --------------------------------------------------------------------------
# Workload description
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class KVShape:
    """Per-token KV shape.  Staging slot = [L, 2, C, H, D]; paged block = [B, H, D]."""
    num_layers: int
    kv_heads: int
    head_dim: int
    elem_bytes: int = 2
    block_size: int = 16
    chunk_tokens: int = 256
    dtype: str = "bf16"

    @property
    def bytes_per_token(self) -> int:
        return 2 * self.num_layers * self.kv_heads * self.head_dim * self.elem_bytes

    @property
    def seg_bytes(self) -> int:
        return self.block_size * self.kv_heads * self.head_dim * self.elem_bytes

    @property
    def slot_bytes(self) -> int:
        return self.chunk_tokens * self.bytes_per_token

    @property
    def blocks_per_chunk(self) -> int:
        return self.chunk_tokens // self.block_size


@dataclass
class Workload:
    name: str
    shape: KVShape
    seed: int
    tokens: np.ndarray            # int32 [sum n_r]
    tok_off: np.ndarray           # int64 [R+1]
    prefix_id: np.ndarray         # int32 [R], -1 = no shared prefix
    prefix_tokens: np.ndarray     # int64 [R], tokens taken from the shared prefix stream
    prefix_streams: List[np.ndarray]   # int32 token streams of the shared prefixes
    prestage_chunks: List[Tuple[int, int]]  # (prefix id, chunk j) resident at start, slot = position
    num_slots: int                # staging capacity in chunks
    num_blocks: int               # paged pool blocks
    block_tables: np.ndarray      # int32 [R, bt_stride], -1 beyond a request's blocks
    staging_in_host: bool = False
    paged_layout: str = "kv_first"    # "kv_first": per layer [2, NB, B, H, D]; "block_first": [NB, 2, B, H, D]
    block_pad: int = 0            # bytes after each [B, H, D] segment of the paged pool (multiple of 16)
    notes: Dict[str, object] = field(default_factory=dict)

    @property
    def num_reqs(self) -> int:
        return int(self.tok_off.size - 1)

    @property
    def lengths(self) -> np.ndarray:
        return np.diff(self.tok_off)

    @property
    def bt_stride(self) -> int:
        return int(self.block_tables.shape[1])

    @property
    def free_slots(self) -> np.ndarray:
        return np.arange(len(self.prestage_chunks), self.num_slots, dtype=np.int32)

    def strides(self) -> Tuple[int, int]:
        """(kv_stride, block_stride) in bytes within one layer's paged tensor."""
        seg = self.shape.seg_bytes + self.block_pad
        if self.paged_layout == "kv_first":
            return self.num_blocks * seg, seg
        if self.paged_layout == "block_first":
            return seg, 2 * seg
        raise ValueError(self.paged_layout)

    def layer_bytes(self) -> int:
        return 2 * self.num_blocks * (self.shape.seg_bytes + self.block_pad)

    def offsets(self):
        """(blk_off, chunk_off) int64 arrays for the ragged hash / lookup outputs."""
        nb = self.lengths // 16
        blk_off = np.zeros(self.num_reqs + 1, np.int64)
        np.cumsum(nb, out=blk_off[1:])
        nc = nb // (self.shape.chunk_tokens // 16)
        chunk_off = np.zeros(self.num_reqs + 1, np.int64)
        np.cumsum(nc, out=chunk_off[1:])
        return blk_off, chunk_off

    def prefix_stream_request(self):
        """The shared prefix streams as a request batch (tokens, tok_off), used to
        compute the keys of the prestaged chunks."""
        lens = np.array([s.size for s in self.prefix_streams], np.int64)
        off = np.zeros(lens.size + 1, np.int64)
        np.cumsum(lens, out=off[1:])
        toks = (np.concatenate(self.prefix_streams) if self.prefix_streams
                else np.zeros(0, np.int32)).astype(np.int32)
        return toks, off

    def staged_bytes(self) -> int:
        return self.num_slots * self.shape.slot_bytes

    def pool_bytes(self) -> int:
        return self.shape.num_layers * self.layer_bytes()

    # buffer tags for the KV content formula
    TAG_STAGING = 1
    TAG_POOL = 2


def _rng(seed: int, purpose: int) -> np.random.Generator:
    return np.random.default_rng([seed, purpose])


def _assemble(name, shape, seed, lengths, prefix_id, prefix_tokens, n_prefixes,
              prestage, num_slots, pool_factor, pool_blocks=None, staging_in_host=False,
              notes=None, paged_layout="kv_first", block_pad=0) -> Workload:
    """Build tokens, streams and block tables from lengths and prefix choices."""
    rng_tok = _rng(seed, _P_TOK)
    lengths = np.asarray(lengths, np.int64)
    R = lengths.size
    stream_len = np.zeros(n_prefixes, np.int64)
    for r in range(R):
        p = prefix_id[r]
        if p >= 0:
            stream_len[p] = max(stream_len[p], prefix_tokens[r])
    streams = [rng_tok.integers(0, 32000, size=int(stream_len[p]), dtype=np.int32)
               for p in range(n_prefixes)]
    parts = []
    for r in range(R):
        n, p, k = int(lengths[r]), int(prefix_id[r]), int(prefix_tokens[r])
        own = rng_tok.integers(0, 32000, size=n - (k if p >= 0 else 0), dtype=np.int32)
        parts.append(np.concatenate([streams[p][:k], own]) if p >= 0 else own)
    tokens = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
    tok_off = np.zeros(R + 1, np.int64)
    np.cumsum(lengths, out=tok_off[1:])

    B = shape.block_size
    need = (lengths + B - 1) // B
    if pool_blocks is None:
        # the factor applies to the tokens; every request also rounds its tail up to a whole block, so many
        # short requests can need more blocks than that: never fewer than the live blocks
        pool_blocks = max(int(math.ceil(pool_factor * lengths.sum() / B)), int(need.sum()))
    assert pool_blocks >= need.sum(), "pool smaller than the live blocks"
    perm = _rng(seed, _P_PERM).permutation(pool_blocks).astype(np.int32)
    bt_stride = int(need.max()) if R else 1
    bt = np.full((R, max(bt_stride, 1)), -1, np.int32)
    pos = 0
    for r in range(R):
        bt[r, :need[r]] = perm[pos:pos + need[r]]
        pos += int(need[r])
    return Workload(name=name, shape=shape, seed=seed, tokens=tokens, tok_off=tok_off,
                    prefix_id=np.asarray(prefix_id, np.int32),
                    prefix_tokens=np.asarray(prefix_tokens, np.int64),
                    prefix_streams=streams, prestage_chunks=list(prestage), num_slots=num_slots,
                    num_blocks=pool_blocks, block_tables=bt, staging_in_host=staging_in_host,
                    paged_layout=paged_layout, block_pad=block_pad, notes=dict(notes or {}))


def repermute_block_tables(w: Workload, purpose_salt: int = 0) -> None:
    """Give every request a fresh random set of pool blocks (same counts)."""
    B = w.shape.block_size
    need = (w.lengths + B - 1) // B
    perm = _rng(w.seed, _P_PERM2 + 16 * purpose_salt).permutation(w.num_blocks).astype(np.int32)
    bt = np.full_like(w.block_tables, -1)
    pos = 0
    for r in range(w.num_reqs):
        bt[r, :need[r]] = perm[pos:pos + need[r]]
        pos += int(need[r])
    w.block_tables = bt


def random_shapes(seed: int, n: int) -> List[KVShape]:
    """n KV shapes for parity sweeps: 1-6 layers, 1-8 KV heads, head sizes 16-128 (80 and 96 included),
    1/2/4-byte elements, blocks of 1-32 tokens, chunks of 1-8 blocks; the chunk is a whole number of 16-token
    hash blocks and a paged segment a whole number of 16-byte vectors."""
    rng = _rng(seed, _P_SHAPES)
    out: List[KVShape] = []
    while len(out) < n:
        L = int(rng.integers(1, 7))
        H = int(rng.choice([1, 2, 3, 4, 8]))
        D = int(rng.choice([16, 32, 64, 80, 96, 128]))
        e = int(rng.choice([1, 2, 4]))
        B = int(rng.choice([1, 2, 4, 8, 16, 32]))
        C = int(B * rng.choice([1, 2, 4, 8]))
        if C % 16 or (B * H * D * e) % 16:
            continue
        out.append(KVShape(L, H, D, e, B, C))
    return out


def random_retrieve_jobs(w: Workload, seed: int, slots_used: int) -> np.ndarray:
    """Retrieve jobs ([n,4] int32, slot/req/chunk/0) for every complete chunk
    of the batch, each reading a random slot among the first ``slots_used``
    (slots repeat: many jobs may read one chunk), in random order, so the list
    is not grouped by slot.  Destinations are distinct (one job per chunk)."""
    rng = _rng(seed, _P_JOBS)
    C = w.shape.chunk_tokens
    rc = [(r, c) for r in range(w.num_reqs) for c in range(int(w.lengths[r]) // C)]
    jobs = np.zeros((len(rc), 4), np.int32)
    if rc:
        jobs[:, 1:3] = np.array(rc, np.int32)
        jobs[:, 0] = rng.integers(0, min(slots_used, w.num_slots), size=len(rc))
        jobs = jobs[rng.permutation(len(rc))]
    return jobs


def _prefix_len(ratio: float, n: int, C: int) -> int:
    """Prefix cache ratio relative to the prompt, kept as complete chunks."""
    return int(math.floor(ratio * n / C)) * C


def _zipf_probs(k: int, s: float) -> np.ndarray:
    w = 1.0 / np.arange(1, k + 1, dtype=np.float64) ** s
    return w / w.sum()


# --------------------------------------------------------------------------
# The configurations
# --------------------------------------------------------------------------

SHAPE_TINY = KVShape(num_layers=2, kv_heads=2, head_dim=64, elem_bytes=2, block_size=16,
                     chunk_tokens=64, dtype="fp16")
SHAPE_32L = KVShape(num_layers=32, kv_heads=8, head_dim=128, elem_bytes=2, block_size=16,
                    chunk_tokens=256, dtype="bf16")
SHAPE_80L = KVShape(num_layers=80, kv_heads=8, head_dim=128, elem_bytes=2, block_size=16,
                    chunk_tokens=256, dtype="bf16")
# 48 layers x 8 KV heads x 128 dims, bf16: 192 KiB per token (a 14B-class model)
SHAPE_48L = KVShape(num_layers=48, kv_heads=8, head_dim=128, elem_bytes=2, block_size=16,
                    chunk_tokens=256, dtype="bf16")


def tiny(seed: int = 1) -> Workload:
    """2 layers, 2 KV heads, head_dim 64, fp16; block 16, chunk 64; 8 requests of
    256 tokens whose first half comes from one shared prefix; 128-block pool
    (exactly the live blocks) with permuted block tables.  Nothing is staged
    at start: the test stores every chunk, then retrieves the hits."""
    R, n = 8, 256
    shape = SHAPE_TINY
    k = _prefix_len(0.5, n, shape.chunk_tokens)
    return _assemble("tiny-l2h2d64-8x256-p50", shape, seed, [n] * R, [0] * R, [k] * R, 1,
                     prestage=[], num_slots=32, pool_factor=1.0)


def l32_uniform(seed: int = 2, shape: KVShape = SHAPE_32L, paged_layout: str = "kv_first",
                block_pad: int = 0) -> Workload:
    """32 layers, 8 KV heads, head_dim 128, bf16 (128 KiB/token); block 16,
    chunk 256; 64 requests x 4096 tokens; 50% prefix ratio from 8 shared
    prefixes (request r uses prefix r mod 8); pool 1.25x live tokens; staging
    holds the 64 prefix chunks plus 512 free slots for the misses.  The same
    batch is also built with another KV shape, paged layout or padded paged
    block stride."""
    R, n, P = 64, 4096, 8
    k = _prefix_len(0.5, n, shape.chunk_tokens)
    pid = [r % P for r in range(R)]
    nck = k // shape.chunk_tokens
    prestage = [(p, j) for p in range(P) for j in range(nck)]
    misses = R * (n // shape.chunk_tokens - nck)
    name = f"l{shape.num_layers}h{shape.kv_heads}d{shape.head_dim}-64x4096-p50"
    if paged_layout != "kv_first":
        name += "-" + paged_layout
    if block_pad:
        name += f"-pad{block_pad}"
    return _assemble(name, shape, seed, [n] * R, pid, [k] * R, P, prestage=prestage,
                     num_slots=len(prestage) + misses, pool_factor=1.25, paged_layout=paged_layout,
                     block_pad=block_pad)


def single_prefix(shape: KVShape, n: int = 65536, in_host: bool = False, seed: int = 6) -> Workload:
    """One request of ``n`` tokens that is entirely a staged prefix: every one
    of its n/C chunks is resident at start, so the pass retrieves all of them
    (64k tokens: 8 GiB of KV at 128 KiB/token, 12 GiB at 192 KiB/token) and
    stores nothing.  Pool 1.25x the request's blocks."""
    k = _prefix_len(1.0, n, shape.chunk_tokens)
    nck = k // shape.chunk_tokens
    name = f"l{shape.num_layers}h{shape.kv_heads}d{shape.head_dim}-1x{n}-p100" + ("-host" if in_host else "")
    return _assemble(name, shape, seed, [n], [0], [k], 1, prestage=[(0, j) for j in range(nck)],
                     num_slots=nck, pool_factor=1.25, staging_in_host=in_host)


def l32_lognormal(ratio: float, seed: int = 3) -> Workload:
    """32-layer bf16 shape; 256 requests, lognormal prompt lengths (sigma 0.8,
    mean 2048, clipped to [256, 8192]); prefix ratio ``ratio`` of each prompt,
    as complete chunks, from 32 shared prefixes drawn Zipf(s=1.1); pool 1.25x
    live.  Every chunk of every used prefix stream is staged at start."""
    R, P, sigma = 256, 32, 0.8
    shape = SHAPE_32L
    mu = math.log(2048.0) - sigma * sigma / 2
    lengths = np.clip(np.rint(_rng(seed, _P_LEN).lognormal(mu, sigma, size=R)), 256, 8192).astype(np.int64)
    pid = _rng(seed, _P_ZIPF).choice(P, size=R, p=_zipf_probs(P, 1.1)).astype(np.int32)
    k = np.array([_prefix_len(ratio, int(n), shape.chunk_tokens) for n in lengths], np.int64)
    C = shape.chunk_tokens
    stream_chunks = np.zeros(P, np.int64)
    for r in range(R):
        stream_chunks[pid[r]] = max(stream_chunks[pid[r]], k[r] // C)
    prestage = [(p, j) for p in range(P) for j in range(int(stream_chunks[p]))]
    misses = int(sum(int(n) // C - int(kk) // C for n, kk in zip(lengths, k)))
    return _assemble(f"l32h8d128-256xlognormal2048-p{int(ratio * 100)}", shape, seed, lengths, pid, k, P,
                     prestage=prestage, num_slots=len(prestage) + misses, pool_factor=1.25,
                     notes={"mean_len": float(lengths.mean()), "ratio": ratio})


def l80_long(seed: int = 4) -> Workload:
    """80 layers, 8 KV heads, head_dim 128, bf16 (320 KiB/token); 32 requests x
    8192 tokens at a 75% prefix ratio, one distinct prefix per request (24
    staged chunks each); pool 1.1x live."""
    R, n = 32, 8192
    shape = SHAPE_80L
    k = _prefix_len(0.75, n, shape.chunk_tokens)
    nck = k // shape.chunk_tokens
    prestage = [(r, j) for r in range(R) for j in range(nck)]
    misses = R * (n // shape.chunk_tokens - nck)
    return _assemble("l80h8d128-32x8192-p75", shape, seed, [n] * R, list(range(R)), [k] * R, R,
                     prestage=prestage, num_slots=len(prestage) + misses, pool_factor=1.1)


def l32_capacity(cap: float, in_host: bool, seed: int = 5, ring_slots: int = 64) -> Workload:
    """32-layer bf16 shape; 1024 requests x 1024 tokens at a 90% prefix ratio
    (768 tokens = 3 complete chunks) from 16 prefixes drawn Zipf(s=1.1).  The
    staging buffer holds ``cap`` (1, 0.5, 0.25) of the unique hit KV, filled by
    popularity rank with whole prefixes first, plus a ring of ``ring_slots``
    free slots for stores; it lives in HBM or in mapped pinned host memory."""
    R, n, P = 1024, 1024, 16
    shape = SHAPE_32L
    k = _prefix_len(0.9, n, shape.chunk_tokens)
    pid = _rng(seed, _P_ZIPF).choice(P, size=R, p=_zipf_probs(P, 1.1)).astype(np.int32)
    nck = k // shape.chunk_tokens
    used = sorted(set(int(p) for p in pid))
    counts = np.bincount(pid, minlength=P)
    by_rank = sorted(used, key=lambda p: (-counts[p], p))
    keep_chunks = int(round(cap * len(used) * nck))
    prestage = []
    for p in by_rank:
        if len(prestage) + nck > keep_chunks:
            break
        prestage += [(p, j) for j in range(nck)]
    tag = "host" if in_host else "hbm"
    return _assemble(f"l32h8d128-1024x1024-p90-cap{int(cap * 100)}-{tag}", shape, seed, [n] * R, pid, [k] * R, P,
                     prestage=prestage, num_slots=len(prestage) + ring_slots, pool_factor=1.1,
                     staging_in_host=in_host, notes={"cap": cap, "unique_prefixes": len(used)})


def small_random(seed: int, shape: KVShape, num_reqs: int, max_len: int, n_prefixes: int = 2,
                 ratio: float = 0.5, pool_factor: float = 1.5, extra_slots: int = 8,
                 paged_layout: str = "kv_first", prestage_all: bool = True, block_pad: int = 0) -> Workload:
    """Small ragged workload for parity tests: random lengths in [0, max_len]
    (including empty, shorter-than-a-block and ragged tails)."""
    rng = _rng(seed, _P_SMALL)
    lengths = rng.integers(0, max_len + 1, size=num_reqs).astype(np.int64)
    if num_reqs:
        lengths[0] = max_len
    pid = rng.integers(-1, n_prefixes, size=num_reqs).astype(np.int32)
    C = shape.chunk_tokens
    k = np.array([_prefix_len(ratio, int(n), C) if p >= 0 else 0 for n, p in zip(lengths, pid)], np.int64)
    stream_chunks = np.zeros(max(n_prefixes, 1), np.int64)
    for r in range(num_reqs):
        if pid[r] >= 0:
            stream_chunks[pid[r]] = max(stream_chunks[pid[r]], k[r] // C)
    prestage = ([(p, j) for p in range(n_prefixes) for j in range(int(stream_chunks[p]))]
                if prestage_all else [])
    misses = int(sum(int(n) // C for n in lengths))
    return _assemble(f"random-s{seed}", shape, seed, lengths, pid, k, n_prefixes,
                     prestage=prestage, num_slots=len(prestage) + misses + extra_slots,
                     pool_factor=pool_factor, pool_blocks=None, paged_layout=paged_layout,
                     block_pad=block_pad)


CONFIGS = {
    "tiny": tiny,
    "l32-64x4096": l32_uniform,
    "l32-lognormal-p25": lambda: l32_lognormal(0.25),
    "l32-lognormal-p50": lambda: l32_lognormal(0.50),
    "l32-lognormal-p75": lambda: l32_lognormal(0.75),
    "l80-32x8192": l80_long,
    "l32-1024x1024-cap100-hbm": lambda: l32_capacity(1.0, False),
    "l32-1024x1024-cap50-hbm": lambda: l32_capacity(0.5, False),
    "l32-1024x1024-cap25-hbm": lambda: l32_capacity(0.25, False),
    "l32-1024x1024-cap100-host": lambda: l32_capacity(1.0, True),
    "l32-1024x1024-cap50-host": lambda: l32_capacity(0.5, True),
    "l32-1024x1024-cap25-host": lambda: l32_capacity(0.25, True),
    "l32-1x65536": lambda: single_prefix(SHAPE_32L),
    "l32-1x65536-host": lambda: single_prefix(SHAPE_32L, in_host=True),
    "l48-1x65536": lambda: single_prefix(SHAPE_48L),
    "l48-64x4096": lambda: l32_uniform(shape=SHAPE_48L),
    "l32-64x4096-block_first": lambda: l32_uniform(paged_layout="block_first"),
    "l32-64x4096-pad4096": lambda: l32_uniform(block_pad=4096),
}


def make(name: str) -> Workload:
    return CONFIGS[name]()


# --------------------------------------------------------------------------
# Controller scenarios (request streams for the commitment simulator)
# --------------------------------------------------------------------------

@dataclass
class StagingScenario:
    """Inputs of one controller simulation: staged objects and a request stream."""
    name: str
    obj_bytes: List[float]
    arrival: List[float]
    manifests: List[List[int]]
    uncached: List[int]
    out_tokens: List[int]


def policy_scenario(ratio: float, seed: int = 7, kv_bytes_per_token: int = 128 * 1024, chunk: int = 256,
                    gap_s: float = 0.5, out_tokens: int = 128, question_tokens: int = 32) -> StagingScenario:
    """Shaped like the paper's policy experiment (Section 5): 12 documents in
    three length groups of 4, together spanning 16,078-67,744 tokens (lengths
    drawn uniformly inside each group, no dataset text), one request per
    document in a fixed random order every ``gap_s`` seconds; the prefix
    ``ratio`` of each document is retained as complete 256-token chunks (each
    an object of chunk x KV bytes per token); the rest of the document plus a
    question is prefilled; ``out_tokens`` are generated."""
    rng = _rng(seed, _P_LEN)
    groups = [(16078, 30000), (30000, 48000), (48000, 67744)]
    lengths = [int(rng.integers(lo, hi + 1)) for lo, hi in groups for _ in range(4)]
    order = _rng(seed, _P_PERM).permutation(len(lengths))
    obj, man, unc, arr = [], [], [], []
    for k, d in enumerate(order):
        n = lengths[d]
        kept = int(math.floor(ratio * n / chunk))
        ids = list(range(len(obj), len(obj) + kept))
        obj += [float(chunk * kv_bytes_per_token)] * kept
        man.append(ids)
        unc.append(n - kept * chunk + question_tokens)
        arr.append(gap_s * k)
    return StagingScenario(f"policy-12docs-p{int(ratio * 100)}", obj, arr, man, unc, [out_tokens] * len(man))


def shared_prefix_scenario(n: int, seed: int = 11, n_prefixes: int = 64, chunks_max: int = 64,
                           chunk_bytes: int = 32 << 20, gap_s: float = 0.05) -> StagingScenario:
    """A long request stream for timing the simulator: ``n`` requests drawing
    Zipf(1.1) over ``n_prefixes`` shared prefixes, each request reusing a
    random number of its prefix's chunks."""
    rng = _rng(seed, _P_ZIPF)
    pid = rng.choice(n_prefixes, size=n, p=_zipf_probs(n_prefixes, 1.1))
    lens = _rng(seed, _P_LEN).integers(1, chunks_max + 1, size=n_prefixes)
    base = np.concatenate([[0], np.cumsum(lens)]).astype(int)
    use = _rng(seed, _P_SMALL).integers(0, chunks_max + 1, size=n)
    man = [list(range(base[p], base[p] + min(int(u), int(lens[p])))) for p, u in zip(pid, use)]
    unc = [int(x) for x in _rng(seed, _P_TOK).integers(100, 4000, size=n)]
    return StagingScenario(f"shared-{n}", [float(chunk_bytes)] * int(base[-1]), [gap_s * i for i in range(n)], man,
                           unc, [64] * n)
