"""CPU oracle for the KV staging path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never does, and
this package imports nothing from the product package.

The arithmetic lives in ``tempokv_oracle.c`` (plain single-threaded C, element
loops); this file compiles it with gcc and marshals numpy arrays into it.
"""
from __future__ import annotations

import ctypes as ct
import os
import subprocess
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tempokv_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib: Optional[ct.CDLL] = None

DEFER, COMMIT, BLOCKED, ORDINARY, EINVAL = 0, 1, 2, 3, -1


def build() -> str:
    """Compile the oracle into ``oracle/liboracle.so`` (always recompiles)."""
    tmp = _LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
                           "-o", tmp, _SRC, "-lm"])
    os.replace(tmp, _LIB)
    return _LIB


class OrLayout(ct.Structure):
    _fields_ = [("L", ct.c_int32), ("H", ct.c_int32), ("D", ct.c_int32), ("e", ct.c_int32),
                ("B", ct.c_int32), ("C", ct.c_int32), ("num_blocks", ct.c_int64),
                ("num_slots", ct.c_int64), ("kv_stride", ct.c_int64), ("block_stride", ct.c_int64)]


def _p(a: np.ndarray, ctype):
    return a.ctypes.data_as(ct.POINTER(ctype))


def lib() -> ct.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    # tests of the pins load a deliberately broken copy of the oracle instead
    override = os.environ.get("TEMPOKV_ORACLE_LIB")
    if override:
        L = ct.CDLL(override)
    else:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ct.CDLL(_LIB)
    u64p, i64p, i32p, u8p = (ct.POINTER(ct.c_uint64), ct.POINTER(ct.c_int64),
                             ct.POINTER(ct.c_int32), ct.POINTER(ct.c_uint8))
    L.or_mix64.restype = ct.c_uint64
    L.or_mix64.argtypes = [ct.c_uint64]
    L.or_splitmix64_next.restype = ct.c_uint64
    L.or_splitmix64_next.argtypes = [u64p]
    L.or_block_digest.restype = ct.c_uint64
    L.or_block_digest.argtypes = [i32p]
    L.or_hash_prefix.restype = ct.c_int
    L.or_hash_prefix.argtypes = [i32p, i64p, ct.c_int32, ct.c_uint64, i64p, u64p]
    L.or_lookup.restype = ct.c_int
    L.or_lookup.argtypes = [u64p, i32p, ct.c_int64, u64p, i64p, ct.c_int32, ct.c_int32, i64p, i32p, i32p]
    L.or_build_jobs.restype = ct.c_int
    L.or_build_jobs.argtypes = [i32p, i32p, u64p, i64p, i64p, ct.c_int32, ct.c_int32, i32p, ct.c_int32,
                                i32p, i32p, i32p, u64p, i32p, i32p]
    L.or_retrieve_scatter.restype = None
    L.or_retrieve_scatter.argtypes = [ct.POINTER(OrLayout), u8p, ct.POINTER(u8p), i32p, ct.c_int32,
                                      ct.c_int32, i32p, ct.c_int32]
    L.or_store_gather.restype = None
    L.or_store_gather.argtypes = L.or_retrieve_scatter.argtypes
    L.or_retrieve_scatter_layer.restype = None
    L.or_retrieve_scatter_layer.argtypes = [ct.POINTER(OrLayout), u8p, u8p, i32p, ct.c_int32, ct.c_int32, i32p,
                                            ct.c_int32]
    L.or_store_gather_layer.restype = None
    L.or_store_gather_layer.argtypes = L.or_retrieve_scatter_layer.argtypes
    L.or_scatter_source.restype = ct.c_int
    L.or_scatter_source.argtypes = [ct.POINTER(OrLayout), i32p, ct.c_int32, ct.c_int32, i32p, ct.c_int32,
                                    ct.c_int32, ct.c_int32, ct.c_int64, i64p]
    L.or_gather_source.restype = ct.c_int
    L.or_gather_source.argtypes = [ct.POINTER(OrLayout), i32p, ct.c_int32, ct.c_int32, i32p, ct.c_int32,
                                   ct.c_int32, ct.c_int32, i32p]
    L.or_validate_jobs.restype = ct.c_int
    L.or_validate_jobs.argtypes = [ct.POINTER(OrLayout), i32p, ct.c_int32, ct.c_int32, i32p, ct.c_int32, ct.c_int]
    L.or_commit_should_stage.restype = ct.c_int
    L.or_commit_should_stage.argtypes = [ct.c_double, ct.c_double, ct.c_uint64, ct.c_uint64, ct.c_uint64,
                                         ct.c_uint64, ct.c_int]
    _lib = L
    return L


# ---------------------------------------------------------------------------
# numpy-facing wrappers
# ---------------------------------------------------------------------------

def mix64(x: int) -> int:
    return int(lib().or_mix64(ct.c_uint64(x & 0xFFFFFFFFFFFFFFFF)))


def splitmix64_sequence(seed: int, n: int) -> list:
    st = ct.c_uint64(seed & 0xFFFFFFFFFFFFFFFF)
    return [int(lib().or_splitmix64_next(ct.byref(st))) for _ in range(n)]


def block_digest(tok16: np.ndarray) -> int:
    t = np.ascontiguousarray(tok16, np.int32)
    assert t.size == 16
    return int(lib().or_block_digest(_p(t, ct.c_int32)))


def block_offsets(tok_off: np.ndarray) -> np.ndarray:
    nb = np.diff(np.asarray(tok_off, np.int64)) // 16
    off = np.zeros(nb.size + 1, np.int64)
    np.cumsum(nb, out=off[1:])
    return off


def chunk_offsets(blk_off: np.ndarray, blocks_per_chunk: int) -> np.ndarray:
    nc = np.diff(np.asarray(blk_off, np.int64)) // blocks_per_chunk
    off = np.zeros(nc.size + 1, np.int64)
    np.cumsum(nc, out=off[1:])
    return off


def hash_prefix(tokens: np.ndarray, tok_off: np.ndarray, seed: int = 0,
                blk_off: Optional[np.ndarray] = None) -> np.ndarray:
    tokens = np.ascontiguousarray(tokens, np.int32)
    tok_off = np.ascontiguousarray(tok_off, np.int64)
    if blk_off is None:
        blk_off = block_offsets(tok_off)
    blk_off = np.ascontiguousarray(blk_off, np.int64)
    out = np.zeros(max(int(blk_off[-1]), 1), np.uint64)
    rc = lib().or_hash_prefix(_p(tokens, ct.c_int32), _p(tok_off, ct.c_int64), tok_off.size - 1,
                              ct.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), _p(blk_off, ct.c_int64),
                              _p(out, ct.c_uint64))
    if rc != 0:
        raise ValueError("or_hash_prefix: inconsistent offsets")
    return out[:int(blk_off[-1])]


def chunk_keys(block_hash: np.ndarray, blk_off: np.ndarray, blocks_per_chunk: int) -> np.ndarray:
    """Chunk keys of every request, in (request, chunk) order."""
    keys = []
    for r in range(blk_off.size - 1):
        nb = int(blk_off[r + 1] - blk_off[r])
        for j in range(nb // blocks_per_chunk):
            keys.append(block_hash[blk_off[r] + (j + 1) * blocks_per_chunk - 1])
    return np.array(keys, np.uint64)


def lookup(index: Dict[int, int], block_hash: np.ndarray, blk_off: np.ndarray,
           blocks_per_chunk: int, chunk_off: Optional[np.ndarray] = None):
    if chunk_off is None:
        chunk_off = chunk_offsets(blk_off, blocks_per_chunk)
    keys = np.array(list(index.keys()), np.uint64)
    slots = np.array(list(index.values()), np.int32)
    keys = np.ascontiguousarray(keys if keys.size else np.zeros(1, np.uint64))
    slots = np.ascontiguousarray(slots if slots.size else np.zeros(1, np.int32))
    bh = np.ascontiguousarray(block_hash if block_hash.size else np.zeros(1, np.uint64), np.uint64)
    R = blk_off.size - 1
    chunk_slot = np.zeros(max(int(chunk_off[-1]), 1), np.int32)
    hits = np.zeros(max(R, 1), np.int32)
    rc = lib().or_lookup(_p(keys, ct.c_uint64), _p(slots, ct.c_int32), len(index), _p(bh, ct.c_uint64),
                         _p(np.ascontiguousarray(blk_off, np.int64), ct.c_int64), R, blocks_per_chunk,
                         _p(np.ascontiguousarray(chunk_off, np.int64), ct.c_int64),
                         _p(chunk_slot, ct.c_int32), _p(hits, ct.c_int32))
    if rc != 0:
        raise ValueError("or_lookup: inconsistent offsets")
    return chunk_slot[:int(chunk_off[-1])], hits[:R]


def build_jobs(hit_chunks, chunk_slot, block_hash, blk_off, chunk_off, blocks_per_chunk, free_slots):
    R = blk_off.size - 1
    nchunks = int(chunk_off[-1])
    hit = np.ascontiguousarray(hit_chunks if R else np.zeros(1), np.int32)
    cs = np.ascontiguousarray(chunk_slot if nchunks else np.zeros(1), np.int32)
    bh = np.ascontiguousarray(block_hash if block_hash.size else np.zeros(1), np.uint64)
    fs = np.ascontiguousarray(free_slots if len(free_slots) else np.zeros(1), np.int32)
    retr = np.zeros((max(nchunks, 1), 4), np.int32)
    store = np.zeros((max(nchunks, 1), 4), np.int32)
    skeys = np.zeros(max(nchunks, 1), np.uint64)
    nr, ns, nd = ct.c_int32(0), ct.c_int32(0), ct.c_int32(0)
    rc = lib().or_build_jobs(_p(hit, ct.c_int32), _p(cs, ct.c_int32), _p(bh, ct.c_uint64),
                             _p(np.ascontiguousarray(blk_off, np.int64), ct.c_int64),
                             _p(np.ascontiguousarray(chunk_off, np.int64), ct.c_int64), R,
                             blocks_per_chunk, _p(fs, ct.c_int32), len(free_slots),
                             _p(retr, ct.c_int32), ct.byref(nr), _p(store, ct.c_int32),
                             _p(skeys, ct.c_uint64), ct.byref(ns), ct.byref(nd))
    if rc != 0:
        raise MemoryError("or_build_jobs")
    return retr[:nr.value].copy(), store[:ns.value].copy(), skeys[:ns.value].copy(), nd.value


def make_layout(shape, num_blocks: int, num_slots: int, kv_stride: int, block_stride: int) -> OrLayout:
    return OrLayout(shape.num_layers, shape.kv_heads, shape.head_dim, shape.elem_bytes,
                    shape.block_size, shape.chunk_tokens, num_blocks, num_slots, kv_stride, block_stride)


def _layer_array(layers: Sequence[np.ndarray]):
    arr = (ct.POINTER(ct.c_uint8) * len(layers))()
    for i, a in enumerate(layers):
        assert a.dtype == np.uint8 and a.flags.c_contiguous
        arr[i] = a.ctypes.data_as(ct.POINTER(ct.c_uint8))
    return arr


def retrieve_scatter(layout: OrLayout, staging: np.ndarray, layers: Sequence[np.ndarray],
                     block_tables: np.ndarray, jobs: np.ndarray) -> None:
    """In place: layers[l] (uint8) receive the staged chunks of ``jobs``."""
    bt = np.ascontiguousarray(block_tables, np.int32)
    jb = np.ascontiguousarray(jobs if len(jobs) else np.zeros((1, 4)), np.int32)
    assert staging.dtype == np.uint8 and staging.flags.c_contiguous
    lib().or_retrieve_scatter(ct.byref(layout), staging.ctypes.data_as(ct.POINTER(ct.c_uint8)),
                              _layer_array(layers), _p(bt, ct.c_int32), bt.shape[1], bt.shape[0],
                              _p(jb, ct.c_int32), len(jobs))


def store_gather(layout: OrLayout, staging: np.ndarray, layers: Sequence[np.ndarray],
                 block_tables: np.ndarray, jobs: np.ndarray) -> None:
    """In place: staging (uint8) receives the paged blocks of ``jobs``."""
    bt = np.ascontiguousarray(block_tables, np.int32)
    jb = np.ascontiguousarray(jobs if len(jobs) else np.zeros((1, 4)), np.int32)
    assert staging.dtype == np.uint8 and staging.flags.c_contiguous
    lib().or_store_gather(ct.byref(layout), staging.ctypes.data_as(ct.POINTER(ct.c_uint8)),
                          _layer_array(layers), _p(bt, ct.c_int32), bt.shape[1], bt.shape[0],
                          _p(jb, ct.c_int32), len(jobs))


def layer_part_bytes(layout: OrLayout) -> int:
    """Bytes of one layer of one staging slot ([2][C][H][D] elements)."""
    return 2 * layout.C * layout.H * layout.D * layout.e


def retrieve_scatter_layer(layout: OrLayout, stg_layer: np.ndarray, paged: np.ndarray,
                           block_tables: np.ndarray, jobs: np.ndarray) -> None:
    """In place: one layer's paged tensor receives that layer's part of the
    staged chunks of ``jobs``; ``stg_layer`` holds the layer's part of every
    slot back to back (slot s at s * layer_part_bytes)."""
    bt = np.ascontiguousarray(block_tables, np.int32)
    jb = np.ascontiguousarray(jobs if len(jobs) else np.zeros((1, 4)), np.int32)
    assert stg_layer.dtype == np.uint8 and stg_layer.flags.c_contiguous
    assert stg_layer.size >= layout.num_slots * layer_part_bytes(layout)
    assert paged.dtype == np.uint8 and paged.flags.c_contiguous
    lib().or_retrieve_scatter_layer(ct.byref(layout), stg_layer.ctypes.data_as(ct.POINTER(ct.c_uint8)),
                                    paged.ctypes.data_as(ct.POINTER(ct.c_uint8)), _p(bt, ct.c_int32), bt.shape[1],
                                    bt.shape[0], _p(jb, ct.c_int32), len(jobs))


def store_gather_layer(layout: OrLayout, stg_layer: np.ndarray, paged: np.ndarray,
                       block_tables: np.ndarray, jobs: np.ndarray) -> None:
    """In place: ``stg_layer`` (one layer's part of every slot) receives that
    layer's paged blocks of ``jobs``."""
    bt = np.ascontiguousarray(block_tables, np.int32)
    jb = np.ascontiguousarray(jobs if len(jobs) else np.zeros((1, 4)), np.int32)
    assert stg_layer.dtype == np.uint8 and stg_layer.flags.c_contiguous
    assert stg_layer.size >= layout.num_slots * layer_part_bytes(layout)
    assert paged.dtype == np.uint8 and paged.flags.c_contiguous
    lib().or_store_gather_layer(ct.byref(layout), stg_layer.ctypes.data_as(ct.POINTER(ct.c_uint8)),
                                paged.ctypes.data_as(ct.POINTER(ct.c_uint8)), _p(bt, ct.c_int32), bt.shape[1],
                                bt.shape[0], _p(jb, ct.c_int32), len(jobs))


def scatter_source(layout: OrLayout, block_tables: np.ndarray, jobs: np.ndarray,
                   layer: int, kv: int, blk: int) -> Optional[int]:
    bt = np.ascontiguousarray(block_tables, np.int32)
    jb = np.ascontiguousarray(jobs if len(jobs) else np.zeros((1, 4)), np.int32)
    off = ct.c_int64(0)
    f = lib().or_scatter_source(ct.byref(layout), _p(bt, ct.c_int32), bt.shape[1], bt.shape[0],
                                _p(jb, ct.c_int32), len(jobs), layer, kv, blk, ct.byref(off))
    return off.value if f else None


def gather_source(layout: OrLayout, block_tables: np.ndarray, jobs: np.ndarray,
                  slot: int, seg: int) -> Optional[int]:
    bt = np.ascontiguousarray(block_tables, np.int32)
    jb = np.ascontiguousarray(jobs if len(jobs) else np.zeros((1, 4)), np.int32)
    blk = ct.c_int32(0)
    f = lib().or_gather_source(ct.byref(layout), _p(bt, ct.c_int32), bt.shape[1], bt.shape[0],
                               _p(jb, ct.c_int32), len(jobs), slot, seg, ct.byref(blk))
    return blk.value if f else None


# outcomes of validate_jobs
VOK, VERANGE, VEDUP = 0, -3, -6


def validate_jobs(layout: OrLayout, block_tables: np.ndarray, jobs: np.ndarray, is_store: bool) -> int:
    """VOK, VERANGE or VEDUP for a job batch against its block tables
    ([num_reqs, bt_stride]): out-of-range fields or block ids, then two jobs
    writing one destination (scatter: a paged block; gather: a staging slot)."""
    bt = np.ascontiguousarray(block_tables, np.int32)
    jb = np.ascontiguousarray(jobs if len(jobs) else np.zeros((1, 4)), np.int32)
    return int(lib().or_validate_jobs(ct.byref(layout), _p(bt, ct.c_int32), bt.shape[1], bt.shape[0],
                                      _p(jb, ct.c_int32), len(jobs), 1 if is_store else 0))


def commit_should_stage(ttu: float, ttr: float, free_protected: int, claim_new: int,
                        claim_total: int, budget: int, retrieval_requested: bool) -> int:
    return int(lib().or_commit_should_stage(ttu, ttr, free_protected, claim_new, claim_total, budget,
                                            1 if retrieval_requested else 0))
