"""Python binding of libtempokv (the C ABI declared in include/tempokv.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels or its native host code.  PyTorch supplies device memory and streams.
The functions keep the C names; tensors are passed where the C call takes a
device pointer, numpy arrays where it takes host memory.  A negative status
raises ``KvError`` (``kv_build_jobs`` returns ``KV_ENOSPC`` instead, since its
outputs stay valid).
"""
from __future__ import annotations

import ctypes as ct
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtempokv.so")

KV_OK, KV_EINVAL, KV_EALIGN, KV_ERANGE, KV_ENOSPC, KV_EHIP, KV_EDUP, KV_ELIMIT = 0, -1, -2, -3, -4, -5, -6, -7
KV_INDEX_STATIC_MAX_PAIRS = 65536
KV_DEFER, KV_COMMIT, KV_BLOCKED, KV_ORDINARY = 0, 1, 2, 3
KV_POLICY_DEMAND, KV_POLICY_IMMEDIATE, KV_POLICY_QUEUE_K, KV_POLICY_TEMPO_STATIC, KV_POLICY_TEMPO = range(5)
KV_RETRIEVE_UNIT, KV_RETRIEVE_PAIR, KV_RETRIEVE_STREAM, KV_RETRIEVE_QUAD = range(4)
RETRIEVE_KIND_NAMES = {KV_RETRIEVE_UNIT: "unit", KV_RETRIEVE_PAIR: "pair", KV_RETRIEVE_STREAM: "stream",
                       KV_RETRIEVE_QUAD: "quad"}
SIM_TRACE_KINDS = ["arrive", "admit", "commit", "ordinary", "ready", "stageready", "transfer", "fetch", "release",
                   "done", "evict"]
KV_MAX_LAYERS = 128
HASH_BLOCK_TOKENS = 16

# every symbol include/tempokv.h declares
EXPORTS = ["kv_hash_prefix", "kv_index_create", "kv_index_destroy", "kv_index_insert", "kv_index_insert_static",
           "kv_index_erase",
           "kv_index_size", "kv_index_find", "kv_lookup", "kv_build_jobs", "kv_retrieve_scatter",
           "kv_retrieve_plan", "kv_retrieve_scatter_as", "kv_store_gather", "kv_group_jobs_by_slot",
           "kv_validate_jobs", "kv_commit_should_stage", "kv_commit_should_stage_n", "kv_strerror",
           "kv_host_device_pointer", "kv_version", "kv_sim_run", "kv_stage_in", "kv_stage_out",
           "kv_pipeline_create", "kv_pipeline_destroy", "kv_retrieve_pipelined", "kv_decide_claims",
           "kv_build_jobs_routed", "kv_ttr_static", "kv_ttr_state_aware", "kv_chunk_keys", "kv_validate_jobs_device",
           "kv_probe_mixed_traffic"]
# the calls that run on the host only (host.cpp, controller.cpp)
HOST_CALLS = ["kv_build_jobs", "kv_build_jobs_routed", "kv_decide_claims", "kv_group_jobs_by_slot",
              "kv_validate_jobs", "kv_commit_should_stage", "kv_commit_should_stage_n", "kv_retrieve_plan",
              "kv_strerror", "kv_version", "kv_sim_run", "kv_ttr_static", "kv_ttr_state_aware", "kv_chunk_keys"]


class KvError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {strerror(status)} ({status})")


class KvLayout(ct.Structure):
    _fields_ = [("num_layers", ct.c_int32), ("kv_heads", ct.c_int32), ("head_dim", ct.c_int32),
                ("elem_bytes", ct.c_int32), ("block_size", ct.c_int32), ("chunk_tokens", ct.c_int32),
                ("num_blocks", ct.c_int64), ("num_slots", ct.c_int64), ("paged_kv_stride", ct.c_int64),
                ("paged_block_stride", ct.c_int64)]


class KvSimConfig(ct.Structure):
    _fields_ = [("budget_bytes", ct.c_double), ("capacity_bytes", ct.c_double), ("stage_rate", ct.c_double),
                ("static_rate", ct.c_double), ("gpu_rate", ct.c_double), ("prefill_s", ct.c_double),
                ("decode_s", ct.c_double), ("tick_s", ct.c_double), ("max_active", ct.c_int32),
                ("policy", ct.c_int32), ("queue_k", ct.c_int32), ("reserved", ct.c_int32)]


class KvSimResult(ct.Structure):
    _fields_ = [("area_byte_s", ct.c_double), ("cost_gib_s_per_request", ct.c_double), ("end_s", ct.c_double),
                ("p_max_bytes", ct.c_double), ("committed", ct.c_int32), ("blocked", ct.c_int32),
                ("ordinary", ct.c_int32), ("reserved", ct.c_int32), ("events", ct.c_int64)]


class KvSimEvent(ct.Structure):
    _fields_ = [("t", ct.c_double), ("kind", ct.c_int32), ("id", ct.c_int32)]


_lib: Optional[ct.CDLL] = None
# Tests only: a separately built copy of the host-only calls (HOST_CALLS) from the same sources, e.g. a
# sanitizer build, used by the host-call wrappers in place of libtempokv.so.
_host_override: Optional[ct.CDLL] = None
_vp, _i32, _i64, _u32, _u64, _dbl = ct.c_void_p, ct.c_int32, ct.c_int64, ct.c_uint32, ct.c_uint64, ct.c_double

SIGNATURES = {
    "kv_hash_prefix": [_vp, _vp, _i32, _u64, _vp, _vp, _vp],
    "kv_index_create": [_i64, ct.POINTER(_vp)],
    "kv_index_destroy": [_vp],
    "kv_index_insert": [_vp, _vp, _vp, _i32, _vp],
    "kv_index_insert_static": [_vp, _vp, _vp, _i32, _vp],
    "kv_index_erase": [_vp, _vp, _i32, _vp],
    "kv_index_size": [_vp, ct.POINTER(_i64)],
    "kv_index_find": [_vp, _u64, ct.POINTER(_i32)],
    "kv_lookup": [_vp, _vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp],
    "kv_build_jobs": [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _i32, _vp, ct.POINTER(_i32), _vp, _vp,
                      ct.POINTER(_i32), ct.POINTER(_i32)],
    "kv_build_jobs_routed": [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _i32, _vp, _vp, _vp, ct.POINTER(_i32), _vp,
                             ct.POINTER(_i32), _vp, _vp, ct.POINTER(_i32), ct.POINTER(_i32)],
    "kv_chunk_keys": [_vp, _vp, _i32, _i32, _vp, _vp],
    "kv_decide_claims": [_i32, _vp, _vp, _vp, _vp, _vp, _vp, _u64, _u64, _i64, _vp, ct.POINTER(_u64), _vp],
    "kv_retrieve_scatter": [ct.POINTER(KvLayout), _vp, _vp, _vp, _i32, _i32, _vp, _i32, _vp],
    "kv_store_gather": [ct.POINTER(KvLayout), _vp, _vp, _vp, _i32, _i32, _vp, _i32, _vp],
    "kv_retrieve_plan": [ct.POINTER(KvLayout), _vp, _i32],
    "kv_retrieve_scatter_as": [_i32, ct.POINTER(KvLayout), _vp, _vp, _vp, _i32, _i32, _vp, _i32, _vp],
    "kv_group_jobs_by_slot": [_vp, _i32],
    "kv_probe_mixed_traffic": [ct.POINTER(KvLayout), _vp, _vp, _vp, _i32, _i32, _vp, _i32, _vp, _i32, _u32, _vp],
    "kv_validate_jobs": [ct.POINTER(KvLayout), _vp, _i32, _i32, _vp, _i32, ct.c_int],
    "kv_validate_jobs_device": [ct.POINTER(KvLayout), _vp, _i32, _i32, _vp, _i32, ct.c_int, _vp, _vp, _vp],
    "kv_commit_should_stage": [_dbl, _dbl, _u64, _u64, _u64, _u64, ct.c_int],
    "kv_commit_should_stage_n": [_i32, _vp, _vp, _u64, _vp, _vp, _u64, _vp, _vp],
    "kv_ttr_static": [_i32, _vp, _i32, _vp, _vp, _dbl, ct.POINTER(_dbl)],
    "kv_ttr_state_aware": [_i32, _vp, _i32, _vp, _vp, _vp, _vp, _dbl, _dbl, _dbl, ct.POINTER(_dbl)],
    "kv_strerror": [ct.c_int],
    "kv_host_device_pointer": [_vp, ct.POINTER(_vp)],
    "kv_version": [],
    "kv_sim_run": [ct.POINTER(KvSimConfig), _vp, _i32, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp,
                   ct.POINTER(KvSimResult), _vp, _i64, ct.POINTER(_i64)],
    "kv_stage_in": [ct.POINTER(KvLayout), _vp, _vp, _vp, _i32, _vp],
    "kv_stage_out": [ct.POINTER(KvLayout), _vp, _vp, _vp, _i32, _vp],
    "kv_pipeline_create": [_i32, ct.POINTER(_vp)],
    "kv_pipeline_destroy": [_vp],
    "kv_retrieve_pipelined": [_vp, ct.POINTER(KvLayout), _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _i32, _i32,
                              _vp, _vp],
}


def declare(L: ct.CDLL, names) -> ct.CDLL:
    """Set the argument and result types of the named calls on a loaded library."""
    for name in names:
        f = getattr(L, name)
        f.argtypes = SIGNATURES[name]
        f.restype = ct.c_int
    if "kv_strerror" in names:
        L.kv_strerror.restype = ct.c_char_p
    if "kv_version" in names:
        L.kv_version.restype = ct.c_char_p
    return L


def lib() -> ct.CDLL:
    """Load libtempokv.so.  Raises if it has not been built: there is no
    fallback implementation."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_35065_amd.build`")
    # torch first: the library then binds to the HIP runtime torch already
    # loaded (same soname), so torch's streams and allocations are its own.
    import torch  # noqa: F401
    _lib = declare(ct.CDLL(LIB_PATH), list(SIGNATURES))
    return _lib


def host_lib() -> ct.CDLL:
    """The library whose host-only calls the wrappers below use: libtempokv.so,
    unless a test installed a separately built copy of those calls."""
    return _host_override if _host_override is not None else lib()


def strerror(status: int) -> str:
    return host_lib().kv_strerror(status).decode()


def kv_version() -> str:
    return host_lib().kv_version().decode()


def _check(rc: int, what: str) -> int:
    if rc < 0:
        raise KvError(rc, what)
    return rc


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------

def _stream(stream) -> int:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dptr(t, dtype=None, what: str = "tensor") -> int:
    """Device pointer of a contiguous CUDA (HIP) tensor, or an int address."""
    if isinstance(t, int):
        return t
    import torch
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def make_layout(num_layers: int, kv_heads: int, head_dim: int, elem_bytes: int, block_size: int,
                chunk_tokens: int, num_blocks: int, num_slots: int, paged_kv_stride: int,
                paged_block_stride: int) -> KvLayout:
    return KvLayout(num_layers, kv_heads, head_dim, elem_bytes, block_size, chunk_tokens, num_blocks, num_slots,
                    paged_kv_stride, paged_block_stride)


# ---------------------------------------------------------------------------
# the C calls
# ---------------------------------------------------------------------------

def kv_hash_prefix(d_tokens, d_tok_off, num_reqs: int, seed: int, d_blk_off, d_block_hash, stream=None) -> None:
    import torch
    _check(lib().kv_hash_prefix(_dptr(d_tokens, torch.int32, "tokens"), _dptr(d_tok_off, torch.int64, "tok_off"),
                                num_reqs, seed & 0xFFFFFFFFFFFFFFFF, _dptr(d_blk_off, torch.int64, "blk_off"),
                                _hash_ptr(d_block_hash), _stream(stream)), "kv_hash_prefix")


def _hash_ptr(t) -> int:
    """Block hashes are 64-bit words; an int64 (or uint64) tensor holds them."""
    if isinstance(t, int):
        return t
    import torch
    if t.dtype not in (torch.int64, getattr(torch, "uint64", torch.int64)):
        raise ValueError(f"block_hash must be a 64-bit integer tensor, got {t.dtype}")
    return _dptr(t, None, "block_hash")


class KvIndex:
    """Owner of a kv_index handle."""

    def __init__(self, max_entries: int):
        h = _vp()
        _check(lib().kv_index_create(max_entries, ct.byref(h)), "kv_index_create")
        self.handle = h
        self.max_entries = max_entries

    def insert(self, keys: np.ndarray, slots: np.ndarray, stream=None) -> None:
        kv_index_insert(self, keys, slots, stream)

    def insert_static(self, keys: np.ndarray, slots: np.ndarray, stream=None) -> None:
        kv_index_insert_static(self, keys, slots, stream)

    def erase(self, keys: np.ndarray, stream=None) -> None:
        kv_index_erase(self, keys, stream)

    def size(self) -> int:
        return kv_index_size(self)

    def find(self, key: int) -> int:
        return kv_index_find(self, key)

    def destroy(self) -> None:
        if self.handle:
            _check(lib().kv_index_destroy(self.handle), "kv_index_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def kv_index_create(max_entries: int) -> KvIndex:
    return KvIndex(max_entries)


def kv_index_destroy(idx: KvIndex) -> None:
    idx.destroy()


def kv_index_insert(idx: KvIndex, keys: np.ndarray, slots: np.ndarray, stream=None) -> None:
    keys = np.ascontiguousarray(keys, np.uint64)
    slots = np.ascontiguousarray(slots, np.int32)
    if keys.size != slots.size:
        raise ValueError("keys and slots differ in length")
    _check(lib().kv_index_insert(idx.handle, keys.ctypes.data, slots.ctypes.data, keys.size, _stream(stream)),
           "kv_index_insert")


def kv_index_insert_static(idx: KvIndex, keys: np.ndarray, slots: np.ndarray, stream=None) -> None:
    """kv_index_insert without any allocation: the device-table update is
    staged in the library's fixed per-GPU array (at most
    KV_INDEX_STATIC_MAX_PAIRS keys per call; calls on one GPU must be ordered
    on one stream)."""
    keys = np.ascontiguousarray(keys, np.uint64)
    slots = np.ascontiguousarray(slots, np.int32)
    if keys.size != slots.size:
        raise ValueError("keys and slots differ in length")
    _check(lib().kv_index_insert_static(idx.handle, keys.ctypes.data, slots.ctypes.data, keys.size,
                                        _stream(stream)), "kv_index_insert_static")


def kv_index_erase(idx: KvIndex, keys: np.ndarray, stream=None) -> None:
    keys = np.ascontiguousarray(keys, np.uint64)
    _check(lib().kv_index_erase(idx.handle, keys.ctypes.data, keys.size, _stream(stream)), "kv_index_erase")


def kv_index_size(idx: KvIndex) -> int:
    n = _i64(0)
    _check(lib().kv_index_size(idx.handle, ct.byref(n)), "kv_index_size")
    return n.value


def kv_index_find(idx: KvIndex, key: int) -> int:
    s = _i32(0)
    _check(lib().kv_index_find(idx.handle, key & 0xFFFFFFFFFFFFFFFF, ct.byref(s)), "kv_index_find")
    return s.value


def kv_lookup(idx: KvIndex, d_block_hash, d_blk_off, num_reqs: int, blocks_per_chunk: int, d_chunk_off,
              d_chunk_slot, d_hit_chunks, stream=None) -> None:
    import torch
    _check(lib().kv_lookup(idx.handle, _hash_ptr(d_block_hash), _dptr(d_blk_off, torch.int64, "blk_off"),
                           num_reqs, blocks_per_chunk, _dptr(d_chunk_off, torch.int64, "chunk_off"),
                           _dptr(d_chunk_slot, torch.int32, "chunk_slot"),
                           _dptr(d_hit_chunks, torch.int32, "hit_chunks"), _stream(stream)), "kv_lookup")


def kv_build_jobs(hit_chunks: np.ndarray, chunk_slot: np.ndarray, block_hash: np.ndarray, blk_off: np.ndarray,
                  chunk_off: np.ndarray, blocks_per_chunk: int, free_slots: np.ndarray):
    """Returns (retrieve [n,4] int32, store [m,4] int32, store_keys [m] uint64, dropped, status)."""
    R = blk_off.size - 1
    nchunks = int(chunk_off[-1]) if R >= 0 and chunk_off.size else 0
    hit = np.ascontiguousarray(hit_chunks, np.int32)
    cs = np.ascontiguousarray(chunk_slot, np.int32)
    bh = np.ascontiguousarray(block_hash, np.uint64)
    bo = np.ascontiguousarray(blk_off, np.int64)
    co = np.ascontiguousarray(chunk_off, np.int64)
    fs = np.ascontiguousarray(free_slots, np.int32)
    retr = np.zeros((max(nchunks, 1), 4), np.int32)
    store = np.zeros((max(nchunks, 1), 4), np.int32)
    keys = np.zeros(max(nchunks, 1), np.uint64)
    nr, ns, nd = _i32(0), _i32(0), _i32(0)
    rc = host_lib().kv_build_jobs(hit.ctypes.data, cs.ctypes.data, bh.ctypes.data, bo.ctypes.data, co.ctypes.data, R,
                             blocks_per_chunk, fs.ctypes.data if fs.size else None, fs.size, retr.ctypes.data,
                             ct.byref(nr), store.ctypes.data, keys.ctypes.data, ct.byref(ns), ct.byref(nd))
    if rc < 0 and rc != KV_ENOSPC:
        raise KvError(rc, "kv_build_jobs")
    return retr[:nr.value].copy(), store[:ns.value].copy(), keys[:ns.value].copy(), nd.value, rc


def kv_chunk_keys(block_hash: np.ndarray, blk_off: np.ndarray, blocks_per_chunk: int,
                  chunk_off: np.ndarray) -> np.ndarray:
    """Chunk keys (uint64, in (request, chunk) order) from host block hashes."""
    R = blk_off.size - 1
    bh = np.ascontiguousarray(block_hash if np.size(block_hash) else np.zeros(1), np.uint64)
    bo = np.ascontiguousarray(blk_off, np.int64)
    co = np.ascontiguousarray(chunk_off, np.int64)
    out = np.zeros(max(int(co[-1]) if co.size else 0, 1), np.uint64)
    _check(host_lib().kv_chunk_keys(bh.ctypes.data, bo.ctypes.data, R, blocks_per_chunk,
                                    co.ctypes.data, out.ctypes.data), "kv_chunk_keys")
    return out[:int(co[-1]) if co.size else 0].copy()


def kv_decide_claims(hit_chunks: np.ndarray, chunk_slot: np.ndarray, chunk_off: np.ndarray, ttu, ttr, requested,
                     slot_bytes: int, budget_bytes: int, num_slots: int, protected: Optional[np.ndarray] = None,
                     reserved_bytes: int = 0):
    """Commitment decisions for the claims of a batch.  Returns (decisions
    int32 [R], protected uint8 [num_slots], reserved bytes); `protected` and
    `reserved_bytes` are the ledger to start from (default: nothing
    protected)."""
    R = chunk_off.size - 1
    hit = np.ascontiguousarray(hit_chunks, np.int32)
    cs = np.ascontiguousarray(chunk_slot, np.int32)
    co = np.ascontiguousarray(chunk_off, np.int64)
    u = np.ascontiguousarray(np.broadcast_to(np.asarray(ttu, np.float64), (R,)))
    t = np.ascontiguousarray(np.broadcast_to(np.asarray(ttr, np.float64), (R,)))
    rq = np.ascontiguousarray(np.broadcast_to(np.asarray(requested).astype(bool), (R,)), np.uint8)
    prot = (np.zeros(num_slots, np.uint8) if protected is None
            else np.ascontiguousarray(protected, np.uint8).copy())
    if prot.size != num_slots:
        raise ValueError("protected must hold one flag per staging slot")
    dec = np.zeros(max(R, 1), np.int32)
    res = _u64(int(reserved_bytes))
    _check(host_lib().kv_decide_claims(R, hit.ctypes.data, cs.ctypes.data, co.ctypes.data, u.ctypes.data,
                                       t.ctypes.data, rq.ctypes.data, int(slot_bytes), int(budget_bytes),
                                       int(num_slots), prot.ctypes.data, ct.byref(res), dec.ctypes.data),
           "kv_decide_claims")
    return dec[:R].copy(), prot, res.value


def kv_build_jobs_routed(hit_chunks: np.ndarray, chunk_slot: np.ndarray, block_hash: np.ndarray,
                         blk_off: np.ndarray, chunk_off: np.ndarray, blocks_per_chunk: int, free_slots: np.ndarray,
                         requested, decisions: np.ndarray):
    """Returns (retrieve [n,4], ordinary [k,4], store [m,4], store_keys [m], dropped, status): the jobs of
    the requests whose retrieval is requested, their matched chunks split by commitment decision."""
    R = blk_off.size - 1
    nchunks = int(chunk_off[-1]) if chunk_off.size else 0
    hit = np.ascontiguousarray(hit_chunks, np.int32)
    cs = np.ascontiguousarray(chunk_slot, np.int32)
    bh = np.ascontiguousarray(block_hash, np.uint64)
    bo = np.ascontiguousarray(blk_off, np.int64)
    co = np.ascontiguousarray(chunk_off, np.int64)
    fs = np.ascontiguousarray(free_slots, np.int32)
    rq = np.ascontiguousarray(np.broadcast_to(np.asarray(requested).astype(bool), (R,)), np.uint8)
    dec = np.ascontiguousarray(decisions, np.int32)
    retr = np.zeros((max(nchunks, 1), 4), np.int32)
    ordn = np.zeros((max(nchunks, 1), 4), np.int32)
    store = np.zeros((max(nchunks, 1), 4), np.int32)
    keys = np.zeros(max(nchunks, 1), np.uint64)
    nr, no, ns, nd = _i32(0), _i32(0), _i32(0), _i32(0)
    rc = host_lib().kv_build_jobs_routed(hit.ctypes.data, cs.ctypes.data, bh.ctypes.data, bo.ctypes.data,
                                         co.ctypes.data, R, blocks_per_chunk, fs.ctypes.data if fs.size else None,
                                         fs.size, rq.ctypes.data, dec.ctypes.data, retr.ctypes.data, ct.byref(nr),
                                         ordn.ctypes.data, ct.byref(no), store.ctypes.data, keys.ctypes.data,
                                         ct.byref(ns), ct.byref(nd))
    if rc < 0 and rc != KV_ENOSPC:
        raise KvError(rc, "kv_build_jobs_routed")
    return (retr[:nr.value].copy(), ordn[:no.value].copy(), store[:ns.value].copy(), keys[:ns.value].copy(),
            nd.value, rc)


def kv_ttr_static(objs, obj_bytes, resident, static_rate: float) -> float:
    """Static TTR of a claim over its distinct objects `objs` (ids into obj_bytes / resident)."""
    o = np.ascontiguousarray(objs, np.int32).reshape(-1)
    b = np.ascontiguousarray(obj_bytes, np.float64).reshape(-1)
    r = np.ascontiguousarray(np.asarray(resident).astype(bool), np.uint8).reshape(-1)
    if r.size != b.size:
        raise ValueError("resident must hold one flag per object")
    out = _dbl(0.0)
    _check(host_lib().kv_ttr_static(o.size, o.ctypes.data, b.size, b.ctypes.data, r.ctypes.data, float(static_rate),
                                    ct.byref(out)), "kv_ttr_static")
    return out.value


def kv_ttr_state_aware(objs, obj_bytes, resident, queued, ready_at, now_s: float, busy_until_s: float,
                       stage_rate: float) -> float:
    """State-aware TTR of a claim against the staging queue's state."""
    o = np.ascontiguousarray(objs, np.int32).reshape(-1)
    b = np.ascontiguousarray(obj_bytes, np.float64).reshape(-1)
    r = np.ascontiguousarray(np.asarray(resident).astype(bool), np.uint8).reshape(-1)
    q = np.ascontiguousarray(np.asarray(queued).astype(bool), np.uint8).reshape(-1)
    t = np.ascontiguousarray(ready_at, np.float64).reshape(-1)
    if not (r.size == q.size == t.size == b.size):
        raise ValueError("per-object arrays must have the same length")
    out = _dbl(0.0)
    _check(host_lib().kv_ttr_state_aware(o.size, o.ctypes.data, b.size, b.ctypes.data, r.ctypes.data,
                                         q.ctypes.data, t.ctypes.data, float(now_s), float(busy_until_s),
                                         float(stage_rate), ct.byref(out)), "kv_ttr_state_aware")
    return out.value


def _layer_array(layers: Sequence) -> ct.Array:
    arr = (_vp * len(layers))()
    for i, t in enumerate(layers):
        arr[i] = _dptr(t, None, f"layer {i}")
    return arr


def kv_retrieve_scatter(layout: KvLayout, d_staging, layers: Sequence, d_block_tables, bt_stride: int,
                        num_reqs: int, d_jobs, num_jobs: int, stream=None) -> None:
    import torch
    if len(layers) != layout.num_layers:
        raise ValueError("one paged tensor per layer is required")
    _check(lib().kv_retrieve_scatter(ct.byref(layout), _dptr(d_staging, None, "staging"), _layer_array(layers),
                                     _dptr(d_block_tables, torch.int32, "block_tables"), bt_stride, num_reqs,
                                     _dptr(d_jobs, torch.int32, "jobs") if num_jobs else None, num_jobs,
                                     _stream(stream)), "kv_retrieve_scatter")


def kv_retrieve_plan(layout: KvLayout, h_jobs: np.ndarray) -> int:
    """The retrieve variant (KV_RETRIEVE_*) for a job list ([n,4] int32, grouped by slot)."""
    hj = np.ascontiguousarray(h_jobs, np.int32).reshape(-1, 4)
    return _check(host_lib().kv_retrieve_plan(ct.byref(layout), hj.ctypes.data if hj.size else None, hj.shape[0]),
                  "kv_retrieve_plan")


def kv_retrieve_scatter_as(kind: int, layout: KvLayout, d_staging, layers: Sequence, d_block_tables,
                           bt_stride: int, num_reqs: int, d_jobs, num_jobs: int, stream=None) -> None:
    """kv_retrieve_scatter with an explicit variant (KV_RETRIEVE_UNIT / PAIR / STREAM / QUAD)."""
    import torch
    if len(layers) != layout.num_layers:
        raise ValueError("one paged tensor per layer is required")
    _check(lib().kv_retrieve_scatter_as(kind, ct.byref(layout), _dptr(d_staging, None, "staging"),
                                        _layer_array(layers), _dptr(d_block_tables, torch.int32, "block_tables"),
                                        bt_stride, num_reqs, _dptr(d_jobs, torch.int32, "jobs") if num_jobs else None,
                                        num_jobs, _stream(stream)), "kv_retrieve_scatter_as")


def kv_store_gather(layout: KvLayout, d_staging, layers: Sequence, d_block_tables, bt_stride: int,
                    num_reqs: int, d_jobs, num_jobs: int, stream=None) -> None:
    import torch
    if len(layers) != layout.num_layers:
        raise ValueError("one paged tensor per layer is required")
    _check(lib().kv_store_gather(ct.byref(layout), _dptr(d_staging, None, "staging"), _layer_array(layers),
                                 _dptr(d_block_tables, torch.int32, "block_tables"), bt_stride, num_reqs,
                                 _dptr(d_jobs, torch.int32, "jobs") if num_jobs else None, num_jobs,
                                 _stream(stream)), "kv_store_gather")


def kv_probe_mixed_traffic(layout: KvLayout, d_staging, layers: Sequence, d_block_tables, bt_stride: int,
                           num_reqs: int, d_jobs, num_jobs: int, d_slots, num_read_slots: int, fill: int,
                           stream=None) -> None:
    """Measurement reference for the retrieve (not part of the path): reads every
    segment of the listed slots and writes `fill` into every destination block of
    the jobs, interleaved in one launch with no data passing between them.
    Overwrites those destination blocks."""
    import torch
    if len(layers) != layout.num_layers:
        raise ValueError("one paged tensor per layer is required")
    _check(lib().kv_probe_mixed_traffic(ct.byref(layout), _dptr(d_staging, None, "staging"), _layer_array(layers),
                                        _dptr(d_block_tables, torch.int32, "block_tables"), bt_stride, num_reqs,
                                        _dptr(d_jobs, torch.int32, "jobs") if num_jobs else None, num_jobs,
                                        _dptr(d_slots, torch.int32, "slots") if num_read_slots else None,
                                        num_read_slots, int(fill) & 0xFFFFFFFF, _stream(stream)),
           "kv_probe_mixed_traffic")


def _hptr(t, what: str = "host buffer") -> int:
    """Address of a pinned host tensor (torch, pin_memory) or an int address."""
    if isinstance(t, int):
        return t
    if t.is_cuda:
        raise ValueError(f"{what} must be in host memory")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if not t.is_pinned():
        raise ValueError(f"{what} must be pinned (asynchronous DMA copies need page-locked memory)")
    return t.data_ptr()


def kv_stage_in(layout: KvLayout, h_lower_tier, d_staging, slots, stream=None) -> None:
    """DMA copies of the listed slots, lower tier (pinned host) -> HBM staging."""
    sl = np.ascontiguousarray(slots, np.int32).reshape(-1)
    _check(lib().kv_stage_in(ct.byref(layout), _hptr(h_lower_tier, "lower tier") if sl.size else None,
                             _dptr(d_staging, None, "staging") if sl.size else None,
                             sl.ctypes.data if sl.size else None, sl.size, _stream(stream)), "kv_stage_in")


def kv_stage_out(layout: KvLayout, d_staging, h_lower_tier, slots, stream=None) -> None:
    """DMA copies of the listed slots, HBM staging -> lower tier (pinned host)."""
    sl = np.ascontiguousarray(slots, np.int32).reshape(-1)
    _check(lib().kv_stage_out(ct.byref(layout), _dptr(d_staging, None, "staging") if sl.size else None,
                              _hptr(h_lower_tier, "lower tier") if sl.size else None,
                              sl.ctypes.data if sl.size else None, sl.size, _stream(stream)), "kv_stage_out")


class KvPipeline:
    """Owner of the events of kv_retrieve_pipelined (kv_pipeline_create)."""

    def __init__(self, max_batches: int = 64):
        h = _vp()
        _check(lib().kv_pipeline_create(max_batches, ct.byref(h)), "kv_pipeline_create")
        self.handle = h.value
        self.max_batches = max_batches

    def close(self) -> None:
        if self.handle:
            _check(lib().kv_pipeline_destroy(self.handle), "kv_pipeline_destroy")
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def kv_retrieve_pipelined(pipeline: KvPipeline, layout: KvLayout, h_lower_tier, d_staging, layers: Sequence,
                          d_block_tables, bt_stride: int, num_reqs: int, h_jobs: np.ndarray, d_jobs,
                          slots_per_batch: int, copy_stream, stream=None) -> None:
    """Retrieve whose chunks start in the lower tier: per batch of slots,
    DMA copy on copy_stream, then the scatter on `stream` once they landed.
    h_jobs ([n,4] int32, grouped by slot) and d_jobs hold the same jobs."""
    import torch
    if len(layers) != layout.num_layers:
        raise ValueError("one paged tensor per layer is required")
    hj = np.ascontiguousarray(h_jobs, np.int32).reshape(-1, 4)
    n = hj.shape[0]
    if n and (d_jobs is None or int(d_jobs.numel()) != 4 * n):
        raise ValueError("d_jobs must hold the same jobs as h_jobs")
    _check(lib().kv_retrieve_pipelined(pipeline.handle, ct.byref(layout), _hptr(h_lower_tier, "lower tier") if n else None,
                                       _dptr(d_staging, None, "staging"), _layer_array(layers),
                                       _dptr(d_block_tables, torch.int32, "block_tables"), bt_stride, num_reqs,
                                       hj.ctypes.data if n else None,
                                       _dptr(d_jobs, torch.int32, "jobs") if n else None, n, slots_per_batch,
                                       _stream(copy_stream), _stream(stream)), "kv_retrieve_pipelined")


def kv_group_jobs_by_slot(jobs: np.ndarray) -> np.ndarray:
    """Returns the jobs ([n,4] int32) stably ordered by slot (a copy)."""
    jb = np.ascontiguousarray(jobs, np.int32).reshape(-1, 4).copy()
    _check(host_lib().kv_group_jobs_by_slot(jb.ctypes.data if jb.size else None, jb.shape[0]), "kv_group_jobs_by_slot")
    return jb


def kv_validate_jobs(layout: KvLayout, block_tables: np.ndarray, jobs: np.ndarray, is_store: bool) -> int:
    """Returns KV_OK, KV_ERANGE or KV_EDUP (other errors raise)."""
    bt = np.ascontiguousarray(block_tables, np.int32)
    jb = np.ascontiguousarray(jobs, np.int32).reshape(-1, 4)
    rc = host_lib().kv_validate_jobs(ct.byref(layout), bt.ctypes.data, bt.shape[1], bt.shape[0], jb.ctypes.data,
                                jb.shape[0], 1 if is_store else 0)
    if rc not in (KV_OK, KV_ERANGE, KV_EDUP):
        raise KvError(rc, "kv_validate_jobs")
    return rc


def kv_validate_jobs_device(layout: KvLayout, d_block_tables, bt_stride: int, num_reqs: int, d_jobs, num_jobs: int,
                            is_store: bool, d_marks, d_status, stream=None) -> None:
    """Enqueue the device form of kv_validate_jobs: d_status (int32 device
    tensor of one element) receives KV_OK, KV_ERANGE or KV_EDUP; d_marks is
    int32 device scratch of 2 + (num_slots if is_store else num_blocks)."""
    import torch
    need = 2 + (layout.num_slots if is_store else layout.num_blocks)
    if not isinstance(d_marks, int) and d_marks.numel() < need:
        raise ValueError(f"d_marks holds {d_marks.numel()} int32, needs {need}")
    _check(lib().kv_validate_jobs_device(ct.byref(layout), _dptr(d_block_tables, torch.int32, "block_tables"),
                                         bt_stride, num_reqs, _dptr(d_jobs, torch.int32, "jobs"), num_jobs,
                                         1 if is_store else 0, _dptr(d_marks, torch.int32, "marks"),
                                         _dptr(d_status, torch.int32, "status"), _stream(stream)),
           "kv_validate_jobs_device")


def kv_commit_should_stage(ttu_s: float, ttr_s: float, free_protected_bytes: int, claim_new_bytes: int,
                           claim_total_bytes: int, budget_bytes: int, retrieval_requested: bool) -> int:
    """Returns a KV_DEFER/KV_COMMIT/KV_BLOCKED/KV_ORDINARY decision or KV_EINVAL."""
    return host_lib().kv_commit_should_stage(ttu_s, ttr_s, free_protected_bytes, claim_new_bytes, claim_total_bytes,
                                        budget_bytes, 1 if retrieval_requested else 0)


def kv_commit_should_stage_n(ttu, ttr, free_protected_bytes: int, claim_new, claim_total, budget_bytes: int,
                             requested) -> np.ndarray:
    """The commitment rule for a batch of claims (int32 decisions, KV_EINVAL
    for an element with invalid inputs)."""
    a = np.ascontiguousarray(ttu, np.float64).reshape(-1)
    n = a.size
    b = np.ascontiguousarray(ttr, np.float64).reshape(-1)
    cn = np.ascontiguousarray(claim_new, np.uint64).reshape(-1)
    ct_ = np.ascontiguousarray(claim_total, np.uint64).reshape(-1)
    rq = np.ascontiguousarray(np.asarray(requested).astype(bool), np.uint8).reshape(-1)
    if not (b.size == cn.size == ct_.size == rq.size == n):
        raise ValueError("all claim arrays must have the same length")
    out = np.zeros(n, np.int32)
    if n:
        _check(host_lib().kv_commit_should_stage_n(n, a.ctypes.data, b.ctypes.data, int(free_protected_bytes),
                                              cn.ctypes.data, ct_.ctypes.data, int(budget_bytes), rq.ctypes.data,
                                              out.ctypes.data), "kv_commit_should_stage_n")
    return out


def kv_host_device_pointer(host_ptr: int) -> int:
    d = _vp()
    _check(lib().kv_host_device_pointer(host_ptr, ct.byref(d)), "kv_host_device_pointer")
    return d.value


def kv_sim_run(config: KvSimConfig, obj_bytes, arrival, manifests, uncached, out_tokens, trace: bool = False):
    """Run the controller simulation.  Returns (result, first_token, done,
    trace) where trace is a list of (t, kind name, id) if requested."""
    ob = np.ascontiguousarray(obj_bytes, np.float64)
    arr = np.ascontiguousarray(arrival, np.float64)
    N = arr.size
    off = np.zeros(N + 1, np.int64)
    np.cumsum([len(m) for m in manifests], out=off[1:])
    objs = np.ascontiguousarray(np.concatenate([np.asarray(m, np.int32) for m in manifests]) if N and off[-1]
                                else np.zeros(1, np.int32), np.int32)
    unc = np.ascontiguousarray(uncached, np.int32)
    out = np.ascontiguousarray(out_tokens, np.int32)
    ft = np.zeros(max(N, 1), np.float64)
    dn = np.zeros(max(N, 1), np.float64)
    res = KvSimResult()
    n_tr = _i64(0)
    buf = None
    cap = 0
    if trace:
        cap = 64 * (N + ob.size) + 1024
        buf = (KvSimEvent * cap)()
    rc = host_lib().kv_sim_run(ct.byref(config), ob.ctypes.data if ob.size else None, ob.size, arr.ctypes.data,
                          off.ctypes.data, objs.ctypes.data, unc.ctypes.data, out.ctypes.data, N, ft.ctypes.data,
                          dn.ctypes.data, ct.byref(res), ct.cast(buf, ct.c_void_p) if buf is not None else None,
                          cap, ct.byref(n_tr))
    _check(rc, "kv_sim_run")
    events = None
    if trace:
        if n_tr.value > cap:
            raise RuntimeError("trace buffer too small")
        events = [(buf[k].t, SIM_TRACE_KINDS[buf[k].kind], buf[k].id) for k in range(n_tr.value)]
    return res, ft[:N].copy(), dn[:N].copy(), events
