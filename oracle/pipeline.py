"""The oracle's version of one pass over a workload -- TEST INFRASTRUCTURE ONLY.

Mirrors the sequence the library runs (hash, prefix lookup, job build,
retrieve scatter, store gather, index update) with the plain C oracle and a
Python dict as the index.  KV bytes come from the workload generator's host
formula, never from the GPU.
"""
from __future__ import annotations

import time
from typing import Dict, List, Optional

import numpy as np

import oracle
from workloads import Workload, kv_bytes_np


class OraclePath:
    def __init__(self, w: Workload, hash_seed: int = 0, with_kv: bool = True, staging_tag: int = 1,
                 pool_tag_base: int = 1000, kv_seed: int = 0, finite: bool = True):
        self.w = w
        self.hash_seed = hash_seed
        kv_stride, block_stride = w.strides()
        self.layout = oracle.make_layout(w.shape, w.num_blocks, w.num_slots, kv_stride, block_stride)
        self.bpc = w.shape.chunk_tokens // 16
        self.set_batch(w)
        self.index: Dict[int, int] = {}
        self.free: List[int] = []
        self.staging: Optional[np.ndarray] = None
        self.layers: Optional[List[np.ndarray]] = None
        if with_kv:
            self.staging = kv_bytes_np(staging_tag, kv_seed, 0, w.staged_bytes(), finite).copy()
            self.layers = [kv_bytes_np(pool_tag_base + l, kv_seed, 0, w.layer_bytes(), finite).copy()
                           for l in range(w.shape.num_layers)]

    def set_batch(self, w: Workload) -> None:
        """Take a new request batch over the same pool and staging buffer."""
        self.batch = w
        self.blk_off = oracle.block_offsets(w.tok_off)
        self.chunk_off = oracle.chunk_offsets(self.blk_off, self.bpc)

    def prestage(self) -> None:
        w = self.w
        toks, off = w.prefix_stream_request()
        boff = oracle.block_offsets(off)
        h = oracle.hash_prefix(toks, off, self.hash_seed, boff)
        for slot, (p, j) in enumerate(w.prestage_chunks):
            self.index[int(h[boff[p] + (j + 1) * self.bpc - 1])] = slot
        self.free = list(range(len(w.prestage_chunks), w.num_slots))

    def run_pass(self, evict_stored: bool = False, timers: Optional[dict] = None) -> dict:
        """One pass.  ``timers``: optional dict; wall seconds of each step are
        added under "hash", "lookup" (lookup and job build), "retrieve" and
        "store"."""
        w = self.batch
        clock = [time.perf_counter()]

        def lap(name):
            if timers is not None:
                now = time.perf_counter()
                timers[name] = timers.get(name, 0.0) + now - clock[0]
                clock[0] = now

        bh = oracle.hash_prefix(w.tokens, w.tok_off, self.hash_seed, self.blk_off)
        lap("hash")
        cs, hit = oracle.lookup(self.index, bh, self.blk_off, self.bpc, self.chunk_off)
        retr, store, skeys, dropped = oracle.build_jobs(hit, cs, bh, self.blk_off, self.chunk_off, self.bpc,
                                                        np.array(self.free, np.int32))
        lap("lookup")
        if self.staging is not None:
            oracle.retrieve_scatter(self.layout, self.staging, self.layers, w.block_tables, retr)
            lap("retrieve")
            oracle.store_gather(self.layout, self.staging, self.layers, w.block_tables, store)
            lap("store")
        for k, s in zip(skeys, store[:, 0]):
            self.index[int(k)] = int(s)
        used = set(int(s) for s in store[:, 0])
        self.free = [s for s in self.free if s not in used]
        if evict_stored:
            for k in skeys:
                self.index.pop(int(k), None)
            self.free = sorted(self.free + sorted(used))
        return dict(block_hash=bh, chunk_slot=cs, hit=hit, retrieve=retr, store=store, store_keys=skeys,
                    dropped=dropped)
