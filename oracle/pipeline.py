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

    def decide_claims(self, hit, chunk_slot, claims) -> List[int]:
        """Commitment decision of every request's claim (Section 3.2).  The
        claim of request r is its matched prefix; its KV objects are the
        distinct slots of those chunks.  Claims whose retrieval is requested
        are considered first, then the others, each in request order, and a
        claim that cannot commit does not hold up the rest ("Commitment and
        replanning").  The protected budget counts each protected object once,
        so a claim newly reserves only its objects not yet protected ("Shared
        staging and resource lifecycle")."""
        w = self.batch
        R = w.num_reqs
        slot_bytes = w.shape.slot_bytes
        requested = [bool(x) for x in claims.requested]
        protected = set()
        reserved = 0
        decision = [None] * R
        order = [r for r in range(R) if requested[r]] + [r for r in range(R) if not requested[r]]
        for r in order:
            objs = []
            for j in range(int(hit[r])):
                s = int(chunk_slot[self.chunk_off[r] + j])
                if s not in objs:
                    objs.append(s)
            total = len(objs) * slot_bytes
            new = sum(slot_bytes for s in objs if s not in protected)
            free = max(claims.budget_bytes - reserved, 0)
            d = oracle.commit_should_stage(float(claims.ttu[r]), float(claims.ttr[r]), free, new, total,
                                           claims.budget_bytes, requested[r])
            decision[r] = d
            if d == oracle.COMMIT:
                protected.update(objs)
                reserved += new
        return decision

    def _running_jobs(self, bh, cs, hit, running):
        """Jobs of the running requests only: the oracle's job build over the
        sub-batch they form, with request ids mapped back to the batch."""
        idx = [r for r in range(self.batch.num_reqs) if running[r]]
        bo, co = self.blk_off, self.chunk_off
        sub_bh = np.concatenate([bh[bo[r]:bo[r + 1]] for r in idx]) if idx else np.zeros(0, np.uint64)
        sub_cs = np.concatenate([cs[co[r]:co[r + 1]] for r in idx]) if idx else np.zeros(0, np.int32)
        sub_bo = np.zeros(len(idx) + 1, np.int64)
        sub_co = np.zeros(len(idx) + 1, np.int64)
        for k, r in enumerate(idx):
            sub_bo[k + 1] = sub_bo[k] + bo[r + 1] - bo[r]
            sub_co[k + 1] = sub_co[k] + co[r + 1] - co[r]
        sub_hit = np.array([hit[r] for r in idx], np.int32)
        retr, store, skeys, dropped = oracle.build_jobs(sub_hit, sub_cs, sub_bh, sub_bo, sub_co, self.bpc,
                                                        np.array(self.free, np.int32))
        back = np.array(idx, np.int32)
        for jobs in (retr, store):
            if len(jobs):
                jobs[:, 1] = back[jobs[:, 1]]
        return retr, store, skeys, dropped

    def run_pass(self, evict_stored: bool = False, timers: Optional[dict] = None, claims=None) -> dict:
        """One pass.  ``timers``: optional dict; wall seconds of each step are
        added under "hash", "lookup" (lookup and job build), "retrieve" and
        "store".  ``claims``: per-request commitment inputs (requested, ttu,
        ttr arrays and budget_bytes); by default every request's retrieval is
        requested now with TTU = TTR = 0 and the whole staging buffer as the
        budget.  Only requests whose retrieval is requested run and get jobs;
        their matched chunks are retrieved on the protected route when the
        claim commits and on the ordinary route otherwise (Section 3.2,
        "Protected capacity and on-demand retrieval"); both routes copy the
        same staged bytes."""
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
        if claims is None:
            decision = [oracle.COMMIT] * w.num_reqs
            running = [True] * w.num_reqs
            retr, store, skeys, dropped = oracle.build_jobs(hit, cs, bh, self.blk_off, self.chunk_off, self.bpc,
                                                            np.array(self.free, np.int32))
        else:
            decision = self.decide_claims(hit, cs, claims)
            running = [bool(x) for x in claims.requested]
            retr, store, skeys, dropped = self._running_jobs(bh, cs, hit, running)
        ordinary = np.array([decision[q[1]] == oracle.ORDINARY for q in retr], bool)
        retr, ordn = retr[~ordinary] if len(retr) else retr, retr[ordinary] if len(retr) else retr
        lap("lookup")
        if self.staging is not None:
            oracle.retrieve_scatter(self.layout, self.staging, self.layers, w.block_tables, retr)
            oracle.retrieve_scatter(self.layout, self.staging, self.layers, w.block_tables, ordn)
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
        return dict(block_hash=bh, chunk_slot=cs, hit=hit, retrieve=retr, ordinary=ordn, store=store,
                    store_keys=skeys, dropped=dropped, decisions=np.array(decision, np.int32))
