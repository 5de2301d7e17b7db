"""One pass of the staging hot path over a batch of requests, on one GPU.

A pass is:  hash (kv_hash_prefix) -> lookup (kv_lookup) -> one device-to-host
copy of the lookup result -> commitment decisions for the requests' claims
(kv_decide_claims) and the host job build that routes each claim by its
decision (kv_build_jobs_routed) -> one host-to-device copy of the jobs ->
retrieve scatter (kv_retrieve_plan picks the copy variant, or the variant
tune_retrieve found faster for that plan on this path's pool;
kv_retrieve_scatter_as runs it) -> store gather (kv_store_gather) ->
index update (kv_index_insert; optionally kv_index_erase of what was just
stored, which returns the batch to its starting state so that passes can be
repeated).

When the workload keeps its staged chunks in host memory, ``lower_tier``
picks how the retrieve reaches them:
  "zero-copy"   the scatter reads the pinned host buffer through its device
                mapping (kv_retrieve_scatter on a host-mapped pointer);
  "pipelined"   host memory is the lower tier and an HBM staging buffer the
                fast tier: chunks not resident in HBM are staged by DMA on a
                second stream, batch by batch, and each batch's scatter waits
                for its copies (kv_retrieve_pipelined);
  "serialized"  the same, with copies and scatters on one stream.
In the two staged modes the store gathers into the HBM staging buffer and
copies the stored slots back to host memory (kv_stage_out).

Commitment (Section 3.2).  Each request's claim is its matched prefix.  A
pass takes, per request, whether retrieval is requested now (the request
runs in this pass), its TTU and TTR estimates, and a protected-capacity
budget (``ClaimInputs``; by default every request runs, TTU = TTR = 0, and the
budget is the whole staging buffer, so every claim commits).  The decisions
route the work:
  KV_COMMIT, requested      the claim's chunks take the protected route: the
                            scatter from the HBM fast tier (staged modes: DMA
                            into HBM first, then the gated scatter);
  KV_ORDINARY               the ordinary retrieval path: the chunks are read
                            where they lie without protection (staged modes:
                            zero-copy from the lower tier, nothing is staged
                            into HBM for them), in a launch of their own;
  KV_COMMIT, not requested  staging begins at commitment: in staged modes the
                            claim's chunks not yet in HBM are copied there;
  KV_BLOCKED, KV_DEFER      the claim stays PLANNED; its request gets no jobs.
Only requests whose retrieval is requested get retrieve or store jobs.
Protection lasts until the pass's retrieval completes, so each pass starts
with nothing protected.

This module only sequences the C calls and owns the buffers they read and
write; it computes nothing itself.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch

from . import (KV_COMMIT, KV_OK, KV_ORDINARY, KV_RETRIEVE_QUAD, KV_RETRIEVE_STREAM, RETRIEVE_KIND_NAMES, KvIndex,
               KvLayout, KvPipeline, kv_build_jobs_routed, kv_chunk_keys, kv_decide_claims,
               kv_group_jobs_by_slot, kv_hash_prefix, kv_host_device_pointer, kv_lookup, kv_retrieve_pipelined,
               kv_retrieve_plan, kv_retrieve_scatter_as, kv_stage_in, kv_stage_out, kv_store_gather,
               kv_validate_jobs_device, make_layout)

LOWER_TIER_MODES = ("zero-copy", "pipelined", "serialized")


@dataclass
class ClaimInputs:
    """Per-request inputs of a pass's commitment decisions (Section 3.2)."""
    requested: np.ndarray        # bool [R]: retrieval requested now (the request runs in this pass)
    ttu: np.ndarray              # float64 [R], seconds until retrieval would begin
    ttr: np.ndarray              # float64 [R], seconds until the claim would be stage-ready
    budget_bytes: int            # protected-capacity budget

    @staticmethod
    def all_now(num_reqs: int, budget_bytes: int) -> "ClaimInputs":
        """Every request runs now (retrieval requested, TTU = TTR = 0)."""
        return ClaimInputs(np.ones(num_reqs, bool), np.zeros(num_reqs), np.zeros(num_reqs), int(budget_bytes))


@dataclass
class PassStats:
    num_retrieve: int = 0        # jobs on the protected route
    num_ordinary: int = 0        # jobs on the ordinary route
    num_store: int = 0
    dropped: int = 0
    retrieve_bytes: int = 0      # payload copied by the scatter, both routes (read = written)
    ordinary_bytes: int = 0      # of which on the ordinary route
    store_bytes: int = 0
    staged_bytes: int = 0        # lower tier -> HBM by DMA (staged modes)
    commits: int = 0
    reserved_bytes: int = 0      # protected bytes reserved by the pass's commitments
    decisions: Dict[int, int] = field(default_factory=dict)


class StagingPath:
    """Device state of one workload: tokens, offsets, block tables, staging
    buffer, per-layer paged KV tensors, the staged-chunk index and the host
    free-slot list.

    Parameters mirror the workload description (``workloads.Workload``): it
    provides shapes, token ids, block tables and which chunks are staged at
    the start.  KV contents are filled by the caller (see ``fill``)."""

    def __init__(self, w, device: str = "cuda", hash_seed: int = 0, stream: Optional[torch.cuda.Stream] = None,
                 lower_tier: str = "zero-copy", slots_per_batch: int = 4, overlap: bool = False):
        if lower_tier not in LOWER_TIER_MODES:
            raise ValueError(f"lower_tier must be one of {LOWER_TIER_MODES}")
        self.w = w
        self.dev = torch.device(device)
        self.hash_seed = hash_seed
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.dev)
        # hash, lookup and index updates; a stream of their own when passes overlap
        self._own_lookup_stream = torch.cuda.Stream(self.dev)
        self.lookup_stream = self._own_lookup_stream if overlap else self.stream
        self._lookup_done = torch.cuda.Event()
        self._parity = 0
        s = w.shape
        kv_stride, block_stride = w.strides()
        self.layout: KvLayout = make_layout(s.num_layers, s.kv_heads, s.head_dim, s.elem_bytes, s.block_size,
                                            s.chunk_tokens, w.num_blocks, w.num_slots, kv_stride, block_stride)
        self.bpc = s.chunk_tokens // 16
        d = self.dev
        self.staged_mode = w.staging_in_host and lower_tier != "zero-copy"
        self.slots_per_batch = slots_per_batch
        self.resident = np.zeros(w.num_slots, bool)   # slots whose HBM copy is current (staged modes)
        with torch.cuda.stream(self.stream):
            self.staging_host = None
            if w.staging_in_host:
                self.staging_host = torch.empty(w.staged_bytes(), dtype=torch.uint8, pin_memory=True)
                self.staging_ptr = kv_host_device_pointer(self.staging_host.data_ptr())
                self.host_mapped_ptr = self.staging_ptr     # the lower tier read in place (ordinary route)
                self.staging = None
                if self.staged_mode:
                    self.staging = torch.empty(w.staged_bytes(), dtype=torch.uint8, device=d)
                    self.staging_ptr = self.staging.data_ptr()
            else:
                self.staging = torch.empty(w.staged_bytes(), dtype=torch.uint8, device=d)
                self.staging_ptr = self.staging.data_ptr()
            self.layers = [torch.empty(w.layer_bytes(), dtype=torch.uint8, device=d) for _ in range(s.num_layers)]
        if self.staged_mode:
            self.copy_stream = (torch.cuda.Stream(self.dev) if lower_tier == "pipelined" else self.stream)
            self.pipeline = KvPipeline(64)
        self.set_batch(w)
        self.index = KvIndex(max(w.num_slots, 1))
        self.free: List[int] = []
        self.last_store_keys = np.zeros(0, np.uint64)
        self.last_store_slots = np.zeros(0, np.int32)
        self.last_retrieve = np.zeros((0, 4), np.int32)
        self.last_ordinary = np.zeros((0, 4), np.int32)
        self.last_store = np.zeros((0, 4), np.int32)
        self.last_decisions = np.zeros(0, np.int32)
        self.retrieve_kind: Optional[int] = None
        self._val_marks: Optional[torch.Tensor] = None   # scratch of the device race check (validate=True)
        # planned retrieve variant -> variant to run instead (set by tune_retrieve)
        self.retrieve_choice: Dict[int, int] = {}
        self._last_nres = 0

    def set_batch(self, w) -> None:
        """Load a new request batch (tokens, offsets, block tables) that uses
        this path's KV shape, pool and staging buffer."""
        assert w.shape == self.w.shape and w.num_blocks == self.w.num_blocks and w.num_slots == self.w.num_slots
        self.batch = w
        R = w.num_reqs
        blk_off, chunk_off = w.offsets()
        self.blk_off_h, self.chunk_off_h = blk_off, chunk_off
        nblk, nch = int(blk_off[-1]), int(chunk_off[-1])
        d = self.dev
        with torch.cuda.stream(self.stream):
            self.tokens = torch.from_numpy(w.tokens if w.tokens.size else np.zeros(1, np.int32)).to(d)
            self.tok_off = torch.from_numpy(w.tok_off).to(d)
            self.blk_off = torch.from_numpy(blk_off).to(d)
            self.chunk_off = torch.from_numpy(chunk_off).to(d)
            self.block_hash = torch.empty(max(nblk, 1), dtype=torch.int64, device=d)
            self.chunk_slot = torch.empty(max(nch, 1), dtype=torch.int32, device=d)
            self.hit = torch.empty(max(R, 1), dtype=torch.int32, device=d)
            self.bt = torch.from_numpy(np.ascontiguousarray(w.block_tables)).to(d)
            self.d_retr = torch.empty((max(nch, 1), 4), dtype=torch.int32, device=d)
            self.d_store = torch.empty((max(nch, 1), 4), dtype=torch.int32, device=d)
        # pinned host mirrors for the one D2H and one H2D copy of a pass
        self.h_block_hash = torch.zeros(max(nblk, 1), dtype=torch.int64, pin_memory=True)
        self.h_chunk_slot = torch.zeros(max(nch, 1), dtype=torch.int32, pin_memory=True)
        self.h_hit = torch.zeros(max(R, 1), dtype=torch.int32, pin_memory=True)
        # job lists, two of each: a pass fills one while the upload of the other may still be queued
        self._h_retr = [torch.zeros((max(nch, 1), 4), dtype=torch.int32, pin_memory=True) for _ in range(2)]
        self._h_store = [torch.zeros((max(nch, 1), 4), dtype=torch.int32, pin_memory=True) for _ in range(2)]
        self._uploaded = [torch.cuda.Event(), torch.cuda.Event()]
        self.stream.synchronize()
        self.lookup_stream.synchronize()

    # ------------------------------------------------------------------
    def staging_view(self) -> torch.Tensor:
        """The authoritative staged chunks: the host buffer when the workload
        keeps them in host memory, else the HBM staging buffer."""
        return self.staging_host if self.staging_host is not None else self.staging

    def set_overlap(self, overlap: bool) -> None:
        """Run hash, lookup and index updates on a stream of their own (passes
        can overlap) or on this path's stream (each pass after the previous
        one's copies).  Waits for all queued work first."""
        self.stream.synchronize()
        self.lookup_stream.synchronize()
        self.lookup_stream = self._own_lookup_stream if overlap else self.stream

    def drop_fast_tier(self) -> None:
        """Forget which slots are resident in HBM (staged modes): the next
        retrieve stages every chunk it reads from host memory again."""
        self.resident[:] = False

    def fill(self, staging_tag: int, pool_tag_base: int, seed: int, finite: bool = True) -> None:
        """Fill staging and pool with the workload KV formula (input generation).
        Layer l of the pool uses tag ``pool_tag_base + l``."""
        from workloads import fill_kv_
        self.resident[:] = False
        with torch.cuda.stream(self.stream):
            if self.staging_host is None:
                fill_kv_(self.staging, staging_tag, seed, finite)
            else:
                # host staging: fill device windows and copy them into the pinned buffer
                n = self.staging_host.numel()
                win = min(n, 1 << 30)
                scratch = torch.empty(win, dtype=torch.uint8, device=self.dev)
                for s0 in range(0, n, win):
                    m = min(win, n - s0)
                    fill_kv_(scratch[:m], staging_tag, seed, finite, byte_start=s0)
                    self.staging_host[s0:s0 + m].copy_(scratch[:m])
                del scratch
            for l, t in enumerate(self.layers):
                fill_kv_(t, pool_tag_base + l, seed, finite)
        self.stream.synchronize()

    def prestage(self) -> None:
        """Index the chunks the workload says are staged at start: hash the
        shared prefix streams with the library and insert their chunk keys
        with slots 0..P-1 in workload order; the other slots are free."""
        w = self.w
        toks, off = w.prefix_stream_request()
        P = len(w.prestage_chunks)
        if P:
            nb = np.diff(off) // 16
            boff = np.zeros(off.size, np.int64)
            np.cumsum(nb, out=boff[1:])
            with torch.cuda.stream(self.stream):
                dt = torch.from_numpy(toks if toks.size else np.zeros(1, np.int32)).to(self.dev)
                doff = torch.from_numpy(off).to(self.dev)
                dboff = torch.from_numpy(boff).to(self.dev)
                dh = torch.empty(max(int(boff[-1]), 1), dtype=torch.int64, device=self.dev)
                kv_hash_prefix(dt, doff, off.size - 1, self.hash_seed, dboff, dh, self.stream)
                h = dh.cpu().numpy().view(np.uint64)
            nc = np.diff(boff) // self.bpc
            coff = np.zeros(off.size, np.int64)
            np.cumsum(nc, out=coff[1:])
            ck = kv_chunk_keys(h, boff, self.bpc, coff)
            keys = np.array([ck[coff[p] + j] for p, j in w.prestage_chunks], np.uint64)
            self.index.insert(keys, np.arange(P, dtype=np.int32), self.lookup_stream)
        self.free = list(range(P, w.num_slots))
        self.stream.synchronize()
        self.lookup_stream.synchronize()

    # ------------------------------------------------------------------
    def run_pass(self, evict_stored: bool = False, validate: bool = False, timers: Optional[dict] = None,
                 claims: Optional[ClaimInputs] = None) -> PassStats:
        """One pass of the hot path over the current batch.

        ``timers``: optional dict; when given, a (start, end) pair of
        torch.cuda.Event is appended under "hash", "lookup", "retrieve",
        "ordinary" and "store" around each launch, recorded on the stream it
        runs on.  ``claims``: the commitment inputs (default: every request
        runs now and the budget is the whole staging buffer).  ``validate``
        (debug): the job lists are checked on the host and, once uploaded, on
        the device (kv_validate_jobs, kv_validate_jobs_device) before any copy
        is launched."""
        self.launch_lookup(timers)
        return self.complete_pass(evict_stored, validate, timers, claims)

    def launch_lookup(self, timers: Optional[dict] = None) -> None:
        """Enqueue the first half of a pass on the lookup stream: hash, lookup
        and the copy of their results to pinned host memory.  It sees every
        index update enqueued before it.  With overlapping passes it runs
        while the copies of the previous pass are still in flight."""
        w = self.batch
        R = w.num_reqs
        ls = self.lookup_stream
        with torch.cuda.stream(ls):
            e = self._ev(timers, "hash", ls)
            kv_hash_prefix(self.tokens, self.tok_off, R, self.hash_seed, self.blk_off, self.block_hash, ls)
            self._ev_end(e, ls)
            e = self._ev(timers, "lookup", ls)
            kv_lookup(self.index, self.block_hash, self.blk_off, R, self.bpc, self.chunk_off, self.chunk_slot,
                      self.hit, ls)
            self._ev_end(e, ls)
            self.h_block_hash.copy_(self.block_hash, non_blocking=True)
            self.h_chunk_slot.copy_(self.chunk_slot, non_blocking=True)
            self.h_hit.copy_(self.hit, non_blocking=True)
            self._lookup_done.record(ls)

    def default_claims(self) -> ClaimInputs:
        return ClaimInputs.all_now(self.batch.num_reqs, self.w.num_slots * self.w.shape.slot_bytes)

    def complete_pass(self, evict_stored: bool = False, validate: bool = False,
                      timers: Optional[dict] = None, claims: Optional[ClaimInputs] = None) -> PassStats:
        """Second half of a pass: wait for the lookup results, decide the
        claims and build the jobs on the host, enqueue the copies on this
        path's stream and the index update on the lookup stream."""
        w = self.batch
        R = w.num_reqs
        st = PassStats()
        nblk, nch = int(self.blk_off_h[-1]), int(self.chunk_off_h[-1])
        self._lookup_done.synchronize()
        bh = self.h_block_hash.numpy()[:nblk].view(np.uint64)
        cs = self.h_chunk_slot.numpy()[:nch]
        hit = self.h_hit.numpy()[:R]
        free = np.array(self.free, np.int32)
        slot_bytes = w.shape.slot_bytes
        cl = claims if claims is not None else self.default_claims()
        dec, protected, reserved = kv_decide_claims(hit, cs, self.chunk_off_h, cl.ttu, cl.ttr, cl.requested,
                                                    slot_bytes, cl.budget_bytes, w.num_slots)
        retr, ordn, store, skeys, dropped, rc = kv_build_jobs_routed(hit, cs, bh, self.blk_off_h, self.chunk_off_h,
                                                                     self.bpc, free, cl.requested, dec)
        st.num_retrieve, st.num_ordinary, st.num_store, st.dropped = len(retr), len(ordn), len(store), dropped
        st.retrieve_bytes = (len(retr) + len(ordn)) * slot_bytes
        st.ordinary_bytes = len(ordn) * slot_bytes
        st.store_bytes = len(store) * slot_bytes
        st.reserved_bytes = reserved
        for d, c in zip(*np.unique(dec, return_counts=True)):
            st.decisions[int(d)] = int(c)
        st.commits = int(np.count_nonzero(dec == KV_COMMIT))
        if validate:
            from . import kv_validate_jobs
            both = np.concatenate([retr, ordn])
            assert kv_validate_jobs(self.layout, w.block_tables, both, False) == 0 or len(both) == 0
            assert kv_validate_jobs(self.layout, w.block_tables, store, True) == 0 or len(store) == 0
        nr, no, ns = len(retr), len(ordn), len(store)
        nres = nr   # jobs whose chunk is already in the staging buffer the scatter reads
        par = self._parity
        self._parity ^= 1
        self._uploaded[par].synchronize()     # the upload that last read these buffers has run
        self.h_retr, self.h_store = self._h_retr[par], self._h_store[par]
        with torch.cuda.stream(self.stream):
            if nr:
                # jobs sharing a staged chunk run back to back (results do not depend on order)
                grouped = kv_group_jobs_by_slot(retr)
                if self.staged_mode:
                    # resident chunks first (plain scatter), then the ones to stage
                    here = self.resident[grouped[:, 0]]
                    grouped = np.concatenate([grouped[here], grouped[~here]])
                    nres = int(here.sum())
                self.h_retr.numpy()[:nr] = grouped
            if no:
                # the ordinary route's jobs follow the protected route's in the same upload
                self.h_retr.numpy()[nr:nr + no] = kv_group_jobs_by_slot(ordn)
            if nr + no:
                self.d_retr[:nr + no].copy_(self.h_retr[:nr + no], non_blocking=True)
            if ns:
                self.h_store.numpy()[:ns] = store
                self.d_store[:ns].copy_(self.h_store[:ns], non_blocking=True)
            self._uploaded[par].record(self.stream)
            if validate:
                self._validate_on_device(nr + no, ns)
            e = self._ev(timers, "retrieve")
            # the copy variant suited to how these jobs share staged chunks
            planned = kv_retrieve_plan(self.layout, self.h_retr.numpy()[:nres])
            self.retrieve_kind = self.retrieve_choice.get(planned, planned)
            self._last_nres = nres
            kv_retrieve_scatter_as(self.retrieve_kind, self.layout, self.staging_ptr, self.layers, self.bt,
                                   w.bt_stride, R, self.d_retr, nres, self.stream)
            if nres < nr:
                h_jobs = self.h_retr.numpy()[nres:nr]
                es = None
                if self.copy_stream is not self.stream:
                    self.copy_stream.wait_stream(self.stream)
                    es = self._ev(timers, "stage", self.copy_stream)   # the copies alone
                kv_retrieve_pipelined(self.pipeline, self.layout, self.staging_host, self.staging, self.layers,
                                      self.bt, w.bt_stride, R, h_jobs, self.d_retr[nres:nr], self.slots_per_batch,
                                      self.copy_stream, self.stream)
                self._ev_end(es, self.copy_stream)
                staged = np.unique(h_jobs[:, 0])
                self.resident[staged] = True
                st.staged_bytes = int(staged.size) * slot_bytes
            self._ev_end(e)
            if no:
                # ordinary retrieval: read in place, unprotected (from the lower tier when there is one)
                e = self._ev(timers, "ordinary")
                src = self.host_mapped_ptr if self.staged_mode else self.staging_ptr
                okind = kv_retrieve_plan(self.layout, self.h_retr.numpy()[nr:nr + no])
                kv_retrieve_scatter_as(okind, self.layout, src, self.layers, self.bt, w.bt_stride, R,
                                       self.d_retr[nr:nr + no], no, self.stream)
                self._ev_end(e)
            if self.staged_mode:
                # staging begins at commitment for claims whose retrieval is not requested yet
                ahead = np.nonzero((protected != 0) & ~self.resident)[0].astype(np.int32)
                if ahead.size:
                    if self.copy_stream is not self.stream:
                        self.copy_stream.wait_stream(self.stream)
                    kv_stage_in(self.layout, self.staging_host, self.staging, ahead, self.copy_stream)
                    # later scatters read these slots as resident: they wait for the copies
                    self.stream.wait_stream(self.copy_stream)
                    self.resident[ahead] = True
                    st.staged_bytes += int(ahead.size) * slot_bytes
            e = self._ev(timers, "store")
            kv_store_gather(self.layout, self.staging_ptr, self.layers, self.bt, w.bt_stride, R, self.d_store, ns,
                            self.stream)
            if self.staged_mode and ns:
                # retain the stored chunks in host memory too; their HBM copy is current
                kv_stage_out(self.layout, self.staging, self.staging_host, np.sort(store[:, 0]), self.stream)
                self.resident[store[:, 0]] = True
            self._ev_end(e)
        if ns:
            self.index.insert(skeys, store[:, 0].copy(), self.lookup_stream)
        used = set(int(x) for x in store[:, 0])
        self.free = [s for s in self.free if s not in used]
        self.last_store_keys, self.last_store_slots = skeys, store[:, 0].copy()
        self.last_retrieve, self.last_ordinary, self.last_store = retr, ordn, store
        self.last_decisions = dec
        if evict_stored and ns:
            self.evict_last()
        return st

    def _validate_on_device(self, n_retr: int, n_store: int) -> None:
        """Debug check of the uploaded job lists on this path's stream
        (kv_validate_jobs_device): raises before any copy of the pass is
        launched if a list names an out-of-range id or two jobs of one launch
        write the same block or slot."""
        w = self.batch
        if self._val_marks is None:
            self._val_marks = torch.empty(2 + max(self.w.num_blocks, self.w.num_slots), dtype=torch.int32,
                                          device=self.dev)
            self._val_status = torch.empty(2, dtype=torch.int32, device=self.dev)
        kv_validate_jobs_device(self.layout, self.bt, w.bt_stride, w.num_reqs, self.d_retr, n_retr, False,
                                self._val_marks, self._val_status[0:1], self.stream)
        kv_validate_jobs_device(self.layout, self.bt, w.bt_stride, w.num_reqs, self.d_store, n_store, True,
                                self._val_marks, self._val_status[1:2], self.stream)
        self.stream.synchronize()
        got = [int(x) for x in self._val_status.cpu()]
        assert got == [KV_OK, KV_OK], f"device job check: retrieve {got[0]}, store {got[1]}"

    def tune_retrieve(self, reps: int = 5) -> Dict[str, float]:
        """Choose, for this path's paged pool, between the planned retrieve and
        the four-job-window retrieve (KV_RETRIEVE_QUAD) by timing both on the
        resident jobs of the last pass: the faster (median of ``reps``
        interleaved launches) is used for that plan from then on.  The
        retrieve is idempotent, so the extra launches leave the pool as the
        pass left it.  Returns the median times in ms by variant name; empty
        when the last pass had no resident retrieve jobs, the plan was the
        streaming retrieve (no staged chunk read twice), or the staged chunks
        are read from host memory in place (zero-copy: every window quarter
        would read its segment over the host link, 5-7x slower)."""
        self.stream.synchronize()
        self.lookup_stream.synchronize()
        n = self._last_nres
        if n == 0 or (self.staging_host is not None and not self.staged_mode):
            return {}
        w = self.batch
        jobs = self.h_retr.numpy()[:n]
        planned = kv_retrieve_plan(self.layout, jobs)
        if planned == KV_RETRIEVE_STREAM:
            return {}
        kinds = [planned, KV_RETRIEVE_QUAD]
        ms: Dict[int, List[float]] = {k: [] for k in kinds}
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for _ in range(reps):
            for k in kinds:
                a.record(self.stream)
                kv_retrieve_scatter_as(k, self.layout, self.staging_ptr, self.layers, self.bt, w.bt_stride,
                                       w.num_reqs, self.d_retr, n, self.stream)
                b.record(self.stream)
                b.synchronize()
                ms[k].append(a.elapsed_time(b))
        med = {k: float(np.median(v)) for k, v in ms.items()}
        self.retrieve_choice[planned] = min(kinds, key=lambda k: med[k])
        return {RETRIEVE_KIND_NAMES[k]: round(v, 4) for k, v in med.items()}

    def _ev(self, timers, name, stream=None):
        if timers is None:
            return None
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream if stream is not None else self.stream)
        timers.setdefault(name, []).append((a, b))
        return b

    def _ev_end(self, b, stream=None) -> None:
        if b is not None:
            b.record(stream if stream is not None else self.stream)

    def evict_last(self) -> None:
        """Erase the keys stored by the last pass and free their slots."""
        if self.last_store_keys.size:
            self.index.erase(self.last_store_keys, self.lookup_stream)
            self.free = sorted(self.free + [int(s) for s in self.last_store_slots])
            self.last_store_keys = np.zeros(0, np.uint64)
            self.last_store_slots = np.zeros(0, np.int32)

