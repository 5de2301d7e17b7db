"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times.

Every configuration:
  * hash, lookup and the job lists are compared in full with the oracle;
  * copies are checked on sampled segments: for a sampled paged block the
    oracle says (one by one) which staged segment, if any, lands there, and
    the expected bytes are recomputed from the input generator's formula; the
    same for sampled staging segments written by the store gather.  Samples
    cover every layer, both planes, the first and last jobs, and blocks that
    no job touches (which must keep their original bytes);
  * complete comparison, one layer at a time: for a layer the oracle's
    one-layer walks rebuild the expected paged tensor and the expected
    staging contents from the input formula and the job lists, and every
    byte of the GPU's layer (written blocks, untouched blocks) and of every
    staging slot's part for that layer (stored, read and untouched slots) is
    compared, with only one layer's buffers per worker held on the host
    (buffers of 20-170 GiB cannot be held twice).  Every layer for one
    configuration of each workload family (EVERY_BYTE; all of them with
    TEMPOKV_EVERY_BYTE_ALL=1, about 1.7 TiB and six and a half minutes), the first and the
    last layer for the others."""
import concurrent.futures as cf
import ctypes
import os
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2609_35065_amd as kv
import workloads as W
from oracle.pipeline import OraclePath
from paper_2609_35065_amd.pipeline import StagingPath

pytestmark = pytest.mark.gpu

STG_TAG, POOL_TAG = 1, 1000


def _seg_view(w, layer_tensor, kv, blk):
    seg = w.shape.seg_bytes
    kvs, bs = w.strides()
    off = kv * kvs + blk * bs
    return layer_tensor[off:off + seg], off


def check_full_size(name, n_samples=600, seed=0, lower_tier="zero-copy", force_kind=None, layers=None):
    """layers: None (samples only), "edges" (also the first and the last layer
    in full) or "all" (also every layer in full)."""
    w = W.make(name)
    print(f"[fullsize] {name}: {w.num_reqs} reqs, pool {w.pool_bytes() / 2**30:.1f} GiB, "
          f"staging {w.staged_bytes() / 2**30:.1f} GiB, lower tier {lower_tier}, retrieve {force_kind}", flush=True)
    g = StagingPath(w, lower_tier=lower_tier)
    if force_kind is not None:
        g.retrieve_choice = {k: force_kind for k in (kv.KV_RETRIEVE_UNIT, kv.KV_RETRIEVE_PAIR, kv.KV_RETRIEVE_STREAM)}
    g.fill(STG_TAG, POOL_TAG, w.seed)
    g.prestage()
    o = OraclePath(w, with_kv=False)
    o.prestage()
    sg = g.run_pass(validate=True)
    so = o.run_pass()
    torch.cuda.synchronize()
    if force_kind is not None:
        assert g.retrieve_kind == force_kind
    nblk, nch, R = int(g.blk_off_h[-1]), int(g.chunk_off_h[-1]), w.num_reqs
    assert np.array_equal(g.h_block_hash.numpy()[:nblk].view(np.uint64), so["block_hash"])
    assert np.array_equal(g.h_chunk_slot.numpy()[:nch], so["chunk_slot"])
    assert np.array_equal(g.h_hit.numpy()[:R], so["hit"])
    assert np.array_equal(g.last_retrieve, so["retrieve"])
    assert np.array_equal(g.last_store, so["store"])
    # the hit counts follow from the workload's construction
    C = w.shape.chunk_tokens
    resident = set(p for p, _ in w.prestage_chunks)
    exp_hit = np.array([w.prefix_tokens[r] // C if w.prefix_id[r] in resident else 0 for r in range(R)])
    assert np.array_equal(so["hit"], exp_hit)

    rng = np.random.default_rng(seed)
    L, seg = w.shape.num_layers, w.shape.seg_bytes
    retr, store = so["retrieve"], so["store"]
    # --- scatter: sampled destination blocks, touched and untouched
    nseg = C // w.shape.block_size
    touched = np.unique(np.concatenate([w.block_tables[q[1], q[2] * nseg:(q[2] + 1) * nseg] for q in retr])) \
        if len(retr) else np.zeros(0, np.int32)
    picks = []
    if len(retr):
        for q in (retr[0], retr[-1]):
            for i in range(nseg):
                picks.append((int(rng.integers(0, L)), int(rng.integers(0, 2)),
                              int(w.block_tables[q[1], q[2] * nseg + i])))
        for b in rng.choice(touched, min(n_samples, touched.size), replace=False):
            picks.append((int(rng.integers(0, L)), int(rng.integers(0, 2)), int(b)))
    for b in rng.integers(0, w.num_blocks, n_samples // 4):
        picks.append((int(rng.integers(0, L)), int(rng.integers(0, 2)), int(b)))
    n_touched = 0
    for l, kvp, blk in picks:
        got, off = _seg_view(w, g.layers[l], kvp, blk)
        got = got.cpu().numpy()
        src = oracle.scatter_source(o.layout, w.block_tables, retr, l, kvp, blk)
        if src is None:
            exp = W.kv_bytes_np(POOL_TAG + l, w.seed, off, seg)
        else:
            n_touched += 1
            exp = W.kv_bytes_np(STG_TAG, w.seed, src, seg)
        assert np.array_equal(got, exp), (name, "scatter", l, kvp, blk)
    if len(retr):
        assert n_touched > 0
    # padded block strides: the bytes between segments keep their original contents
    if w.block_pad:
        for blk in list(touched[:200]) + [int(b) for b in rng.integers(0, w.num_blocks, 50)]:
            l, kvp = int(rng.integers(0, L)), int(rng.integers(0, 2))
            _, off = _seg_view(w, g.layers[l], kvp, int(blk))
            got = g.layers[l][off + seg:off + seg + w.block_pad].cpu().numpy()
            assert np.array_equal(got, W.kv_bytes_np(POOL_TAG + l, w.seed, off + seg, w.block_pad)), (name, "pad")
    # --- gather: sampled staging segments of the stored slots
    if len(store):
        slots = [int(store[0, 0]), int(store[-1, 0])] + [int(s) for s in rng.choice(store[:, 0], min(40, len(store)))]
        stg = g.staging_view()
        for s in slots:
            for _ in range(8):
                l, kvp, i = int(rng.integers(0, L)), int(rng.integers(0, 2)), int(rng.integers(0, nseg))
                so_off = s * w.shape.slot_bytes + ((l * 2 + kvp) * nseg + i) * seg
                got = stg[so_off:so_off + seg].cpu().numpy()
                blk = oracle.gather_source(o.layout, w.block_tables, store, s, i)
                assert blk is not None
                _, poff = _seg_view(w, g.layers[l], kvp, blk)
                exp = W.kv_bytes_np(POOL_TAG + l, w.seed, poff, seg)
                assert np.array_equal(got, exp), (name, "gather", s, l, kvp, i)
    if layers is not None:
        # every byte of the chosen layers: pool and every staging slot
        t0 = time.perf_counter()
        sel = range(L) if layers == "all" else sorted({0, L - 1})
        n = _check_layers(w, g, o, retr, store, sel, 8 if layers == "all" else 2)
        print(f"[fullsize] {name}: {len(sel)} of {L} layers compared in full ({n / 2**30:.1f} GiB, "
              f"{time.perf_counter() - t0:.0f} s)", flush=True)
    del g
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return sg, so


FULL = ["l32-64x4096", "l32-lognormal-p25", "l32-lognormal-p50", "l32-lognormal-p75", "l80-32x8192",
        "l32-1024x1024-cap100-hbm", "l32-1024x1024-cap50-hbm", "l32-1024x1024-cap25-hbm",
        "l32-1024x1024-cap25-host", "l32-1x65536", "l48-1x65536", "l48-64x4096", "l32-64x4096-block_first",
        "l32-64x4096-pad4096"]


HOST_ZERO_COPY = ["l32-1024x1024-cap50-host", "l32-1024x1024-cap100-host", "l32-1x65536-host"]
# every byte of every layer: one configuration of each workload family in every run
EVERY_BYTE = ["l32-64x4096", "l48-64x4096", "l80-32x8192", "l32-lognormal-p50", "l32-1024x1024-cap25-hbm",
              "l32-1x65536", "l48-1x65536", "l32-1x65536-host"]
if os.environ.get("TEMPOKV_EVERY_BYTE_ALL"):
    EVERY_BYTE = FULL + HOST_ZERO_COPY


def _layers(name):
    return "all" if name in EVERY_BYTE else "edges"


@pytest.mark.parametrize("name", FULL)
def test_full_size(name):
    check_full_size(name, layers=_layers(name))


@pytest.mark.parametrize("name", ["l32-1x65536-host", "l32-1024x1024-cap100-host"])
def test_full_size_sampled_pipelined_from_host(name):
    # the staged chunks start in pinned host memory and reach HBM by DMA,
    # batch by batch, before each batch's scatter
    sg, _ = check_full_size(name, lower_tier="pipelined")
    assert sg.staged_bytes > 0


@pytest.mark.parametrize("name", ["l32-64x4096", "l48-64x4096", "l32-lognormal-p75", "l32-1024x1024-cap25-hbm",
                                  "l32-64x4096-pad4096"])
def test_full_size_quad_retrieve(name):
    # the four-job-window retrieve, which tune_retrieve may choose for a pool (on the 32-layer batch it
    # usually does, so there it is compared in full)
    check_full_size(name, force_kind=kv.KV_RETRIEVE_QUAD, layers="all" if name == "l32-64x4096" or os.environ.get("TEMPOKV_EVERY_BYTE_ALL") else "edges")


# ---------------------------------------------------------------------------
# complete comparison, streamed one layer at a time
# ---------------------------------------------------------------------------

_libc = ctypes.CDLL(None)
_libc.memcmp.restype = ctypes.c_int
_libc.memcmp.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t]


def _same(got: np.ndarray, exp: np.ndarray) -> bool:
    """Byte equality of two contiguous uint8 arrays (memcmp: no temporary the
    size of the buffers, and the GIL is released while it runs)."""
    assert got.dtype == exp.dtype == np.uint8 and got.flags.c_contiguous and exp.flags.c_contiguous
    return got.size == exp.size and _libc.memcmp(got.ctypes.data, exp.ctypes.data, got.size) == 0


def _first_difference(got: np.ndarray, exp: np.ndarray) -> int:
    return int(np.flatnonzero(got != exp)[0])


def _layer_check(w, g, o, retr, store, l, bufs):
    """Compare layer l of the pool and of every staging slot with the oracle's
    one-layer walks over the formula's bytes.  Returns the bytes compared."""
    L, S = w.shape.num_layers, w.num_slots
    part = oracle.layer_part_bytes(o.layout)
    exp_pool, exp_stg, got_pool, got_stg = bufs
    # expected: the pool formula with the retrieve's bytes scattered in, then the store's bytes gathered out
    W.kv_words_np(POOL_TAG + l, w.seed, 0, exp_pool.size // 4, out=exp_pool.view(np.uint32))
    for s in range(S):
        W.kv_words_np(STG_TAG, w.seed, (s * w.shape.slot_bytes + l * part) // 4, part // 4,
                      out=exp_stg[s * part:(s + 1) * part].view(np.uint32))
    oracle.retrieve_scatter_layer(o.layout, exp_stg, exp_pool, w.block_tables, retr)
    oracle.store_gather_layer(o.layout, exp_stg, exp_pool, w.block_tables, store)
    got_pool.copy_(g.layers[l])
    got_stg.copy_(g.staging_view().view(S, L, part)[:, l, :].reshape(-1))
    gp, gs = got_pool.numpy(), got_stg.numpy()
    assert _same(gp, exp_pool), f"layer {l}: paged tensor differs at byte {_first_difference(gp, exp_pool)}"
    assert _same(gs, exp_stg), f"layer {l}: staging differs at byte {_first_difference(gs, exp_stg)}"
    return exp_pool.size + exp_stg.size


def _check_layers(w, g, o, retr, store, layers, workers):
    """_layer_check over `layers`, `workers` layers at a time; returns the bytes compared."""
    L, S = w.shape.num_layers, w.num_slots
    part = oracle.layer_part_bytes(o.layout)
    nw = max(1, min(workers, (os.cpu_count() or 4), len(layers)))
    pools = [(np.empty(w.layer_bytes(), np.uint8), np.empty(S * part, np.uint8),
              torch.from_numpy(np.empty(w.layer_bytes(), np.uint8)),
              torch.from_numpy(np.empty(S * part, np.uint8))) for _ in range(nw)]
    free = list(range(nw))
    total = 0

    def one(l, k):
        with torch.cuda.stream(torch.cuda.Stream()):
            n = _layer_check(w, g, o, retr, store, l, pools[k])
            torch.cuda.current_stream().synchronize()
        return n

    with cf.ThreadPoolExecutor(nw) as ex:
        pending = {}
        for l in layers:
            if not free:
                done, _ = cf.wait(pending, return_when=cf.FIRST_COMPLETED)
                for f in done:
                    total += f.result()
                    free.append(pending.pop(f))
            k = free.pop()
            pending[ex.submit(one, l, k)] = k
        for f in cf.as_completed(pending):
            total += f.result()
    return total


@pytest.mark.parametrize("name", HOST_ZERO_COPY)
def test_full_size_zero_copy_from_host(name):
    # host-staged workloads in the bench's default mode: the scatter reads the pinned buffer in place
    check_full_size(name, lower_tier="zero-copy", layers=_layers(name))
