"""GPU parity of passes whose claims do not all commit (Section 3.2).

A tight protected-capacity budget and a mix of requests whose retrieval is
requested now and requests only eligible (or not) by their TTU/TTR estimates
produce every outcome: KV_COMMIT (protected route), KV_ORDINARY (ordinary
route, read in place), KV_BLOCKED and KV_DEFER (no jobs).  Every pass is
compared with the oracle's: decisions, both retrieve lists, store jobs, and
every byte of the staging buffer (or lower tier) and the paged pool.  In the
staged lower-tier modes the ordinary route reads the lower tier in place and
stages nothing, while committed claims whose retrieval is not requested yet
are staged into HBM ahead of use."""
import numpy as np
import pytest
import torch

import paper_2609_35065_amd as kv
import workloads as W
from oracle.pipeline import OraclePath
from paper_2609_35065_amd.pipeline import ClaimInputs, StagingPath

pytestmark = pytest.mark.gpu

STG_TAG, POOL_TAG = 1, 1000


def _claims(rng, R, slot_bytes, slots_in_budget):
    requested = rng.random(R) < 0.55
    ttu = rng.choice([-1.0, 0.0, 0.5, 3.0], R)
    ttr = rng.choice([0.0, 1.0, 2.0], R)
    return ClaimInputs(requested, ttu, ttr, slots_in_budget * slot_bytes)


@pytest.mark.parametrize("mode", ["hbm", "zero-copy", "pipelined", "serialized"])
@pytest.mark.parametrize("seed", [5, 6])
def test_commitment_routes_match_oracle(mode, seed):
    shape = W.KVShape(2, 8, 128, 2, 16, 64)
    w = W.small_random(seed, shape, num_reqs=14, max_len=520, n_prefixes=3)
    if mode != "hbm":
        w.staging_in_host = True
    print(f"[claims] mode {mode}, seed {seed}: {w.num_reqs} requests, {w.num_slots} slots", flush=True)
    g = StagingPath(w, lower_tier="zero-copy" if mode == "hbm" else mode, slots_per_batch=2)
    g.fill(STG_TAG, POOL_TAG, w.seed)
    g.prestage()
    o = OraclePath(w, kv_seed=w.seed, staging_tag=STG_TAG, pool_tag_base=POOL_TAG)
    o.prestage()
    rng = np.random.default_rng(seed)
    seen = set()
    for p in range(6):
        cl = _claims(rng, w.num_reqs, w.shape.slot_bytes, int(rng.integers(0, 5)))
        sg, so = g.run_pass(validate=True, claims=cl), o.run_pass(claims=cl)
        torch.cuda.synchronize()
        assert np.array_equal(g.last_decisions, so["decisions"]), p
        assert np.array_equal(g.last_retrieve, so["retrieve"]), p
        assert np.array_equal(g.last_ordinary, so["ordinary"]), p
        assert np.array_equal(g.last_store, so["store"]), p
        assert sg.num_ordinary == len(so["ordinary"])
        assert np.array_equal(g.staging_view().cpu().numpy(), o.staging), p
        for l in range(len(g.layers)):
            assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l]), (p, l)
        if g.staged_mode:
            hb = g.staging.cpu().numpy().reshape(w.num_slots, -1)
            hh = g.staging_host.numpy().reshape(w.num_slots, -1)
            assert np.array_equal(hb[g.resident], hh[g.resident]), "a resident HBM slot differs from host"
        seen |= set(int(d) for d in so["decisions"])
        g.drop_fast_tier()
    assert {kv.KV_COMMIT, kv.KV_ORDINARY, kv.KV_BLOCKED, kv.KV_DEFER} <= seen, seen


def test_default_claims_all_commit_and_match_previous_jobs():
    # with the default inputs (everything requested now, the whole staging buffer as budget) every claim
    # commits and the jobs are those of kv_build_jobs
    w = W.small_random(9, W.KVShape(2, 2, 64, 2, 16, 64), num_reqs=10, max_len=400)
    g = StagingPath(w)
    g.fill(STG_TAG, POOL_TAG, w.seed)
    g.prestage()
    o = OraclePath(w, kv_seed=w.seed, staging_tag=STG_TAG, pool_tag_base=POOL_TAG)
    o.prestage()
    for _ in range(2):
        sg, so = g.run_pass(validate=True), o.run_pass()
        torch.cuda.synchronize()
        assert np.all(g.last_decisions == kv.KV_COMMIT) and sg.num_ordinary == 0
        assert np.array_equal(g.last_retrieve, so["retrieve"]) and np.array_equal(g.last_store, so["store"])
        for l in range(len(g.layers)):
            assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l])


def test_random_shapes_modes_and_claims():
    # TEMPOKV_CLAIM_SHAPES random shapes (40 by default) drawn from TEMPOKV_CLAIM_SEED (777 by default), each
    # in one of the four modes with a random batch, pipeline batch size, overlapped or serial passes, paged
    # layout and padding; three passes with random commitment inputs and eviction, each compared in full.
    import os
    n = int(os.environ.get("TEMPOKV_CLAIM_SHAPES", "40"))
    seed = int(os.environ.get("TEMPOKV_CLAIM_SEED", "777"))
    modes = ["hbm", "zero-copy", "pipelined", "serialized"]
    seen = set()
    for k, shape in enumerate(W.random_shapes(seed, n)):
        rng = np.random.default_rng(seed * 11 + k)
        mode = modes[k % 4]
        w = W.small_random(seed * 13 + k, shape, num_reqs=int(rng.integers(2, 16)),
                           max_len=int(rng.integers(1, 5)) * shape.chunk_tokens + int(rng.integers(0, 40)),
                           n_prefixes=int(rng.integers(1, 4)), paged_layout=["kv_first", "block_first"][k % 2],
                           block_pad=[0, 16, 4096][k % 3])
        if mode != "hbm":
            w.staging_in_host = True
        g = StagingPath(w, lower_tier="zero-copy" if mode == "hbm" else mode,
                        slots_per_batch=int(rng.integers(1, 5)), overlap=bool(k % 3 == 0))
        g.fill(STG_TAG, POOL_TAG, w.seed)
        g.prestage()
        o = OraclePath(w, kv_seed=w.seed, staging_tag=STG_TAG, pool_tag_base=POOL_TAG)
        o.prestage()
        for p in range(3):
            R = w.num_reqs
            cl = ClaimInputs(rng.random(R) < 0.6, rng.choice([-1.0, 0.0, 0.5, 3.0], R),
                             rng.choice([0.0, 1.0, 2.0], R), int(rng.integers(0, 6)) * w.shape.slot_bytes)
            evict = bool(rng.random() < 0.5)
            g.run_pass(validate=True, claims=cl, evict_stored=evict)
            so = o.run_pass(claims=cl, evict_stored=evict)
            torch.cuda.synchronize()
            tag = (k, mode, p, shape)
            assert np.array_equal(g.last_decisions, so["decisions"]), tag
            assert np.array_equal(g.last_retrieve, so["retrieve"]), tag
            assert np.array_equal(g.last_ordinary, so["ordinary"]), tag
            assert np.array_equal(g.last_store, so["store"]), tag
            assert np.array_equal(g.staging_view().cpu().numpy(), o.staging), tag
            for l in range(len(g.layers)):
                assert np.array_equal(g.layers[l].cpu().numpy(), o.layers[l]), tag + (l,)
            if g.staged_mode:
                hb = g.staging.cpu().numpy().reshape(w.num_slots, -1)
                hh = g.staging_host.numpy().reshape(w.num_slots, -1)
                assert np.array_equal(hb[g.resident], hh[g.resident]), tag
            seen |= set(int(d) for d in so["decisions"])
            if rng.random() < 0.5:
                g.drop_fast_tier()
        del g, o
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        if k % 100 == 99:
            print(f"[claims] {k + 1}/{n} shapes ok", flush=True)
    if n >= 40:
        assert {kv.KV_COMMIT, kv.KV_ORDINARY, kv.KV_BLOCKED, kv.KV_DEFER} <= seen, seen
