"""Pins for the controller oracle: the commitment rules of Section 3.2 and the
cost metric of Section 5, checked on scenarios whose outcome follows from the
text alone."""
import math

import numpy as np
import pytest

from oracle import controller as ct

GiB = 1 << 30
MiB = 1 << 20


def cfg(**kw):
    d = dict(budget=50 * GiB, capacity=100 * GiB, stage_rate=11 * GiB, static_rate=11 * GiB, gpu_rate=50 * GiB,
             prefill_s=1e-4, decode_s=0.02, max_active=4, tick=0.05, policy=ct.TEMPO)
    d.update(kw)
    return ct.SimConfig(**d)


def events(res, kind):
    return [(t, a) for t, k, a in res["trace"] if k == kind]


def small_workload(n=6, chunks=8, share=False, gap=0.5):
    obj, man = [], []
    for i in range(n):
        if share and i:
            man.append(list(man[0]))
            continue
        ids = list(range(len(obj), len(obj) + chunks))
        obj += [32 * MiB] * chunks
        man.append(ids)
    arr = [gap * i for i in range(n)]
    return obj, arr, man, [500] * n, [64] * n


def test_single_request_immediate_closed_form():
    obj, arr, man, unc, out = small_workload(n=1, chunks=4)
    c = cfg(policy=ct.IMMEDIATE)
    r = ct.simulate(c, obj, arr, man, unc, out)
    B = 4 * 32 * MiB
    ready = B / c.stage_rate                    # staged back to back from t=0
    t_end = ready + B / c.gpu_rate              # transfer starts once stage-ready, then protection ends
    assert math.isclose(r["area"], B * t_end, rel_tol=1e-12)
    assert math.isclose(r["C"], B * t_end / GiB, rel_tol=1e-12)
    assert math.isclose(r["ttft"][0], t_end + 500 * c.prefill_s, rel_tol=1e-12)


def test_immediate_commits_at_report_and_demand_at_admission():
    # two slots and arrivals every 0.1 s: requests queue, so the policies differ
    obj, arr, man, unc, out = small_workload(n=8, gap=0.1)
    imm = ct.simulate(cfg(policy=ct.IMMEDIATE, max_active=2), obj, arr, man, unc, out)
    for t, i in events(imm, "commit"):
        assert t == arr[i]
    dem = ct.simulate(cfg(policy=ct.DEMAND, max_active=2), obj, arr, man, unc, out)
    admit = dict((i, t) for t, i in events(dem, "admit"))
    for t, i in events(dem, "commit"):
        assert t == admit[i]
    # advance staging hides latency but reserves capacity longer
    assert imm["C"] > dem["C"]
    assert np.mean(imm["ttft"]) <= np.mean(dem["ttft"])


def test_queue_k_commits_when_among_first_k():
    obj, arr, man, unc, out = small_workload(n=10, gap=0.1)
    r = ct.simulate(cfg(policy=ct.QUEUE_K, queue_k=1), obj, arr, man, unc, out)
    commits = dict((i, t) for t, i in events(r, "commit"))
    assert len(commits) == 10
    # request i >= max_active + 1 waits in the queue and commits before its admission
    admit = dict((i, t) for t, i in events(r, "admit"))
    assert any(commits[i] < admit[i] for i in range(5, 10))


def test_reserved_capacity_never_exceeds_budget_and_shared_objects_count_once():
    obj, arr, man, unc, out = small_workload(n=6, chunks=8, share=True)
    r = ct.simulate(cfg(policy=ct.IMMEDIATE), obj, arr, man, unc, out)
    assert r["P_max"] == 8 * 32 * MiB           # six claims on the same eight objects
    obj, arr, man, unc, out = small_workload(n=12, chunks=40)
    for pol in range(5):
        r = ct.simulate(cfg(policy=pol, budget=4 * GiB), obj, arr, man, unc, out)
        assert r["P_max"] <= 4 * GiB


def test_blocked_stays_planned_and_requested_takes_ordinary_path():
    # footprints of 1.25 GiB against a 2 GiB budget: only one claim fits at a time
    obj, arr, man, unc, out = small_workload(n=5, chunks=40, gap=0.0)
    r = ct.simulate(cfg(policy=ct.IMMEDIATE, budget=2 * GiB), obj, arr, man, unc, out)
    assert r["blocked"] >= 1
    assert r["ordinary"] >= 1
    ordinary = set(i for _, i in events(r, "ordinary"))
    committed = set(i for _, i in events(r, "commit"))
    assert not (ordinary & committed)            # exclusive paths
    for i in committed:
        assert r["final_state"][i] == ct.RELEASED     # a commitment is never revoked
    # a footprint larger than the whole budget can never commit
    obj, arr, man, unc, out = small_workload(n=2, chunks=40)
    r = ct.simulate(cfg(policy=ct.DEMAND, budget=1 * GiB), obj, arr, man, unc, out)
    assert r["ordinary"] == 2 and r["committed"] == 0


def test_tempo_commits_at_the_first_control_point_with_nonpositive_laxity():
    # one long request occupies the only slot; the second waits behind it
    obj = [32 * MiB] * 64
    man = [list(range(0, 32)), list(range(32, 64))]
    arr, unc, out = [0.0, 0.1], [100, 100], [400, 10]
    c = cfg(policy=ct.TEMPO, max_active=1, decode_s=0.02)
    r = ct.simulate(c, obj, arr, man, unc, out)
    commits = dict((i, t) for t, i in events(r, "commit"))
    admit = dict((i, t) for t, i in events(r, "admit"))
    # request 1's retrieval starts when request 0 ends; TTR = its 1 GiB at the staging rate
    B = 32 * 32 * MiB
    end0 = r["done"][0]
    ttr = B / c.stage_rate
    tc = commits[1]
    assert tc < admit[1]
    assert end0 - tc <= ttr + 1e-9                      # laxity <= 0 when committed
    assert end0 - (tc - c.tick) > ttr - 1e-9            # still positive one tick earlier
    # committing at the first control point with laxity <= 0 makes readiness
    # just in time or late by less than one control interval: the transfer
    # starts when staging completes, within one tick of admission
    t_x = events(r, "transfer")[-1][0]
    assert math.isclose(t_x, max(admit[1], tc + ttr), rel_tol=1e-12)
    assert 0.0 <= t_x - admit[1] < c.tick


def test_state_aware_ttr_sees_the_queue():
    # two claims committed back to back share the staging device: the second's
    # state-aware TTR includes the first's outstanding reads, the static one does not
    obj = [32 * MiB] * 64
    man = [list(range(0, 32)), list(range(32, 64)), list(range(0, 32))]
    arr, unc, out = [0.0, 0.0, 0.05], [100] * 3, [50] * 3
    st = ct.simulate(cfg(policy=ct.TEMPO_STATIC, max_active=1), obj, arr, man, unc, out)
    sa = ct.simulate(cfg(policy=ct.TEMPO, max_active=1), obj, arr, man, unc, out)
    c_st = dict((i, t) for t, i in events(st, "commit"))
    c_sa = dict((i, t) for t, i in events(sa, "commit"))
    assert c_sa[1] <= c_st[1]
