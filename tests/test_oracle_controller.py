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
    # six claims on the same eight objects, all reported at t=0 and committed together
    obj, arr, man, unc, out = small_workload(n=6, chunks=8, share=True, gap=0.0)
    r = ct.simulate(cfg(policy=ct.IMMEDIATE), obj, arr, man, unc, out)
    assert r["committed"] == 6 and len(set(t for t, _ in events(r, "commit"))) == 1
    assert r["P_max"] == 8 * 32 * MiB
    # staging of a shared object is coalesced: each object is read from the device once
    assert sorted(o for _, o in events(r, "ready")) == list(range(8))
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
    c = cfg(policy=ct.DEMAND, budget=1 * GiB)
    r = ct.simulate(c, obj, arr, man, unc, out)
    assert r["ordinary"] == 2 and r["committed"] == 0
    # the ordinary path still reads its objects through the staging device before the transfer
    B = 40 * 32 * MiB
    assert math.isclose(r["ttft"][0], B / c.stage_rate + B / c.gpu_rate + 500 * c.prefill_s, rel_tol=1e-12)



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


def test_bytes_already_protected_need_no_free_capacity():
    # the budget holds exactly one footprint; a second claim on the same objects reserves nothing new and
    # commits at once instead of waiting for the first to release
    obj, arr, man, unc, out = small_workload(n=2, chunks=8, share=True, gap=0.0)
    r = ct.simulate(cfg(policy=ct.IMMEDIATE, budget=8 * 32 * MiB), obj, arr, man, unc, out)
    commits = dict((i, t) for t, i in events(r, "commit"))
    assert commits == {0: 0.0, 1: 0.0} and r["blocked"] == 0


def test_queue_k_commits_only_within_the_first_k_waiting():
    obj, arr, man, unc, out = small_workload(n=10, gap=0.1)
    for k in (1, 2, 3):
        r = ct.simulate(cfg(policy=ct.QUEUE_K, queue_k=k, max_active=2), obj, arr, man, unc, out)
        arrive = dict((i, t) for t, i in events(r, "arrive"))
        admit = dict((i, t) for t, i in events(r, "admit"))
        for tc, i in events(r, "commit"):
            if admit[i] <= tc:
                continue                       # committed once requested
            # FCFS position among requests that have arrived and are not admitted at tc
            pos = sum(1 for j in range(i) if arrive[j] <= tc and admit[j] > tc)
            assert pos < k, (k, i, pos)


def test_cost_is_per_request():
    # two identical requests far apart cost what one costs (C is the reserved byte-time per request)
    obj1, arr1, man1, unc1, out1 = small_workload(n=1, chunks=4)
    one = ct.simulate(cfg(policy=ct.IMMEDIATE), obj1, arr1, man1, unc1, out1)
    obj, man = obj1 * 2, [man1[0], [o + 4 for o in man1[0]]]
    two = ct.simulate(cfg(policy=ct.IMMEDIATE), obj, [0.0, 100.0], man, unc1 * 2, out1 * 2)
    assert math.isclose(two["C"], one["C"], rel_tol=1e-12)
    assert math.isclose(two["area"], 2 * one["area"], rel_tol=1e-12)


def test_state_aware_ttr_commits_behind_a_busy_device_earlier():
    # one slot: request 0 runs ~1 s; request 1 (4 GiB) commits when its laxity reaches zero and keeps the
    # staging device busy until request 0 ends; request 2 (2 GiB) follows request 1, whose service (0.11 s) is
    # shorter than request 2's staging (0.18 s).  With the state-aware TTR request 2's reads wait behind request
    # 1's, so its laxity is already negative when request 1 commits; the static TTR ignores the queue and
    # commits it about TTR1 + svc1 - TTR2 = 0.29 s later.
    obj = [32 * MiB] * (1 + 128 + 64)
    man = [[0], list(range(1, 129)), list(range(129, 193))]
    arr, unc, out = [0.0, 0.0, 0.0], [100, 100, 100], [50, 1, 1]
    c = dict(max_active=1, decode_s=0.02)
    st = ct.simulate(cfg(policy=ct.TEMPO_STATIC, **c), obj, arr, man, unc, out)
    sa = ct.simulate(cfg(policy=ct.TEMPO, **c), obj, arr, man, unc, out)
    c_st = dict((i, t) for t, i in events(st, "commit"))
    c_sa = dict((i, t) for t, i in events(sa, "commit"))
    assert c_sa[2] <= c_sa[1] + 0.05 + 1e-9           # at request 1's commit or the next control point
    assert c_st[2] - c_sa[2] > 0.2
