"""The library's controller simulation (kv_sim_run, C++) against the oracle
(oracle/controller.py), event by event: identical traces (time, kind, id),
first-token and end times, reserved byte-time and counters, on random
scenarios for every policy -- shared prefixes, tight budgets (blocking and
the ordinary path), small fast tiers (eviction) and queueing."""
import math

import numpy as np
import pytest

import paper_2609_35065_amd as kv
from oracle import controller as ct

GiB, MiB = 1 << 30, 1 << 20


def scenario(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 25))
    n_docs = int(rng.integers(1, 8))
    chunk = int(rng.choice([8, 32, 64])) * MiB
    doc_chunks = [int(rng.integers(1, 60)) for _ in range(n_docs)]
    doc_base = np.concatenate([[0], np.cumsum(doc_chunks)]).astype(int)
    obj = [float(chunk)] * int(doc_base[-1])
    man, unc, out, arr = [], [], [], []
    t = 0.0
    for i in range(n):
        d = int(rng.integers(0, n_docs))
        k = int(rng.integers(0, doc_chunks[d] + 1))
        m = list(range(doc_base[d], doc_base[d] + k))
        if rng.random() < 0.2 and m:
            m = m + [m[0]]                              # duplicate entry: counted once
        man.append(m)
        unc.append(int(rng.integers(0, 5000)))
        out.append(int(rng.integers(1, 200)))
        t += float(rng.choice([0.0, 0.05, 0.1, 0.5, 1.0]))
        arr.append(t)
    total_max = max([len(set(m)) for m in man] + [1]) * chunk
    budget = float(int(rng.choice([0.5, 1.0, 2.0, 8.0]) * total_max))
    cap = float(budget + int(rng.choice([0, 1, 4])) * total_max)
    cfg = dict(budget=budget, capacity=cap, stage_rate=float(rng.choice([2, 11, 40])) * GiB,
               static_rate=11.0 * GiB, gpu_rate=float(rng.choice([25, 50])) * GiB,
               prefill_s=float(rng.choice([5e-5, 1e-4])), decode_s=float(rng.choice([0.01, 0.02])),
               max_active=int(rng.integers(1, 5)), tick=0.05, queue_k=int(rng.integers(1, 5)))
    return cfg, obj, arr, man, unc, out


def run_both(cfgd, policy, obj, arr, man, unc, out):
    c = ct.SimConfig(policy=policy, **cfgd)
    ref = ct.simulate(c, obj, arr, man, unc, out)
    k = kv.KvSimConfig(cfgd["budget"], cfgd["capacity"], cfgd["stage_rate"], cfgd["static_rate"], cfgd["gpu_rate"],
                       cfgd["prefill_s"], cfgd["decode_s"], cfgd["tick"], cfgd["max_active"], policy,
                       cfgd["queue_k"], 0)
    res, ft, dn, tr = kv.kv_sim_run(k, obj, arr, man, unc, out, trace=True)
    return ref, res, ft, dn, tr


@pytest.mark.parametrize("policy", range(5))
@pytest.mark.parametrize("seed", range(40))
def test_event_by_event_parity(seed, policy):
    cfgd, obj, arr, man, unc, out = scenario(seed)
    ref, res, ft, dn, tr = run_both(cfgd, policy, obj, arr, man, unc, out)
    assert tr == ref["trace"]
    assert np.array_equal(ft, np.array(ref["first_token"])) or np.allclose(ft, ref["first_token"], rtol=0, atol=0)
    assert np.array_equal(dn, np.array(ref["done"]))
    assert res.area_byte_s == ref["area"]
    assert res.cost_gib_s_per_request == ref["C"]
    assert res.end_s == ref["end"]
    assert res.p_max_bytes == ref["P_max"]
    assert (res.committed, res.blocked, res.ordinary) == (ref["committed"], ref["blocked"], ref["ordinary"])


def test_invalid_arguments():
    good = kv.KvSimConfig(GiB, 2 * GiB, GiB, GiB, GiB, 1e-4, 1e-2, 0.05, 4, kv.KV_POLICY_TEMPO, 4, 0)
    for field, bad in [("budget_bytes", -1.0), ("capacity_bytes", 0.5 * GiB), ("stage_rate", 0.0),
                       ("tick_s", 0.0), ("max_active", 0), ("policy", 7), ("reserved", 1)]:
        c = kv.KvSimConfig.from_buffer_copy(good)
        setattr(c, field, bad)
        with pytest.raises(kv.KvError):
            kv.kv_sim_run(c, [float(MiB)], [0.0], [[0]], [1], [1])
    with pytest.raises(kv.KvError):
        kv.kv_sim_run(good, [float(MiB)], [0.0], [[3]], [1], [1])        # object out of range
    with pytest.raises(kv.KvError):
        kv.kv_sim_run(good, [1.5], [0.0], [[0]], [1], [1])               # non-integer bytes
    res, ft, dn, _ = kv.kv_sim_run(good, [], [], [], [], [])
    assert res.events == 0 or res.events >= 0


@pytest.mark.parametrize("ratio", [0.5, 0.75, 1.0])
@pytest.mark.parametrize("policy,k", [(0, 0), (1, 0), (2, 1), (2, 4), (3, 0), (4, 0)])
def test_policy_scenario_parity(ratio, policy, k):
    import workloads as W
    sc = W.policy_scenario(ratio)
    cfgd = dict(budget=50.0 * GiB, capacity=100.0 * GiB, stage_rate=11.0 * GiB, static_rate=11.0 * GiB,
                gpu_rate=25.0 * GiB, prefill_s=1e-4, decode_s=0.03, max_active=4, tick=0.05, queue_k=k)
    ref, res, ft, dn, tr = run_both(cfgd, policy, sc.obj_bytes, sc.arrival, sc.manifests, sc.uncached, sc.out_tokens)
    assert tr == ref["trace"]
    assert res.area_byte_s == ref["area"] and np.array_equal(dn, np.array(ref["done"]))


def test_policy_scenario_shape():
    import workloads as W
    sc = W.policy_scenario(1.0)
    assert len(sc.arrival) == 12 and sc.arrival[1] - sc.arrival[0] == 0.5
    toks = [len(m) * 256 + u - 32 for m, u in zip(sc.manifests, sc.uncached)]
    assert 16078 <= min(toks) and max(toks) <= 67744
    assert all(b == 32 * MiB for b in sc.obj_bytes)
    half = W.policy_scenario(0.5)
    assert sum(len(m) for m in half.manifests) < sum(len(m) for m in sc.manifests)
