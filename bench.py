#!/usr/bin/env python3
"""Benchmark of the KV staging hot path on one MI355X.

One step is one pass of the whole path over the batch: prefix hash, lookup,
one device-to-host copy of the lookup result, host job build and commitment
decisions, one host-to-device copy of the jobs, the retrieve scatter, the
store gather, and the index update (the chunks stored in the step are evicted
again at its end, so every step does the same work).  Inputs (tokens, block
tables, staging and pool contents) are resident in HBM before timing starts.
Steps overlap as in a serving loop: the hash and lookup of step i+1 run on a
stream of their own, and its jobs are built on the host, while the copies of
step i are in flight (--serial runs them back to back).  After the warm-up
steps, and outside the timed region, the retrieve variant for this pool is
chosen by timing the planned one against the four-job-window one (--no-tune
keeps the plan).

Prints one JSON line: the whole-step payload rate in GB/s (bytes read plus
bytes written by the scatter and the gather, divided by wall time per step),
per-kernel rates measured with HIP events on the launch stream, the roofline
of the dominant copy kernel against MI355X's 8 TB/s HBM peak, and the CPU
oracle timed on a bounded sample of the same workload shape.

    python bench.py [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "paged-KV scatter/gather GB/s (% of HBM peak); prefix-hash Mtok/s"
HBM_PEAK_GBS = 8000.0
STG_TAG, POOL_TAG = 1, 1000
PROFILES = os.path.join(ROOT, "profiles")


def _src_digest() -> str:
    h = hashlib.sha256()
    for f in ("copy.hip", "internal.h"):
        with open(os.path.join(ROOT, "paper_2609_35065_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _load_traffic(kernel: str, workload: str):
    """HBM bytes per launch measured by rocprofv3 counters, if a summary for
    this kernel and workload exists and was taken from the current source."""
    path = os.path.join(PROFILES, f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    kvs = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.strip().split("=", 1)
            kvs[k.strip()] = v.strip()
    if kvs.get("source_digest") != _src_digest():
        return None
    try:
        return float(kvs["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _cpu_baseline(shape):
    """The CPU oracle on a bounded sample with the benchmark's KV shape:
    8 requests x 4096 tokens, 50% prefix from 2 shared prefixes (64 retrieve
    and 64 store jobs per pass, 8 GiB moved per pass at 32 layers), two passes
    (stored chunks are evicted after each, as in the benchmark), single
    thread."""
    import workloads as W
    from oracle.pipeline import OraclePath
    R, passes = 8, 2
    w = W._assemble("cpu-sample", shape, 2, [4096] * R, [r % 2 for r in range(R)], [2048] * R, 2,
                    prestage=[(p, j) for p in range(2) for j in range(8)], num_slots=16 + 8 * R, pool_factor=1.25)
    o = OraclePath(w, kv_seed=2)
    o.prestage()
    moved = r_moved = s_moved = 0
    laps: dict = {}
    # the oracle is single-threaded; pin the process to one core while it runs
    prev = os.sched_getaffinity(0) if hasattr(os, "sched_getaffinity") else None
    if prev:
        os.sched_setaffinity(0, {min(prev)})
    try:
        t0 = time.perf_counter()
        for _ in range(passes):
            so = o.run_pass(evict_stored=True, timers=laps)
            r_moved += 2 * len(so["retrieve"]) * shape.slot_bytes
            s_moved += 2 * len(so["store"]) * shape.slot_bytes
        dt = time.perf_counter() - t0
    finally:
        if prev:
            os.sched_setaffinity(0, prev)
    moved = r_moved + s_moved
    per_op = {"hash_Mtok/s": round(passes * w.tokens.size / laps["hash"] / 1e6, 3),
              "lookup_and_job_build_ms": round(laps["lookup"] * 1e3 / passes, 3),
              "retrieve_GB/s": round(r_moved / laps["retrieve"] / 1e9, 4),
              "store_GB/s": round(s_moved / laps["store"] / 1e9, 4)}
    return {"value": round(moved / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "per_op": per_op, "host_cpu": _cpu_model(), "host_nproc": os.cpu_count(),
            "sample": (f"{passes} oracle passes (hash, lookup, job build, scatter, gather) over {R} requests x 4096 "
                       f"tokens of the {shape.num_layers}-layer bf16 KV shape, 50% prefix from 2 shared prefixes: "
                       f"{len(so['retrieve'])} retrieve + {len(so['store'])} store jobs per pass, "
                       f"{moved / 2**30:.1f} GiB moved in {dt:.2f} s, single-threaded C")}


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _retrieve_write_bound(path, torch, reps: int = 5):
    """The timed retrieve's writes on their own: the same jobs, variant and
    destination blocks, but every job reading one staged chunk (which stays in
    L2), so HBM sees only the scattered 32 KiB writes.  Its time bounds the
    retrieve on this pool from below; it runs after the timed steps and
    leaves the written blocks holding that chunk."""
    import numpy as np
    import paper_2609_35065_amd as kv
    n = path._last_nres
    # (the streaming retrieve's non-temporal loads would not keep the one chunk in L2)
    if n == 0 or path.staging_host is not None or path.retrieve_kind not in (
            kv.KV_RETRIEVE_UNIT, kv.KV_RETRIEVE_PAIR, kv.KV_RETRIEVE_QUAD):
        return None
    w = path.batch
    jobs = path.h_retr.numpy()[:n].copy()
    jobs[:, 0] = jobs[0, 0]
    d_jobs = torch.from_numpy(jobs).to(path.dev)
    s = path.stream
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ms = []
    for _ in range(reps):
        a.record(s)
        kv.kv_retrieve_scatter_as(path.retrieve_kind, path.layout, path.staging_ptr, path.layers, path.bt,
                                  w.bt_stride, w.num_reqs, d_jobs, n, s)
        b.record(s)
        b.synchronize()
        ms.append(a.elapsed_time(b))
    t = float(np.median(ms))
    written = n * w.shape.slot_bytes
    return {"ms": round(t, 4), "GB/s_written": round(written / (t * 1e-3) / 1e9, 1),
            "what": "the timed retrieve's jobs and variant with every job reading one staged chunk: its "
                    "scattered writes alone (median of 5)"}


def _calibration_copy(torch, reps: int = 5) -> dict:
    """A plain contiguous copy of known size, run by the library's own copy
    kernel: one layer, block size == chunk size, block_first paged layout and
    an identity block table make the retrieve scatter a 4 GiB memcpy (the
    paged block [2][B][H][D] and the staged chunk [1][2][C][H][D] are the same
    bytes).  Used to scale hardware byte counters.  Launches no other kernel."""
    import numpy as np
    import paper_2609_35065_amd as kv
    n, seg = 4096, 256 * 8 * 128 * 2          # 4096 slots of 1 MiB; segment = one plane of a chunk
    lo = kv.make_layout(1, 8, 128, 2, 256, 256, n, n, seg, 2 * seg)
    stg = torch.empty(n * 2 * seg, dtype=torch.uint8, device="cuda")
    pool = torch.empty(n * 2 * seg, dtype=torch.uint8, device="cuda")
    bt = torch.from_numpy(np.arange(n, dtype=np.int32).reshape(n, 1)).cuda()
    jobs = torch.from_numpy(np.stack([np.arange(n), np.arange(n), np.zeros(n), np.zeros(n)], 1)
                            .astype(np.int32)).cuda()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    kv.kv_retrieve_scatter(lo, stg, [pool], bt, 1, n, jobs, n)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        kv.kv_retrieve_scatter(lo, stg, [pool], bt, 1, n, jobs, n)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    return {"calibration": "contiguous copy by kv_copy_retrieve", "bytes_read_per_dispatch": n * 2 * seg,
            "bytes_written_per_dispatch": n * 2 * seg, "dispatches": reps + 1, "ms": round(ms, 4),
            "GB/s_rw": round(2 * n * 2 * seg / (ms * 1e-3) / 1e9, 1)}


def _controller_bench() -> dict:
    """The claim/commitment controller simulation: the six policy
    configurations of the paper's policy comparison on a request stream shaped
    like its workload (three prefix ratios), plus the library's simulator
    timed against the oracle's on one long shared-prefix stream."""
    import numpy as np
    import paper_2609_35065_amd as kv
    import workloads as W
    from oracle import controller as ct
    GiB = float(1 << 30)
    base = dict(budget=50 * GiB, capacity=100 * GiB, stage_rate=11 * GiB, static_rate=11 * GiB, gpu_rate=25 * GiB,
                prefill_s=1e-4, decode_s=0.03, tick=0.05, max_active=4)
    configs = [("Demand", kv.KV_POLICY_DEMAND, 0), ("Immediate", kv.KV_POLICY_IMMEDIATE, 0),
               ("Queue-1", kv.KV_POLICY_QUEUE_K, 1), ("Queue-4", kv.KV_POLICY_QUEUE_K, 4),
               ("TempoKV-Static", kv.KV_POLICY_TEMPO_STATIC, 0), ("TempoKV", kv.KV_POLICY_TEMPO, 0)]

    def kcfg(policy, k, **over):
        d = dict(base, **over)
        return kv.KvSimConfig(d["budget"], d["capacity"], d["stage_rate"], d["static_rate"], d["gpu_rate"],
                              d["prefill_s"], d["decode_s"], d["tick"], d["max_active"], policy, k, 0)

    out = {"policies": {}, "capacity_sweep": {}}
    for ratio in (0.5, 0.75, 1.0):
        sc = W.policy_scenario(ratio)
        rows = {}
        for name, pol, k in configs:
            res, ft, dn, _ = kv.kv_sim_run(kcfg(pol, k), sc.obj_bytes, sc.arrival, sc.manifests, sc.uncached,
                                           sc.out_tokens)
            ttft = np.array(ft) - np.array(sc.arrival)
            tput = sum(sc.out_tokens) / (max(dn) - min(sc.arrival))
            rows[name] = {"C_GiBs_per_req": round(res.cost_gib_s_per_request, 3),
                          "p95_ttft_s": round(float(np.percentile(ttft, 95)), 3),
                          "out_tok_per_s": round(tput, 2), "blocked": res.blocked, "ordinary": res.ordinary}
        imm, tk = rows["Immediate"]["C_GiBs_per_req"], rows["TempoKV"]["C_GiBs_per_req"]
        rows["TempoKV_C_reduction_vs_Immediate"] = round(1 - tk / imm, 3) if imm else None
        out["policies"][f"ratio_{int(ratio * 100)}"] = rows
    sc = W.policy_scenario(1.0)
    for cap in (100, 50, 25):
        rows = {}
        for name, pol, k in configs:
            res, ft, dn, _ = kv.kv_sim_run(kcfg(pol, k, capacity=cap * GiB, budget=cap / 2 * GiB), sc.obj_bytes,
                                           sc.arrival, sc.manifests, sc.uncached, sc.out_tokens)
            ttft = np.array(ft) - np.array(sc.arrival)
            rows[name] = {"C_GiBs_per_req": round(res.cost_gib_s_per_request, 3),
                          "p95_ttft_s": round(float(np.percentile(ttft, 95)), 3), "blocked": res.blocked}
        out["capacity_sweep"][f"fast_tier_{cap}GiB"] = rows
    # simulator speed on one long stream; the oracle timed on the same stream is this mode's CPU baseline
    sc = W.shared_prefix_scenario(400)
    c = ct.SimConfig(policy=ct.TEMPO, queue_k=4, **base)
    t0 = time.perf_counter()
    ref = ct.simulate(c, sc.obj_bytes, sc.arrival, sc.manifests, sc.uncached, sc.out_tokens)
    t_py = time.perf_counter() - t0
    t0 = time.perf_counter()
    res, ft, dn, _ = kv.kv_sim_run(kcfg(kv.KV_POLICY_TEMPO, 4), sc.obj_bytes, sc.arrival, sc.manifests, sc.uncached,
                                   sc.out_tokens)
    t_cc = time.perf_counter() - t0
    assert res.area_byte_s == ref["area"], "simulator and oracle disagree"
    out["simulator_speed"] = {"scenario": sc.name, "events": res.events, "library_s": round(t_cc, 4),
                              "library_events_per_s": round(res.events / t_cc), "speedup_vs_oracle": round(t_py / t_cc, 1)}
    out["cpu_baseline"] = {"value": round(res.events / t_py), "unit": "events/s", "cores": 1, "kind": "oracle",
                           "sample": f"the oracle's simulation of {sc.name} ({res.events} events) in {t_py:.3f} s"}
    return out


def _host_link_gbs(torch, nbytes: int = 1 << 30, reps: int = 3) -> dict:
    """Host-link context for workloads staged in host memory: a DMA copy of a
    pinned buffer into HBM, and the library's copy kernel reading the same
    buffer through its device mapping (the calibration layout of
    _calibration_copy: contiguous, identity table)."""
    import numpy as np
    import paper_2609_35065_amd as kv
    host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    host.fill_(3)
    dev = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    dev.copy_(host, non_blocking=True)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        dev.copy_(host, non_blocking=True)
    e.record()
    torch.cuda.synchronize()
    dma = nbytes / (s.elapsed_time(e) / reps * 1e-3) / 1e9
    n, seg = nbytes // (1 << 20), 256 * 8 * 128 * 2
    lo = kv.make_layout(1, 8, 128, 2, 256, 256, n, n, seg, 2 * seg)
    bt = torch.from_numpy(np.arange(n, dtype=np.int32).reshape(n, 1)).cuda()
    jobs = torch.from_numpy(np.stack([np.arange(n), np.arange(n), np.zeros(n), np.zeros(n)], 1)
                            .astype(np.int32)).cuda()
    mapped = kv.kv_host_device_pointer(host.data_ptr())
    kv.kv_retrieve_scatter(lo, mapped, [dev], bt, 1, n, jobs, n)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        kv.kv_retrieve_scatter(lo, mapped, [dev], bt, 1, n, jobs, n)
    e.record()
    torch.cuda.synchronize()
    zc = nbytes / (s.elapsed_time(e) / reps * 1e-3) / 1e9
    del host, dev
    torch.cuda.empty_cache()
    return {"host_to_hbm_dma_GB/s": round(dma, 1), "zero_copy_kernel_read_GB/s": round(zc, 1)}


def _clocks():
    """rocm-smi's clock report, if the tool is available (context only)."""
    import shutil
    import subprocess
    exe = shutil.which("rocm-smi")
    if not exe:
        return None
    try:
        r = subprocess.run([exe, "--showclocks", "--json"], capture_output=True, text=True, timeout=20)
        return json.loads(r.stdout) if r.returncode == 0 else None
    except (OSError, ValueError, subprocess.SubprocessError):
        return None


def _device_copy_gbs(torch, nbytes: int = 4 << 30, reps: int = 5) -> float:
    """Plain device-to-device copy rate (read + write bytes / time): practical-peak context."""
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    b.copy_(a)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    del a, b
    torch.cuda.empty_cache()
    return 2 * nbytes / (ms * 1e-3) / 1e9


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="l32-64x4096")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--controller", action="store_true",
                    help="run the claim/commitment controller simulation (host only) and exit")
    ap.add_argument("--calib-copy", action="store_true",
                    help="only run a plain 4 GiB contiguous copy (counter calibration) and exit")
    ap.add_argument("--lower-tier", default="zero-copy", choices=("zero-copy", "pipelined", "serialized"),
                    help="workloads whose staged chunks live in host memory: read them in place (zero-copy), or "
                         "stage them into HBM by DMA batch by batch, overlapped with the scatter on a second "
                         "stream (pipelined) or on the same stream (serialized); staged modes start every step "
                         "with no chunk resident in HBM")
    ap.add_argument("--slots-per-batch", type=int, default=4,
                    help="staged modes: distinct staged chunks per copy/scatter batch")
    ap.add_argument("--serial", action="store_true",
                    help="run each step's hash and lookup after the previous step's copies instead of overlapping "
                         "them (with the host job build) with those copies")
    ap.add_argument("--no-tune", action="store_true",
                    help="run the planned retrieve variant without timing it against the four-job-window one")
    ap.add_argument("--no-fill", action="store_true",
                    help="leave KV buffers uninitialised (hardware-counter runs: no generator kernels run; the "
                         "copies move the same bytes) and skip the device-copy and CPU-baseline extras")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the staging path shards by request with no exchange between "
              "GPUs, so multi-GPU runs are not part of this benchmark (use --gpus 1).", file=sys.stderr)
        return 2

    if args.controller:
        print(json.dumps({"controller": _controller_bench()}))
        return 0

    import numpy as np
    import torch
    import workloads as W
    from paper_2609_35065_amd import RETRIEVE_KIND_NAMES
    from paper_2609_35065_amd.pipeline import StagingPath

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    if args.calib_copy:
        print(json.dumps(_calibration_copy(torch)))
        return 0

    w = W.make(args.workload)
    print(f"[bench] workload {w.name}: {w.num_reqs} requests, pool {w.pool_bytes() / 2**30:.1f} GiB, "
          f"staging {w.staged_bytes() / 2**30:.1f} GiB", file=sys.stderr, flush=True)
    path = StagingPath(w, lower_tier=args.lower_tier, slots_per_batch=args.slots_per_batch,
                       overlap=not args.serial)
    if not args.no_fill:
        path.fill(STG_TAG, POOL_TAG, w.seed)
    path.prestage()

    def steps(n, timers=None):
        # Step i+1's hash and lookup are enqueued (on their own stream) as soon
        # as step i's copies and index update are, so they and step i+1's host
        # job build overlap step i's copies.  Every step still does all its work.
        out = None
        if n:
            path.launch_lookup(timers)
        for i in range(n):
            path.drop_fast_tier()          # staged modes: every step stages its chunks again
            out = path.complete_pass(evict_stored=True, timers=timers)
            if i + 1 < n:
                path.launch_lookup(timers)
        return out

    steps(args.warmup)
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)
    # pick the retrieve variant for this pool by timing (outside the timed steps)
    tuning = path.tune_retrieve() if args.warmup and not args.no_tune else {}

    timers: dict = {}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    stats = steps(args.steps, timers)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    print(f"[bench] timed {args.steps} steps", file=sys.stderr, flush=True)

    # hash and lookup once more on an otherwise idle GPU: in the overlapped
    # steps they share the CUs with the previous step's copies
    iso: dict = {}
    path.set_overlap(False)
    for _ in range(5):
        path.drop_fast_tier()
        path.run_pass(evict_stored=True, timers=iso)
    torch.cuda.synchronize()

    def iso_ms(name):
        ev = [a.elapsed_time(b) for a, b in iso.get(name, [])]
        return float(np.median(ev)) if ev else 0.0

    def avg_ms(name):
        ev = timers.get(name, [])
        return float(np.mean([a.elapsed_time(b) for a, b in ev])) if ev else 0.0

    def spread(name):
        ev = [a.elapsed_time(b) for a, b in timers.get(name, [])]
        return {"ms_median": round(float(np.median(ev)), 4), "ms_min": round(float(np.min(ev)), 4)} if ev else {}

    ms_step = (t1 - t0) * 1e3 / args.steps
    r_bytes = 2 * stats.retrieve_bytes          # read + write per step
    s_bytes = 2 * stats.store_bytes
    value = (r_bytes + s_bytes) / (ms_step * 1e-3) / 1e9
    k_ms = {k: avg_ms(k) for k in ("hash", "lookup", "retrieve", "store", "stage")}
    r_gbs = r_bytes / (k_ms["retrieve"] * 1e-3) / 1e9 if k_ms["retrieve"] else 0.0
    s_gbs = s_bytes / (k_ms["store"] * 1e-3) / 1e9 if k_ms["store"] else 0.0
    n_tok = int(w.tokens.size)
    hash_iso = iso_ms("hash")
    hash_mtok = n_tok / (hash_iso * 1e-3) / 1e6 if hash_iso else 0.0

    # unique staged bytes a retrieve must read at least once + bytes written:
    # its algorithmic HBM bytes when requests share staged chunks (the
    # counters measure within 0.2 % of this); the payload counts every read
    uniq = len(set(int(q[0]) for q in path.last_retrieve)) * w.shape.slot_bytes
    r_alg = uniq + stats.retrieve_bytes
    r_hbm = r_alg / (k_ms["retrieve"] * 1e-3) / 1e9 if k_ms["retrieve"] else 0.0
    dom = "retrieve" if k_ms["retrieve"] * 1 >= k_ms["store"] else "store"
    dom_kernel = "kv_copy_retrieve" if dom == "retrieve" else "kv_copy_store"
    achieved = r_hbm if dom == "retrieve" else s_gbs
    traffic = _load_traffic(dom_kernel, args.workload)
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "layers": w.shape.num_layers, "kv_heads": w.shape.kv_heads,
                   "head_dim": w.shape.head_dim, "block_size": w.shape.block_size,
                   "chunk_tokens": w.shape.chunk_tokens, "requests": w.num_reqs, "tokens": n_tok,
                   "pool_blocks": w.num_blocks, "staging_slots": w.num_slots,
                   "retrieve_jobs": stats.num_retrieve, "store_jobs": stats.num_store,
                   "steps_overlap": not args.serial,
                   "retrieve_variant": RETRIEVE_KIND_NAMES.get(path.retrieve_kind),
                   "retrieve_tuning_ms": tuning},
        "roofline": {"bound": "hbm", "kernel": dom_kernel, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic},
        "kernels": {
            "retrieve_scatter": {"ms": round(k_ms["retrieve"], 4), "GB/s": round(r_hbm, 1),
                                 "frac_of_peak": round(r_hbm / HBM_PEAK_GBS, 4), "algorithmic_bytes": r_alg,
                                 "payload_GB/s": round(r_gbs, 1), "payload_bytes_rw": r_bytes},
            "store_gather": {"ms": round(k_ms["store"], 4), "GB/s": round(s_gbs, 1),
                             "frac_of_peak": round(s_gbs / HBM_PEAK_GBS, 4), "payload_bytes_rw": s_bytes},
            "hash_prefix": {"ms": round(k_ms["hash"], 4), "isolated_ms": round(hash_iso, 4),
                            "Mtok/s": round(hash_mtok, 1),
                            "ns_per_chain_step": round(hash_iso * 1e6 / max(1, int(w.lengths.max()) // 16), 2)},
            "lookup": {"ms": round(k_ms["lookup"], 4), "isolated_ms": round(iso_ms("lookup"), 4)},
        },
        "timing": "HIP events on the launch stream around every launch of the timed steps (ms = mean); hash "
                  "and lookup also on an idle GPU after the timed steps (isolated_ms = median of 5, used for "
                  "Mtok/s)",
        "source_digest": _src_digest(),
    }
    if not w.staging_in_host:
        # the same step in HBM terms: unique staged reads + writes of the retrieve, reads + writes of the store
        line["step_hbm_GB/s"] = round((r_alg + s_bytes) / (ms_step * 1e-3) / 1e9, 1)
    for name, key in (("retrieve", "retrieve_scatter"), ("store", "store_gather"), ("hash", "hash_prefix"),
                      ("lookup", "lookup")):
        line["kernels"][key].update(spread(name))
    if w.staging_in_host:
        lt = {"mode": args.lower_tier, "staged_bytes_per_step": stats.staged_bytes}
        if path.staged_mode:
            lt["slots_per_batch"] = args.slots_per_batch
            lt["retrieve_ms_includes_staging"] = True
            if k_ms["stage"]:
                lt["stage_ms"] = round(k_ms["stage"], 4)
                lt["stage_GB/s"] = round(stats.staged_bytes / (k_ms["stage"] * 1e-3) / 1e9, 1)
        line["config"]["lower_tier"] = lt
    wb = _retrieve_write_bound(path, torch) if not args.no_fill else None
    del path
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if not args.no_fill:
        line["practical_peak"] = {"torch_device_copy_GB/s": round(_device_copy_gbs(torch), 1),
                                  "library_contiguous_copy_GB/s": _calibration_copy(torch)["GB/s_rw"]}
        if wb:
            # the retrieve's algorithmic bytes moved at the pool's own scattered-write rate
            wb["alg_bytes_at_this_rate_ms"] = round(r_alg / (wb["GB/s_written"] * 1e9) * 1e3, 4)
            wb["retrieve_frac_of_this_rate"] = round(wb["alg_bytes_at_this_rate_ms"] / k_ms["retrieve"], 4)
            line["practical_peak"]["retrieve_writes_only"] = wb
        if w.staging_in_host:
            line["practical_peak"].update(_host_link_gbs(torch))
        props = torch.cuda.get_device_properties(0)
        line["gpu"] = {"name": props.name, "compute_units": props.multi_processor_count,
                       "memory_GiB": round(props.total_memory / 2**30, 1), "clocks": _clocks()}
    if not args.no_cpu_baseline and not args.no_fill:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        line["cpu_baseline"] = _cpu_baseline(w.shape)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
