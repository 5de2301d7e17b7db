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

Prints one JSON line: the whole step's HBM bytes per second (the
retrieve's unique staged reads and its writes plus the store's reads and
writes, divided by wall time per step; the payload rate, which counts every
job's read, is reported beside it), per-kernel rates measured with HIP events
on the launch stream, the roofline of the dominant copy kernel against
MI355X's 8 TB/s HBM peak (both copy kernels are listed), same-pool ceilings,
and the CPU oracle timed on a bounded sample of the same workload shape.

    python bench.py [--steps K] [--warmup W] [--workload NAME]
    python bench.py --summarize-trace DIR --workload NAME --command CMD   (rocprofv3 output -> profiles/)
    python bench.py --summarize-traffic DIR --workload NAME               (FETCH_SIZE / WRITE_SIZE -> profiles/)
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
# the same-pool ceiling: launches of each of its two measurements (writes alone, writes with the unique reads)
CEILING_REPS = 5
CEILING_LAUNCHES = 2 * CEILING_REPS


def _src_digest() -> str:
    h = hashlib.sha256()
    for f in ("copy.hip", "internal.h"):
        with open(os.path.join(ROOT, "paper_2609_35065_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _load_traffic(kernel: str, workload: str, variant: str = None):
    """HBM bytes per launch measured by rocprofv3 counters, if a summary for
    this kernel (retrieve: and variant) and workload exists and was taken from
    the current source."""
    if kernel == "kv_copy_retrieve" and variant is None:
        return None
    tag = f"{kernel}_{variant}" if kernel == "kv_copy_retrieve" else kernel
    path = os.path.join(PROFILES, f"traffic_{tag}_{workload}.txt")
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


# ---------------------------------------------------------------------------
# Kernel symbols, and the summaries of rocprofv3 output committed under profiles/
# ---------------------------------------------------------------------------

def _rows_of(seg_bytes: int, row_bytes: int) -> int:
    """Rows of `row_bytes` per segment when that is 1, 2, 4, 8 or 16 (the copy kernels' fast paths)."""
    if seg_bytes % row_bytes:
        return 0
    r = seg_bytes // row_bytes
    return r if r in (1, 2, 4, 8, 16) else 0


def _symbol(kind: str, w) -> str:
    """The __global__ function (copy.hip) a copy launch of this kind runs for the workload's segment size."""
    seg = w.shape.seg_bytes
    if kind in ("unit", "pair", "quad"):
        r = _rows_of(seg, 256 * 16)
        if kind == "pair" and r != 8:
            kind = "unit"
        if r:
            return {"unit": "retrieve_unit_kernel", "pair": "retrieve_pair_kernel",
                    "quad": "retrieve_quad_kernel"}[kind] + f"<{r}>"
        return "copy_generic_kernel<true>"
    retrieve = kind == "stream"
    for t in (1024, 512, 256):
        r = _rows_of(seg, t * 16)
        if r:
            return f"group_copy_kernel<{t}, {r}, {'true' if retrieve else 'false'}>"
    return f"copy_generic_kernel<{'true' if retrieve else 'false'}>"


def _label(symbol: str) -> str:
    """What a library kernel does, from its symbol."""
    for key, text in (("retrieve_unit_kernel", "retrieve scatter, unit walk (KV_RETRIEVE_UNIT)"),
                      ("retrieve_pair_kernel", "retrieve scatter, pair walk (KV_RETRIEVE_PAIR)"),
                      ("retrieve_quad_kernel", "retrieve scatter, four-job window (KV_RETRIEVE_QUAD)"),
                      ("copy_generic_kernel<true>", "retrieve scatter, generic path"),
                      ("copy_generic_kernel<false>", "store gather, generic path"),
                      ("hash_kernel", "prefix hash (kv_hash_prefix)"),
                      ("lookup_kernel", "lookup (kv_lookup)"),
                      ("index_apply_kernel", "index update (kv_index_insert / erase)"),
                      ("mixed_traffic_kernel", "measurement reference: the retrieve's bytes, no dependence "
                                               "(kv_probe_mixed_traffic)")):
        if key in symbol:
            return text
    if "group_copy_kernel" in symbol:
        return ("retrieve scatter, streaming (KV_RETRIEVE_STREAM)" if "true>" in symbol
                else "store gather (kv_store_gather)")
    return "other"


def _short_symbol(name: str) -> str:
    """rocprofv3's demangled kernel name without namespaces and argument list."""
    base = name.split("(tkv::")[0].split("(long")[0].split("(const")[0]
    if base.endswith(")") and "(" in base and "<" not in base.split("(")[-1]:
        base = base[:base.rfind("(")]
    base = base.replace("tkv::(anonymous namespace)::", "").replace("(anonymous namespace)::", "").strip()
    return base[5:] if base.startswith("void ") else base


def _csv_rows(directory: str, suffix: str):
    import csv
    import glob
    files = sorted(glob.glob(os.path.join(directory, "**", f"*{suffix}"), recursive=True))
    if not files:
        raise FileNotFoundError(f"no *{suffix} under {directory}")
    rows = []
    for f in files:
        rows += list(csv.DictReader(open(f)))
    return rows


def _bench_json(log: str):
    if not os.path.exists(log):
        return None
    js = [l for l in open(log) if l.startswith("{")]
    return json.loads(js[-1]) if js else None


def profile_commands(workload: str, out: str) -> list:
    """The rocprofv3 runs behind profiles/*_{workload}.*: (name, command) pairs,
    each writing under `out`/name (every counter pass is a run of its own)."""
    b3 = f"python3 bench.py --steps 3 --warmup 1 --no-fill --workload {workload}"
    pmc = {"sq": "SQ_INSTS_VMEM_RD SQ_INSTS_VMEM_WR SQ_INSTS_SMEM SQ_WAVES SQ_INSTS_VALU SQ_INSTS_SALU "
                 "SQ_BUSY_CYCLES SQ_WAVE_CYCLES",
           "tcc": "TCC_HIT_sum TCC_MISS_sum TCC_EA0_WRREQ_sum TCC_EA0_RDREQ_sum",
           "tlb": "TCP_UTCL1_TRANSLATION_MISS_sum TCP_UTCL1_TRANSLATION_HIT_sum GRBM_GUI_ACTIVE GRBM_COUNT",
           "occ": "OccupancyPercent",
           "pmc_fetch": "FETCH_SIZE", "pmc_write": "WRITE_SIZE"}
    cmds = [("ktrace", f"rocprofv3 --kernel-trace --stats -f csv -d {out}/ktrace -o c -- python3 bench.py "
                       f"--no-cpu-baseline --no-extras --workload {workload}")]
    for name, ctrs in pmc.items():
        cmds.append((name, f"rocprofv3 --pmc {ctrs} --kernel-include-regex tkv -f csv -d {out}/{name} -o c -- {b3}"))
    for name, ctr in (("cal_fetch", "FETCH_SIZE"), ("cal_write", "WRITE_SIZE")):
        cmds.append((name, f"rocprofv3 --pmc {ctr} -f csv -d {out}/{name} -o c -- python3 bench.py --calib-copy"))
    # the retrieve's same-pool ceiling alone (every kernel counted: its reads are torch reductions)
    cc = f"python3 bench.py --warmup 1 --no-fill --ceiling-only --workload {workload}"
    for name, ctr in (("ceil_fetch", "FETCH_SIZE"), ("ceil_write", "WRITE_SIZE")):
        cmds.append((name, f"rocprofv3 --pmc {ctr} -f csv -d {out}/{name} -o c -- {cc}"))
    return cmds


def summarize_trace(directory: str, workload: str, command: str) -> str:
    """profiles/kernel_trace_{workload}.md from a rocprofv3 --kernel-trace --stats run."""
    rows = _csv_rows(directory, "_kernel_stats.csv")
    lines = [f"# Kernel trace summary: {workload}", "", "Command (repository root, one MI355X):", "", "```", command,
             "```", "", "Made by `python bench.py --summarize-trace`: the rows of rocprofv3's kernel statistics whose "
             "kernel is one of the library's, with the kernel's symbol as rocprofv3 printed it "
             "(namespaces and argument list dropped); all other rows are the input generator and runtime copies.",
             "", "| kernel | symbol (copy.hip, hash.hip, index.hip) | calls | avg us | min us | max us | total ms |",
             "|---|---|---:|---:|---:|---:|---:|"]
    ours = [r for r in rows if _label(_short_symbol(r["Name"])) != "other"]
    for r in sorted(ours, key=lambda r: -float(r["TotalDurationNs"])):
        sym = _short_symbol(r["Name"])
        lines.append(f"| {_label(sym)} | `{sym}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} |")
    other = [r for r in rows if _label(_short_symbol(r["Name"])) == "other"]
    lines += ["", f"Other kernels: {len(other)} names, "
                  f"{sum(float(r['TotalDurationNs']) for r in other) / 1e6:.1f} ms in total."]
    d = _bench_json(os.path.join(directory, "bench.log"))
    if d:
        k = d["kernels"]
        tun = d["config"].get("retrieve_tuning_ms") or {}
        lines += ["", f"The timed steps ran the `{d['config'].get('retrieve_variant')}` retrieve "
                      f"(`{d['roofline']['per_kernel']['retrieve_scatter']['symbol']}`)."]
        if tun:
            lines[-1] += (" Before them the bench timed the candidates on this pool (medians: "
                          + ", ".join(f"{n} {v:.3f} ms" for n, v in tun.items()) + "), so both appear above.")
        lines += ["", "HIP-event timings the same run printed (mean over its timed steps): "
                      f"retrieve {k['retrieve_scatter']['ms']:.3f} ms, store {k['store_gather']['ms']:.3f} ms; "
                      f"hash {k['hash_prefix'].get('isolated_ms', 0) * 1e3:.1f} us and lookup "
                      f"{k['lookup'].get('isolated_ms', 0) * 1e3:.1f} us on an idle GPU."]
    path = os.path.join(PROFILES, f"kernel_trace_{workload}.md")
    open(path, "w").write("\n".join(lines) + "\n")
    return path


def _counter_medians(directory: str):
    import statistics
    from collections import defaultdict
    agg = defaultdict(list)
    for r in _csv_rows(directory, "_counter_collection.csv"):
        agg[(_short_symbol(r["Kernel_Name"]), r["Counter_Name"])].append(float(r["Counter_Value"]))
    return {k: statistics.median(v) for k, v in agg.items()}


def _calibration_scales(cal_dir: str):
    """FETCH_SIZE and WRITE_SIZE scale factors from the calibration copy (4 GiB each way)."""
    w_cal = 4 << 30
    cf = [v for (k, c), v in _counter_medians(os.path.join(cal_dir, "cal_fetch")).items() if "copy_generic" in k]
    cw = [v for (k, c), v in _counter_medians(os.path.join(cal_dir, "cal_write")).items() if "copy_generic" in k]
    return w_cal / 1024 / cf[0], w_cal / 1024 / cw[0], cf[0], cw[0]


def summarize_traffic(directory: str, workload: str, calibration: str = None) -> list:
    """profiles/traffic_*_{workload}.txt: FETCH_SIZE and WRITE_SIZE per launch
    of the store and of the retrieve variant the timed steps ran, scaled by
    what the same counters read for the calibration copy of known size."""
    cal_dir = calibration or directory
    cmds = dict(profile_commands(workload, "gpurun_out/prof_" + workload))
    cal_wl = os.path.basename(os.path.normpath(cal_dir))[len("prof_"):] or workload
    cmds.update({k: v for k, v in profile_commands(cal_wl, "gpurun_out/prof_" + cal_wl) if k.startswith("cal_")})
    fe, wr = _counter_medians(os.path.join(directory, "pmc_fetch")), _counter_medians(os.path.join(directory, "pmc_write"))
    f_fetch, f_write, cf, cw = _calibration_scales(cal_dir)
    d = _bench_json(os.path.join(directory, "pmc_fetch.log"))
    variant = d["config"]["retrieve_variant"]
    import workloads as W
    w = W.make(workload)
    out = []
    kinds = [("kv_copy_store", _symbol("store", w))]
    for v in ("unit", "pair", "quad", "stream"):
        # the timed variant, and the candidate the retrieve tuning also launched in the same run
        if _symbol(v, w) not in [k for k, _ in kinds]:
            kinds.append((f"kv_copy_retrieve_{v}", _symbol(v, w)))
    for kern, sym in kinds:
        fk = [v for (k, c), v in fe.items() if k == sym and c == "FETCH_SIZE"]
        wk = [v for (k, c), v in wr.items() if k == sym and c == "WRITE_SIZE"]
        if not fk or not wk:
            continue
        fk, wk = fk[0], wk[0]
        txt = [f"# HBM traffic per launch of {_label(sym)}, workload {workload}",
               "# Made by `python bench.py --summarize-traffic` from these runs (repository root, one MI355X):",
               *[f"#   {cmds[n]}" for n in ("pmc_fetch", "pmc_write", "cal_fetch", "cal_write")],
               "# Each counter is the median over the kernel's launches, in KiB per dispatch, scaled by the same",
               "# counter's reading for the calibration: a 4 GiB contiguous copy (4 GiB read, 4 GiB written) by",
               "# copy_generic_kernel<true>.  --no-fill: the KV buffers are not initialised (the copies move the",
               "# same bytes); the input fill is never run under --pmc.",
               f"kernel={kern}", f"symbol={sym}", f"workload={workload}", f"source_digest={_src_digest()}",
               f"timed_variant={variant}" + ("" if kern == "kv_copy_store" or kern.endswith(variant) else
                                              " (this variant ran in the retrieve tuning before the timed steps)"),
               f"fetch_kib_per_dispatch={fk:.1f}", f"write_kib_per_dispatch={wk:.1f}",
               f"calibration_fetch_kib={cf:.1f}", f"calibration_write_kib={cw:.1f}",
               f"fetch_scale={f_fetch:.4f}", f"write_scale={f_write:.4f}",
               f"hbm_read_bytes_per_launch={fk * f_fetch * 1024:.0f}",
               f"hbm_write_bytes_per_launch={wk * f_write * 1024:.0f}",
               f"traffic_bytes_per_launch={(fk * f_fetch + wk * f_write) * 1024:.0f}"]
        path = os.path.join(PROFILES, f"traffic_{kern}_{workload}.txt")
        open(path, "w").write("\n".join(txt) + "\n")
        out.append(path)
    return out


def summarize_ceiling(directory: str, workload: str, calibration: str = None):
    """profiles/traffic_retrieve_ceiling_{workload}.txt: HBM bytes of the
    retrieve's same-pool ceiling, from a --ceiling-only run under FETCH_SIZE
    and one under WRITE_SIZE.  The ceiling's retrieve launches (every job
    reading one staged chunk) are the last CEILING_LAUNCHES launches of the
    retrieve kernel in the run; its reads of the unique staged chunks are the
    torch reduction kernels (CEILING_LAUNCHES passes over the chunks).
    Returns the path, or None when the run measured no ceiling."""
    import statistics
    from collections import defaultdict
    cal_dir = calibration or directory
    d = _bench_json(os.path.join(directory, "ceil_fetch.log"))
    if not d or not d.get("ceiling"):
        return None
    n = int(d["ceiling_launches"])
    variant = d["config"]["retrieve_variant"]
    import workloads as W
    sym = _symbol(variant, W.make(workload))
    f_fetch, f_write, cf, cw = _calibration_scales(cal_dir)
    res = {}
    for kind, ctr, scale in (("ceil_fetch", "FETCH_SIZE", f_fetch), ("ceil_write", "WRITE_SIZE", f_write)):
        rows = [r for r in _csv_rows(os.path.join(directory, kind), "_counter_collection.csv")
                if r["Counter_Name"] == ctr]
        mine = sorted((int(r["Dispatch_Id"]), float(r["Counter_Value"])) for r in rows
                      if _short_symbol(r["Kernel_Name"]) == sym)
        if len(mine) < n:
            raise ValueError(f"{kind}: {len(mine)} launches of {sym}, expected at least {n}")
        per_reader = defaultdict(float)
        for r in rows:
            if "reduce_kernel" in r["Kernel_Name"]:
                per_reader[_short_symbol(r["Kernel_Name"]).split("<")[0]] += float(r["Counter_Value"])
        mixed = [float(r["Counter_Value"]) for r in rows if _short_symbol(r["Kernel_Name"]) == "mixed_traffic_kernel"]
        res[kind] = (statistics.median(v for _, v in mine[-n:]) * scale * 1024,
                     sum(per_reader.values()) / n * scale * 1024, len(mine),
                     statistics.median(mixed) * scale * 1024 if mixed else None)
    c = d["ceiling"]
    cmds = dict(profile_commands(workload, "gpurun_out/prof_" + workload))
    cal_wl = os.path.basename(os.path.normpath(cal_dir))[len("prof_"):] or workload
    cmds.update({k: v for k, v in profile_commands(cal_wl, "gpurun_out/prof_" + cal_wl) if k.startswith("cal_")})
    wo_read, rd_read, nl, ix_read = res["ceil_fetch"]
    wo_write, rd_write, _, ix_write = res["ceil_write"]
    txt = [f"# HBM traffic of the retrieve's same-pool ceiling, workload {workload}",
           "# Made by `python bench.py --summarize-ceiling` from these runs (repository root, one MI355X):",
           *[f"#   {cmds[k]}" for k in ("ceil_fetch", "ceil_write", "cal_fetch", "cal_write")],
           "# The ceiling re-runs the retrieve's own jobs, variant and destination blocks with every job reading",
           "# one staged chunk (its scattered writes alone), and reads the retrieve's unique staged chunks with",
           "# torch reductions, alone and concurrently with those writes.  Counters: the median over the last",
           f"# {n} launches of the retrieve kernel (the ceiling's; the warm-up pass and the tuning launch it",
           "# before them) and the reductions' sum divided by the number of read passes, scaled by the calibration",
           "# copy's readings as in the traffic files of the copy kernels.",
           f"workload={workload}", f"symbol={sym}", f"retrieve_variant={variant}",
           f"retrieve_launches_in_run={nl}", f"ceiling_launches={n}",
           f"fetch_scale={f_fetch:.4f}", f"write_scale={f_write:.4f}",
           f"writes_only_hbm_read_bytes_per_launch={wo_read:.0f}",
           f"writes_only_hbm_write_bytes_per_launch={wo_write:.0f}",
           f"unique_read_hbm_read_bytes_per_pass={rd_read:.0f}",
           f"unique_read_hbm_write_bytes_per_pass={rd_write:.0f}",
           f"ceiling_traffic_bytes={wo_read + wo_write + rd_read + rd_write:.0f}"]
    if ix_read is not None and ix_write is not None:
        txt += ["# kv_probe_mixed_traffic (mixed_traffic_kernel, the same algorithmic bytes in one launch with no",
                "# dependence between its reads and writes): median over its launches in the run",
                f"independent_mix_hbm_read_bytes_per_launch={ix_read:.0f}",
                f"independent_mix_hbm_write_bytes_per_launch={ix_write:.0f}"]
    if isinstance(c, dict) and "writes_with_unique_read" in c:
        txt.append(f"# timings of this run are not quoted: counter collection serialises the two streams")
    path = os.path.join(PROFILES, f"traffic_retrieve_ceiling_{workload}.txt")
    open(path, "w").write("\n".join(txt) + "\n")
    return path


def summarize_counters(directory: str, workload: str) -> str:
    """profiles/counters_{workload}.md: memory instructions, L2 traffic and hit
    rate, address translation and occupancy per launch of each copy kernel."""
    cmds = dict(profile_commands(workload, "gpurun_out/prof_" + workload))
    c = {}
    for kind in ("sq", "tcc", "tlb", "occ"):
        c.update(_counter_medians(os.path.join(directory, kind)))
    d = _bench_json(os.path.join(directory, "sq.log"))
    lines = [f"# Hardware counters per launch: workload {workload}", "",
             "Commands (repository root, one MI355X; one counter group per run):", "", "```",
             *[cmds[k] for k in ("sq", "tcc", "tlb", "occ")], "```", "",
             "Made by `python bench.py --summarize-counters`: medians over each kernel's launches.  "
             "TCC_EA0_RDREQ counts 128-byte and TCC_EA0_WRREQ 64-byte requests leaving the L2 (hits in the memory-side "
             "cache included).  --no-fill: KV buffers uninitialised, same bytes moved."]
    if d:
        lines[-1] += (f"  The timed steps ran the `{d['config'].get('retrieve_variant')}` retrieve; the tuning before "
                      "them launches both candidates, so both appear.")
    syms = sorted({k for (k, cn) in c if cn == "SQ_WAVES" and _label(k) != "other"})
    for sym in syms:
        g = lambda n, sym=sym: c.get((sym, n), float("nan"))
        waves = g("SQ_WAVES")
        hit, miss = g("TCC_HIT_sum"), g("TCC_MISS_sum")
        th, tm = g("TCP_UTCL1_TRANSLATION_HIT_sum"), g("TCP_UTCL1_TRANSLATION_MISS_sum")
        lines += ["", f"## {_label(sym)}: `{sym}`", "", "| quantity | value | per wave or bytes |", "|---|---:|---|",
                  f"| SQ_WAVES | {waves:.0f} | |",
                  f"| SQ_INSTS_VMEM_RD | {g('SQ_INSTS_VMEM_RD'):.0f} | x 1 KiB = {g('SQ_INSTS_VMEM_RD') * 1024 / 1e9:.3f} GB |",
                  f"| SQ_INSTS_VMEM_WR | {g('SQ_INSTS_VMEM_WR'):.0f} | x 1 KiB = {g('SQ_INSTS_VMEM_WR') * 1024 / 1e9:.3f} GB |",
                  f"| SQ_INSTS_SMEM | {g('SQ_INSTS_SMEM'):.0f} | {g('SQ_INSTS_SMEM') / waves:.1f} per wave |",
                  f"| SQ_INSTS_VALU / SQ_INSTS_SALU | {g('SQ_INSTS_VALU'):.0f} / {g('SQ_INSTS_SALU'):.0f} | "
                  f"{g('SQ_INSTS_VALU') / waves:.0f} / {g('SQ_INSTS_SALU') / waves:.0f} per wave |",
                  f"| TCC_EA0_RDREQ_sum | {g('TCC_EA0_RDREQ_sum'):.0f} | x 128 B = {g('TCC_EA0_RDREQ_sum') * 128 / 1e9:.3f} GB |",
                  f"| TCC_EA0_WRREQ_sum | {g('TCC_EA0_WRREQ_sum'):.0f} | x 64 B = {g('TCC_EA0_WRREQ_sum') * 64 / 1e9:.3f} GB |",
                  f"| L2 hit rate | {hit / (hit + miss) * 100:.1f} % | TCC_HIT_sum {hit:.0f}, TCC_MISS_sum {miss:.0f} |",
                  f"| UTCL1 translation misses | {tm:.0f} | of {th + tm:.0f} ({tm / (th + tm) * 100:.3f} %) |",
                  f"| OccupancyPercent | {g('OccupancyPercent'):.1f} % | |"]
    path = os.path.join(PROFILES, f"counters_{workload}.md")
    open(path, "w").write("\n".join(lines) + "\n")
    return path


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


def _retrieve_write_bound(path, torch, reps: int = CEILING_REPS):
    """The timed retrieve's writes on their own: the same jobs, variant and
    destination blocks, but every job reading one staged chunk (which stays in
    L2), so HBM sees only the scattered 32 KiB writes.  Its time bounds the
    retrieve on this pool from below; it runs after the timed steps and
    leaves the written blocks holding that chunk.  Before it, the same
    algorithmic bytes are moved by kv_probe_mixed_traffic (reads and writes
    interleaved in one launch with no dependence between them), and after
    it the writes run together with a read of the unique chunks on a second
    stream."""
    import numpy as np
    import paper_2609_35065_amd as kv
    n = path._last_nres
    # (the streaming retrieve's non-temporal loads would not keep the one chunk in L2)
    if n == 0 or path.staging_host is not None or path.retrieve_kind not in (
            kv.KV_RETRIEVE_UNIT, kv.KV_RETRIEVE_PAIR, kv.KV_RETRIEVE_QUAD):
        return None
    w = path.batch
    s = path.stream
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    slots = np.unique(path.h_retr.numpy()[:n, 0])
    sb = w.shape.slot_bytes
    uniq = int(slots.size) * sb
    written = n * sb
    # First, the same algorithmic bytes with no dependence between reads and writes, in one launch
    # (kv_probe_mixed_traffic: the unique staged chunks read, the destination blocks written with a
    # filler, interleaved).  It overwrites the destinations; the writes-only launches below rewrite them.
    d_slots = torch.from_numpy(slots.astype(np.int32)).to(path.dev)
    mix = []
    for _ in range(reps):
        a.record(s)
        kv.kv_probe_mixed_traffic(path.layout, path.staging_ptr, path.layers, path.bt, w.bt_stride, w.num_reqs,
                                  path.d_retr, n, d_slots, int(slots.size), 0x5A5A5A5A, s)
        b.record(s)
        b.synchronize()
        mix.append(a.elapsed_time(b))
    t_ix = float(np.median(mix))
    jobs = path.h_retr.numpy()[:n].copy()
    jobs[:, 0] = jobs[0, 0]
    d_jobs = torch.from_numpy(jobs).to(path.dev)
    ms = []
    for _ in range(reps):
        a.record(s)
        kv.kv_retrieve_scatter_as(path.retrieve_kind, path.layout, path.staging_ptr, path.layers, path.bt,
                                  w.bt_stride, w.num_reqs, d_jobs, n, s)
        b.record(s)
        b.synchronize()
        ms.append(a.elapsed_time(b))
    t = float(np.median(ms))
    out = {"ms": round(t, 4), "GB/s_written": round(written / (t * 1e-3) / 1e9, 1),
           "what": "the timed retrieve's jobs and variant with every job reading one staged chunk: its "
                   f"scattered writes alone (median of {reps})"}
    out["independent_mix"] = {
        "ms": round(t_ix, 4), "GB/s_alg": round((uniq + written) / (t_ix * 1e-3) / 1e9, 1),
        "what": "kv_probe_mixed_traffic: the unique staged chunks read and the destination blocks written, "
                f"interleaved in one launch with no data passing between them (median of {reps})"}
    # The same writes with the unique staged chunks read from HBM at the same time, on a second stream:
    # the retrieve's algorithmic bytes (unique reads + writes) with no kernel of ours reading them.  The
    # reads are torch reductions over the contiguous runs of the chunks' slots.
    runs, start = [], int(slots[0])
    for prev, cur in zip(slots[:-1], slots[1:]):
        if cur != prev + 1:
            runs.append((start, int(prev) + 1))
            start = int(cur)
    runs.append((start, int(slots[-1]) + 1))
    views = [path.staging[r0 * sb:r1 * sb].view(torch.int64) for r0, r1 in runs]
    s2 = torch.cuda.Stream()
    sink = torch.zeros(len(views), dtype=torch.int64, device=path.dev)

    def read_unique(stream):
        with torch.cuda.stream(stream):
            for k, v in enumerate(views):
                torch.sum(v, dim=0, out=sink[k])

    rd, mixed = [], []
    for _ in range(reps):
        a.record(s)
        read_unique(s)
        b.record(s)
        b.synchronize()
        rd.append(a.elapsed_time(b))
        c = torch.cuda.Event(enable_timing=True)
        a.record(s)
        s2.wait_event(a)
        read_unique(s2)
        kv.kv_retrieve_scatter_as(path.retrieve_kind, path.layout, path.staging_ptr, path.layers, path.bt,
                                  w.bt_stride, w.num_reqs, d_jobs, n, s)
        c.record(s2)
        s.wait_event(c)
        b.record(s)
        b.synchronize()
        mixed.append(a.elapsed_time(b))
    t_rd, t_mx = float(np.median(rd)), float(np.median(mixed))
    out["unique_read"] = {"ms": round(t_rd, 4), "GB/s": round(uniq / (t_rd * 1e-3) / 1e9, 1),
                          "what": "the retrieve's unique staged chunks read once (torch reductions), idle GPU"}
    out["writes_with_unique_read"] = {
        "ms": round(t_mx, 4), "GB/s_alg": round((uniq + written) / (t_mx * 1e-3) / 1e9, 1),
        "what": f"the scattered writes alone and the unique reads, concurrently on two streams (median of {reps}): "
                "the retrieve's algorithmic bytes on this pool without the retrieve's own reads"}
    return out


def _store_shape_copy(torch, reps: int = 5) -> dict:
    """A plain contiguous copy run by the store gather's own kernel shape
    (1024-lane workgroups, 16 non-temporal 16-byte loads per lane, then the
    stores): one layer, 8 heads x 128 dims bf16, 16-token blocks, 256-token
    chunks, the [2][NB][B][H][D] paged layout and an identity block table, so
    that each staged chunk's K and V halves are 512 KiB contiguous runs of the
    paged tensor.  4 GiB read and 4 GiB written per launch: the practical
    ceiling of a dense copy in the shape the store runs."""
    import numpy as np
    import paper_2609_35065_amd as kv
    n, seg = 4096, 16 * 8 * 128 * 2            # 4096 chunks of 1 MiB; 32 KiB segments
    nb = 16 * n
    lo = kv.make_layout(1, 8, 128, 2, 16, 256, nb, n, nb * seg, seg)
    stg = torch.empty(n * 32 * seg, dtype=torch.uint8, device="cuda")
    pool = torch.empty(2 * nb * seg, dtype=torch.uint8, device="cuda")
    bt = torch.from_numpy(np.arange(nb, dtype=np.int32).reshape(n, 16)).cuda()
    jobs = torch.from_numpy(np.stack([np.arange(n), np.arange(n), np.zeros(n), np.zeros(n)], 1)
                            .astype(np.int32)).cuda()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    kv.kv_store_gather(lo, stg, [pool], bt, 16, n, jobs, n)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        kv.kv_store_gather(lo, stg, [pool], bt, 16, n, jobs, n)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    del stg, pool
    torch.cuda.empty_cache()
    return {"ms": round(ms, 4), "GB/s_rw": round(2 * n * 32 * seg / (ms * 1e-3) / 1e9, 1),
            "what": "4 GiB contiguous copy by the store gather's kernel (1024-lane workgroups, non-temporal)"}


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
    return {"calibration": "contiguous copy by copy_generic_kernel<true> (the retrieve's generic path, cached "
                           "loads)", "bytes_read_per_dispatch": n * 2 * seg,
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
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the same-pool ceilings and practical-peak copies after the timed steps (kernel "
                         "traces: every launch of a copy kernel is then a step's, a tuning or an idle-GPU pass's)")
    ap.add_argument("--ceiling-only", action="store_true",
                    help="after the warm-up (and the retrieve tuning) run only the retrieve's same-pool ceiling "
                         "launches, print them and exit (the counter passes behind that ceiling)")
    ap.add_argument("--profile-commands", metavar="OUTDIR",
                    help="print the rocprofv3 runs behind the profiles of --workload, writing under OUTDIR "
                         "(name<TAB>command per line), and exit")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="write profiles/kernel_trace_<workload>.md from a rocprofv3 kernel-trace run in DIR "
                         "(with its bench output in DIR/bench.log) and exit; --command names the run")
    ap.add_argument("--summarize-traffic", metavar="DIR",
                    help="write profiles/traffic_*_<workload>.txt from the pmc_fetch, pmc_write, cal_fetch and "
                         "cal_write runs under DIR and exit")
    ap.add_argument("--summarize-ceiling", metavar="DIR",
                    help="write profiles/traffic_retrieve_ceiling_<workload>.txt from the ceil_fetch and ceil_write "
                         "runs under DIR (calibration from --calibration or DIR) and exit")
    ap.add_argument("--summarize-counters", metavar="DIR",
                    help="write profiles/counters_<workload>.md from the sq, tcc, tlb and occ runs under DIR and exit")
    ap.add_argument("--command", default="", help="the command a --summarize-trace run was made with")
    ap.add_argument("--calibration", default=None,
                    help="--summarize-traffic: directory holding the cal_fetch / cal_write runs (default: DIR)")
    args = ap.parse_args()

    if args.profile_commands:
        for name, cmd in profile_commands(args.workload, args.profile_commands):
            print(f"{name}\t{cmd}")
        return 0
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, args.workload, args.command))
        return 0
    if args.summarize_traffic:
        print("\n".join(summarize_traffic(args.summarize_traffic, args.workload, args.calibration)))
        return 0
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters, args.workload))
        return 0
    if args.summarize_ceiling:
        print(summarize_ceiling(args.summarize_ceiling, args.workload, args.calibration))
        return 0

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
    if args.ceiling_only:
        # the last CEILING_LAUNCHES launches of the retrieve kernel in this process are the ceiling's
        print(json.dumps({"workload": w.name, "config": {"retrieve_variant": RETRIEVE_KIND_NAMES.get(path.retrieve_kind),
                                                        "retrieve_tuning_ms": tuning},
                          "ceiling_launches": CEILING_LAUNCHES,
                          "ceiling": _retrieve_write_bound(path, torch, reps=CEILING_REPS)}))
        return 0

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
    payload_rate = (r_bytes + s_bytes) / (ms_step * 1e-3) / 1e9
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
    # the step in HBM bytes: unique staged reads + writes of the retrieve, reads + writes of the store (with
    # the staging buffer in host memory the retrieve's reads cross the host link instead: payload rate)
    hbm_rate = (r_alg + s_bytes) / (ms_step * 1e-3) / 1e9
    value = payload_rate if w.staging_in_host else hbm_rate
    dom = "retrieve" if k_ms["retrieve"] * 1 >= k_ms["store"] else "store"
    dom_kernel = "kv_copy_retrieve" if dom == "retrieve" else "kv_copy_store"
    achieved = r_hbm if dom == "retrieve" else s_gbs
    variant = RETRIEVE_KIND_NAMES.get(path.retrieve_kind)
    traffic = _load_traffic(dom_kernel, args.workload, variant)
    per_kernel = {
        "store_gather": {"symbol": _symbol("store", w), "achieved": round(s_gbs, 1),
                         "frac": round(s_gbs / HBM_PEAK_GBS, 4), "traffic": _load_traffic("kv_copy_store", args.workload)},
        "retrieve_scatter": {"symbol": _symbol(variant, w) if variant else None, "achieved": round(r_hbm, 1),
                             "frac": round(r_hbm / HBM_PEAK_GBS, 4),
                             "traffic": _load_traffic("kv_copy_retrieve", args.workload, variant)},
    }
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
                   "retrieve_variant": variant,
                   "retrieve_tuning_ms": tuning},
        "value_basis": ("payload bytes (staging in host memory) per second of step" if w.staging_in_host else
                        "HBM bytes per second of step: unique staged reads + writes of the retrieve, reads + "
                        "writes of the store"),
        "payload_GB/s": round(payload_rate, 1),
        "roofline": {"bound": "hbm", "kernel": dom_kernel, "symbol": per_kernel[
                         "retrieve_scatter" if dom == "retrieve" else "store_gather"]["symbol"],
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "per_kernel": per_kernel,
                     "min_frac": round(min(v["frac"] for v in per_kernel.values() if v["achieved"]) if any(
                         v["achieved"] for v in per_kernel.values()) else 0.0, 4)},
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
        line["step_hbm_GB/s"] = round(hbm_rate, 1)
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
    extras = not args.no_fill and not args.no_extras
    wb = _retrieve_write_bound(path, torch) if extras else None
    del path
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if extras:
        sc = _store_shape_copy(torch)
        line["practical_peak"] = {"store_shape_copy_GB/s": sc["GB/s_rw"],
                                  "store_frac_of_store_shape_copy": round(s_gbs / sc["GB/s_rw"], 4),
                                  "torch_device_copy_GB/s": round(_device_copy_gbs(torch), 1),
                                  "generic_copy_GB/s": _calibration_copy(torch)["GB/s_rw"]}
        if wb:
            # the retrieve's algorithmic bytes moved at the pool's own scattered-write rate
            wb["alg_bytes_at_this_rate_ms"] = round(r_alg / (wb["GB/s_written"] * 1e9) * 1e3, 4)
            wb["retrieve_frac_of_this_rate"] = round(wb["alg_bytes_at_this_rate_ms"] / k_ms["retrieve"], 4)
            mx = wb["writes_with_unique_read"]
            mx["retrieve_frac_of_this_ceiling"] = round(mx["ms"] / k_ms["retrieve"], 4)
            ix = wb["independent_mix"]
            ix["retrieve_speedup_over_this"] = round(ix["ms"] / k_ms["retrieve"], 4)
            line["practical_peak"]["retrieve_writes_only"] = wb
        if w.staging_in_host:
            line["practical_peak"].update(_host_link_gbs(torch))
        props = torch.cuda.get_device_properties(0)
        line["gpu"] = {"name": props.name, "compute_units": props.multi_processor_count,
                       "memory_GiB": round(props.total_memory / 2**30, 1), "clocks": _clocks()}
    if not args.no_cpu_baseline and not args.no_fill:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cb = _cpu_baseline(w.shape)
        # why a sample: the oracle at this rate would take this long for one whole step of the workload
        full_s = (r_bytes + s_bytes) / (cb["value"] * 1e9) if cb["value"] else None
        cb["full_step_estimate_s"] = round(full_s, 1) if full_s else None
        cb["sample"] += (f"; bounded so that the default run stays within minutes: one whole step of "
                         f"{w.name} moves {(r_bytes + s_bytes) / 2**30:.0f} GiB, about {full_s:.0f} s of single-core "
                         f"oracle work per step at this rate, with {w.pool_bytes() / 2**30 + w.staged_bytes() / 2**30:.0f}"
                         f" GiB of host buffers" if full_s else "")
        line["cpu_baseline"] = cb
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
