"""The profile summaries under profiles/ are made from rocprofv3 output by
bench.py (--summarize-trace, --summarize-traffic, --summarize-counters); these
tests check, without a GPU, that every kernel they name is a __global__
function of the library's sources and that the summaries scale and label
rocprofv3's numbers as documented."""
import csv
import os
import re
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import workloads as W  # noqa: E402

CSRC = os.path.join(ROOT, "paper_2609_35065_amd", "csrc")


def _globals():
    names = set()
    for f in os.listdir(CSRC):
        if f.endswith(".hip"):
            text = open(os.path.join(CSRC, f)).read()
            names |= set(re.findall(r"__global__\s+(?:__launch_bounds__\(\w+\)\s+)?void\s+(\w+)\s*\(", text))
    return names


@pytest.mark.parametrize("name", sorted(W.CONFIGS))
def test_every_symbol_is_a_kernel_of_the_library(name):
    w = W.make(name)
    kernels = _globals()
    for kind in ("store", "unit", "pair", "quad", "stream"):
        sym = bench._symbol(kind, w)
        assert sym.split("<")[0] in kernels, (kind, sym)
        assert bench._label(sym) != "other"


def test_symbols_follow_the_segment_size():
    w = W.make("l32-64x4096")                        # 32 KiB segments
    assert bench._symbol("store", w) == "group_copy_kernel<1024, 2, false>"
    assert bench._symbol("quad", w) == "retrieve_quad_kernel<8>"
    t = W.tiny()                                     # 4 KiB segments
    assert bench._symbol("pair", t) == "retrieve_unit_kernel<1>"   # the pair walk runs at 32 KiB only
    assert bench._symbol("stream", t) == "group_copy_kernel<256, 1, true>"


def _write_csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=list(rows[0]))
        wr.writeheader()
        wr.writerows(rows)


def test_trace_summary_names_label_and_symbol(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    d = tmp_path / "ktrace"
    _write_csv(str(d / "host" / "c_kernel_stats.csv"), [
        {"Name": "tkv::(anonymous namespace)::group_copy_kernel<1024, 2, false>(tkv::CopyParams)", "Calls": "10",
         "TotalDurationNs": "57000000", "AverageNs": "5700000", "MinNs": "5600000", "MaxNs": "5800000"},
        {"Name": "void at::native::elementwise_kernel<128, 4>(int, float)", "Calls": "3",
         "TotalDurationNs": "3000", "AverageNs": "1000", "MinNs": "900", "MaxNs": "1100"}])
    path = bench.summarize_trace(str(d), "w", "rocprofv3 ... -- python3 bench.py")
    text = open(path).read()
    assert "| store gather (kv_store_gather) | `group_copy_kernel<1024, 2, false>` | 10 | 5700.0 |" in text
    assert "Other kernels: 1 names" in text


def test_traffic_summary_scales_by_the_calibration(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    d = tmp_path / "prof"
    store = "tkv::(anonymous namespace)::group_copy_kernel<1024, 2, false>(tkv::CopyParams)"
    quad = "tkv::(anonymous namespace)::retrieve_quad_kernel<8>(tkv::CopyParams)"
    cal = "tkv::(anonymous namespace)::copy_generic_kernel<true>(tkv::CopyParams)"
    row = lambda k, c, v: {"Kernel_Name": k, "Counter_Name": c, "Counter_Value": str(v)}
    _write_csv(str(d / "pmc_fetch" / "c_counter_collection.csv"), [row(store, "FETCH_SIZE", 100), row(quad, "FETCH_SIZE", 10)])
    _write_csv(str(d / "pmc_write" / "c_counter_collection.csv"), [row(store, "WRITE_SIZE", 200), row(quad, "WRITE_SIZE", 50)])
    _write_csv(str(d / "cal_fetch" / "c_counter_collection.csv"), [row(cal, "FETCH_SIZE", (4 << 20) / 2)])
    _write_csv(str(d / "cal_write" / "c_counter_collection.csv"), [row(cal, "WRITE_SIZE", 4 << 20)])
    (d / "pmc_fetch.log").write_text('{"config": {"retrieve_variant": "quad"}}\n')
    paths = bench.summarize_traffic(str(d), "l32-64x4096")
    vals = {}
    for p in paths:
        kv = dict(l.strip().split("=", 1) for l in open(p) if "=" in l and not l.startswith("#"))
        vals[kv["kernel"]] = kv
    # FETCH_SIZE reads half the calibration's bytes: scale 2; WRITE_SIZE exact: scale 1
    assert float(vals["kv_copy_store"]["hbm_read_bytes_per_launch"]) == 200 * 1024
    assert float(vals["kv_copy_store"]["hbm_write_bytes_per_launch"]) == 200 * 1024
    assert vals["kv_copy_retrieve_quad"]["symbol"] == "retrieve_quad_kernel<8>"
    assert float(vals["kv_copy_retrieve_quad"]["traffic_bytes_per_launch"]) == (20 + 50) * 1024
    # the bench line reads them back only while the copy sources are unchanged
    assert bench._load_traffic("kv_copy_retrieve", "l32-64x4096", "quad") == (20 + 50) * 1024
    assert bench._load_traffic("kv_copy_retrieve", "l32-64x4096", "pair") is None


def test_ceiling_summary_takes_the_ceiling_launches(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    d = tmp_path / "prof"
    quad = "tkv::(anonymous namespace)::retrieve_quad_kernel<8>(tkv::CopyParams)"
    red = "void at::native::reduce_kernel<512, 1>(at::native::ReduceOp<long>)"
    cal = "tkv::(anonymous namespace)::copy_generic_kernel<true>(tkv::CopyParams)"
    n = bench.CEILING_LAUNCHES

    def rows(ctr, real, ceil, reader):
        out, i = [], 0
        for v in [real] * 5 + [ceil] * n:          # warm-up and tuning launches first, then the ceiling's
            i += 1
            out.append({"Dispatch_Id": str(i), "Kernel_Name": quad, "Counter_Name": ctr, "Counter_Value": str(v)})
        for _ in range(n):                          # one reduction per read pass
            i += 1
            out.append({"Dispatch_Id": str(i), "Kernel_Name": red, "Counter_Name": ctr, "Counter_Value": str(reader)})
        for v in mixed:                             # the independent-mix probe's launches
            i += 1
            out.append({"Dispatch_Id": str(i), "Kernel_Name": mix, "Counter_Name": ctr, "Counter_Value": str(v)})
        return out

    mix = ("tkv::(anonymous namespace)::mixed_traffic_kernel(tkv::CopyParams, int const*, int, long, long, "
           "unsigned int)")
    mixed = [120, 100, 110]
    _write_csv(str(d / "ceil_fetch" / "c_counter_collection.csv"), rows("FETCH_SIZE", 1000, 10, 100))
    mixed = [4100, 4100, 4000]
    _write_csv(str(d / "ceil_write" / "c_counter_collection.csv"), rows("WRITE_SIZE", 4000, 4000, 0))
    row = lambda c, v: {"Dispatch_Id": "1", "Kernel_Name": cal, "Counter_Name": c, "Counter_Value": str(v)}
    _write_csv(str(d / "cal_fetch" / "c_counter_collection.csv"), [row("FETCH_SIZE", (4 << 20) / 2)])
    _write_csv(str(d / "cal_write" / "c_counter_collection.csv"), [row("WRITE_SIZE", 4 << 20)])
    (d / "ceil_fetch.log").write_text('{"config": {"retrieve_variant": "quad"}, "ceiling_launches": %d, '
                                      '"ceiling": {"ms": 3.2}}\n' % n)
    path = bench.summarize_ceiling(str(d), "l32-64x4096")
    kv = dict(l.strip().split("=", 1) for l in open(path) if "=" in l and not l.startswith("#"))
    assert kv["symbol"] == "retrieve_quad_kernel<8>"
    assert float(kv["writes_only_hbm_read_bytes_per_launch"]) == 10 * 2 * 1024      # FETCH_SIZE scale 2
    assert float(kv["writes_only_hbm_write_bytes_per_launch"]) == 4000 * 1024
    assert float(kv["unique_read_hbm_read_bytes_per_pass"]) == 100 * 2 * 1024
    assert int(kv["retrieve_launches_in_run"]) == 5 + n
    assert float(kv["independent_mix_hbm_read_bytes_per_launch"]) == 110 * 2 * 1024     # median, scaled
    assert float(kv["independent_mix_hbm_write_bytes_per_launch"]) == 4100 * 1024
    assert bench._label("mixed_traffic_kernel") != "other"
    # no ceiling measured (streaming retrieve, or staged chunks in host memory): no file
    (d / "ceil_fetch.log").write_text('{"config": {"retrieve_variant": "stream"}, "ceiling_launches": %d, '
                                      '"ceiling": null}\n' % n)
    assert bench.summarize_ceiling(str(d), "l32-64x4096") is None
