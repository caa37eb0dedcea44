"""Host-side logic of bench.py: argument handling that must not touch the GPU,
the counter-summary arithmetic (scaling each counter by the copy kernel's
reading for a known byte count) and the labelling of kernel-trace groups."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def _write_counters(path, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, cname, val in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": cname, "Counter_Value": val})


def test_summarize_pmc_scales_by_the_copy_kernel(tmp_path, monkeypatch):
    wl = workloads.WORKLOADS["classifier_4096x1000"]
    kib_each_way = 4.0 * wl.elements / 1024.0
    soft = "void smx::k_wave_row<4, true>(float const*, float*, long, long)"
    copy = "smx::k_copy4(float const*, float*, long)"
    # FETCH_SIZE reads half the bytes for both kernels; the softmax kernel
    # fetches 1% more than the copy.  WRITE_SIZE reads the bytes written.
    _write_counters(tmp_path / "fetch",
                    [(soft, "FETCH_SIZE", 0.505 * kib_each_way)] * 3
                    + [(copy, "FETCH_SIZE", 0.5 * kib_each_way)] * 3)
    _write_counters(tmp_path / "write",
                    [(soft, "WRITE_SIZE", kib_each_way)] * 3
                    + [(copy, "WRITE_SIZE", kib_each_way)] * 3)
    _write_counters(tmp_path / "occ",
                    [(soft, "OccupancyPercent", 40.0), (soft, "SQ_WAVES", 4096.0),
                     (soft, "GRBM_GUI_ACTIVE", 1e4), (copy, "OccupancyPercent", 50.0),
                     (copy, "SQ_WAVES", 4000.0), (copy, "GRBM_GUI_ACTIVE", 1.2e4)])
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path / "profiles"))
    doc = bench.summarize_pmc(str(tmp_path), wl, "cmd")
    assert doc["scale_fetch"] == pytest.approx(2.0)
    assert doc["scale_write"] == pytest.approx(1.0)
    assert doc["traffic_fetch_bytes_per_launch"] == pytest.approx(1.01 * 4 * wl.elements)
    assert doc["traffic_write_bytes_per_launch"] == pytest.approx(4 * wl.elements)
    assert doc["traffic_over_algorithmic"] == pytest.approx(1.005)
    assert doc["softmax_occupancy_percent"] == 40.0
    assert doc["copy_sq_waves_per_dispatch"] == 4000.0
    with open(tmp_path / "profiles" / f"pmc_{wl.key}.json") as f:
        assert json.load(f)["source_sha256"] == bench.kernel_source_sha256()
    md = (tmp_path / "profiles" / f"pmc_{wl.key}.md").read_text()
    assert "k_wave_row" in md and "Occupancy" in md


def test_traffic_is_withheld_when_sources_changed(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    with open(tmp_path / "pmc_x.json", "w") as f:
        json.dump({"source_sha256": "0" * 64, "traffic_bytes_per_launch": 1.0}, f)
    assert bench.load_traffic("x") == (None, "kernel changed since the counters were taken")
    with open(tmp_path / "pmc_x.json", "w") as f:
        json.dump({"source_sha256": bench.kernel_source_sha256(),
                   "traffic_bytes_per_launch": 5.0}, f)
    assert bench.load_traffic("x") == (5.0, None)
    assert bench.load_traffic("missing") == (None, None)


def _write_trace(path, rows):
    os.makedirs(path, exist_ok=True)
    fields = ["Kernel_Name", "Grid_Size_X", "Start_Timestamp", "End_Timestamp", "VGPR_Count",
              "SGPR_Count", "LDS_Block_Size", "Scratch_Size"]
    with open(os.path.join(path, "run_kernel_trace.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        for name, grid, b, e in rows:
            w.writerow({"Kernel_Name": name, "Grid_Size_X": grid, "Start_Timestamp": b,
                        "End_Timestamp": e, "VGPR_Count": 56, "SGPR_Count": 32,
                        "LDS_Block_Size": 512, "Scratch_Size": 0})
    with open(os.path.join(path, "run_kernel_stats.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "AverageNs", "MinNs", "MaxNs"])
        w.writeheader()
        w.writerow({"Name": rows[0][0], "Calls": len(rows), "AverageNs": 1000, "MinNs": 900,
                    "MaxNs": 1100})


def test_summarize_trace_and_lookup(tmp_path, monkeypatch):
    """Dispatch durations are grouped by (kernel, grid) into runs, written to
    the trace JSON, and read back for a plan's kernel while the sources are
    unchanged."""
    # as the profiler prints it: every row kernel ends with its row-phase flag
    name = "smx::k_split_onepass<256, 8, true, 0, false>"
    full = f"void {name}(float const*, float*)"
    # 10 calls of 20..29 us, then (after a 1 s gap) 5 more of 40 us
    rows = [(full, 524288, 1000 + i * 100_000, 1000 + i * 100_000 + (20 + i) * 1000)
            for i in range(10)]
    rows += [(full, 524288, 2_000_000_000 + i * 100_000, 2_000_000_000 + i * 100_000 + 40_000)
             for i in range(5)]
    rows += [("Cijk_other_library_kernel", 64, 0, 5000)]
    _write_trace(tmp_path / "trace", rows)
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path / "profiles"))
    monkeypatch.setattr(bench, "TRACE_JSON", str(tmp_path / "profiles" / "trace_bench.json"))
    bench.summarize_trace(str(tmp_path / "trace"), "cmd", None)
    doc = json.load(open(tmp_path / "profiles" / "trace_bench.json"))
    runs = [k for k in doc["kernels"] if k["kernel"] == name]
    assert [r["calls"] for r in runs] == [10, 5]
    assert runs[0]["median_us"] == pytest.approx(24.5)
    plan = {"kernel_name": "split_row", "elems_per_lane": 32, "vec_width": 4,
            "block_threads": 256, "lanes_per_row": 256}
    assert bench.plan_kernel_name(plan, 32768) == name
    assert bench.plan_kernel_name(plan, 32765) == "smx::k_split_onepass<256, 8, true, 0, true>"
    assert bench.plan_kernel_name(dict(plan, vec_width=1), 32765).endswith("false, 0, false>")
    wave = {"kernel_name": "wave_row", "elems_per_lane": 16, "vec_width": 4,
            "block_threads": 256, "lanes_per_row": 64}
    assert bench.plan_kernel_name(wave, 1000) == "smx::k_wave_row<4, true, 0, false>"
    packed = {"kernel_name": "packed", "elems_per_lane": 13, "vec_width": 4,
              "block_threads": 256, "lanes_per_row": 4}
    assert bench.plan_kernel_name(packed, 50) == "smx::k_packed<4, 13, true, 0>"
    st = bench.kernel_trace_stats(name, 524288)
    assert st["calls"] == 10 and st["p10_us"] < st["median_us"] < st["p90_us"]
    doc["source_sha256"] = "0" * 64
    json.dump(doc, open(tmp_path / "profiles" / "trace_bench.json", "w"))
    assert "note" in bench.kernel_trace_stats(name, 524288)
