"""Host-side logic of bench.py (CPU only): the rocprofv3 counter summary with
its copy calibration, the source-hash gate on reported traffic, the kernel-trace
summary and the algorithmic byte counts."""
import csv
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _counter_csv(path, rows):
    """rows of (kernel, counter, value, dispatch id)"""
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                           "Counter_Value"])
        w.writeheader()
        for k, c, v, d in rows:
            w.writerow({"Dispatch_Id": d, "Kernel_Name": k, "Counter_Name": c,
                        "Counter_Value": v})


def test_pmc_summary_scales_by_the_copy(tmp_path):
    """A 1 MiB copy that reads 512 KiB (FETCH) and writes 1024 KiB (WRITE) gives
    factors 2 and 1; a kernel's HBM bytes are the scaled sum of its first
    dispatch's counters (the timed step's; rows may come in any order)."""
    f, w = tmp_path / "f.csv", tmp_path / "w.csv"
    sym = bench.PMC_KERNELS["k_kahn"][0]
    _counter_csv(f, [("__amd_rocclr_copyBuffer", "FETCH_SIZE", 512.0, 1),
                     (sym + "int)", "FETCH_SIZE", 300.0, 9), (sym + "int)", "FETCH_SIZE", 100.0, 4)])
    _counter_csv(w, [("__amd_rocclr_copyBuffer", "WRITE_SIZE", 1024.0, 1),
                     (sym + "int)", "WRITE_SIZE", 70.0, 9), (sym + "int)", "WRITE_SIZE", 50.0, 4)])
    out = bench.pmc_summary(str(f), str(w), 1)
    assert "factors fetch 2.0000 write 1.0000" in out
    row = next(line for line in out.splitlines() if line.startswith("| k_kahn |"))
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[1] == bench.source_hash(bench.PMC_KERNELS["k_kahn"][1])
    assert cells[2] == "2" and float(cells[3]) == 100.0 and float(cells[4]) == 50.0
    assert float(cells[5]) == (100.0 * 2 + 50.0 * 1) * 1024


def test_traffic_only_while_the_sources_match(tmp_path, monkeypatch):
    h = bench.source_hash(bench.PMC_KERNELS["k_kahn"][1])
    p = tmp_path / "t.md"
    p.write_text(f"| k_kahn | {h} | 1 | 1 | 1 | 12345 | |\n"
                 f"| k_place | 0000000000000000 | 1 | 1 | 1 | 777 | |\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILES", [str(p)])
    assert bench.load_traffic("k_kahn") == 12345.0
    assert bench.load_traffic("k_place") is None          # stale hash
    assert bench.load_traffic("k_makespan_one") is None  # no row
    assert bench.load_traffic("not_a_kernel") is None


def test_stats_summary_orders_by_total(tmp_path):
    p = tmp_path / "s.csv"
    with open(p, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs"])
        w.writeheader()
        w.writerow({"Name": "a(int)", "Calls": 2, "TotalDurationNs": 2e6, "AverageNs": 1e6})
        w.writerow({"Name": "b(int)", "Calls": 1, "TotalDurationNs": 5e6, "AverageNs": 5e6})
    lines = bench.stats_summary(str(p)).splitlines()
    assert lines[2].startswith("| b |") and lines[3].startswith("| a |")
    assert "| 5.000 | 5000.0 |" in lines[2]


def test_algorithmic_bytes():
    n, m = 1000, 3000
    assert bench.algorithmic_bytes("k_blevel_sweep", n, m, 1) == 32 * n + 12 * m
    assert bench.algorithmic_bytes("k_makespan_one", n, m, 1) == 33 * n + 21 * m
    assert bench.algorithmic_bytes("k_makespan_batch", n, m, 5) == 24 * n + 12 * m + 5 * (9 * n + 9 * m)
    assert bench.algorithmic_bytes("k_kahn", n, m, 1) is None
