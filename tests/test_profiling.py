"""The rocprofv3 summarizers behind the committed profiles (CPU): the traffic
calibration picks the 1 GiB copy among copies of other sizes and scales each
counter by it; the utilization summary turns GRBM/SQ counters into clock, MFMA
busy share, executed work and LDS activity; the kernel statistics table and the
source-hash guard of the traffic file."""
from __future__ import annotations

import csv
import json
import os

import pytest

from paper_2607_14952_amd import profiling as P

CC_FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
             "End_Timestamp"]


def _write_counters(directory, rows):
    os.makedirs(directory, exist_ok=True)
    with open(os.path.join(directory, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=CC_FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(CC_FIELDS, r)))


def _dispatches(counter, values):
    """[(dispatch, kernel, total)] -> rows, each total split over two per-XCD rows."""
    rows = []
    for d, name, v in values:
        rows.append((d, name, counter, v / 2, 0, 1000))
        rows.append((d, name, counter, v / 2, 0, 1000))
    return rows


def test_traffic_calibration_and_scaling(tmp_path):
    gib = 1 << 30
    copy = "__amd_rocclr_copyBuffer"
    fetch = [(1, copy, gib / 2 / 1024), (2, "kernel_a", 1000.0), (3, "kernel_a", 1200.0),
             (4, copy, 4 * gib / 2 / 1024)]
    write = [(1, copy, gib / 1024), (2, "kernel_a", 500.0), (3, "kernel_a", 500.0),
             (4, copy, 4 * gib / 1024)]
    _write_counters(tmp_path / "f", _dispatches("FETCH_SIZE", fetch))
    _write_counters(tmp_path / "w", _dispatches("WRITE_SIZE", write))
    out = tmp_path / "traffic.json"
    doc = P.write_traffic(str(tmp_path / "f"), str(tmp_path / "w"), str(out), gib, "cmd")
    assert doc["scale"]["FETCH_SIZE"] == pytest.approx(2.0)      # the 1 GiB copy, not the 4 GiB one
    assert doc["scale"]["WRITE_SIZE"] == pytest.approx(1.0)
    a = doc["kernels"]["kernel_a"]
    assert a["dispatches"] == 2
    assert a["hbm_bytes_per_dispatch"] == pytest.approx(1100 * 1024 * 2 + 500 * 1024)
    # the guard: bytes for the current sources, none once the hash differs
    assert P.traffic_for("kernel_a", str(out)) == pytest.approx(a["hbm_bytes_per_dispatch"])
    stale = json.loads(out.read_text())
    stale["source_hash"] = "0" * 16
    out.write_text(json.dumps(stale))
    assert P.traffic_for("kernel_a", str(out)) is None
    assert P.traffic_for("kernel_a", str(tmp_path / "missing.json")) is None


def test_util_summary(tmp_path):
    ns = 10_000_000                       # one 10 ms dispatch
    gui = 1.8e9 * 1e-2                    # cycles per XCD at 1.8 GHz
    vals = {"GRBM_GUI_ACTIVE": 8 * gui, "SQ_VALU_MFMA_BUSY_CYCLES": 0.5 * 1024 * gui,
            "SQ_INSTS_VALU_MFMA_MOPS_BF16": 10e12 / 512, "SQ_BUSY_CYCLES": 1.0,
            "SQ_LDS_IDX_ACTIVE": 0.3 * 256 * gui, "SQ_LDS_BANK_CONFLICT": 0.01 * 256 * gui}
    rows = [(7, "the_kernel", c, v, 0, ns) for c, v in vals.items()]
    _write_counters(tmp_path / "u", rows)
    out = tmp_path / "util.md"
    P.write_util_md(str(tmp_path / "u"), str(out), "cmd", "title")
    line = [l for l in out.read_text().splitlines() if l.startswith("| `the_kernel`")][0]
    cells = [c.strip() for c in line.strip("|").split("|")]
    # kernel | dispatches | ms | clock | busy % | TFLOP | TFLOP/s | % of peak at clock | LDS % | conflict %
    assert cells[1:] == ["1", "10.000", "1.80", "50.0", "10.00", "1000", "53.3", "30.0", "1.00"]


def test_stats_table(tmp_path):
    d = tmp_path / "s"
    d.mkdir()
    with open(d / "run_kernel_stats.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "MinNs", "MaxNs", "Percentage"])
        w.writerow(["k_fast", 3, 3_000_000, 1_000_000, 900_000, 1_100_000, 25.0])
        w.writerow(["k_slow", 2, 9_000_000, 4_500_000, 4_000_000, 5_000_000, 75.0])
    with open(d / "run_kernel_trace.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        for s, e in ((0, 900_000), (10, 1_000_010), (20, 1_100_020)):
            w.writerow(["k_fast", s, e])
        for s, e in ((0, 4_000_000), (0, 5_000_000)):
            w.writerow(["k_slow", s, e])
    out = tmp_path / "stats.md"
    P.write_stats_md(str(d), str(out), "cmd", "title")
    text = out.read_text()
    assert "cmd" in text and P.source_hash() in text
    rows = [l for l in text.splitlines() if l.startswith("| `k_")]
    assert rows[0].startswith("| `k_slow`"), "sorted by total time"
    fast = [c.strip() for c in rows[1].strip("|").split("|")]
    assert fast[1:4] == ["3", "1.000", "1.000"]                   # calls, average, median
    assert "long launches" not in text                            # no kernel of mixed sizes


def test_long_launches():
    ms = 1e6
    # three shard-sized launches and one short one over the response keys
    assert P.long_launches([22 * ms, 21 * ms, 23 * ms, 0.3 * ms]) == (3, pytest.approx(22 * ms))
    assert P.long_launches([22 * ms, 21 * ms]) is None            # one size
    assert P.long_launches([0.5 * ms, 0.01 * ms]) is None         # all short
    assert P.long_launches([]) is None
