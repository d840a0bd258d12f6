"""The rocprofv3 summariser that writes the traffic figures under profiles/ (CPU only, synthetic CSVs).

Counter files record no grid shape, so launches of one kernel that cover different stage counts are
told apart by how much they fetch: the dispatches kept are those within 1/4 of the algorithmic bytes
(scaled by the device copy's reading of the same counter), and the write run's dispatches at the same
ordinals. Kernel traces do record grid shapes and select by grid y."""
import csv
import os

import pytest

from paper_2605_30852_amd import profsum as ps

K = "k_sgemv<unsigned short, 3>"


def _csv(path, rows, header):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        for r in rows:
            w.writerow(r)
    return str(path)


def _counters(tmp_path, fetch_kib, write_kib):
    hdr = ["Kernel_Name", "Counter_Name", "Counter_Value"]
    f = _csv(tmp_path / "f.csv", [["__amd_rocclr_copyBuffer", "FETCH_SIZE", 524288.0]] +
             [[f"void spd::{K}(spd::Ctx, spd::Rows)", "FETCH_SIZE", v] for v in fetch_kib], hdr)
    w = _csv(tmp_path / "w.csv", [["__amd_rocclr_copyBuffer", "WRITE_SIZE", 1048576.0]] +
             [[f"void spd::{K}(spd::Ctx, spd::Rows)", "WRITE_SIZE", v] for v in write_kib], hdr)
    return f, w


def _kv(text):
    return dict(line.split("=", 1) for line in text.splitlines() if "=" in line)


def test_traffic_keeps_the_launches_near_the_algorithmic_bytes(tmp_path):
    # two-stage launches (~97500 KiB fetched), one-stage (half) and four-stage (double) launches mixed
    fetch = [97500, 48750, 97510, 195000, 97490]
    write = [150, 75, 152, 300, 154]
    f, w = _counters(tmp_path, fetch, write)
    algo = 2 * 97500 * 1024  # the copy reads 512 MiB for 1 GiB: fetch scale 2
    out = _kv(ps.traffic(f, w, K, 2, algo, None))
    assert out["dispatches_fetch"] == "3" and out["dispatches_write"] == "3"
    assert float(out["fetch_kib_median"]) == 97500 and float(out["write_kib_median"]) == 152
    assert float(out["scale_fetch"]) == pytest.approx(2.0)
    assert float(out["hbm_bytes_per_launch"]) == pytest.approx((97500 * 2 + 152) * 1024)


def test_traffic_without_algorithmic_bytes_takes_the_largest_cluster(tmp_path):
    f, w = _counters(tmp_path, [100, 98, 50, 99], [1, 2, 3, 4])
    out = _kv(ps.traffic(f, w, K, 2, None, None))
    assert out["selection"].startswith("largest-value cluster")
    assert out["dispatches_fetch"] == "3" and float(out["write_kib_median"]) == 2


def test_traffic_reports_mismatched_runs(tmp_path):
    f, w = _counters(tmp_path, [100, 98], [1])
    assert ps.traffic(f, w, K, 2, 100 * 2 * 1024, None).startswith("incomplete")


def test_trace_selects_by_grid_y(tmp_path):
    hdr = ["Kernel_Name", "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z", "Workgroup_Size_X",
           "Start_Timestamp", "End_Timestamp"]
    rows = [[f"void spd::{K}(spd::Ctx, spd::Rows)", 1024 * 256, y, 1, 256, 0, d * 1000]
            for y, d in [(2, 40), (2, 42), (4, 73), (1, 20)]]
    t = _csv(tmp_path / "t.csv", rows, hdr)
    out = _kv(ps.trace(t, K, 2))
    assert out["dispatches"] == "2" and float(out["mean_us"]) == pytest.approx(41.0)
