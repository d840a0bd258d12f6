"""The rocprofv3 summariser that writes the traffic figures under profiles/ (CPU only, synthetic CSVs).

Counter files record only a dispatch's total grid size, which is the same for a stage launch over one,
two or four stages (every stage launch has the same number of workgroups), so a selection by grid y
takes the dispatch ids of the matching dispatches from the kernel trace of the same counter run, which
records the grid shape, or keeps the dispatches of one measured phase, which a profiling run brackets
with marker dispatches of the read-probe kernel. Nothing is selected by the measured values
themselves."""
import csv

import pytest

from paper_2605_30852_amd import profsum as ps

K = "k_sgemv<unsigned short, 3>"
NAME = f"void spd::{K}(spd::Ctx, spd::Rows)"


def _csv(path, rows, header):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        for r in rows:
            w.writerow(r)
    return str(path)


def _run(tmp_path, tag, counter, copy_value, dispatches):
    """dispatches: (dispatch id, grid y, counter value) of the kernel; returns (counter csv, trace csv)."""
    hdr = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value"]
    rows = [[1, 1 << 28, "__amd_rocclr_copyBuffer", counter, copy_value]]
    rows += [[i, 1024 * 256, NAME, counter, v] for i, _, v in dispatches]
    c = _csv(tmp_path / f"{tag}_counter.csv", rows, hdr)
    thdr = ["Dispatch_Id", "Kernel_Name", "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z", "Start_Timestamp",
            "End_Timestamp"]
    trows = [[1, "__amd_rocclr_copyBuffer", 1 << 28, 1, 1, 0, 10]]
    trows += [[i, NAME, 1024 * 256 // y, y, 1, 0, 10] for i, y, _ in dispatches]
    t = _csv(tmp_path / f"{tag}_trace.csv", trows, thdr)
    return c, t


def _kv(text):
    return dict(line.split("=", 1) for line in text.splitlines() if "=" in line)


def test_traffic_selects_dispatches_by_id_from_the_same_runs_trace(tmp_path):
    # four-stage (grid y 4), two-stage and one-stage launches mixed; the fetch run and the write run
    # issue their dispatches under different ids
    f, ft = _run(tmp_path, "f", "FETCH_SIZE", 524288.0,
                 [(10, 4, 195000), (11, 2, 97500), (12, 4, 195010), (13, 1, 48000), (14, 4, 194990)])
    w, wt = _run(tmp_path, "w", "WRITE_SIZE", 1048576.0,
                 [(20, 4, 300), (21, 2, 150), (22, 4, 302), (23, 1, 75), (24, 4, 304)])
    algo = 2 * 195000 * 1024
    out = _kv(ps.traffic(f, w, K, 4, algo, None, ft, wt))
    assert out["dispatches_fetch"] == "3" and out["dispatches_write"] == "3"
    assert float(out["fetch_kib_median"]) == 195000 and float(out["write_kib_median"]) == 302
    assert float(out["scale_fetch"]) == pytest.approx(2.0) and float(out["scale_write"]) == pytest.approx(1.0)
    assert float(out["hbm_bytes_per_launch"]) == pytest.approx((195000 * 2 + 302) * 1024)
    assert "dispatch id" in out["selection"]


def test_traffic_refuses_a_grid_selection_without_traces(tmp_path):
    f, _ = _run(tmp_path, "f", "FETCH_SIZE", 524288.0, [(10, 4, 195000), (11, 2, 97500)])
    w, _ = _run(tmp_path, "w", "WRITE_SIZE", 1048576.0, [(20, 4, 300), (21, 2, 150)])
    assert ps.traffic(f, w, K, 4, None, None).startswith("incomplete")


def test_traffic_of_every_dispatch(tmp_path):
    f, _ = _run(tmp_path, "f", "FETCH_SIZE", 524288.0, [(10, 1, 100), (11, 1, 98), (12, 1, 99)])
    w, _ = _run(tmp_path, "w", "WRITE_SIZE", 1048576.0, [(20, 1, 1), (21, 1, 2), (22, 1, 3)])
    out = _kv(ps.traffic(f, w, K, None, None, None))
    assert out["selection"] == "all dispatches" and out["dispatches_fetch"] == "3"
    assert float(out["write_kib_median"]) == 2


def test_trace_selects_by_grid_y(tmp_path):
    hdr = ["Kernel_Name", "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z", "Workgroup_Size_X",
           "Start_Timestamp", "End_Timestamp"]
    rows = [[NAME, 1024 * 256, y, 1, 256, 0, d * 1000] for y, d in [(2, 40), (2, 42), (4, 73), (1, 20)]]
    t = _csv(tmp_path / "t.csv", rows, hdr)
    out = _kv(ps.trace(t, K, 2))
    assert out["dispatches"] == "2" and float(out["mean_us"]) == pytest.approx(41.0)


def test_traffic_selects_a_phase_between_markers(tmp_path):
    """Phase k lies between marker groups 2k and 2k+1 (runs of consecutive read-probe dispatches):
    same-named dispatches before, between and after the phases are left out, whatever their values."""
    hdr = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value"]
    probe = "void spd::k_read_probe(uint4 const*, unsigned long, float*)"

    def run(tag, counter, copy_value, scale):
        rows = [[1, 1 << 28, "__amd_rocclr_copyBuffer", counter, copy_value]]
        seq = [("k", 50), ("m", 0), ("m", 0), ("k", 100), ("k", 102), ("m", 0), ("m", 0), ("k", 7),
               ("m", 0), ("m", 0), ("k", 400), ("k", 404), ("k", 399), ("m", 0), ("m", 0), ("k", 50),
               ("m", 0), ("m", 0)]  # the last pair: the closing probe
        for i, (what, v) in enumerate(seq):
            rows.append([10 + i, 1024 * 256, NAME if what == "k" else probe, counter, v * scale])
        rows.reverse()  # the file's row order is not the dispatch order
        return _csv(tmp_path / f"{tag}.csv", rows, hdr)

    f = run("f", "FETCH_SIZE", 524288.0, 1000)
    w = run("w", "WRITE_SIZE", 1048576.0, 1)
    out0 = _kv(ps.traffic(f, w, K, None, None, None, phase=0))
    assert out0["dispatches_fetch"] == "2" and float(out0["fetch_kib_median"]) == 101000
    out1 = _kv(ps.traffic(f, w, K, None, None, None, phase=1))
    assert out1["dispatches_write"] == "3" and float(out1["write_kib_median"]) == 400
    assert "phase 1" in out1["selection"]
    assert ps.traffic(f, w, K, None, None, None, phase=2).startswith("incomplete")


def test_counters_summary_with_mfma_share(tmp_path):
    """Several counters per dispatch (one row each): medians per counter, the MFMA busy share of the
    dispatch's active cycles on every SIMD, and the MOPS counter scaled to operations."""
    hdr = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value"]
    rows = []
    for i, (busy, active, mops) in enumerate([(400, 10, 100), (600, 10, 300), (500, 10, 200)]):
        for name, v in (("SQ_VALU_MFMA_BUSY_CYCLES", busy), ("GRBM_GUI_ACTIVE", active),
                        ("SQ_INSTS_VALU_MFMA_MOPS_F32", mops)):
            rows.append([100 + i, 256, NAME, name, v])
    rows.append([200, 256, "other", "GRBM_GUI_ACTIVE", 1])
    c = _csv(tmp_path / "m.csv", rows, hdr)
    out = _kv(ps.counters(c, K, None, 100))
    assert out["GRBM_GUI_ACTIVE_dispatches"] == "3"
    assert float(out["mfma_busy_share_median"]) == pytest.approx(0.5)
    assert float(out["f32_mfma_flop_median"]) == 512 * 200
