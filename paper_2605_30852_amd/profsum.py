"""Condense rocprofv3 CSV output (``-f csv``) into the short text summaries kept with the project.

    python -m paper_2605_30852_amd.profsum stats KERNEL_STATS.csv [--top N]
    python -m paper_2605_30852_amd.profsum trace KERNEL_TRACE.csv --kernel NAME [--grid-y Y]
    python -m paper_2605_30852_amd.profsum counters COUNTERS.csv --kernel NAME [--phase K] [--simds N]
    python -m paper_2605_30852_amd.profsum traffic FETCH.csv WRITE.csv --kernel NAME
        [--phase K | --grid-y Y --fetch-trace KT.csv --write-trace KT.csv] [--algo-bytes B] [--source CSRC_DIR]

`stats` prints the per-kernel table; `trace` the duration of the dispatches of one kernel (a
substring of its name, optionally only those whose grid has Y workgroups in y, e.g. the two-stage
group launches); `traffic` the HBM bytes per dispatch of that kernel from a FETCH_SIZE run and a
WRITE_SIZE run, each scaled by what the same counter reads for the largest device copy in the run
(a 1 GiB copy reads and writes 2^30 bytes), as key=value lines. The counter files record only the
total grid size, which is the same for a stage launch over one, two or four stages, so dispatches
are selected by identity: `--phase K` keeps those of the run's K-th measured phase, which a
profiling run of bench.py brackets with marker dispatches of the library's read-probe kernel; a
grid-y selection takes the dispatch ids from a kernel trace of the same run. Pure text processing:
it reads the CSV files only."""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import statistics
import sys

GIB_KIB = float(1 << 20)


def _rows(path):
    with open(path, newline="") as f:
        yield from csv.DictReader(f)


def _grid_y(r):
    for k in ("Grid_Size_Y", "Grid_Y"):
        if k in r and r[k] not in (None, ""):
            return int(r[k])
    return None


def _match(r, kernel, grid_y):
    if kernel not in r.get("Kernel_Name", ""):
        return False
    return grid_y is None or _grid_y(r) == grid_y


def stats(path, top):
    rows = list(_rows(path))
    out = ["| kernel | calls | average us | total ms | share |", "|---|---:|---:|---:|---:|"]
    for r in rows[:top]:
        out.append(f"| `{r['Name']}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f}% |")
    return "\n".join(out)


def trace(path, kernel, grid_y):
    d = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in _rows(path) if _match(r, kernel, grid_y)]
    if not d:
        return f"no dispatch of {kernel!r} (grid y {grid_y})"
    return (f"kernel={kernel}\ngrid_y={grid_y}\ndispatches={len(d)}\nmean_us={statistics.mean(d):.2f}\n"
            f"median_us={statistics.median(d):.2f}\nmin_us={min(d):.2f}\nmax_us={max(d):.2f}")


def _dispatch_ids(trace_path, kernel, grid_y):
    """Dispatch ids of the kernel's dispatches with grid_y workgroups in y, from a kernel trace."""
    return {r["Dispatch_Id"] for r in _rows(trace_path) if _match(r, kernel, grid_y)}


def _counter(path, kernel, grid_y, ids=None):
    """Values of the kernel's dispatches in dispatch order and the largest device copy's value. With
    ids (dispatch ids from a kernel trace of the same run) only those dispatches count; otherwise the
    grid-y selection needs grid dimensions in the file itself (None if it has none)."""
    vals, copies, has_y = [], [], False
    for r in _rows(path):
        v = float(r["Counter_Value"])
        has_y = has_y or _grid_y(r) is not None
        if ids is not None:
            if kernel in r.get("Kernel_Name", "") and r["Dispatch_Id"] in ids:
                vals.append(v)
        elif _match(r, kernel, grid_y if _grid_y(r) is not None else None):
            vals.append(v)
        if "copyBuffer" in r.get("Kernel_Name", ""):
            copies.append(v)
    if grid_y is not None and ids is None and not has_y:
        return None, (max(copies) if copies else None)
    return vals, (max(copies) if copies else None)


MARKER = "k_read_probe"


def _phase_ids(path, phase):
    """Dispatch ids between the run's phase markers: the dispatches of the library's read-probe kernel
    that a profiling run issues around each measured phase (one group of consecutive probe dispatches
    before the phase, one after). Phase k lies between marker groups 2k and 2k + 1, in dispatch
    order; the selection depends on dispatch order and kernel names only."""
    rows = sorted(_rows(path), key=lambda r: int(r["Dispatch_Id"]))
    groups, cur = [], None  # (first index, last index) of each run of marker dispatches
    for i, r in enumerate(rows):
        if MARKER in r.get("Kernel_Name", ""):
            if cur is not None and cur[1] == i - 1:
                cur[1] = i
            else:
                cur = [i, i]
                groups.append(cur)
    if len(groups) < 2 * phase + 2:
        return None
    lo, hi = groups[2 * phase][1], groups[2 * phase + 1][0]
    return {rows[i]["Dispatch_Id"] for i in range(lo + 1, hi)}


def counters(path, kernel, phase=None, simds=None):
    """Median per dispatch of every counter in a counter file, over the kernel's dispatches (those of
    measured phase k with phase=k). With simds (the GPU's SIMD count), SQ_VALU_MFMA_BUSY_CYCLES is also
    given as a share of the dispatch's GRBM_GUI_ACTIVE cycles on every SIMD, and the MFMA floating
    point operations from the MOPS counters (each counts 512 operations)."""
    ids = _phase_ids(path, phase) if phase is not None else None
    if phase is not None and ids is None:
        return f"incomplete: fewer than {2 * phase + 2} phase markers"
    per = {}
    for r in _rows(path):
        if kernel not in r.get("Kernel_Name", "") or (ids is not None and r["Dispatch_Id"] not in ids):
            continue
        per.setdefault(r["Counter_Name"], {}).setdefault(r["Dispatch_Id"], 0.0)
        per[r["Counter_Name"]][r["Dispatch_Id"]] += float(r["Counter_Value"])
    if not per:
        return f"no dispatch of {kernel!r}"
    lines = [f"kernel={kernel}", "selection=" + (f"phase {phase}" if phase is not None else "all dispatches")]
    for name in sorted(per):
        v = list(per[name].values())
        lines.append(f"{name}_dispatches={len(v)}")
        lines.append(f"{name}_median={statistics.median(v):.1f}")
    if simds and "SQ_VALU_MFMA_BUSY_CYCLES" in per and "GRBM_GUI_ACTIVE" in per:
        util = [per["SQ_VALU_MFMA_BUSY_CYCLES"][i] / (per["GRBM_GUI_ACTIVE"][i] * simds)
                for i in per["SQ_VALU_MFMA_BUSY_CYCLES"] if per["GRBM_GUI_ACTIVE"].get(i)]
        lines.append(f"mfma_busy_share_median={statistics.median(util):.4f}")
    for name in sorted(per):
        if name.startswith("SQ_INSTS_VALU_MFMA_MOPS_"):
            lines.append(f"{name[len('SQ_INSTS_VALU_MFMA_MOPS_'):].lower()}_mfma_flop_median="
                         f"{512 * statistics.median(per[name].values()):.0f}")
    return "\n".join(lines)


def kernel_sources_digest(csrc):
    """First 16 hex digits of the SHA-256 over the device sources in directory csrc (every .hip and .h
    file, in name order): the counters describe these sources only."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode())
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()[:16]


def traffic(fetch, write, kernel, grid_y, algo, source, fetch_trace=None, write_trace=None, phase=None):
    if phase is not None:
        fids, wids = _phase_ids(fetch, phase), _phase_ids(write, phase)
        if fids is None or wids is None:
            return f"incomplete: fewer than {2 * phase + 2} phase markers in a counter file"
    else:
        fids = _dispatch_ids(fetch_trace, kernel, grid_y) if fetch_trace else None
        wids = _dispatch_ids(write_trace, kernel, grid_y) if write_trace else None
    fv, fc = _counter(fetch, kernel, grid_y, fids)
    wv, wc = _counter(write, kernel, grid_y, wids)
    if fv is None or wv is None:
        return "incomplete: the counter files hold no grid shape; give the kernel traces of the same runs"
    if not fv or not wv or not fc or not wc:
        return "incomplete: " + repr((len(fv), len(wv), fc, wc))
    sf, sw = GIB_KIB / fc, GIB_KIB / wc
    if phase is not None:
        how = f"phase {phase}: the dispatches between the run's phase markers {2 * phase} and {2 * phase + 1}"
    else:
        how = "all dispatches" if grid_y is None else (
            f"grid y = {grid_y}, by dispatch id from the kernel trace of each counter run" if fids is not None
            else f"grid y = {grid_y}")
    fk, wk = statistics.median(fv), statistics.median(wv)
    hbm = (fk * sf + wk * sw) * 1024.0
    lines = [f"kernel={kernel}", f"selection={how}", f"dispatches_fetch={len(fv)}", f"dispatches_write={len(wv)}",
             f"fetch_kib_median={fk:.1f}", f"write_kib_median={wk:.1f}",
             f"copy_fetch_kib={fc:.1f}", f"copy_write_kib={wc:.1f}",
             f"scale_fetch={sf:.4f}", f"scale_write={sw:.4f}", f"hbm_bytes_per_launch={hbm:.0f}"]
    if algo:
        lines.append(f"algorithmic_bytes_per_launch={algo:.0f}")
        lines.append(f"traffic_over_algorithmic={hbm / algo:.4f}")
    if source:
        lines.append("kernels_sha256=" + kernel_sources_digest(source))
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("csv")
    a.add_argument("--top", type=int, default=24)
    b = sub.add_parser("trace")
    b.add_argument("csv")
    b.add_argument("--kernel", required=True)
    b.add_argument("--grid-y", type=int, default=None)
    m = sub.add_parser("counters")
    m.add_argument("csv")
    m.add_argument("--kernel", required=True)
    m.add_argument("--phase", type=int, default=None)
    m.add_argument("--simds", type=int, default=None, help="SIMDs of the GPU (MI355X: 1024)")
    c = sub.add_parser("traffic")
    c.add_argument("fetch")
    c.add_argument("write")
    c.add_argument("--kernel", required=True)
    c.add_argument("--grid-y", type=int, default=None)
    c.add_argument("--fetch-trace", default=None, help="kernel trace CSV of the FETCH_SIZE run")
    c.add_argument("--write-trace", default=None, help="kernel trace CSV of the WRITE_SIZE run")
    c.add_argument("--algo-bytes", type=float, default=None)
    c.add_argument("--source", default=None, help="the kernel source directory (csrc)")
    c.add_argument("--phase", type=int, default=None,
                   help="only the dispatches of measured phase k (between phase markers 2k and 2k+1)")
    args = ap.parse_args(argv)
    if args.cmd == "stats":
        print(stats(args.csv, args.top))
    elif args.cmd == "trace":
        print(trace(args.csv, args.kernel, args.grid_y))
    elif args.cmd == "counters":
        print(counters(args.csv, args.kernel, args.phase, args.simds))
    else:
        print(traffic(args.fetch, args.write, args.kernel, args.grid_y, args.algo_bytes, args.source,
                      args.fetch_trace, args.write_trace, args.phase))
    return 0


if __name__ == "__main__":
    sys.exit(main())
