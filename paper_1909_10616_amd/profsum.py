"""Summaries of rocprofv3 CSV output for the tuned GEMM kernels.

  python -m paper_1909_10616_amd.profsum trace DIR PREFIX [--kernel SUBSTR] [--grid N] [--lds B] [--last R]
      kernel-trace statistics per (kernel, grid, workgroup, LDS): dispatches and
      mean/min/max duration; with filters, the mean of the last R matching
      dispatches (the re-timed best configuration at the end of a bench step).
  python -m paper_1909_10616_amd.profsum pmc DIR PREFIX [--kernel SUBSTR] [--grid N] [--lds B]
      per-dispatch mean of every collected counter for the matching kernels.
  python -m paper_1909_10616_amd.profsum traffic FETCH_DIR WRITE_DIR COPY_FETCH_DIR COPY_WRITE_DIR
      --copy-bytes N --kernel SUBSTR [--grid N] [--lds B]
      HBM traffic per launch: FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the
      kernel, each scaled by (known copy bytes / what the same counter reads for
      a plain device copy of that size).
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import os
import statistics


def _rows(d, prefix, kind):
    paths = glob.glob(os.path.join(d, "**", f"{prefix}_{kind}.csv"), recursive=True)
    if not paths:
        paths = glob.glob(os.path.join(d, "**", f"*{kind}.csv"), recursive=True)
    rows = []
    for p in paths:
        with open(p) as f:
            rows.extend(csv.DictReader(f))
    return rows


def _grid(r):
    return int(r.get("Grid_Size_X") or r.get("Grid_Size") or 0)


def _match(r, kernel, grid, lds):
    if kernel and kernel not in r["Kernel_Name"]:
        return False
    if grid and _grid(r) != grid:
        return False
    if lds and int(r["LDS_Block_Size"]) not in (0, lds):  # dynamic LDS is reported as 0
        return False
    return True


def trace(d, prefix, kernel=None, grid=0, lds=0, last=0):
    rows = _rows(d, prefix, "kernel_trace")
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    groups = collections.OrderedDict()
    for r in rows:
        key = (r["Kernel_Name"], _grid(r), int(r.get("Workgroup_Size_X") or r.get("Workgroup_Size") or 0),
               int(r["LDS_Block_Size"]))
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        groups.setdefault(key, []).append(dur)
    out = ["dispatches  mean_us   min_us   max_us  grid_items  wg  lds  kernel"]
    for (name, g, wg, l), v in sorted(groups.items(), key=lambda kv: -sum(kv[1]))[:25]:
        out.append(f"{len(v):10d} {statistics.mean(v):8.2f} {min(v):8.2f} {max(v):8.2f} "
                   f"{g:11d} {wg:3d} {l:6d}  {name[:100]}")
    if kernel or grid or lds:
        sel = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows
               if _match(r, kernel, grid, lds)]
        if last:
            sel = sel[-last:]
        if sel:
            out.append(f"selected: {len(sel)} dispatches, mean {statistics.mean(sel):.2f} us, "
                       f"median {statistics.median(sel):.2f} us")
    return "\n".join(out)


def pmc(d, prefix, kernel=None, grid=0, lds=0):
    rows = [r for r in _rows(d, prefix, "counter_collection") if _match(r, kernel, grid, lds)]
    per = collections.defaultdict(list)
    for r in rows:
        per[(r["Kernel_Name"][:80], r["Counter_Name"])].append(float(r["Counter_Value"]))
    return {k: statistics.mean(v) for k, v in per.items()}, len(rows)


def _counter(d, name, kernel, grid, lds):
    vals, _ = pmc(d, "*", kernel, grid, lds)
    got = [v for (k, c), v in vals.items() if c == name]
    return statistics.mean(got) if got else float("nan")


def traffic(fetch_dir, write_dir, cfetch_dir, cwrite_dir, copy_bytes, kernel, grid=0, lds=0,
            copy_kernel="copy"):
    f_k = _counter(fetch_dir, "FETCH_SIZE", kernel, grid, lds)
    w_k = _counter(write_dir, "WRITE_SIZE", kernel, grid, lds)
    f_c = _counter(cfetch_dir, "FETCH_SIZE", copy_kernel, 0, 0)
    w_c = _counter(cwrite_dir, "WRITE_SIZE", copy_kernel, 0, 0)
    ff = copy_bytes / (f_c * 1024.0)
    wf = copy_bytes / (w_c * 1024.0)
    return {"fetch_kib": f_k, "write_kib": w_k, "copy_fetch_kib": f_c, "copy_write_kib": w_c,
            "fetch_factor": ff, "write_factor": wf,
            "fetch_bytes": f_k * 1024.0 * ff, "write_bytes": w_k * 1024.0 * wf,
            "traffic_bytes": f_k * 1024.0 * ff + w_k * 1024.0 * wf}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("mode", choices=["trace", "pmc", "traffic"])
    ap.add_argument("dirs", nargs="+")
    ap.add_argument("--kernel", default=None)
    ap.add_argument("--grid", type=int, default=0)
    ap.add_argument("--lds", type=int, default=0)
    ap.add_argument("--last", type=int, default=0)
    ap.add_argument("--copy-bytes", type=float, default=0)
    ap.add_argument("--copy-kernel", default="copy")
    a = ap.parse_args()
    if a.mode == "trace":
        print(trace(a.dirs[0], a.dirs[1], a.kernel, a.grid, a.lds, a.last))
    elif a.mode == "pmc":
        vals, n = pmc(a.dirs[0], a.dirs[1], a.kernel, a.grid, a.lds)
        print(f"{n} counter rows")
        for (k, c), v in sorted(vals.items()):
            print(f"{c:32s} {v:16.1f}  {k}")
    else:
        t = traffic(*a.dirs[:4], a.copy_bytes, a.kernel, a.grid, a.lds, a.copy_kernel)
        for k, v in t.items():
            print(f"{k:16s} {v:.4g}")


if __name__ == "__main__":
    main()
