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
  python -m paper_1909_10616_amd.profsum bestcfg BENCH_JSON
      the best configuration of a bench line, as the JSON bench.py --replay takes.
  python -m paper_1909_10616_amd.profsum report OUT [--args "EXTRA BENCH ARGUMENTS"]
      markdown summary of a profile_bench.sh output folder (run with those
      extra bench.py arguments), ending with the line for profiles/traffic.txt.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import json
import os
import re
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


def best_cfg(bench_json):
    d = _last_line_json(bench_json)
    m = re.match(r"m(\[.*?\])k(\[.*?\])n(\[.*?\])mfma(\d+)", d["config"]["best_config"])
    return [json.loads(m.group(1)), json.loads(m.group(2)), json.loads(m.group(3)), int(m.group(4))]


def _last_line_json(path):
    with open(path) as f:
        lines = [l for l in f if l.strip().startswith("{")]
    return json.loads(lines[-1])


def report(out, copy_bytes=1 << 30, extra=""):
    b = _last_line_json(os.path.join(out, "bench_traced.json"))
    c = b["config"]
    kname = c["kernel_name"]
    info = c["kernel"]
    grid = info["grid_x"] * 64 * info["waves"]
    rows = [r for r in _rows(os.path.join(out, "trace"), "bench", "kernel_trace")]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    sel = [r for r in rows if _match(r, kname, grid, info["lds_bytes"])
           and int(r.get("Grid_Size_Y") or 1) == info["grid_y"]]
    last = sel[-200:]
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in last]
    t = traffic(*(os.path.join(out, d) for d in ("fetch", "write", "cfetch", "cwrite")),
                copy_bytes, kname, grid, info["lds_bytes"])
    u, _ = pmc(os.path.join(out, "util"), "u", kname, grid, info["lds_bytes"])
    uc = {cn: v for (k, cn), v in u.items()}
    w = c["workload"]
    flops = 2.0 * c["M"] * c["N"] * c["K"]
    mean_us = statistics.mean(dur)
    L = []
    L.append(f"# {w}: {kname}, {info['BM']}x{info['BN']}x{info['BK']} tile, {info['waves']} wavefronts")
    L.append("")
    L.append("Commands (from the repository root on the GPU host; OUT is the output folder):")
    L.append("")
    x = (" " + extra) if extra else ""
    L.append(f"    paper_1909_10616_amd/profile_bench.sh OUT{x}")
    L.append("      = rocprofv3 --kernel-trace --stats --output-format csv -d OUT/trace -o bench -- "
             f"python3 bench.py --no-cpu-baseline{x}")
    L.append(f"        rocprofv3 --pmc FETCH_SIZE   (then WRITE_SIZE) ... -- python3 bench.py{x} --replay CFG --repeat 20")
    L.append("        rocprofv3 --pmc FETCH_SIZE   (then WRITE_SIZE) ... -- python3 bench.py --calibrate-copy 1024 --repeat 5")
    L.append("        rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE SQ_LDS_BANK_CONFLICT "
             f"SQ_LDS_IDX_ACTIVE SQ_WAVE_CYCLES SQ_WAIT_ANY ... -- python3 bench.py{x} --replay CFG --repeat 20")
    L.append("    python3 paper_1909_10616_amd/profsum.py report OUT" + (f' --args "{extra}"' if extra else ""))
    L.append("")
    L.append(f"Best configuration of the traced search: `{c['best_config']}` (CFG), "
             f"{c['configs_timed']} configurations timed of {c['space_size']} "
             f"({c['fraction_of_space_pct']:.6f}% of the space), search {c['search_wall_s']} s.")
    L.append(f"Launch: `{c['launch_signature']}`, kernel sources `{c['kernel_source']}`.")
    if last:
        r0 = last[-1]
        vg = r0.get('VGPR_Count')
        L.append(f"Registers per lane (kernel trace fields): VGPR_Count {vg}, Accum_VGPR_Count "
                 f"{r0.get('Accum_VGPR_Count')}, SGPR_Count {r0.get('SGPR_Count')}; scratch "
                 f"{r0.get('Scratch_Size')} B. The trace counts the descriptor's VGPR allocation "
                 f"granules as 4 registers each; gfx950 allocates 8 per granule, so the wavefront "
                 f"holds {2 * int(vg) if str(vg).isdigit() else '2x that'} VGPRs.")
    L.append("")
    L.append("## Kernel trace vs. bench timing")
    L.append("")
    L.append("| source | launches | mean µs | TFLOP/s |")
    L.append("|---|---|---|---|")
    L.append(f"| kernel trace, last {len(dur)} dispatches of CFG | {len(dur)} | {mean_us:.2f} | "
             f"{flops / (mean_us * 1e-6) / 1e12:.1f} |")
    L.append(f"| bench.py HIP events around the same {len(dur)} launches (best_ms) | {len(dur)} | "
             f"{b['config']['best_ms'] * 1e3:.2f} | {b['value']:.1f} |")
    L.append(f"| median of the traced dispatches | | {statistics.median(dur):.2f} | |")
    L.append("")
    rf = b["roofline"]
    L.append(f"Roofline ({rf.get('bound', 'mfma')} bound): {rf.get('achieved')} {rf.get('unit', 'TFLOP/s')} "
             f"of {rf['peak']} {rf.get('unit', 'TFLOP/s')}, fraction {rf['frac']:.4f}"
             + (f"; MFMA fraction {rf['mfma_frac']:.4f}" if "mfma_frac" in rf else "") + ".")
    L.append("")
    L.append("## HBM traffic per launch (FETCH_SIZE, WRITE_SIZE; scaled by a 1 GiB copy)")
    L.append("")
    L.append("| counter | kernel KiB/dispatch | copy KiB/dispatch | scale | bytes |")
    L.append("|---|---|---|---|---|")
    L.append(f"| FETCH_SIZE | {t['fetch_kib']:.0f} | {t['copy_fetch_kib']:.0f} | {t['fetch_factor']:.3f} | "
             f"{t['fetch_bytes']:.4g} |")
    L.append(f"| WRITE_SIZE | {t['write_kib']:.0f} | {t['copy_write_kib']:.0f} | {t['write_factor']:.3f} | "
             f"{t['write_bytes']:.4g} |")
    alg = b["roofline"]["algorithmic_bytes"]
    L.append("")
    L.append(f"Total {t['traffic_bytes']:.4g} B per launch against {alg} algorithmic bytes "
             f"(A and B read once, C written once): {t['traffic_bytes'] / alg:.2f}x. "
             f"At the traced mean that is {t['traffic_bytes'] / (mean_us * 1e-6) / 1e9:.0f} GB/s of HBM.")
    L.append("")
    L.append("## Utilisation counters (mean per dispatch of CFG)")
    L.append("")
    for k in sorted(uc):
        L.append(f"- {k}: {uc[k]:.0f}")
    L.append("")
    L.append("## Line for profiles/traffic.txt")
    L.append("")
    L.append(f"    {c['launch_signature']} | source={c['kernel_source']} traffic_bytes={t['traffic_bytes']:.0f}")
    return "\n".join(L)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("mode", choices=["trace", "pmc", "traffic", "bestcfg", "report"])
    ap.add_argument("dirs", nargs="+")
    ap.add_argument("--kernel", default=None)
    ap.add_argument("--grid", type=int, default=0)
    ap.add_argument("--lds", type=int, default=0)
    ap.add_argument("--last", type=int, default=0)
    ap.add_argument("--copy-bytes", type=float, default=0)
    ap.add_argument("--copy-kernel", default="copy")
    ap.add_argument("--args", default="", help="report: the extra bench.py arguments of the profile")
    a = ap.parse_args()
    if a.mode == "bestcfg":
        print(json.dumps(best_cfg(a.dirs[0])))
    elif a.mode == "report":
        print(report(a.dirs[0], extra=a.args))
    elif a.mode == "trace":
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
