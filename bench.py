"""Benchmark: tuned GEMM found by G-BFS on one MI355X.

A step is one pass of the whole path on the resident synthetic inputs: a
G-BFS search (§4.2 Alg.1) over the tiling space with its budget of timed
configurations — enumeration/rank, legitimacy, neighbours, ρ-sampling,
lowering, every candidate GEMM run and timed on the GPU and checked against
the reference — followed by the report: s* and the next TOPK − 1 configurations of
the search log by cost, each re-timed over REPEAT back-to-back launches
between HIP events on the bench stream; the fastest is the reported
configuration, and it is re-timed once more (REPEAT launches) for the value.

value   = TFLOP/s of the reported configuration (2·M·N·K per run) from that
          last re-timing;
ms_per_step = wall time of one step (search + report).

Prints ONE JSON line (rank 0). Only one GPU: --gpus above 1 exits.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "best-found GEMM TFLOP/s (% of MFMA peak); configs timed / % of space"
# MI355X published dense peaks (TFLOP/s) and HBM bandwidth (GB/s)
PEAK = {"bf16": 2516.6, "f32": 157.3}
HBM_GBS = 8000.0
REPEAT = 200
TOPK = 4


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def hand_s0(w):
    from paper_1909_10616_amd.gemmtune import hand_start
    return hand_start(w.M, w.N, w.K, w.d, w.mfma_coord)


def fmt_cfg(c):
    from paper_1909_10616_amd.gemmtune import fmt_cfg as f
    return f(c)


def kernel_name(w, info):
    """Symbol of the kernel instantiation a lowered configuration launches."""
    dt = 1 if w.dtype == "bf16" else 0
    cpr = info["BK"] // (8 if w.dtype == "bf16" else 4) if info["fast"] else 0
    if info["dl"]:
        return f"gt::gemm_kernel_dl<{info['I']}, {info['TM']}, {info['TN']}, {cpr}>"
    return f"gt::gemm_kernel<{dt}, {info['I']}, {info['TM']}, {info['TN']}, {cpr}>"


def _code_only(text: str) -> str:
    """C++ source without its comments, trailing blanks and empty lines (no
    string literal in these sources holds a comment marker)."""
    import re
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(line.rstrip() for line in text.splitlines() if line.strip())


def kernel_source_hash():
    """Fingerprint of the code of the sources that hold the GPU kernels
    (comments and layout do not count; how a configuration lowers is part
    of the launch signature)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("gemm_kernel.hpp", "gemm_inst.hip", "aux_kernels.hip"):
        with open(os.path.join(ROOT, "paper_1909_10616_amd", "csrc", f)) as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def launch_signature(w, info):
    return (f"{w.name} {kernel_name(w, info).replace(' ', '')} grid={info['grid_x']}x{info['grid_y']} "
            f"waves={info['waves']} lds={info['lds_bytes']} dl={info['dl']}/{info['ring']}")


def measured_traffic(w, info):
    """HBM bytes per launch from profiles/traffic.txt, when the counters were
    taken on this exact launch signature with the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.txt")
    if not os.path.exists(path):
        return None
    want = launch_signature(w, info)
    src = kernel_source_hash()
    for line in open(path):
        if line.startswith("#") or "|" not in line:
            continue
        sig, rest = (x.strip() for x in line.split("|", 1))
        kv = dict(t.split("=", 1) for t in rest.split())
        if sig == want and kv.get("source") == src:
            return int(float(kv["traffic_bytes"]))
    return None


def roofline(dtype, M, N, K, alg_bytes, tflops, hbm_gbs, traffic):
    """The bench line's roofline: the bound is the one the workload's
    arithmetic intensity (2MNK / algorithmic bytes) puts it under — MFMA at
    or above the ridge (the dtype's MFMA peak over the HBM bandwidth), HBM
    below it; the other unit's fraction is given beside it."""
    flops = 2.0 * M * N * K
    peak = PEAK[dtype]
    ridge = peak * 1e12 / (HBM_GBS * 1e9)
    if flops / alg_bytes >= ridge:
        r = {"bound": "mfma", "achieved": round(tflops, 2), "peak": peak, "unit": "TFLOP/s",
             "frac": round(tflops / peak, 4)}
        other = {"hbm_gbs_at_algorithmic_bytes": round(hbm_gbs, 1),
                 "hbm_frac": round(hbm_gbs / HBM_GBS, 4)}
    else:
        r = {"bound": "hbm", "achieved": round(hbm_gbs, 1), "peak": HBM_GBS, "unit": "GB/s",
             "frac": round(hbm_gbs / HBM_GBS, 4)}
        other = {"mfma_tflops": round(tflops, 2), "mfma_frac": round(tflops / peak, 4)}
    r.update({"traffic": traffic, "algorithmic_bytes": alg_bytes,
              "arithmetic_intensity": round(flops / alg_bytes, 1), "ridge": round(ridge, 1)})
    r.update(other)
    return r


def flushed_timing(run, stream, mib, runs=50):
    """Median time of `run` with a `mib` MiB buffer read on the stream before
    each launch (more than the 256 MiB last-level cache, so A and B come from
    HBM; the buffer is written once beforehand, so the lines it leaves in the
    cache are clean and evicting them costs no write-back), each launch
    between its own pair of events."""
    import torch
    buf = torch.ones(mib << 18, dtype=torch.float32, device="cuda:0")
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(runs)]
    with torch.cuda.stream(stream):
        for e0, e1 in evs:
            buf.sum()
            e0.record(stream)
            run()
            e1.record(stream)
    torch.cuda.synchronize()
    d = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    del buf
    return d[runs // 2] if runs % 2 else 0.5 * (d[runs // 2 - 1] + d[runs // 2])


def host_info():
    """The host the CPU baseline runs on: logical CPUs, the CPUs this process
    may use, and the CPU model."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "cpu_model": model}


def cpu_threads():
    """Threads for the oracle: the CPU share the job is given (OMP_NUM_THREADS
    when set, as a scheduler does for each GPU's share of the host), else
    every CPU this process may use."""
    aff = len(os.sched_getaffinity(0))
    return max(1, min(int(os.environ.get("OMP_NUM_THREADS", "0")) or aff, aff))


def cpu_baseline(w, A, B, target_s: float):
    """The oracle (plain fp64 three-loop GEMM) on host cores, in TFLOP/s: the
    whole product when a 64-row sample says it fits in target_s, otherwise
    that many rows. Returns the record and the product (None for a sample)."""
    import oracle
    from workloads import raw_bytes
    threads = cpu_threads()
    Bb = raw_bytes(B)
    rows = min(w.M, 64)
    t = time.perf_counter()
    oracle.gemm(raw_bytes(A[:rows]), Bb, rows, w.N, w.K, w.dtype, nthreads=threads)
    cal = time.perf_counter() - t
    est_full = cal * w.M / rows
    if est_full <= target_s:
        rows = w.M
    else:
        rows = int(min(w.M, max(rows, rows * target_s / max(cal, 1e-3))))
        rows = max(threads, rows - rows % threads)
    t = time.perf_counter()
    C = oracle.gemm(raw_bytes(A[:rows]), Bb, rows, w.N, w.K, w.dtype, nthreads=threads)
    dt = time.perf_counter() - t
    flops = 2.0 * rows * w.N * w.K
    what = "all rows" if rows == w.M else f"rows 0..{rows - 1}"
    rec = {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
           "sample": f"{what} of C ({rows}x{w.N}x{w.K}, fp64 three-loop, {threads} threads), "
                     f"{dt:.1f} s", "host": host_info()}
    return rec, (C if rows == w.M else None)


def componentwise_error(w, A, B, C_gpu, C_oracle):
    """max |C − C*| / (|A|·|B|) elementwise, the oracle computing |A|·|B| on
    the sign-cleared input bytes (exact for fp32 and bf16 alike)."""
    import oracle
    from workloads import raw_bytes
    absab = oracle.gemm(raw_bytes(A.abs()), raw_bytes(B.abs()), w.M, w.N, w.K, w.dtype,
                        nthreads=cpu_threads())
    d = np.abs(C_gpu.astype(np.float64) - C_oracle)
    return float((d / np.maximum(absab, np.finfo(np.float64).tiny)).max())


def single_core_oracle():
    """The oracle on one core at the two small workload shapes (256³ and
    1024³ fp32): seconds and GFLOP/s per core."""
    import oracle
    from workloads import make_inputs, raw_bytes
    out = {}
    for n in (256, 1024):
        A, B = make_inputs(n, n, n, "f32", 0, "uniform")
        t = time.perf_counter()
        oracle.gemm(raw_bytes(A), raw_bytes(B), n, n, n, "f32", nthreads=1)
        dt = time.perf_counter() - t
        out[f"{n}^3_f32"] = {"seconds": round(dt, 3), "gflops_per_core": round(2.0 * n ** 3 / dt / 1e9, 3)}
    return out


def device_info():
    """Name, compute units and maximum shader clock of GPU 0 as rocminfo
    reports them, and the dense bf16 / fp32 MFMA peaks they imply (4096 and
    256 flop per clock per CU)."""
    import subprocess
    import torch
    p = torch.cuda.get_device_properties(0)
    out = {"name": p.name, "arch": getattr(p, "gcnArchName", ""), "cus": p.multi_processor_count}
    try:
        txt = subprocess.run(["rocminfo"], capture_output=True, text=True, timeout=30).stdout
        agent = next(a for a in txt.split("*******") if "gfx950" in a and "Compute Unit" in a)
        for line in agent.splitlines():
            if "Max Clock Freq. (MHz)" in line:
                out["max_sclk_mhz"] = int(line.split(":")[1].split()[0])
            if line.strip().startswith("Compute Unit:"):
                out["cus"] = int(line.split(":")[1].split()[0])
    except Exception as e:  # rocminfo missing or unparsable: report what torch gives
        out["rocminfo_error"] = str(e)[:200]
    if "max_sclk_mhz" in out:
        ghz = out["max_sclk_mhz"] / 1000.0
        out["peak_bf16_tflops_at_max_sclk"] = round(out["cus"] * ghz * 4096 / 1000.0, 1)
        out["peak_f32_tflops_at_max_sclk"] = round(out["cus"] * ghz * 256 / 1000.0, 1)
    return out


def library_enumeration(sp):
    """The library's full enumeration of the space with J (a1, a2), streamed
    in chunks through enumerate_configs."""
    from paper_1909_10616_amd import gemmtune as gt
    chunk = 4_000_000
    buf = (gt.gt_config * chunk)()
    n = ctypes.c_uint64()
    size, legit = sp.size(), 0
    off = gt.gt_config.legit.offset
    t = time.perf_counter()
    for start in range(0, size, chunk):
        gt._check(gt.lib().enumerate_configs(ctypes.byref(sp.c), start, buf, chunk, ctypes.byref(n)),
                  "enumerate_configs")
        raw = np.frombuffer(buf, dtype=np.uint8).reshape(chunk, ctypes.sizeof(gt.gt_config))
        legit += int(raw[:n.value, off:off + 4].copy().view(np.int32).sum())
    return {"configs": size, "legitimate": legit, "seconds": round(time.perf_counter() - t, 2)}


def oracle_side(w, mode, s0, res, rho, seed):
    """The oracle's other two host steps on the same workload: the full
    enumeration of the space with J (a1, a2), and Alg.1 fed the costs the GPU
    search logged (a3, a4, a8), which must retrace the GPU search exactly."""
    import oracle
    osp = oracle.Space(w.M, w.N, w.K, w.d, w.dtype, w.mfma_coord,
                       mode=oracle.ADJACENT if mode == "adjacent" else oracle.ANY_PAIR)
    size = osp.size()
    t = time.perf_counter()
    legit, chunk = 0, 2_000_000
    for start in range(0, size, chunk):
        raw = osp.enumerate_raw(start, min(chunk, size - start))
        legit += int(raw[:, 100:104].copy().view(np.int32).sum())
    t_enum = time.perf_counter() - t
    table = {e["rank"]: e["cost_ms"] for e in res["log"]}
    t = time.perf_counter()
    rep = oracle.gbfs(osp, s0, rho, len(res["log"]), seed, lambda c, r: table.get(r, math.inf))
    t_rep = time.perf_counter() - t
    return {"enumeration": {"configs": size, "legitimate": legit, "seconds": round(t_enum, 2),
                            "threads": 1},
            "gbfs_replay": {"seconds": round(t_rep, 3),
                            "same_trajectory": rep["log_ranks"] == [e["rank"] for e in res["log"]],
                            "same_best": rep["best"] == res["search_best"]}}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="gemm4096_bf16")
    ap.add_argument("--budget", type=int, default=None)
    ap.add_argument("--s0", choices=["hand", "paper"], default="hand")
    ap.add_argument("--rho", type=int, default=5)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--mode", choices=["adjacent", "any"], default="adjacent")
    ap.add_argument("--progress", type=float, default=0.0,
                    help="> 0: a search progress line on stderr at most this often (s)")
    ap.add_argument("--t-max", type=float, default=0.0,
                    help="> 0: search time limit in seconds (T_max of Alg.1)")
    ap.add_argument("--no-enumeration", action="store_true",
                    help="skip the timed full enumeration of the space")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--flush-mib", type=int, default=0,
                    help="> 0: also time the reported configuration with this many MiB read "
                         "before each launch (larger than the 256 MiB last-level cache)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--log-out", default=None, help="write the search log (JSON) here")
    ap.add_argument("--replay", default=None,
                    help="skip the search: launch this configuration (JSON) --repeat times")
    ap.add_argument("--repeat", type=int, default=REPEAT)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="launch a plain device copy of MIB MiB --repeat times (counter scale)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); splitting the search's "
              "candidates or the GEMM's grid over several GPUs is not built.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_1909_10616_amd import gemmtune as gt
    from workloads import WORKLOADS, workload_inputs

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    gt.lib()  # loud failure when the HIP library is missing
    if args.calibrate_copy:
        n = args.calibrate_copy << 18  # floats
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.repeat):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes_read": n * 4, "bytes_written": n * 4,
                          "launches": args.repeat}))
        return
    w = WORKLOADS[args.workload]
    budget = args.budget or w.budget
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream()
    log(f"workload {w.name}: {w.M}x{w.N}x{w.K} {w.dtype}, budget {budget}")
    A, B = workload_inputs(w)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty(w.M, w.N, device=dev, dtype=torch.float32)
    Cref = torch.empty_like(C)
    torch.cuda.synchronize()
    mode = gt.ADJACENT if args.mode == "adjacent" else gt.ANY_PAIR
    sp = gt.Space(w.M, w.N, w.K, w.d, w.dtype, w.mfma_coord, mode=mode)
    size = sp.size()
    s0 = hand_s0(w) if args.s0 == "hand" else sp.paper_s0()
    assert sp.legit(s0), s0

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)

    if args.replay:
        cfg = tuple(tuple(x) if isinstance(x, list) else x for x in json.loads(args.replay))
        assert sp.legit(cfg), cfg
        with torch.cuda.stream(stream):
            gt.gemm_run(cfg, Ad, Bd, C, stream=stream)
            ev0.record(stream)
            for _ in range(args.repeat):
                gt.gemm_run(cfg, Ad, Bd, C, stream=stream)
            ev1.record(stream)
            ev1.synchronize()
        ms = ev0.elapsed_time(ev1) / args.repeat
        info = gt.lower(cfg, w.M, w.N, w.K, w.dtype)
        print(json.dumps({"replay": fmt_cfg(cfg), "ms": ms, "tflops": gt.tflops(w.M, w.N, w.K, ms),
                          "launches": args.repeat + 1, "grid_x": info["grid_x"],
                          "lds_bytes": info["lds_bytes"]}))
        return

    def retime(cfg):
        gt.gemm_run(cfg, Ad, Bd, C, stream=stream)   # warm the kernel
        ev0.record(stream)
        for _ in range(REPEAT):
            gt.gemm_run(cfg, Ad, Bd, C, stream=stream)
        ev1.record(stream)
        ev1.synchronize()
        return ev0.elapsed_time(ev1) / REPEAT

    def step():
        with torch.cuda.stream(stream):
            res = gt.tune_gbfs(sp, budget=budget, s0=s0, rho=args.rho, seed=args.seed,
                               A=Ad, B=Bd, C=C, c_ref=Cref, stream=stream,
                               progress_s=args.progress, t_max_s=args.t_max)
            # report: the TOPK configurations of the log with the lowest
            # (10-run) costs are re-timed over REPEAT launches each, s* first;
            # the fastest is the reported configuration
            ok = sorted((e["cost_ms"], e["rank"]) for e in res["log"] if e["status"] == "ok")
            ranks = [res["best_rank"]] + [r for _, r in ok if r != res["best_rank"]][:TOPK - 1]
            # untimed warm-up: REPEAT launches of s* right after the search's
            # many short runs, so that every re-timing starts from the same
            # sustained-load state of the board
            for _ in range(REPEAT):
                gt.gemm_run(res["best"], Ad, Bd, C, stream=stream)
            top = []
            for r in ranks:
                cfg = sp.unrank(r)
                top.append((retime(cfg), r, cfg))
            _, best_rank, best = min(top)
            # the reported time is a fresh re-timing of the chosen configuration
            # (not the minimum the choice was made on), and the trace's last
            # dispatches are the reported configuration's
            best_ms = retime(best)
        res["search_best"], res["search_best_rank"] = res["best"], res["best_rank"]
        res["best"], res["best_rank"], res["best_ms"] = best, best_rank, best_ms
        res["top"] = [(fmt_cfg(c), round(ms * 1e3, 2)) for ms, _, c in top]
        return res

    for i in range(args.warmup):
        t = time.perf_counter()
        r = step()
        log(f"warmup {i}: best {fmt_cfg(r['best'])} {gt.tflops(w.M, w.N, w.K, r['best_ms']):.1f} "
            f"TFLOP/s, {r['timed']} timed, {time.perf_counter() - t:.1f}s")

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    results = []
    for i in range(args.steps):
        ts = time.perf_counter()
        r = step()
        results.append(r)
        log(f"step {i}: best {fmt_cfg(r['best'])} {gt.tflops(w.M, w.N, w.K, r['best_ms']):.1f} "
            f"TFLOP/s, {r['timed']} timed, {time.perf_counter() - ts:.1f}s")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    last = results[-1]
    best_ms = last["best_ms"]
    info = gt.lower(last["best"], w.M, w.N, w.K, w.dtype)
    peak = PEAK[w.dtype]
    fig = gt.report(w.M, w.N, w.K, w.dtype, best_ms, last["timed"], size, peak)
    value = fig["tflops"]
    # C holds the reported configuration's output (its last re-timing)
    rel = gt.gt_compare(C, Cref, stream=stream)
    C_host = C.cpu().numpy()
    alg_bytes = fig["algorithmic_bytes"]
    # where a search's wall time goes: timing the candidates (their device
    # time, then launch, wait and check overhead) and the host's own steps
    # between candidates (neighbours, sampling, queue, lowering)
    timed_n = max(last["timed"], 1)
    search_split = {
        "wall_s": round(last["wall_s"], 3), "eval_s": round(last["eval_s"], 3),
        "device_s": round(last["device_s"], 3),
        "host_between_candidates_us": round((last["wall_s"] - last["eval_s"]) / timed_n * 1e6, 1),
        "eval_overhead_us": round((last["eval_s"] - last["device_s"]) / timed_n * 1e6, 1),
        "device_share": round(last["device_s"] / max(last["wall_s"], 1e-9), 4),
    }

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed * 1e3 / args.steps, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": w.name, "M": w.M, "N": w.N, "K": w.K,
            "inputs": f"{w.dtype}, seed {w.seed}, {w.dist}", "accumulate": "f32", "output": "f32",
            "levels_mkn": list(w.d), "mfma_coordinate": w.mfma_coord, "neighbours": args.mode,
            "rho": args.rho, "search_seed": args.seed, "s0": fmt_cfg(s0), "s0_kind": args.s0,
            "budget": budget, "configs_timed": last["timed"], "space_size": size,
            "fraction_of_space_pct": fig["fraction_of_space_pct"],
            "best_config": fmt_cfg(last["best"]), "best_rank": last["best_rank"],
            "pct_of_peak": round(fig["pct_of_peak"], 2),
            "search_best_config": fmt_cfg(last["search_best"]),
            "search_best_cost_ms": last["best_cost"], "best_ms": best_ms,
            "retimed_top_us": last["top"],
            # internal consistency of the search (a 10-run cost against a
            # 200-launch re-timing of the same s*)
            "s_star_retime_within_5pct": abs(last["top"][0][1] * 1e-3 / last["best_cost"] - 1.0) <= 0.05,
            "search_wall_s": round(last["wall_s"], 2), "failed": last["failed"],
            "stop": last["stop_reason"], "best_rel_diff_vs_reference": rel,
            "search_time_split": search_split,
            "kernel": {k: info[k] for k in ("I", "TM", "TN", "fast", "dl", "ring", "waves", "BM",
                                            "BN", "BK", "dbuf", "lds_bytes", "grid_x", "grid_y")},
            "kernel_name": kernel_name(w, info), "launch_signature": launch_signature(w, info),
            "kernel_source": kernel_source_hash(),
        },
        "roofline": roofline(w.dtype, w.M, w.N, w.K, alg_bytes, value, fig["hbm_gbs"],
                             measured_traffic(w, info)),
    }
    if args.flush_mib > 0:
        log(f"timing with {args.flush_mib} MiB read before each launch ...")
        fl_ms = flushed_timing(lambda: gt.gemm_run(last["best"], Ad, Bd, C, stream=stream), stream,
                               args.flush_mib)
        out["config"]["flushed"] = {
            "flush_mib": args.flush_mib, "flush": "read", "runs": 50, "median_ms": fl_ms,
            "tflops": round(gt.tflops(w.M, w.N, w.K, fl_ms), 2),
            "hbm_gbs_at_algorithmic_bytes": round(alg_bytes / (fl_ms * 1e-3) / 1e9, 1)}
    out["device"] = device_info()
    if not args.no_enumeration:
        log("library enumeration of the space ...")
        out["library_enumeration"] = library_enumeration(sp)
    if args.log_out:
        with open(args.log_out, "w") as f:
            json.dump({"config": out["config"], "log": last["log"]}, f)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"], C_oracle = cpu_baseline(w, A, B, args.cpu_seconds)
        if C_oracle is not None:
            # the reported configuration's whole output against the fp64 oracle
            err = float(np.abs(C_host.astype(np.float64) - C_oracle).max() / np.abs(C_oracle).max())
            out["rel_err_vs_oracle"] = err
            out["rel_err_tolerance"] = 2e-3 if w.dtype == "bf16" else 1e-5 * math.sqrt(w.K)
            out["matches_oracle"] = err <= out["rel_err_tolerance"]
            # secondary, not graded: the error against the sum of |products|
            out["rel_err_componentwise_vs_oracle"] = componentwise_error(w, A, B, C_host, C_oracle)
            del C_oracle
        log("oracle single-core figures, enumeration and G-BFS replay ...")
        out["cpu_baseline"]["single_core"] = single_core_oracle()
        out["cpu_baseline"].update(oracle_side(w, args.mode, s0, last, args.rho, args.seed))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
