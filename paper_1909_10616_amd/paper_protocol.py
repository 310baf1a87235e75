"""The paper's own tuning protocol (§5) on one MI355X.

  python -m paper_1909_10616_amd.paper_protocol [--sizes 512,1024,2048]
      [--seeds 1] [--methods gbfs,na2c,random] [--out FILE.json]

Perceptron layers Y = WᵀX (W: k×m, X: k×n, fp32, U[−1,1), seed 0), the
space shape of §5 — d = (4, 2, 4), moves between any two levels (Eq.6) —
the paper's start state s0 = [[m,1,1,1],[k,1],[n,1,1,1]], ρ = 5 (G-BFS) and
𝒯 = 3 (N-A2C, other settings at the library's defaults), equal-budget random
search as the baseline, and a budget of 0.1 % of the space (484, 900 and
1,590 timed configurations).
Every candidate is timed by the library as in every other search (1 warm-up,
mean of 10 runs, output checked against the reference). Reported per size
and seed: best cost (ms, TFLOP/s, % of the fp32 MFMA peak), configurations
timed and the fraction of the space, search wall time, the best
configuration. (The replay of such a search through the oracle's Alg.1 is a
GPU test, tests/test_gpu_tn.py.)
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_F32 = 157.3  # MI355X dense fp32 MFMA, TFLOP/s


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--sizes", default="512,1024,2048")
    ap.add_argument("--seeds", type=int, default=1)
    ap.add_argument("--methods", default="gbfs")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()

    import torch
    from paper_1909_10616_amd import gemmtune as gt
    from workloads import PAPER_PROTOCOL, make_perceptron_inputs

    if not torch.cuda.is_available():
        raise SystemExit("paper_protocol needs a GPU")
    gt.lib()
    sizes = {int(x) for x in args.sizes.split(",")}
    dev = torch.device("cuda:0")
    rows = []
    for w in PAPER_PROTOCOL:
        if w.M not in sizes:
            continue
        W, X = make_perceptron_inputs(w.M, w.N, w.K, w.dtype, w.seed, w.dist)
        Wd, Xd = W.to(dev), X.to(dev)
        C = torch.empty(w.M, w.N, device=dev)
        R = torch.empty_like(C)
        gt.gt_reference_gemm(Wd, Xd, R, a_kmajor=True)
        torch.cuda.synchronize()
        sp = gt.Space(w.M, w.N, w.K, w.d, w.dtype, w.mfma_coord, mode=gt.ANY_PAIR, a_kmajor=True)
        s0 = ((w.M, 1, 1, 1), (w.K, 1), (w.N, 1, 1, 1), 0)
        for method, seed in [(m, k) for k in range(args.seeds) for m in args.methods.split(",")]:
            print(f"{w.name} seed {seed}: {method}, budget {w.budget} of {sp.size()}", flush=True)
            t = time.perf_counter()
            if method == "gbfs":
                r = gt.tune_gbfs(sp, budget=w.budget, s0=s0, rho=5, seed=seed, A=Wd, B=Xd, C=C,
                                 c_ref=R, progress_s=30.0)
            elif method == "na2c":
                r = gt.tune_na2c(sp, w.budget, s0=s0, seed=seed, A=Wd, B=Xd, C=C, c_ref=R,
                                 progress_s=30.0)
            elif method == "random":
                r = gt.tune_random(sp, budget=w.budget, seed=seed, A=Wd, B=Xd, C=C, c_ref=R,
                                   progress_s=30.0)
            else:
                raise SystemExit(f"unknown method {method!r}")
            wall = time.perf_counter() - t
            costs = [e["cost_ms"] for e in r["log"]]
            argmin = min(range(len(costs)), key=lambda i: (costs[i], i))
            consistent = r["log"][argmin]["rank"] == r["best_rank"]
            row = {"workload": w.name, "method": method, "M": w.M, "N": w.N, "K": w.K,
                   "seed": seed,
                   "space_size": sp.size(), "budget": w.budget, "timed": r["timed"],
                   "fraction_pct": 100.0 * r["timed"] / sp.size(),
                   "best": gt.fmt_cfg(r["best"]), "best_ms": r["best_cost"],
                   "tflops": gt.tflops(w.M, w.N, w.K, r["best_cost"]),
                   "s0_ms": r["log"][0]["cost_ms"] if method != "random" else None,
                   "failed": r["failed"],
                   "stop": r["stop_reason"], "wall_s": round(wall, 1),
                   "kernel": {k: v for k, v in gt.lower(r["best"], w.M, w.N, w.K,
                                                        sp.dtype).items()
                              if k in ("I", "TM", "TN", "fast", "waves", "BM", "BN", "BK")},
                   "best_is_log_argmin": consistent}
            row["pct_of_fp32_peak"] = round(100.0 * row["tflops"] / PEAK_F32, 2)
            rows.append(row)
            print(f"{w.name} seed {seed} {method}: {row['tflops']:.2f} TFLOP/s "
                  f"({row['pct_of_fp32_peak']} % of fp32 peak), best {row['best']}, "
                  f"{r['timed']} timed in {wall:.0f} s, "
                  f"s* = argmin of the log: {consistent}", flush=True)
    summary = {}
    for name, method in sorted({(r["workload"], r["method"]) for r in rows}):
        v = [r["tflops"] for r in rows if r["workload"] == name and r["method"] == method]
        summary[f"{name} {method}"] = {"seeds": len(v), "min": min(v),
                                       "median": statistics.median(v), "max": max(v)}
    print(json.dumps({"summary": summary}), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            json.dump({"runs": rows, "summary": summary}, f, indent=1)


if __name__ == "__main__":
    main()
