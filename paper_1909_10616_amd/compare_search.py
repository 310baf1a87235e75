"""G-BFS against equal-budget random search and N-A2C, several seeds, one GPU (§5).

  python -m paper_1909_10616_amd.compare_search --workload gemm4096_bf16 --seeds 10
      [--budget N] [--t-max S] [--s0 hand|paper] [--methods gbfs,random,na2c] [--out FILE.json]

For every seed the chosen searches run on the same resident inputs and the same
reference product (computed once); every candidate is timed the same way
(1 warm-up + 10 event-timed runs, output checked). Reported per seed: the
best cost found (ms, TFLOP/s), configurations timed, search wall time; then
min / median / max over seeds. With --t-max each search also stops after that
many seconds (the paper's variance study uses a 750 s time budget); random
draws at large sizes include kernels whose single launch takes seconds, so
an equal configuration budget can take random search many minutes.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="gemm4096_bf16")
    ap.add_argument("--seeds", type=int, default=10)
    ap.add_argument("--budget", type=int, default=0, help="0: the workload's budget")
    ap.add_argument("--t-max", type=float, default=0.0)
    ap.add_argument("--s0", choices=["hand", "paper"], default="hand")
    ap.add_argument("--rho", type=int, default=5)
    ap.add_argument("--methods", default="gbfs,random",
                    help="comma-separated subset of gbfs,random,na2c (random search has no s0)")
    ap.add_argument("--out", default=None)
    ap.add_argument("--progress", type=float, default=0.0,
                    help="> 0: a progress line on stderr at most this often (s)")
    ap.add_argument("--trace", action="store_true",
                    help="name every candidate on stderr before it is launched")
    args = ap.parse_args()
    methods = [m for m in args.methods.split(",") if m]
    if not methods or any(m not in ("gbfs", "random", "na2c") for m in methods):
        raise SystemExit("--methods: a comma-separated subset of gbfs,random,na2c")

    import torch
    from paper_1909_10616_amd import gemmtune as gt
    from workloads import WORKLOADS, workload_inputs

    if not torch.cuda.is_available():
        raise SystemExit("compare_search needs a GPU")
    gt.lib()
    w = WORKLOADS[args.workload]
    budget = args.budget or w.budget
    dev = torch.device("cuda:0")
    A, B = workload_inputs(w)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty(w.M, w.N, device=dev)
    R = torch.empty_like(C)
    gt.gt_reference_gemm(Ad, Bd, R)
    torch.cuda.synchronize()
    sp = gt.Space(w.M, w.N, w.K, w.d, w.dtype, w.mfma_coord)
    s0 = gt.hand_start(w.M, w.N, w.K, w.d, w.mfma_coord) if args.s0 == "hand" else sp.paper_s0()
    runs = []
    for seed in range(args.seeds):
        row = {"seed": seed}
        for name, fn in (("gbfs", gt.tune_gbfs), ("random", gt.tune_random),
                         ("na2c", gt.tune_na2c)):
            if name not in methods:
                continue
            # every candidate is named on stderr before it is launched
            kw = dict(budget=budget, seed=seed, t_max_s=args.t_max, A=Ad, B=Bd, C=C, c_ref=R,
                      trace_fd=2 if args.trace else -1, progress_s=args.progress)
            if name == "gbfs":
                kw.update(s0=s0, rho=args.rho)
            elif name == "na2c":
                kw.update(s0=s0)
            print(f"seed {seed} {name}: searching", flush=True)
            r = fn(sp, **kw)
            row[name] = {"best": gt.fmt_cfg(r["best"]), "best_ms": r["best_cost"],
                         "tflops": gt.tflops(w.M, w.N, w.K, r["best_cost"]), "timed": r["timed"],
                         "failed": r["failed"], "wall_s": round(r["wall_s"], 2),
                         "stop": r["stop_reason"]}
            print(f"seed {seed} {name:6s} {row[name]['tflops']:8.1f} TFLOP/s after "
                  f"{r['timed']} timings in {r['wall_s']:.1f} s: {row[name]['best']}", flush=True)
        runs.append(row)

    def stats(name):
        v = [r[name]["tflops"] for r in runs]
        return {"min": min(v), "median": statistics.median(v), "max": max(v),
                "mean_wall_s": statistics.mean(r[name]["wall_s"] for r in runs)}

    summary = {"workload": w.name, "budget": budget, "t_max_s": args.t_max, "s0": gt.fmt_cfg(s0),
               "s0_kind": args.s0, "space_size": sp.size(), "seeds": args.seeds,
               **{m: stats(m) for m in methods}, "runs": runs}
    print(json.dumps({k: v for k, v in summary.items() if k != "runs"}), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            json.dump(summary, f, indent=1)


if __name__ == "__main__":
    main()
