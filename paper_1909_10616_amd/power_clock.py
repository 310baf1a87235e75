"""Board power and shader clock while one GEMM configuration runs back to back.

  python -m paper_1909_10616_amd.power_clock [--workload gemm4096_bf16]
      [--cfg JSON] [--seconds 12] [--vendor] [--out FILE.json]

A sampler child process (``amd-smi metric -p -c --json`` every ~0.3 s) is
started before this process touches the GPU; then the configuration is
launched in bursts of 500 for ``--seconds`` (per-launch time of every burst
from HIP events), and with ``--vendor`` torch.mm with fp32 output runs the
same way afterwards for scale. Reported per phase: launch time, socket
power and the mean / min / max over the XCDs of the shader clock, from the
samples taken in the second half of the phase (after the clock has settled).
The package power limit (``rocm-smi --showmaxpower``) is recorded too.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

SAMPLER = ("while true; do echo \"T $(date +%s.%N)\"; timeout -k 2 5 amd-smi metric -p -c --json; "
           "sleep 0.25; done")


def parse_samples(text):
    """(time, socket power W, [gfx clocks MHz]) per sample."""
    out = []
    for chunk in ("\n" + text).split("\nT ")[1:]:
        head, _, body = chunk.partition("\n")
        try:
            g = json.loads(body[body.index("{"):])["gpu_data"][0]
            clk = [v["clk"]["value"] for k, v in g["clock"].items()
                   if k.startswith("gfx_") and isinstance(v, dict) and isinstance(v.get("clk"), dict)]
            out.append((float(head), float(g["power"]["socket_power"]["value"]), clk))
        except (ValueError, KeyError, IndexError, TypeError):
            continue
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="gemm4096_bf16")
    ap.add_argument("--cfg", default=None, help="configuration as JSON (default: the known best)")
    ap.add_argument("--seconds", type=float, default=12.0)
    ap.add_argument("--vendor", action="store_true")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()

    limit = subprocess.run(["rocm-smi", "--showmaxpower", "--json"], capture_output=True, text=True)
    samples_path = (args.out or "power_clock.json") + ".samples"
    with open(samples_path, "w") as sf:
        sampler = subprocess.Popen(["bash", "-c", SAMPLER], stdout=sf, stderr=subprocess.STDOUT)
    try:
        phases = run_load(args)
    finally:
        sampler.terminate()
        sampler.wait(timeout=30)
    samples = parse_samples(open(samples_path).read())
    rows = []
    for name, t0, t1, us in phases:
        mid = t0 + (t1 - t0) / 2
        sel = [s for s in samples if mid <= s[0] <= t1]
        clk = [c for s in sel for c in s[2]]
        rows.append({"phase": name, "us_per_launch_median": statistics.median(us),
                     "samples": len(sel),
                     "socket_power_w": [min(s[1] for s in sel), max(s[1] for s in sel)] if sel else None,
                     "gfx_clock_mhz_mean": round(statistics.mean(clk)) if clk else None,
                     "gfx_clock_mhz_range": [min(clk), max(clk)] if clk else None})
        print(json.dumps(rows[-1]), flush=True)
    res = {"max_package_power": limit.stdout.strip(), "phases": rows}
    print(json.dumps(res), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            json.dump(res, f, indent=1)


def run_load(args):
    import torch
    from paper_1909_10616_amd import gemmtune as gt
    from workloads import WORKLOADS, workload_inputs

    if not torch.cuda.is_available():
        raise SystemExit("power_clock needs a GPU")
    gt.lib()
    w = WORKLOADS[args.workload]
    cfg = ((16, 2, 1, 128), (128, 1, 1, 32), (16, 4, 1, 64), 16)
    if args.cfg:
        cfg = tuple(tuple(x) if isinstance(x, list) else x for x in json.loads(args.cfg))
    dev = torch.device("cuda:0")
    A, B = workload_inputs(w)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty(w.M, w.N, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def phase(name, f):
        t0, us = time.time(), []
        while time.time() - t0 < args.seconds:
            e0.record()
            for _ in range(500):
                f()
            e1.record()
            e1.synchronize()
            us.append(e0.elapsed_time(e1) / 500 * 1e3)
            print(f"{name}: {us[-1]:.1f} us per launch", flush=True)
        return name, t0, time.time(), us[1:] or us

    out = [phase(f"{w.name} {gt.fmt_cfg(cfg)}", lambda: gt.gemm_run(cfg, Ad, Bd, C))]
    if args.vendor:
        time.sleep(3)
        out.append(phase("torch.mm fp32 out", lambda: torch.mm(Ad, Bd, out_dtype=torch.float32)))
    return out


if __name__ == "__main__":
    main()
