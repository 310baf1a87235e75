"""Build libgemmtune.so (HIP, gfx950) in-tree.

Every source is compiled with hipcc for gfx950 into ``_build/`` in parallel
and linked into ``paper_1909_10616_amd/_lib/libgemmtune.so``. The kernel
family is split into one translation unit per (dtype, MFMA size, path).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "libgemmtune.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 vector ops stay off on this target
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-munsafe-fp-atomics",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _units():
    units = [
        ("space", "space.cpp", []),
        ("search", "search.cpp", []),
        ("runtime", "runtime.cpp", []),
        ("aux_kernels", "aux_kernels.hip", []),
        ("noalloc", "noalloc.hip", []),
    ]
    units.append(("gemm_lookup", "gemm_lookup.cpp", []))
    for dt, dn in ((0, "f32"), (1, "bf16")):
        for i in (16, 32):
            # CPR 0 is the generic path; the fast path needs CPR >= 64 / I
            for cpr in (0, 2, 4, 8, 16):
                if cpr and cpr < 64 // i:
                    continue
                units.append((f"gemm_{dn}_{i}_c{cpr}", "gemm_inst.hip",
                              [f"-DGT_DT={dt}", f"-DGT_I={i}", f"-DGT_CPR={cpr}"]))
                if cpr and dt == 0:  # fp32 fast path for a K-major A
                    units.append((f"gemm_{dn}_{i}_c{cpr}_akm", "gemm_inst.hip",
                                  [f"-DGT_DT={dt}", f"-DGT_I={i}", f"-DGT_CPR={cpr}",
                                   "-DGT_AKM=1"]))
    return units


def _deps(src):
    """Headers a source depends on: its own #include "…" lines, followed
    through csrc/ and include/ (local headers only)."""
    seen, todo = set(), [os.path.join(CSRC, src)]
    while todo:
        path = todo.pop()
        with open(path) as fh:
            for line in fh:
                line = line.strip()
                if not line.startswith('#include "'):
                    continue
                name = line.split('"')[1]
                for d in (CSRC, os.path.join(ROOT, "include")):
                    h = os.path.join(d, name)
                    if os.path.exists(h) and h not in seen:
                        seen.add(h)
                        todo.append(h)
    return seen


def _compile(unit, incremental=False):
    name, src, defs = unit
    obj = os.path.join(BUILD, name + ".o")
    if incremental and os.path.exists(obj):
        t = os.path.getmtime(obj)
        srcs = [os.path.join(CSRC, src), *_deps(src)]
        if all(t > os.path.getmtime(f) for f in srcs):
            return obj
    cmd = [HIPCC, *COMMON, "-x", "hip", *defs, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compile {name} failed:\n{err}")
    return obj


def build(jobs: int | None = None, verbose: bool = True, incremental: bool = False) -> str:
    """Compile every unit (incremental=True: only units older than their
    source or a header it includes) and link libgemmtune.so."""
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    jobs = jobs or min(16, os.cpu_count() or 4)
    units = _units()
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda u: _compile(u, incremental), units))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


def clean():
    shutil.rmtree(BUILD, ignore_errors=True)


if __name__ == "__main__":
    build()
