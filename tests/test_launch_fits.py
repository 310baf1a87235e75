"""The hardware clauses of J (§3.3, Eq.5 allows such constraints) checked
against the kernels the build actually produced, not against the oracle's
copy of the same formulas. For every legitimate configuration of several
spaces the test lowers the configuration, finds the instantiation it
launches in the gfx950 code objects, reads that kernel's metadata (register
allocation, largest workgroup, static LDS) and checks that the launch fits
the hardware:

* 64·W threads ≤ the kernel's `.max_flat_workgroup_size`;
* ⌈W/4⌉ wavefronts per SIMD × the kernel's registers per lane (VGPRs and
  AGPRs, in granules of 8) ≤ 512, the unified register file of a SIMD;
* dynamic LDS of the launch + the kernel's static LDS ≤ 160 KiB per
  workgroup.

J is a sufficient condition: a configuration it admits always fits. (It is
conservative: some configurations it rejects would also fit.)"""
import math
import os
import random
import subprocess

import pytest
import yaml

LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"
LDS_BYTES = 160 * 1024
REGS_PER_SIMD_LANE = 512


@pytest.fixture(scope="module")
def gt():
    from paper_1909_10616_amd import gemmtune
    if not os.path.exists(gemmtune.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    gemmtune.lib()
    return gemmtune


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    """Mangled kernel name → its metadata, from every GEMM object built."""
    from paper_1909_10616_amd import build
    paths = [os.path.join(build.BUILD, u[0] + ".o") for u in build._units()
             if u[0].startswith("gemm_") and u[1].endswith(".hip")]
    if not all(os.path.exists(p) for p in paths):
        build.build(incremental=True, verbose=False)
    tmp = tmp_path_factory.mktemp("co")
    fb, co = tmp / "fatbin", tmp / "device.co"
    out = {}
    for obj in paths:
        subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fb}", obj], check=True)
        subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o",
                        f"--input={fb}", f"--targets={TARGET}", f"--output={co}"], check=True)
        notes = subprocess.run([f"{LLVM}/llvm-readelf", "--notes", str(co)], check=True,
                               capture_output=True, text=True).stdout
        doc = notes[notes.index("---"):]
        doc = doc[:doc.index("\n...")] if "\n..." in doc else doc
        for k in yaml.safe_load(doc)["amdhsa.kernels"]:
            out[k[".name"]] = k
    assert len(out) > 500
    return out


def symbol(info, dtype, akm):
    """Mangled name of the instantiation a lowered configuration launches."""
    dt = 1 if dtype == "bf16" else 0
    cpr = info["BK"] // (8 if dtype == "bf16" else 4) if info["fast"] else 0
    I, TM, TN = info["I"], info["TM"], info["TN"]
    if info["dl"]:
        return f"_ZN2gt14gemm_kernel_dlILi{I}ELi{TM}ELi{TN}ELi{cpr}EEEvNS_5KArgsE"
    name = "15gemm_kernel_akm" if akm and info["fast"] else "11gemm_kernel"
    return f"_ZN2gt{name}ILi{dt}ELi{I}ELi{TM}ELi{TN}ELi{cpr}EEEvNS_5KArgsE"


def fits(k, info):
    W = info["waves"]
    regs = math.ceil(k[".vgpr_count"] / 8) * 8
    return (64 * W <= k[".max_flat_workgroup_size"]
            and math.ceil(W / 4) * regs <= REGS_PER_SIMD_LANE
            and info["lds_bytes"] + k[".group_segment_fixed_size"] <= LDS_BYTES)


SPACES = [
    # (M, N, K, d, dtype, mfma_coord, a_kmajor, samples)
    (4096, 4096, 4096, (4, 4, 4), "bf16", True, False, 3000),
    (4096, 11008, 4096, (4, 4, 4), "bf16", True, False, 2000),
    (64, 4096, 4096, (4, 4, 4), "bf16", True, False, 2000),
    (1024, 1024, 1024, (4, 4, 4), "f32", False, False, 2000),
    (2048, 2048, 2048, (4, 4, 4), "f32", False, False, 2000),
    (2048, 2048, 2048, (4, 2, 4), "f32", False, True, 2000),
    (256, 256, 512, (4, 4, 4), "bf16", True, True, 1000),
    (96, 80, 48, (4, 3, 4), "bf16", True, False, 1000),
]


@pytest.mark.parametrize("space", SPACES, ids=[f"{s[0]}x{s[1]}x{s[2]}-{s[4]}{'-kmajor' if s[6] else ''}"
                                               for s in SPACES])
def test_every_legitimate_launch_fits_its_compiled_kernel(gt, kernels, space):
    M, N, K, d, dt, mc, akm, samples = space
    sp = gt.Space(M, N, K, d, dt, mc, a_kmajor=akm)
    code = gt.dtype_code(dt) | (gt.A_KMAJOR if akm else 0)
    rng = random.Random(M + 3 * N + 7 * K + akm)
    size = sp.size()
    legit = tries = 0
    while legit < samples and tries < 200 * samples:
        tries += 1
        c = sp.unrank(rng.randrange(size))
        if not sp.legit(c):
            continue          # the library does not lower these
        legit += 1
        info = gt.lower(c, M, N, K, code)
        k = kernels.get(symbol(info, dt, akm))
        assert k is not None, (c, info)   # the lowering table and the objects agree
        assert fits(k, info), (c, info, {f: k[f] for f in (".vgpr_count", ".agpr_count",
                               ".max_flat_workgroup_size", ".group_segment_fixed_size")})
    assert legit == samples


def test_the_fastest_configurations_fit(gt, kernels):
    """The configurations the searches settle on at the workload shapes."""
    cases = [
        (4096, 4096, 4096, "bf16", ((16, 2, 8, 16), (128, 1, 1, 32), (16, 4, 2, 32), 16)),
        (4096, 11008, 4096, "bf16", ((16, 2, 4, 32), (128, 1, 1, 32), (43, 4, 2, 32), 16)),
        (64, 4096, 4096, "bf16", ((2, 2, 1, 16), (32, 1, 4, 32), (128, 2, 1, 16), 16)),
        (1024, 1024, 1024, "f32", ((32, 2, 1, 16), (16, 1, 8, 8), (16, 2, 1, 32), 0)),
    ]
    for M, N, K, dt, c in cases:
        info = gt.lower(c, M, N, K, dt)
        k = kernels[symbol(info, dt, False)]
        assert fits(k, info), (c, info)
        assert k[".private_segment_fixed_size"] == 0, c   # and none of them spills
