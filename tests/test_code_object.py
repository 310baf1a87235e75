"""The direct-load kernels set m0 inside inline assembly (the LDS address of
global_load_lds_dwordx4) and list it as clobbered, a register the compiler
reserves for itself. That is sound only while the compiler keeps no value of
its own in m0 across those statements. This test disassembles the gfx950 code
of every direct-load instantiation in the built objects and checks that m0 is
written only by the statement's own s_mov_b32, that the very next instruction
is the load that reads it, and that no instruction which reads m0 implicitly
(indexed register moves, messages, GWS, append/consume, LDS-DMA buffer loads,
interpolation) appears anywhere in those kernels."""
import os
import re
import subprocess

import pytest

LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"
IMPLICIT_M0 = re.compile(r"^\s*(v_movrel|s_movrel|s_sendmsg|ds_gws|ds_append|ds_consume|v_interp|"
                         r"s_set_gpr_idx|buffer_load_\w+.*\blds\b)")


@pytest.fixture(scope="module")
def objects():
    from paper_1909_10616_amd import build
    units = [u for u in build._units() if u[0].startswith("gemm_bf16_") and not u[0].endswith("_c0")]
    paths = [os.path.join(build.BUILD, u[0] + ".o") for u in units]
    if not all(os.path.exists(p) for p in paths):
        build.build(incremental=True, verbose=False)
    return paths


def _disassemble(obj, tmp_path):
    fb, co = tmp_path / "fatbin", tmp_path / "device.co"
    subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fb}", obj], check=True)
    subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o", f"--input={fb}",
                    f"--targets={TARGET}", f"--output={co}"], check=True)
    return subprocess.run([f"{LLVM}/llvm-objdump", "-d", str(co)], check=True,
                          capture_output=True, text=True).stdout.splitlines()


def test_direct_load_kernels_own_m0(objects, tmp_path):
    kernels = loads = 0
    for obj in objects:
        fn, prev = None, None
        for line in _disassemble(obj, tmp_path):
            m = re.match(r"^[0-9a-f]+ <(\w+)>:$", line)
            if m:
                fn, prev = m.group(1), None
                kernels += "gemm_kernel_dl" in fn
                continue
            if not fn or "gemm_kernel_dl" not in fn or not line.startswith("\t"):
                continue
            ins = line.split("//")[0].strip()
            where = f"{os.path.basename(obj)} {fn}: {ins}"
            assert not IMPLICIT_M0.match(ins), where
            if prev is not None and prev.startswith("s_mov_b32 m0,"):
                assert ins.startswith("global_load_lds_dwordx4 "), where
                loads += 1
            elif ins.startswith("global_load_lds"):
                raise AssertionError(f"load without its m0 write: {where}")
            if re.search(r"\bm0\b", ins):
                assert ins.startswith("s_mov_b32 m0,"), where
            prev = ins
    assert kernels >= 80 and loads > kernels
