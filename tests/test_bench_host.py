"""Host-side pieces of bench.py: the one-GPU guard, the kernel naming and
launch signature the profiles are keyed by, and the traffic lookup that
must only answer for the current kernel sources."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    sys.path.insert(0, ROOT)
    import bench as b
    from paper_1909_10616_amd import gemmtune
    if not os.path.exists(gemmtune.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return b


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_signature_and_traffic_lookup(bench, tmp_path, monkeypatch):
    from paper_1909_10616_amd import gemmtune as gt
    from workloads import WORKLOADS
    w = WORKLOADS["gemm4096_bf16"]
    cfg = ((16, 2, 1, 128), (128, 1, 1, 32), (16, 4, 1, 64), 16)
    info = gt.lower(cfg, w.M, w.N, w.K, w.dtype)
    assert bench.kernel_name(w, info) == "gt::gemm_kernel_dl<16, 8, 4, 4>"
    sig = bench.launch_signature(w, info)
    assert sig == ("gemm4096_bf16 gt::gemm_kernel_dl<16,8,4,4> grid=256x1 waves=8 "
                   "lds=163840 dl=1/5")
    # a private profiles/traffic.txt: the line counts only with the current source hash
    prof = tmp_path / "profiles"
    prof.mkdir()
    src = bench.kernel_source_hash()
    (prof / "traffic.txt").write_text(
        "# comment | not a record\n"
        f"{sig} | source=0000000000000000 traffic_bytes=1\n"
        f"{sig} | source={src} traffic_bytes=268905035\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: src)
    assert bench.measured_traffic(w, info) == 268905035
    (prof / "traffic.txt").write_text(f"{sig} | source=0000000000000000 traffic_bytes=1\n")
    assert bench.measured_traffic(w, info) is None
    other = dict(info, grid_y=2)
    (prof / "traffic.txt").write_text(f"{sig} | source={src} traffic_bytes=5\n")
    assert bench.measured_traffic(w, other) is None


def test_committed_traffic_line_matches_the_sources(bench):
    """profiles/traffic.txt holds a line for the bench's usual winner under the
    kernel sources in the tree (it is refreshed whenever they change)."""
    lines = [l for l in open(os.path.join(ROOT, "profiles", "traffic.txt"))
             if not l.startswith("#") and "|" in l]
    assert any(f"source={bench.kernel_source_hash()}" in l for l in lines)


def test_roofline_bound_follows_arithmetic_intensity(bench):
    """MFMA-bound at or above the ridge (peak over 8 TB/s), HBM-bound below
    it, with the other unit's fraction beside it."""
    # 4096³ bf16: 2·4096³ flop over 134,217,728 B = 1024 flop/B, ridge 314.6
    r = bench.roofline("bf16", 4096, 4096, 4096, 134217728, 1238.36, 1209.3, 269026764)
    assert (r["bound"], r["unit"], r["peak"], r["achieved"]) == ("mfma", "TFLOP/s", 2516.6, 1238.36)
    assert r["frac"] == round(1238.36 / 2516.6, 4) and r["hbm_frac"] == round(1209.3 / 8000, 4)
    assert (r["arithmetic_intensity"], r["ridge"], r["traffic"]) == (1024.0, 314.6, 269026764)
    # 64×4096×4096 bf16: (64·4096 + 4096²)·2 + 64·4096·4 = 35,127,296 B, 61.1 flop/B
    alg = (64 * 4096 + 4096 * 4096) * 2 + 64 * 4096 * 4
    ms = 0.0142
    tf, gbs = 2 * 64 * 4096 * 4096 / (ms * 1e-3) / 1e12, alg / (ms * 1e-3) / 1e9
    r = bench.roofline("bf16", 64, 4096, 4096, alg, tf, gbs, None)
    assert (r["bound"], r["unit"], r["peak"]) == ("hbm", "GB/s", 8000.0)
    assert r["achieved"] == round(gbs, 1) and r["frac"] == round(gbs / 8000, 4)
    assert r["mfma_frac"] == round(tf / 2516.6, 4) and r["arithmetic_intensity"] == 61.1
    # 2048³ fp32: 341.3 flop/B against a ridge of 19.7
    r = bench.roofline("f32", 2048, 2048, 2048, 3 * 2048 * 2048 * 4, 110.0, 500.0, None)
    assert r["bound"] == "mfma" and r["ridge"] == 19.7 and r["arithmetic_intensity"] == 341.3


def test_hand_start_is_legitimate_on_every_workload(bench):
    """The hand-crafted start: 128×128 workgroup tiles (2×2 wavefronts of
    2×2 32-wide blocks) where 128 divides M and N, else 64×64 (one block per
    wavefront); 32-deep K stages; legitimate in every workload's space."""
    from paper_1909_10616_amd import gemmtune as gt
    from workloads import WORKLOADS
    for w in WORKLOADS.values():
        s0 = bench.hand_s0(w)
        sp = gt.Space(w.M, w.N, w.K, w.d, w.dtype, w.mfma_coord)
        assert sp.legit(s0), (w.name, s0)
        m, k, n, mfma = s0
        assert mfma == (32 if w.mfma_coord else 0)
        if tuple(w.d) == (4, 4, 4):
            tile = 128 if w.M % 128 == 0 and w.N % 128 == 0 else 64
            assert m[1:] == ((2, 2, 32) if tile == 128 else (2, 1, 32)) or w.M < 64
            assert n[1:] == ((2, 2, 32) if tile == 128 else (2, 1, 32))
            assert m[0] * tile == w.M and n[0] * tile == w.N and k == (w.K // 32, 1, 2, 16)
    assert bench.hand_s0(WORKLOADS["gemm4096_bf16"]) == \
        ((32, 2, 2, 32), (128, 1, 2, 16), (32, 2, 2, 32), 32)
    assert bench.hand_s0(WORKLOADS["skinny64x4096x4096_bf16"]) == \
        ((1, 2, 1, 32), (128, 1, 2, 16), (64, 2, 1, 32), 32)


def test_componentwise_error(bench):
    """max |C − C*| / (|A|·|B|): rounding the oracle's fp64 product to fp32
    stays within 2^-24 (|fl(c) − c| ≤ 2^-24·|c| ≤ 2^-24·(|A|·|B|)); an error
    planted in one element is seen at its own scale."""
    import numpy as np
    import oracle
    from workloads import make_inputs, raw_bytes

    class W:
        M, N, K, dtype = 48, 40, 64, "bf16"
    A, B = make_inputs(W.M, W.N, W.K, W.dtype, 5, "normal")
    C = oracle.gemm(raw_bytes(A), raw_bytes(B), W.M, W.N, W.K, W.dtype)
    assert bench.componentwise_error(W, A, B, C.astype(np.float32), C) <= 2.0 ** -24
    absab = np.abs(A.float().numpy().astype(np.float64)) @ np.abs(B.float().numpy().astype(np.float64))
    Cg = C.copy()
    Cg[7, 9] += 1e-3 * absab[7, 9]
    assert abs(bench.componentwise_error(W, A, B, Cg, C) - 1e-3) <= 1e-9


@pytest.mark.parametrize("methods,ok", [("gbfs,na2c", True), ("random", True), ("gbfs,bogus", False),
                                        (",", False)])
def test_compare_search_methods_are_checked_before_any_gpu_work(methods, ok):
    """compare_search refuses an unknown search before it touches torch or a
    GPU; a valid list passes that check and stops later, at the missing GPU
    or at the unknown workload name (so no search ever starts here)."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, "-m", "paper_1909_10616_amd.compare_search", "--methods", methods,
                        "--workload", "no_such_workload"],
                       capture_output=True, text=True, timeout=300,
                       cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    assert r.returncode != 0
    assert ("--methods:" in r.stderr) == (not ok), r.stderr[-500:]


def test_kernel_fingerprint_ignores_comments_not_code(bench):
    """The kernel-source fingerprint reads code only: comments and layout do
    not change it, a changed token does."""
    code = "int f(int a) {  // doubles\n  /* the\n     body */\n  return 2 * a;\n}\n\n"
    assert bench._code_only(code) == bench._code_only(code.replace("doubles", "twice")
                                                      .replace("the\n", "a\n") + "\n// end\n")
    assert bench._code_only(code) != bench._code_only(code.replace("2 * a", "3 * a"))
    assert "//" not in bench._code_only(code) and "/*" not in bench._code_only(code)
