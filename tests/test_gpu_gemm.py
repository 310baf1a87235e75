"""GPU parity of the HIP kernel family against the fp64 oracle (through the C ABI).

Tolerances (normwise max relative error against the oracle on the exact
input bytes): fp32 ≤ 1e-5·√K, bf16 inputs with fp32 accumulation ≤ 2e-3.
Small-integer inputs make every partial sum exact in fp32, so those cases
must match bit-exactly, whatever the summation order (split-K atomics too).
"""
import os
import sys

import numpy as np
import pytest
import torch

from workloads import make_inputs, make_large_smallint_inputs, raw_bytes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gt():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_1909_10616_amd import gemmtune
    gemmtune.lib()
    return gemmtune


def tol(dtype, K):
    return 1e-5 * K ** 0.5 if dtype == "f32" else 2e-3


def rel_err(C, ref):
    return float(np.abs(C.astype(np.float64) - ref).max() / max(np.abs(ref).max(), 1e-300))


def run(gt, cfg, A, B):
    dev = torch.device("cuda:0")
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.full((A.shape[0], B.shape[1]), float("nan"), device=dev, dtype=torch.float32)
    gt.gemm_run(cfg, Ad, Bd, C)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


SINGLE_TILE = [
    # (dtype, M, N, K, config) — one wavefront, one MFMA tile
    ("bf16", 32, 32, 16, ((1, 1, 1, 32), (1, 1, 1, 16), (1, 1, 1, 32), 32)),
    ("bf16", 32, 32, 32, ((2, 1, 1, 16), (1, 1, 1, 32), (2, 1, 1, 16), 32)),
    ("bf16", 16, 16, 32, ((1, 1, 1, 16), (1, 1, 1, 32), (1, 1, 1, 16), 16)),
    ("bf16", 16, 16, 64, ((1, 1, 1, 16), (2, 1, 1, 32), (1, 1, 1, 16), 16)),
    ("f32", 32, 32, 8, ((1, 1, 1, 32), (1, 1, 1, 8), (1, 1, 1, 32), 0)),
    ("f32", 16, 16, 16, ((1, 1, 1, 16), (1, 1, 1, 16), (1, 1, 1, 16), 0)),
    ("f32", 16, 16, 4, ((1, 1, 1, 16), (4, 1, 1, 1), (1, 1, 1, 16), 0)),
]


@pytest.mark.parametrize("case", SINGLE_TILE, ids=[f"{c[0]}-{c[1]}x{c[2]}x{c[3]}-{i}"
                                                    for i, c in enumerate(SINGLE_TILE)])
def test_single_tile_bit_exact(gt, orc, case):
    dt, M, N, K, cfg = case
    info = gt.lower(cfg, M, N, K, dt)
    note(f"single tile {dt} {M}x{N}x{K} {cfg} fast={info['fast']}")
    A, B = make_inputs(M, N, K, dt, 21, "smallint")
    C = run(gt, cfg, A, B)
    ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, dt)
    assert np.array_equal(C.astype(np.float64), ref), rel_err(C, ref)


def _sample_configs(gt, orc, space_args, n, seed, extra=()):
    M, N, K, d, dt, mc = space_args
    ls = gt.Space(M, N, K, d, dt, mc)
    os_ = orc.Space(M, N, K, d, dt, mc)
    size = ls.size()
    rng = np.random.default_rng(seed)
    out = list(extra)
    tries = 0
    while len(out) < n + len(extra) and tries < 200000:
        tries += 1
        c = ls.unrank(int(rng.integers(0, size)))
        if not ls.legit(c):
            continue
        info = gt.lower(c, M, N, K, dt)
        # keep the sample cheap: skip configurations with huge grids of tiny tiles
        if info["grid_x"] * info["grid_y"] > 1 << 16:
            continue
        out.append(c)
    for c in out:
        assert ls.legit(c) and os_.legit(c)
    return out


SPACES = {
    "gemm256_f32": (256, 256, 256, (3, 3, 3), "f32", False),
    "bf16_256x256x512": (256, 256, 512, (4, 4, 4), "bf16", True),
    "bf16_odd96x80x48": (96, 80, 48, (4, 3, 4), "bf16", True),
    "f32_odd192x320x128": (192, 320, 128, (4, 4, 4), "f32", False),
}

EXTRA = {
    "gemm256_f32": [((256, 1, 1), (256, 1, 1), (256, 1, 1), 0),        # paper start state
                    ((2, 2, 64), (8, 4, 8), (2, 2, 64), 0),
                    ((4, 2, 32), (16, 4, 4), (4, 2, 32), 0)],
    "bf16_256x256x512": [((2, 2, 2, 32), (8, 1, 4, 16), (2, 2, 2, 32), 32),
                         ((2, 2, 4, 16), (4, 2, 2, 32), (2, 2, 2, 32), 16),
                         ((4, 2, 1, 32), (2, 4, 4, 16), (2, 2, 2, 32), 32),
                         ((256, 1, 1, 1), (512, 1, 1, 1), (256, 1, 1, 1), 16)],
    "bf16_odd96x80x48": [((3, 1, 1, 32), (3, 1, 16), (5, 1, 1, 16), 16),
                         ((3, 2, 1, 16), (3, 2, 8), (5, 1, 2, 8), 32)],
    "f32_odd192x320x128": [((3, 2, 1, 32), (4, 2, 4, 4), (5, 2, 2, 16), 0)],
}


@pytest.mark.parametrize("inputs", ["random", "smallint"])
@pytest.mark.parametrize("space", list(SPACES))
def test_sampled_configurations_match_oracle(gt, orc, space, inputs):
    M, N, K, d, dt, mc = SPACES[space]
    dist = "smallint" if inputs == "smallint" else ("normal" if dt == "bf16" else "uniform")
    A, B = make_inputs(M, N, K, dt, 5, dist)
    ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, dt)
    cfgs = _sample_configs(gt, orc, SPACES[space], 30, 100 + len(space), EXTRA.get(space, ()))
    n_fast = 0
    for cfg in cfgs:
        info = gt.lower(cfg, M, N, K, dt)
        n_fast += info["fast"]
        note(f"{space} {inputs} {cfg} fast={info['fast']} I={info['I']} TM={info['TM']} "
             f"TN={info['TN']} split={info['grid_y']}")
        C = run(gt, cfg, A, B)
        if inputs == "smallint":
            assert np.array_equal(C.astype(np.float64), ref), (cfg, rel_err(C, ref))
        else:
            e = rel_err(C, ref)
            assert e <= tol(dt, K), (cfg, e)
    note(f"{space}: {len(cfgs)} configurations, {n_fast} on the fast path")


def _rowcol_property(C, A, B, dt, orc):
    # C·1 = A·(B·1) and 1ᵀ·C = (1ᵀ·A)·B, evaluated in fp64 from the exact inputs
    a = orc.widen(raw_bytes(A), dt).reshape(A.shape)
    b = orc.widen(raw_bytes(B), dt).reshape(B.shape)
    C64 = C.astype(np.float64)
    rows = a @ b.sum(axis=1)
    cols = a.sum(axis=0) @ b
    rscale = np.abs(C64).sum(axis=1) + 1e-30
    cscale = np.abs(C64).sum(axis=0) + 1e-30
    assert np.all(np.abs(C64.sum(axis=1) - rows) <= 1e-4 * rscale)
    assert np.all(np.abs(C64.sum(axis=0) - cols) <= 1e-4 * cscale)


FULL = [
    # (workload name, configuration)
    ("gemm4096_bf16", ((16, 2, 4, 32), (64, 1, 4, 16), (16, 2, 4, 32), 32)),
    ("gemm4096_bf16", ((32, 2, 2, 32), (64, 1, 2, 32), (16, 2, 4, 32), 32)),
    ("gemm4096_bf16", ((32, 2, 4, 16), (128, 1, 1, 32), (32, 2, 4, 16), 16)),
    # 256x256x32 tiles, 8 wavefronts, direct-load ring of 5 stages (both MFMA sizes)
    ("gemm4096_bf16", ((16, 4, 2, 32), (128, 1, 2, 16), (16, 2, 4, 32), 32)),
    ("gemm4096_bf16", ((16, 2, 8, 16), (128, 1, 1, 32), (16, 4, 1, 64), 16)),
    ("mlp4096x11008x4096_bf16", ((16, 2, 4, 32), (64, 1, 4, 16), (43, 2, 4, 32), 32)),
    ("skinny64x4096x4096_bf16", ((1, 1, 2, 32), (16, 8, 2, 16), (32, 2, 2, 32), 32)),
    # 64x64 tiles, four K slices (8 wavefronts, direct-load ring)
    ("skinny64x4096x4096_bf16", ((1, 2, 2, 16), (8, 4, 1, 128), (64, 4, 1, 16), 16)),
    ("gemm1024_f32", ((8, 2, 2, 32), (32, 1, 4, 8), (8, 2, 2, 32), 0)),
    ("gemm2048_f32", ((16, 2, 2, 32), (64, 1, 4, 8), (16, 2, 2, 32), 0)),
    # one GPU's share of 4096³ split eight ways, along M and along M and N
    ("slab512x4096x4096_bf16", ((8, 1, 2, 32), (64, 1, 4, 16), (32, 4, 1, 32), 32)),
    ("slab1024x2048x4096_bf16", ((8, 2, 2, 32), (64, 1, 2, 32), (32, 2, 2, 16), 16)),
]


_FULL_REF = {}


def _oracle_threads():
    aff = len(os.sched_getaffinity(0))
    return max(1, min(int(os.environ.get("OMP_NUM_THREADS", "0")) or aff, aff))


def _full_oracle(orc, w, A, B):
    """The whole fp64 oracle product of a workload (kept for the module:
    several configurations share a workload)."""
    if w.name not in _FULL_REF:
        _FULL_REF.clear()
        _FULL_REF[w.name] = orc.gemm(raw_bytes(A), raw_bytes(B), w.M, w.N, w.K, w.dtype,
                                     nthreads=_oracle_threads())
    return _FULL_REF[w.name]


@pytest.mark.parametrize("case", FULL, ids=[f"{c[0]}-{i}" for i, c in enumerate(FULL)])
def test_full_size_every_element(gt, orc, case):
    """Every element of C at the workload list's full shapes against the fp64
    oracle's whole product (normwise max relative error within the dtype's
    tolerance), plus the row- and column-sum identities."""
    from workloads import WORKLOADS, workload_inputs
    w = WORKLOADS[case[0]]
    cfg = case[1]
    sp = gt.Space(w.M, w.N, w.K, w.d, w.dtype, w.mfma_coord)
    assert sp.legit(cfg)
    note(f"full size {w.name} {cfg} {gt.lower(cfg, w.M, w.N, w.K, w.dtype)}")
    A, B = workload_inputs(w)
    C = run(gt, cfg, A, B)
    assert np.isfinite(C).all()
    ref = _full_oracle(orc, w, A, B)
    e = rel_err(C, ref)
    note(f"  max |C - C*| / max |C*| = {e:.3e}")
    assert e <= tol(w.dtype, w.K), e
    _rowcol_property(C, A, B, w.dtype, orc)


def test_split_k_smallint_bit_exact(gt, orc):
    M, N, K = 64, 256, 1024
    A, B = make_inputs(M, N, K, "bf16", 8, "smallint")
    ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, "bf16")
    for cfg in [((1, 1, 2, 32), (4, 8, 2, 16), (4, 2, 1, 32), 32),
                ((2, 2, 1, 16), (2, 64, 1, 8), (2, 2, 2, 32), 16),
                ((64, 1, 1, 1), (1, 1024, 1, 1), (256, 1, 1, 1), 16),
                # 256 accumulators per lane (AGPRs)
                ((1, 1, 2, 32), (8, 4, 2, 16), (1, 1, 8, 32), 32)]:
        note(f"split-K {cfg} {gt.lower(cfg, M, N, K, 'bf16')}")
        C = run(gt, cfg, A, B)
        assert np.array_equal(C.astype(np.float64), ref), cfg


SPLITK_PATHS = [
    # (dtype, configuration, (fast, dl)) at 64x256x1024, split K
    ("bf16", ((2, 1, 2, 16), (16, 4, 4, 4), (2, 2, 2, 32), 16), (0, 0)),   # generic
    ("f32", ((2, 1, 2, 16), (16, 4, 4, 4), (2, 2, 2, 32), 16), (1, 0)),    # register-staged
    ("f32", ((2, 2, 1, 16), (4, 4, 8, 8), (4, 2, 2, 16), 0), (1, 0)),
    ("bf16", ((1, 1, 2, 32), (4, 8, 2, 16), (4, 2, 1, 32), 32), (1, 1)),   # direct-load
    ("bf16", ((1, 1, 2, 32), (8, 4, 4, 8), (4, 1, 2, 32), 32), (0, 0)),
]


@pytest.mark.parametrize("case", SPLITK_PATHS, ids=[f"{c[0]}-{i}" for i, c in enumerate(SPLITK_PATHS)])
def test_split_k_every_path_bit_exact(gt, orc, case):
    """Split K on each kernel path (the clear of C, then fp32 atomics from
    every slice), exact on small integers in any order of the adds."""
    dt, cfg, path = case
    M, N, K = 64, 256, 1024
    info = gt.lower(cfg, M, N, K, dt)
    note(f"split-K {dt} {cfg} {info}")
    assert (info["fast"], info["dl"]) == path and info["grid_y"] > 1
    A, B = make_inputs(M, N, K, dt, 9, "smallint")
    ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, dt)
    C = run(gt, cfg, A, B)
    assert np.array_equal(C.astype(np.float64), ref), cfg


def test_reference_compare_and_measure(gt, orc):
    dev = torch.device("cuda:0")
    M = N = K = 512
    A, B = make_inputs(M, N, K, "bf16", 2, "normal")
    ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, "bf16")
    Ad, Bd = A.to(dev), B.to(dev)
    R = torch.empty(M, N, device=dev)
    gt.gt_reference_gemm(Ad, Bd, R)
    torch.cuda.synchronize()
    assert rel_err(R.cpu().numpy(), ref) <= 2e-3
    assert gt.gt_compare(R, R) == 0.0
    C = torch.empty_like(R)
    cfg = ((4, 2, 2, 32), (8, 1, 4, 16), (4, 2, 2, 32), 32)
    m = gt.gt_measure(cfg, Ad, Bd, C, warmup=1, runs=10)
    assert m["mean_ms"] > 0 and not m["aborted"]
    assert gt.gt_compare(C, R) <= 2e-3
    C2 = C.clone()
    C2[3, 7] += 0.1 * float(R.abs().max())
    assert gt.gt_compare(C2, R) > 1e-2
    # early abort: a threshold below any kernel time stops after the warm-up
    m = gt.gt_measure(cfg, Ad, Bd, C, warmup=1, runs=10, abort_ms=1e-9)
    assert m["aborted"] and m["mean_ms"] == m["first_ms"]


@pytest.mark.parametrize("shape", [(512, 512, 1024), (256, 768, 512)])
def test_direct_load_path_bit_exact(gt, orc, shape):
    """Sampled configurations that lower to the direct-to-LDS ring path (bf16),
    small-integer inputs: every product must match the oracle bit-exactly."""
    M, N, K = shape
    sp = gt.Space(M, N, K, (4, 4, 4), "bf16", True)
    A, B = make_inputs(M, N, K, "bf16", 13, "smallint")
    ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, "bf16")
    rng = np.random.default_rng(M + N + K)
    seen, rings, tries = [], set(), 0
    while len(seen) < 24 and tries < 400000:
        tries += 1
        c = sp.unrank(int(rng.integers(0, sp.size())))
        if not sp.legit(c):
            continue
        info = gt.lower(c, M, N, K, "bf16")
        if not info["dl"]:
            continue
        seen.append(c)
        rings.add(info["ring"])
    assert len(seen) >= 8 and len(rings) >= 2, (len(seen), rings)
    for c in seen:
        info = gt.lower(c, M, N, K, "bf16")
        note(f"direct-load {shape} {c} ring={info['ring']} W={info['waves']} "
             f"{info['BM']}x{info['BN']}x{info['BK']} split={info['grid_y']}")
        C = run(gt, c, A, B)
        assert np.array_equal(C.astype(np.float64), ref), c



def test_shutdown_releases_and_library_stays_usable(gt, orc):
    """gt_shutdown frees the comparison buffers; calling it twice is fine and
    the library allocates again on the next use."""
    dev = torch.device("cuda:0")
    M = N = K = 256
    A, B = make_inputs(M, N, K, "f32", 3, "smallint")
    ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, "f32")
    Ad, Bd = A.to(dev), B.to(dev)
    R = torch.empty(M, N, device=dev)
    gt.gt_reference_gemm(Ad, Bd, R)
    assert gt.gt_compare(R, R) == 0.0          # allocates the buffer
    gt.gt_shutdown()
    gt.gt_shutdown()
    cfg = ((4, 2, 2, 16), (16, 1, 4, 4), (4, 2, 2, 16), 0)
    C = torch.full((M, N), float("nan"), device=dev)
    gt.gemm_run(cfg, Ad, Bd, C)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy().astype(np.float64), ref)
    assert gt.gt_compare(C, R) == 0.0          # allocates again
    gt.gt_shutdown()


def test_search_rejects_a_bad_reference_buffer(gt):
    """c_ref receives M·N fp32 values: a wrong size, dtype, device or layout
    is refused before the library sees it."""
    dev = torch.device("cuda:0")
    M = N = K = 64
    sp = gt.Space(M, N, K, (3, 3, 3), "f32", False)
    A = torch.zeros(M, K, device=dev)
    B = torch.zeros(K, N, device=dev)
    C = torch.zeros(M, N, device=dev)
    for bad in (torch.zeros(M * N - 1, device=dev), torch.zeros(M, N, device=dev, dtype=torch.bfloat16),
                torch.zeros(M, N), torch.zeros(N, M, device=dev).t()):
        with pytest.raises(ValueError):
            gt.tune_gbfs(sp, budget=2, A=A, B=B, C=C, c_ref=bad)


def test_operands_beyond_4_gib(gt, orc):
    """Operands of several GiB, split 256 ways along K (M = N = 256, bf16).
    At K = 9·2^20 (A and B 4.5 GiB each) byte offsets from each operand's
    start pass 2^32, which the register-staged and generic kernels address
    with 64-bit offsets; the direct-load ring, whose per-lane offsets from a
    stage origin are 32-bit, is not chosen there. At K = 7·2^20 the ring is
    chosen and its lane offsets reach 3.74 GB, near their 2^32 limit. Inputs
    in {-1, 0, 1}, so every partial sum, in any order, is an integer of at
    most K < 2^24 in magnitude and exact in fp32: sampled entries, the last
    rows and columns among them, equal the oracle exactly."""
    M = N = 256
    cases = [(9 << 20, [((1, 2, 4, 32), None, (1, 4, 2, 32), 16, 1, 32, (1, 0)),     # register-staged
                        ((1, 2, 4, 32), None, (1, 4, 2, 32), 16, 8, 4, (0, 0))]),    # generic
             (7 << 20, [((1, 2, 4, 32), None, (1, 4, 2, 32), 16, 1, 32, (1, 1))])]   # direct-load
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(4)
    rows = np.concatenate([[0, M - 1, M - 1, 0], rng.integers(0, M, 60)])
    cols = np.concatenate([[0, N - 1, 0, N - 1], rng.integers(0, N, 60)])
    for K, cfgs in cases:
        note(f"K = {K}: drawing 2 x {M * K * 2 / 2 ** 30:.2f} GiB of small-integer inputs")
        A, B = make_large_smallint_inputs(M, N, K, "bf16", 31, bound=1)
        Ad, Bd = A.to(dev), B.to(dev)
        ref = orc.gemm_entries(raw_bytes(A), raw_bytes(B), M, N, K, "bf16", rows, cols)
        del A, B
        for m, _, n, mfma, ksub, kblk, path in cfgs:
            cfg = (m, (K // (ksub * kblk) // 256, 256, ksub, kblk), n, mfma)
            info = gt.lower(cfg, M, N, K, "bf16")
            note(f"  {gt.fmt_cfg(cfg)} fast={info['fast']} dl={info['dl']} split={info['grid_y']}")
            assert (info["fast"], info["dl"]) == path and info["grid_y"] == 256
            C = torch.full((M, N), float("nan"), device=dev)
            gt.gemm_run(cfg, Ad, Bd, C)
            torch.cuda.synchronize()
            got = C.cpu().numpy().astype(np.float64)[rows, cols]
            assert np.array_equal(got, ref), cfg
        del Ad, Bd
        torch.cuda.empty_cache()


def test_reference_product_of_a_tall_shape(gt, orc):
    """The check product the searches compare candidates with, on a shape
    with more rows than one grid dimension holds blocks of four (393,216 rows
    > 4·65,535): the kernel strides over the rest. Small integers: sampled
    entries, the last row among them, equal the oracle exactly."""
    M, N, K = 3 << 17, 64, 64
    A, B = make_inputs(M, N, K, "bf16", 41, "smallint")
    dev = torch.device("cuda:0")
    R = torch.full((M, N), float("nan"), device=dev)
    gt.gt_reference_gemm(A.to(dev), B.to(dev), R)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    rows = np.concatenate([[M - 1, M - 1, 4 * 65535, 0], rng.integers(0, M, 124)])
    cols = np.concatenate([[0, N - 1, 7, 0], rng.integers(0, N, 124)])
    ref = orc.gemm_entries(raw_bytes(A), raw_bytes(B), M, N, K, "bf16", rows, cols)
    got = R.cpu().numpy().astype(np.float64)
    assert np.array_equal(got[rows, cols], ref)
    assert not np.isnan(got).any()
