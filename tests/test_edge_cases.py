"""Edge cases of the space, the search and the kernels: empty extents, the
one-point space, prime and odd extents, single-level spaces, the largest
extents the space accepts, and the smallest products on the GPU.

An empty extent has no factorisation into positive integers (Eq.2-4 take the
factors from the positive integers), so both the oracle and the library
reject it instead of returning an empty space."""
import ctypes
import os

import numpy as np
import pytest
import torch

from workloads import make_inputs, raw_bytes


@pytest.fixture(scope="module")
def gt():
    from paper_1909_10616_amd import gemmtune
    if not os.path.exists(gemmtune.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    gemmtune.lib()
    return gemmtune


def _orc_size(orc, M, N, K, d=(4, 4, 4)):
    sp = orc.Space(M, N, K, d)
    out = ctypes.c_uint64()
    rc = orc.lib().or_space_size(ctypes.byref(sp._s), ctypes.byref(out))
    return rc, int(out.value)


@pytest.mark.parametrize("dims", [(0, 16, 16), (16, 0, 16), (16, 16, 0)])
def test_empty_extent_rejected_by_both(gt, orc, dims):
    rc, _ = _orc_size(orc, *dims)
    assert rc != 0
    with pytest.raises(gt.GemmTuneError):
        gt.Space(*dims, (4, 4, 4), "f32", False).size()


def test_extent_limits(gt, orc):
    # the library bounds extents to [1, 2^40]; the closed form still holds there
    big = 1 << 40
    sp = gt.Space(big, 1, 1, (2, 1, 1), "f32", False)
    assert sp.size() == 41                      # C(40 + 1, 1) tuples for d = 2
    rc, n = _orc_size(orc, big, 1, 1, (2, 1, 1))
    assert rc == 0 and n == 41
    with pytest.raises(gt.GemmTuneError):
        gt.Space(big + 2, 1, 1, (2, 1, 1), "f32", False).size()
    with pytest.raises(gt.GemmTuneError):
        gt.Space(16, 16, 16, (5, 4, 4), "f32", False).size()


@pytest.mark.parametrize("mfma", [False, True])
def test_one_point_space(gt, orc, mfma):
    """M = N = K = 1: one tuple per dimension; the only moves are the MFMA
    toggle (when the coordinate exists). G-BFS times s0 (and the toggle) and
    stops on an empty queue."""
    dt = "bf16" if mfma else "f32"
    sp = gt.Space(1, 1, 1, (4, 4, 4), dt, mfma)
    osp = orc.Space(1, 1, 1, (4, 4, 4), dt, mfma)
    n = 2 if mfma else 1
    assert sp.size() == osp.size() == n
    lib_all = sp.enumerate()
    orc_all = osp.enumerate()
    assert [c for c, _ in lib_all] == [c for c, _ in orc_all]
    ones = (1, 1, 1, 1)
    assert lib_all[0][0][:3] == (ones, ones, ones)
    s0 = lib_all[0][0]
    assert sp.legit(s0) and osp.legit(s0)
    lib_nb = [c for c, _ in sp.neighbours(s0)]
    orc_nb = [c for c, _ in osp.neighbours(s0)]
    assert lib_nb == orc_nb == ([(ones, ones, ones, 32)] if mfma else [])
    r = gt.tune_gbfs(sp, budget=10, s0=s0, cost_fn=lambda c, rank: 1.0 + rank)
    assert r["timed"] == n and r["stop_reason"] == "queue-empty"
    assert r["best"] == s0
    o = orc.gbfs(osp, s0, 5, 10, 0, lambda c, rank: 1.0 + rank)
    assert o["timed"] == n and tuple(o["best"]) == s0


@pytest.mark.parametrize("dims", [(7, 3, 5), (1, 11, 13), (97, 1, 1)])
def test_odd_extents_single_tuple(gt, orc, dims):
    """Extents without a factor of two leave only [D, 1, ..., 1] per dimension."""
    M, N, K = dims
    sp = gt.Space(M, N, K, (4, 3, 2), "f32", False)
    osp = orc.Space(M, N, K, (4, 3, 2), "f32", False)
    assert sp.size() == osp.size() == 1
    (cfg, _), = sp.enumerate()
    assert cfg == ((M, 1, 1, 1), (K, 1, 1), (N, 1), 0)
    assert [c for c, _ in sp.neighbours(cfg)] == [] == [c for c, _ in osp.neighbours(cfg)]


def test_single_level_spaces(gt, orc):
    sp = gt.Space(64, 32, 128, (1, 1, 1), "bf16", True)
    osp = orc.Space(64, 32, 128, (1, 1, 1), "bf16", True)
    assert sp.size() == osp.size() == 2
    assert [c for c, _ in sp.enumerate()] == [c for c, _ in osp.enumerate()]


# ---------------------------------------------------------------------------
# GPU: the smallest products and odd shapes, through the C ABI
# ---------------------------------------------------------------------------

def _run(gt, cfg, A, B):
    dev = torch.device("cuda:0")
    C = torch.full((A.shape[0], B.shape[1]), float("nan"), device=dev, dtype=torch.float32)
    gt.gemm_run(cfg, A.to(dev), B.to(dev), C)
    torch.cuda.synchronize()
    return C.cpu().numpy()


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dims", [(1, 1, 1), (7, 5, 3), (1, 64, 96), (33, 1, 17)])
def test_tiny_and_odd_products_exact(gt, orc, dtype, dims):
    """Every configuration of a small space on small-integer inputs: the
    products are exact in fp32 accumulation, so C must equal the oracle bit
    for bit (this covers blocks smaller than the MFMA tile, single-element
    rows and columns, and K shorter than one MFMA step)."""
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    M, N, K = dims
    mf = dtype == "bf16"
    sp = gt.Space(M, N, K, (2, 2, 2), dtype, mf)
    A, B = make_inputs(M, N, K, dtype, 23, "smallint")
    ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, dtype)
    ran = 0
    for cfg, legit in sp.enumerate():
        if not legit:
            continue
        print(f"tiny {dtype} {dims} {cfg}", flush=True)
        C = _run(gt, cfg, A, B)
        assert np.array_equal(C.astype(np.float64), ref), cfg
        ran += 1
    assert ran >= 1
