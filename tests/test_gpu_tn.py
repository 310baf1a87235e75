"""GPU parity of the K-major-A layout (the perceptron product Y = WᵀX of §5)
against the fp64 oracle, through the C ABI: sampled configurations of small
spaces (generic path, fp32 fast path with the K-major kernel), bit-exact on
small-integer inputs; sampled entries at 2048³; and a G-BFS on the paper's
space shape (d = (4, 2, 4), neighbours between any two levels) replayed
through the oracle's Alg.1."""
import math
import sys

import numpy as np
import pytest
import torch

from workloads import make_perceptron_inputs, raw_bytes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gt():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_1909_10616_amd import gemmtune
    gemmtune.lib()
    return gemmtune


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_tn(gt, cfg, W, X):
    dev = torch.device("cuda:0")
    K, M = W.shape
    C = torch.full((M, X.shape[1]), float("nan"), device=dev, dtype=torch.float32)
    gt.gemm_run(cfg, W.to(dev), X.to(dev), C, a_kmajor=True)
    torch.cuda.synchronize()
    return C.cpu().numpy()


SPACES = {
    # (M, N, K, d, dtype, mfma_coord)
    "f32_256_d424": (256, 256, 256, (4, 2, 4), "f32", False),
    "f32_odd192x320x128": (192, 320, 128, (4, 4, 4), "f32", False),
    "bf16_128x256x256": (128, 256, 256, (4, 4, 4), "bf16", True),
}
EXTRA = {  # fp32 fast-path configurations (K-major kernel), both MFMA sizes
    "f32_256_d424": [((2, 2, 2, 32), (16, 16), (2, 2, 2, 32), 0),
                     ((4, 2, 2, 16), (8, 32), (4, 1, 4, 16), 0),
                     ((2, 2, 1, 64), (4, 64), (2, 1, 2, 64), 0),
                     ((256, 1, 1, 1), (256, 1), (256, 1, 1, 1), 0)],   # the paper's s0
    "f32_odd192x320x128": [((3, 2, 1, 32), (4, 2, 4, 4), (5, 2, 2, 16), 0),
                           ((3, 2, 2, 16), (2, 2, 2, 16), (5, 1, 4, 16), 0)],
}


def _sample(gt, space_args, n, seed, extra, mode):
    M, N, K, d, dt, mc = space_args
    sp = gt.Space(M, N, K, d, dt, mc, mode=mode, a_kmajor=True)
    rng = np.random.default_rng(seed)
    out = list(extra)
    code = gt.dtype_code(dt) | gt.A_KMAJOR
    while len(out) < n + len(extra):
        c = sp.unrank(int(rng.integers(0, sp.size())))
        if not sp.legit(c):
            continue
        info = gt.lower(c, M, N, K, code)
        if info["grid_x"] * info["grid_y"] > 1 << 16:
            continue
        out.append(c)
    assert all(sp.legit(c) for c in out)
    return out, code


@pytest.mark.parametrize("inputs", ["random", "smallint"])
@pytest.mark.parametrize("space", list(SPACES))
def test_tn_sampled_configurations_match_oracle(gt, orc, space, inputs):
    M, N, K, d, dt, mc = SPACES[space]
    dist = "smallint" if inputs == "smallint" else ("normal" if dt == "bf16" else "uniform")
    W, X = make_perceptron_inputs(M, N, K, dt, 7, dist)
    ref = orc.gemm_tn(raw_bytes(W), raw_bytes(X), M, N, K, dt)
    cfgs, code = _sample(gt, SPACES[space], 24, 300 + len(space), EXTRA.get(space, ()),
                         gt.ANY_PAIR)
    n_fast = 0
    for cfg in cfgs:
        info = gt.lower(cfg, M, N, K, code)
        assert info["dl"] == 0
        n_fast += info["fast"]
        note(f"tn {space} {inputs} {cfg} fast={info['fast']} I={info['I']} split={info['grid_y']}")
        C = run_tn(gt, cfg, W, X)
        if inputs == "smallint":
            assert np.array_equal(C.astype(np.float64), ref), cfg
        else:
            e = np.abs(C.astype(np.float64) - ref).max() / np.abs(ref).max()
            assert e <= (1e-5 * K ** 0.5 if dt == "f32" else 2e-3), (cfg, e)
    if dt == "f32" and space in EXTRA:
        assert n_fast >= 2
    note(f"tn {space}: {len(cfgs)} configurations, {n_fast} on the fast path")


def test_tn_full_size_sampled_entries(gt, orc):
    """2048³ fp32 perceptron inputs, two fast-path configurations: sampled
    entries against the oracle, computed one by one."""
    M = N = K = 2048
    W, X = make_perceptron_inputs(M, N, K, "f32", 0, "uniform")
    A_bytes = raw_bytes(W.t().contiguous())   # A = Wᵀ element by element
    rng = np.random.default_rng(2)
    rows = np.concatenate([[0, M - 1], rng.integers(0, M, 126)])
    cols = np.concatenate([[0, N - 1], rng.integers(0, N, 126)])
    ref = orc.gemm_entries(A_bytes, raw_bytes(X), M, N, K, "f32", rows, cols)
    for cfg in [((16, 2, 2, 32), (256, 8), (16, 2, 2, 32), 0),
                ((16, 2, 4, 16), (128, 16), (8, 2, 4, 32), 0)]:
        info = gt.lower(cfg, M, N, K, gt.dtype_code("f32") | gt.A_KMAJOR)
        note(f"tn full size {cfg} {info}")
        assert info["fast"] == 1
        C = run_tn(gt, cfg, W, X)
        got = C[rows, cols].astype(np.float64)
        assert np.abs(got - ref).max() / np.abs(ref).max() <= 1e-5 * K ** 0.5


def test_tn_gbfs_paper_space_replays_in_oracle(gt, orc):
    """G-BFS on a 256³ perceptron space of the paper's shape from its s0
    [[m,1,1,1],[k,1],[n,1,1,1]]: every timed output matched the reference,
    and the oracle's Alg.1 fed the logged costs takes the same trajectory."""
    M = N = K = 256
    dev = torch.device("cuda:0")
    W, X = make_perceptron_inputs(M, N, K, "f32", 0, "uniform")
    Wd, Xd = W.to(dev), X.to(dev)
    C = torch.empty(M, N, device=dev)
    sp = gt.Space(M, N, K, (4, 2, 4), "f32", False, mode=gt.ANY_PAIR, a_kmajor=True)
    s0 = ((M, 1, 1, 1), (K, 1), (N, 1, 1, 1), 0)
    note("tn gbfs 256^3 budget 60")
    res = gt.tune_gbfs(sp, budget=60, s0=s0, rho=5, seed=4, A=Wd, B=Xd, C=C)
    log = res["log"]
    assert all(e["status"] in ("ok", "early-abort") for e in log)
    osp = orc.Space(M, N, K, (4, 2, 4), "f32", False, mode=orc.ANY_PAIR)
    table = {e["rank"]: e["cost_ms"] for e in log}
    rep = orc.gbfs(osp, s0, 5, 60, 4, lambda c, r: table.get(r, math.inf))
    assert rep["log_ranks"] == [e["rank"] for e in log] and rep["best"] == res["best"]
    gt.gemm_run(res["best"], Wd, Xd, C, a_kmajor=True)
    torch.cuda.synchronize()
    ref = orc.gemm_tn(raw_bytes(W), raw_bytes(X), M, N, K, "f32")
    e = np.abs(C.cpu().numpy().astype(np.float64) - ref).max() / np.abs(ref).max()
    assert e <= 1e-5 * K ** 0.5
    note(f"tn gbfs best {res['best']} {gt.tflops(M, N, K, res['best_cost']):.2f} TFLOP/s")
