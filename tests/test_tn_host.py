"""The perceptron layout of §5 (Y = WᵀX, W given K×M) on the host side:
the oracle's product pinned to independent facts, the library's lowering of
K-major-A configurations, and the paper-protocol budgets."""
import math
import os

import numpy as np
import pytest

from workloads import PAPER_PROTOCOL, make_perceptron_inputs, raw_bytes


@pytest.fixture(scope="module")
def gt():
    from paper_1909_10616_amd import gemmtune
    if not os.path.exists(gemmtune.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    gemmtune.lib()
    return gemmtune


def _f32_bytes(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint8).reshape(-1)


def test_oracle_tn_identity_and_permutation(orc):
    """W = I gives Y = X; W a permutation matrix P gives Y = PᵀX, i.e. row i
    of Y is row p(i) of X, exactly."""
    rng = np.random.default_rng(0)
    K, N = 24, 40
    X = rng.uniform(-1, 1, (K, N)).astype(np.float32)
    Y = orc.gemm_tn(_f32_bytes(np.eye(K)), _f32_bytes(X), K, N, K, "f32")
    assert np.array_equal(Y, X.astype(np.float64))
    perm = rng.permutation(K)
    P = np.zeros((K, K), dtype=np.float32)
    P[perm, np.arange(K)] = 1.0          # column i of P has its one in row perm[i]
    Y = orc.gemm_tn(_f32_bytes(P), _f32_bytes(X), K, N, K, "f32")
    assert np.array_equal(Y, X[perm].astype(np.float64))


def test_oracle_tn_brute_force_rectangular(orc):
    """A rectangular case (M ≠ K) against a pure-Python triple loop over the
    definition Y[i][j] = Σ_l W[l][i]·X[l][j], in both input dtypes."""
    M, N, K = 5, 3, 7
    for dt in ("f32", "bf16"):
        W, X = make_perceptron_inputs(M, N, K, dt, 3, "smallint")
        w = orc.widen(raw_bytes(W), dt).reshape(K, M)
        x = orc.widen(raw_bytes(X), dt).reshape(K, N)
        want = [[sum(w[l][i] * x[l][j] for l in range(K)) for j in range(N)] for i in range(M)]
        got = orc.gemm_tn(raw_bytes(W), raw_bytes(X), M, N, K, dt)
        assert np.array_equal(got, np.array(want))


def test_paper_protocol_budgets(orc):
    """0.1 % of the spaces whose sizes §5 prints (484,000; 899,756; 1,589,952)."""
    printed = {512: 484000, 1024: 899756, 2048: 1589952}
    for w in PAPER_PROTOCOL:
        sp = orc.Space(w.M, w.N, w.K, w.d, w.dtype, w.mfma_coord, mode=orc.ANY_PAIR)
        assert sp.size() == printed[w.M]
        assert w.budget == math.ceil(sp.size() / 1000)
        s0 = sp.paper_s0()
        assert s0[:3] == ((w.M, 1, 1, 1), (w.K, 1), (w.N, 1, 1, 1)) and sp.legit(s0)


def test_lowering_k_major(gt):
    """K-major A: fp32 fast-path configurations keep the fast path (with the
    K-major kernel), the direct-load path is never chosen, bf16 falls back to
    the generic path; J and the tile shape do not depend on the layout."""
    M = N = K = 1024
    tn32 = gt.dtype_code("f32") | gt.A_KMAJOR
    tn16 = gt.dtype_code("bf16") | gt.A_KMAJOR
    cfg = ((8, 2, 2, 32), (32, 1, 4, 8), (8, 2, 2, 32), 0)
    nn, tn = gt.lower(cfg, M, N, K, "f32"), gt.lower(cfg, M, N, K, tn32)
    assert nn["fast"] == tn["fast"] == 1 and tn["dl"] == 0
    assert {k: v for k, v in nn.items()} == {k: v for k, v in tn.items()}
    bcfg = ((4, 2, 4, 32), (16, 1, 4, 16), (4, 2, 4, 32), 32)
    nn, tn = gt.lower(bcfg, M, N, K, "bf16"), gt.lower(bcfg, M, N, K, tn16)
    assert nn["dl"] == 1 and tn["fast"] == 0 and tn["dl"] == 0
    sp_nn = gt.Space(M, N, K, (4, 4, 4), "bf16", True)
    sp_tn = gt.Space(M, N, K, (4, 4, 4), "bf16", True, a_kmajor=True)
    assert sp_tn.a_kmajor and sp_nn.size() == sp_tn.size()
    for r in range(0, sp_nn.size(), sp_nn.size() // 97):
        c = sp_nn.unrank(r)
        assert sp_nn.legit(c) == sp_tn.legit(c)
    with pytest.raises(gt.GemmTuneError):  # not a dtype, with or without the flag
        gt.Space(16, 16, 16, (4, 4, 4), 2 | gt.A_KMAJOR, False).size()
