"""Host-side parity of libgemmtune against the oracle — CPU only.

The space functions (size, enumeration, rank/unrank, J, neighbours) must match
the oracle bit-exactly, and tune_gbfs with a synthetic cost callback (the
CPU fake backend) must reproduce the oracle's G-BFS trajectory exactly.
"""
import ctypes
import math
import os
import re
import subprocess
import sys
import zlib

import numpy as np
import pytest

from workloads import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

LIB_DT = np.dtype([("d", "<i4", 3), ("mfma", "<i4"), ("m", "<i8", 4), ("k", "<i8", 4),
                   ("n", "<i8", 4), ("legit", "<i4"), ("res", "<i4")])
ORC_DT = np.dtype([("f", "<i8", (3, 4)), ("mfma", "<i4"), ("legit", "<i4")])


@pytest.fixture(scope="session")
def gt():
    from paper_1909_10616_amd import gemmtune
    if not os.path.exists(gemmtune.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    gemmtune.lib()
    return gemmtune


def _spaces():
    out = []
    for w in WORKLOADS.values():
        out.append((w.name, (w.M, w.N, w.K, w.d, w.dtype, w.mfma_coord)))
    for D in (512, 1024, 2048):
        out.append((f"paper{D}_d424", (D, D, D, (4, 2, 4), "f32", False)))
    out.append(("odd96x80x48", (96, 80, 48, (4, 3, 4), "bf16", True)))
    out.append(("tiny", (8, 4, 16, (3, 2, 3), "f32", False)))
    return out


SPACES = _spaces()


def test_header_symbols_are_exported(gt):
    hdr = open(os.path.join(ROOT, "include", "gemmtune.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    decl = set(re.findall(r"^\s*(?:int|const\s+char\s*\*)\s*([a-z_0-9]+)\s*\(", hdr, re.M))
    assert {"gemm_run", "tune_gbfs", "enumerate_configs", "neighbours"} <= decl
    out = subprocess.run(["nm", "-D", "--defined-only", gt.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    assert decl <= exported, decl - exported
    assert decl == set(gt.EXPORTS)
    for name in decl:
        getattr(gt.lib(), name)


@pytest.mark.parametrize("name,args", SPACES, ids=[s[0] for s in SPACES])
def test_space_size_matches_oracle(gt, orc, name, args):
    M, N, K, d, dt, mc = args
    assert gt.Space(M, N, K, d, dt, mc).size() == orc.Space(M, N, K, d, dt, mc).size()


def _compare_window(gt, orc, args, start, count):
    M, N, K, d, dt, mc = args
    ls, os_ = gt.Space(M, N, K, d, dt, mc), orc.Space(M, N, K, d, dt, mc)
    buf, n = ls.enumerate_raw(start, count)
    assert n == count
    a = np.frombuffer(buf, dtype=LIB_DT, count=n)
    b = np.frombuffer(os_.enumerate_raw(start, count).tobytes(), dtype=ORC_DT, count=n)
    assert np.array_equal(a["m"], b["f"][:, 0]) and np.array_equal(a["k"], b["f"][:, 1])
    assert np.array_equal(a["n"], b["f"][:, 2]) and np.array_equal(a["mfma"], b["mfma"])
    assert np.array_equal(a["legit"], b["legit"])
    assert np.all(a["d"] == np.array(d, dtype=np.int32))
    return int(a["legit"].sum())


@pytest.mark.parametrize("name", ["tiny", "odd96x80x48", "gemm256_f32", "paper512_d424"])
def test_full_enumeration_bit_exact(gt, orc, name):
    args = dict(SPACES)[name]
    size = gt.Space(*args).size()
    step = 1 << 20
    for start in range(0, size, step):
        _compare_window(gt, orc, args, start, min(step, size - start))


def test_full_enumeration_gemm1024(gt, orc):
    # 23,393,656 configurations compared in windows of 2^21
    args = dict(SPACES)["gemm1024_f32"]
    size = gt.Space(*args).size()
    legit = 0
    for start in range(0, size, 1 << 21):
        legit += _compare_window(gt, orc, args, start, min(1 << 21, size - start))
    assert 0 < legit < size


@pytest.mark.parametrize("name,args", SPACES, ids=[s[0] for s in SPACES])
def test_sampled_windows_bit_exact(gt, orc, name, args):
    size = gt.Space(*args).size()
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    starts = [0, max(0, size - 4096)] + [int(x) for x in rng.integers(0, max(1, size - 4096), 8)]
    for st in starts:
        _compare_window(gt, orc, args, st, min(4096, size - st))


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("name,args", SPACES, ids=[s[0] for s in SPACES])
def test_neighbours_and_rank_match_oracle(gt, orc, mode, name, args):
    M, N, K, d, dt, mc = args
    ls = gt.Space(M, N, K, d, dt, mc, mode=mode)
    os_ = orc.Space(M, N, K, d, dt, mc, mode=mode)
    size = ls.size()
    rng = np.random.default_rng(7 + mode)
    ranks = [0, size - 1] + [int(x) for x in rng.integers(0, size, 60)]
    for r in ranks:
        c = ls.unrank(r)
        assert c == os_.unrank(r)
        assert ls.rank(c) == r == os_.rank(c)
        assert ls.legit(c) == os_.legit(c)
        assert ls.neighbours(c) == os_.neighbours(c)


def _rand_cost(seed):
    M64 = (1 << 64) - 1

    def f(cfg, rank):
        z = ((rank ^ seed) + 0x9E3779B97F4A7C15) & M64
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
        return 1.0 + (z ^ (z >> 31)) / 2.0 ** 64
    return f


@pytest.mark.parametrize("case", [
    ("gemm256_f32", 5, 64, 0, 0, None),
    ("gemm1024_f32", 5, 200, 1, 0, None),
    ("gemm4096_bf16", 5, 1000, 3, 0, None),
    ("mlp4096x11008x4096_bf16", 5, 300, 4, 0, None),
    ("skinny64x4096x4096_bf16", 3, 300, 4, 1, None),
    ("paper1024_d424", 5, 900, 11, 1, None),
    ("gemm4096_bf16", 5, 400, 9, 0, ((64, 2, 1, 32), (64, 1, 2, 32), (64, 2, 1, 32), 16)),
])
def test_tune_gbfs_synthetic_trajectory_matches_oracle(gt, orc, case):
    name, rho, budget, seed, mode, s0 = case
    M, N, K, d, dt, mc = dict(SPACES)[name]
    ls = gt.Space(M, N, K, d, dt, mc, mode=mode)
    os_ = orc.Space(M, N, K, d, dt, mc, mode=mode)
    cost = _rand_cost(seed * 1000 + 17)
    start = s0 if s0 is not None else ls.paper_s0()
    got = gt.tune_gbfs(ls, budget=budget, s0=s0, rho=rho, seed=seed, cost_fn=cost)
    exp = orc.gbfs(os_, start, rho, budget, seed, cost)
    assert [e["rank"] for e in got["log"]] == exp["log_ranks"]
    assert got["best"] == exp["best"] and got["best_cost"] == exp["best_cost"]
    assert got["timed"] == exp["timed"] and got["popped"] == exp["popped"]


def test_tune_gbfs_unimodal_and_infinite_costs_match_oracle(gt, orc):
    args = (64, 64, 64, (4, 4, 4), "bf16", True)
    ls, os_ = gt.Space(*args), orc.Space(*args)
    target = ((4, 2, 2, 4), (8, 1, 2, 4), (2, 4, 1, 8), 32)

    def cost(cfg, rank):
        if rank % 7 == 3:
            return math.inf           # failures are counted, visited and never expanded
        e = [int(math.log2(v)) for lv in cfg[:3] for v in lv] + [cfg[3] // 32]
        t = [int(math.log2(v)) for lv in target[:3] for v in lv] + [1]
        return 1.0 + sum(abs(a - b) for a, b in zip(e, t))

    got = gt.tune_gbfs(ls, budget=3000, rho=5, seed=5, cost_fn=cost)
    exp = orc.gbfs(os_, ls.paper_s0(), 5, 3000, 5, cost)
    assert [e["rank"] for e in got["log"]] == exp["log_ranks"]
    assert got["failed"] == sum(1 for c in exp["log_costs"] if math.isinf(c))
    assert got["best"] == exp["best"]


def test_tune_gbfs_argument_errors(gt):
    ls = gt.Space(256, 256, 256, (3, 3, 3), "f32", False)
    with pytest.raises(gt.GemmTuneError):
        gt.tune_gbfs(ls, budget=0, cost_fn=lambda c, r: 1.0)
    with pytest.raises(gt.GemmTuneError):
        gt.tune_gbfs(ls, budget=5, rho=0, cost_fn=lambda c, r: 1.0)
    with pytest.raises(gt.GemmTuneError):   # 32 waves: illegitimate start
        gt.tune_gbfs(ls, budget=5, s0=((1, 16, 16), (256, 1, 1), (1, 2, 128), 0),
                     cost_fn=lambda c, r: 1.0)
    with pytest.raises(gt.GemmTuneError):   # not a member (products)
        gt.tune_gbfs(ls, budget=5, s0=((2, 16, 16), (256, 1, 1), (1, 2, 128), 0),
                     cost_fn=lambda c, r: 1.0)
    with pytest.raises(gt.GemmTuneError):   # bad space
        gt.Space(0, 4, 4).size()


def test_tune_gbfs_time_limit(gt):
    import time
    ls = gt.Space(1024, 1024, 1024, (4, 4, 4), "f32", False)

    def slow(cfg, rank):
        time.sleep(0.01)
        return 1.0 + (rank % 1000) / 1000.0

    r = gt.tune_gbfs(ls, budget=10 ** 6, t_max_s=0.2, cost_fn=slow)
    assert r["stop_reason"] == "time-limit" and 1 <= r["timed"] < 200


def test_gemm_run_rejects_before_launch(gt):
    # legitimacy and shape are checked on the host, before any HIP call
    lib = gt.lib()
    bad = gt.to_c(((1, 16, 16), (256, 1, 1), (1, 2, 128), 0))       # 32 waves
    rc = lib.gemm_run(ctypes.byref(bad), 16, 16, 16, 256, 256, 256, gt.F32, None)
    assert rc == -3 and b"legitimate" in lib.gt_last_error()
    wrong = gt.to_c(((2, 8, 16), (256, 1, 1), (1, 2, 128), 0))      # products 256 != 128*...
    rc = lib.gemm_run(ctypes.byref(wrong), 16, 16, 16, 128, 256, 256, gt.F32, None)
    assert rc == -2
    rc = lib.gemm_run(ctypes.byref(bad), None, 16, 16, 256, 256, 256, gt.F32, None)
    assert rc == -1


def test_lowering_of_known_configs(gt):
    info = gt.lower(((16, 2, 4, 32), (64, 1, 4, 16), (16, 2, 4, 32), 32), 4096, 4096, 4096, "bf16")
    assert (info["I"], info["TM"], info["TN"], info["waves"], info["fast"]) == (32, 4, 4, 4, 1)
    assert (info["BM"], info["BN"], info["BK"], info["dbuf"]) == (256, 256, 64, 1)
    assert (info["grid_x"], info["grid_y"], info["lds_bytes"]) == (256, 1, 131072)
    s0 = gt.Space(4096, 4096, 4096, (4, 4, 4), "bf16", True).paper_s0()
    info = gt.lower(s0, 4096, 4096, 4096, "bf16")
    assert (info["I"], info["TM"], info["TN"], info["fast"], info["grid_x"]) == (16, 1, 1, 0,
                                                                                4096 * 4096)
    # split-K and padded blocks take the generic path
    info = gt.lower(((2, 1, 1, 32), (16, 8, 2, 16), (64, 2, 1, 32), 32), 64, 4096, 4096, "bf16")
    assert info["grid_y"] == 8 and info["fast"] == 1
    info = gt.lower(((8, 2, 1, 16), (16, 1, 4, 16), (8, 2, 1, 16), 32), 256, 256, 1024, "bf16")
    assert info["fast"] == 0 and info["TM"] == 1


RANDOM_CASES = [
    # (M, N, K, d, dtype, mfma, budget, seed)
    (256, 256, 256, (3, 3, 3), "f32", False, 64, 0),
    (1024, 1024, 1024, (4, 4, 4), "f32", False, 200, 5),
    (4096, 4096, 4096, (4, 4, 4), "bf16", True, 300, 3),
    (64, 11008, 4096, (4, 4, 4), "bf16", True, 150, 11),
    (1, 1, 1, (4, 4, 4), "f32", False, 4, 0),
]


@pytest.mark.parametrize("case", RANDOM_CASES, ids=[f"{c[0]}x{c[1]}x{c[2]}-{c[4]}" for c in RANDOM_CASES])
def test_tune_random_synthetic_trajectory_matches_oracle(gt, orc, case):
    M, N, K, d, dt, mc, budget, seed = case
    sp = gt.Space(M, N, K, d, dt, mc)
    osp = orc.Space(M, N, K, d, dt, mc)
    cost = lambda c, r: float((r * 2654435761) % 100003) / 7.0   # noqa: E731
    res = gt.tune_random(sp, budget=budget, seed=seed, cost_fn=cost)
    ref = orc.random_search(osp, budget, seed, cost)
    assert [e["rank"] for e in res["log"]] == ref["log_ranks"]
    assert [e["cost_ms"] for e in res["log"]] == ref["log_costs"]
    assert res["timed"] == ref["timed"] and res["popped"] == ref["popped"]
    assert res["best"] == ref["best"] and res["best_cost"] == ref["best_cost"]
    assert res["skipped_illegit"] + res["skipped_visited"] + res["timed"] == res["popped"]
    want = "budget" if res["timed"] == budget else "draws-exhausted"
    assert res["stop_reason"] == want


def test_tune_random_errors_and_time_limit(gt):
    sp = gt.Space(256, 256, 256, (3, 3, 3), "f32", False)
    with pytest.raises(gt.GemmTuneError):
        gt.tune_random(sp, budget=0, cost_fn=lambda c, r: 1.0)
    # GPU mode (no callback) without operands is refused by the C ABI itself
    lib = gt.lib()
    o = gt.gt_tune_opts()
    assert lib.gt_tune_opts_init(ctypes.byref(o)) == 0
    res = gt.gt_tune_result()
    rc = lib.tune_random(ctypes.byref(sp.c), ctypes.byref(o), gt.gt_cost_fn(), None, ctypes.byref(res))
    assert rc == -1 and b"A, B and C" in lib.gt_last_error()
    ls = gt.Space(1024, 1024, 1024, (4, 4, 4), "f32", False)
    import time

    def slow(cfg, rank):
        time.sleep(0.01)
        return 1.0

    r = gt.tune_random(ls, budget=10 ** 6, t_max_s=0.2, cost_fn=slow)
    assert r["stop_reason"] == "time-limit" and 1 <= r["timed"] < 200


NA2C_CASES = [
    # (M, N, K, d, dtype, mfma, mode, budget, seed, params)
    (512, 512, 512, (4, 2, 4), "f32", False, 1, 300, 0, None),        # the paper's space shape
    (1024, 1024, 1024, (4, 2, 4), "f32", False, 1, 300, 7, {"B": 4, "T": 2}),
    (256, 256, 512, (4, 4, 4), "bf16", True, 0, 250, 3, {"eps": 0.5, "mem": 64}),
    (96, 80, 48, (4, 3, 4), "bf16", True, 1, 200, 1, {"H": 8, "lr": 0.05}),
    (64, 32, 64, (3, 2, 3), "f32", False, 1, 400, 2, None),           # small: walks lengthen
    # the variants: clipped log-ratio reward, ε halving after empty episodes
    (512, 512, 512, (4, 2, 4), "f32", False, 1, 300, 4, {"reward": 1}),
    (64, 32, 64, (3, 2, 3), "f32", False, 1, 400, 5, {"eps_halving": 1}),
    (256, 256, 512, (4, 4, 4), "bf16", True, 0, 250, 6, {"reward": 1, "eps_halving": 1}),
]


@pytest.mark.parametrize("cost_kind", ["random", "unimodal"])
@pytest.mark.parametrize("case", NA2C_CASES, ids=[f"{c[0]}x{c[1]}x{c[2]}-{c[4]}-{i}"
                                                  for i, c in enumerate(NA2C_CASES)])
def test_tune_na2c_synthetic_trajectory_matches_oracle(gt, orc, case, cost_kind):
    """The library's N-A2C and the oracle's, fed the same synthetic costs,
    time the identical sequence of configurations (which exercises the walk,
    the policy sampling, the memory and every training step bit for bit)."""
    M, N, K, d, dt, mc, mode, budget, seed, params = case
    sp = gt.Space(M, N, K, d, dt, mc, mode=mode)
    osp = orc.Space(M, N, K, d, dt, mc, mode=mode)
    s0 = osp.paper_s0()
    if cost_kind == "random":
        cost = lambda c, r: 1.0 + ((r * 2654435761 + seed) % 997) / 997.0   # noqa: E731
    else:
        tgt = [e // 2 for e in range(sum(d))]

        def cost(c, r):
            e = [v.bit_length() - 1 for t in c[:3] for v in t]
            return 1.0 + sum(abs(a - b) for a, b in zip(e, tgt))
    res = gt.tune_na2c(sp, budget, s0=s0, seed=seed, cost_fn=cost, params=params)
    ref = orc.na2c(osp, s0, budget, seed, cost, params)
    assert [e["rank"] for e in res["log"]] == ref["log_ranks"]
    assert [e["cost_ms"] for e in res["log"]] == ref["log_costs"]
    assert res["timed"] == ref["timed"] and res["popped"] == ref["popped"]
    assert res["best"] == ref["best"] and res["best_cost"] == ref["best_cost"]


@pytest.mark.parametrize("search", ["gbfs", "random", "na2c"])
def test_nan_cost_is_a_failed_candidate(gt, orc, search):
    """A cost that is not a number is no measurement: the library and the
    oracle both take it as +∞ (a failed candidate), log it as such and count
    it in `failed`; G-BFS used to order its queue by the NaN itself and left
    the oracle's trajectory."""
    sp = gt.Space(256, 256, 256, (3, 3, 3), "f32", False)
    osp = orc.Space(256, 256, 256, (3, 3, 3), "f32", False)

    def cost(c, r):
        h = (r * 2654435761) % 997
        return float("nan") if h % 5 == 0 else 1.0 + h / 997

    s0 = sp.paper_s0()
    if search == "gbfs":
        res, ref = gt.tune_gbfs(sp, 150, s0=s0, rho=3, seed=4, cost_fn=cost), \
            orc.gbfs(osp, s0, 3, 150, 4, cost)
    elif search == "random":
        res, ref = gt.tune_random(sp, 150, seed=4, cost_fn=cost), orc.random_search(osp, 150, 4, cost)
    else:
        res, ref = gt.tune_na2c(sp, 150, s0=s0, seed=4, cost_fn=cost), orc.na2c(osp, s0, 150, 4, cost)
    costs = [e["cost_ms"] for e in res["log"]]
    assert [e["rank"] for e in res["log"]] == ref["log_ranks"] and costs == ref["log_costs"]
    assert res["best"] == ref["best"] and res["best_cost"] == ref["best_cost"]
    nan_ranks = [e["rank"] for e in res["log"] if (e["rank"] * 2654435761) % 997 % 5 == 0]
    assert nan_ranks and res["failed"] == len(nan_ranks) == costs.count(math.inf)
    assert all(e["status"] == "launch-failure" for e in res["log"] if e["rank"] in nan_ranks)


@pytest.mark.parametrize("args", [(3, 5, 7, (2, 2, 2), "f32", False),
                                  (64, 32, 64, (1, 1, 1), "bf16", False)])
@pytest.mark.parametrize("params", [None, {"eps": 1.0}, {"eps": 0.0, "eps_halving": 1}])
def test_tune_na2c_on_a_space_without_moves(gt, orc, args, params):
    """A space of one configuration and no MFMA coordinate offers no action
    in any state: every walk ends where it starts, so N-A2C times s0, spends
    the episodes T … T+8 finding nothing and stops (the library and the
    oracle once divided by the zero count of available actions here)."""
    sp, osp = gt.Space(*args), orc.Space(*args)
    assert sp.size() == 1 and sp.neighbours(sp.unrank(0)) == []
    s0 = sp.unrank(0)
    cost = lambda c, r: 2.5   # noqa: E731
    res = gt.tune_na2c(sp, 40, s0=s0, seed=11, cost_fn=cost, params=params)
    ref = orc.na2c(osp, s0, 40, 11, cost, params)
    assert res["timed"] == ref["timed"] == 1 and res["best"] == ref["best"] == s0
    assert res["popped"] == ref["popped"] == 9
    assert res["stop_reason"] == "neighbourhood-exhausted"


def test_tune_na2c_errors(gt):
    sp = gt.Space(256, 256, 256, (3, 3, 3), "f32", False)
    for bad in ({"T": 0}, {"B": 0}, {"H": 65}, {"mem": 0}, {"max_walks": 0}, {"eps": 1.5},
                {"lr": -1.0}, {"r_clip": 0.0}, {"reward": 2}, {"eps_halving": -1}):
        with pytest.raises(gt.GemmTuneError):
            gt.tune_na2c(sp, 10, cost_fn=lambda c, r: 1.0, params=bad)
    with pytest.raises(gt.GemmTuneError):   # s0 not in the space
        gt.tune_na2c(sp, 10, s0=((128, 1, 1), (256, 1, 1), (256, 1, 1), 0),
                     cost_fn=lambda c, r: 1.0)
    r = gt.tune_na2c(sp, 1, cost_fn=lambda c, r: 1.0)   # default s0 = [D,1,1]
    assert r["timed"] == 1 and r["best"] == ((256, 1, 1), (256, 1, 1), (256, 1, 1), 0)


@pytest.mark.parametrize("name", ["gemm2048_f32", "gemm4096_bf16", "mlp4096x11008x4096_bf16",
                                  "skinny64x4096x4096_bf16", "paper1024_d424", "paper2048_d424"])
def test_full_enumeration_every_workload_space(gt, orc, name):
    """Every configuration of the remaining workload spaces (up to
    188,392,750), library against oracle, in windows of 2^22."""
    args = dict(SPACES)[name]
    size = gt.Space(*args).size()
    legit = 0
    for start in range(0, size, 1 << 22):
        legit += _compare_window(gt, orc, args, start, min(1 << 22, size - start))
    assert 0 < legit < size


def test_report_arithmetic_exact(gt):
    """The report's figures against exact rational arithmetic: TFLOP/s =
    2MNK / cost, % of peak, timed / |ξ| (the whole space), HBM GB/s at the
    algorithmic bytes; each within one rounding of the exact value."""
    from fractions import Fraction as F

    def close(x, q):
        assert abs(F(x) - q) <= abs(q) * F(1, 2 ** 50), (x, float(q))

    cases = [(4096, 4096, 4096, "bf16", 0.11514, 1000, 188392750, 2516.6),
             (256, 256, 256, "f32", 0.0063, 64, 91125, 157.3),
             (4096, 11008, 4096, "bf16", 0.331, 1000, 68318250, 2516.6),
             (64, 4096, 4096, "bf16", 0.0146, 1000, 34780200, 2516.6),
             (1024, 1024, 1024, "f32", 0.0285, 200, 23393656, 157.3)]
    for M, N, K, dt, ms, timed, size, peak in cases:
        r = gt.report(M, N, K, dt, ms, timed, size, peak)
        t = F(2 * M * N * K) / (F(ms) / 1000) / 10 ** 12
        close(r["tflops"], t)
        close(r["pct_of_peak"], 100 * t / F(peak))
        close(r["fraction_of_space_pct"], F(100 * timed, size))
        esz = 2 if dt == "bf16" else 4
        assert r["algorithmic_bytes"] == (M * K + K * N) * esz + M * N * 4
        close(r["hbm_gbs"], F(r["algorithmic_bytes"]) / (F(ms) / 1000) / 10 ** 9)
    # the workload list's budgets as shares of their spaces (exact values)
    assert gt.report(4096, 4096, 4096, "bf16", 1.0, 1000, 188392750, 1)["fraction_of_space_pct"] \
        == 100 * 1000 / 188392750
    assert F(1000, 188392750) < F(1, 100)     # the search explores under 1 % of the space
    # 1 ms at 4096³: 137.438953472 TFLOP/s exactly
    assert gt.report(4096, 4096, 4096, "bf16", 1.0, 1, 1, 1)["tflops"] == 137.438953472


def test_one_hip_runtime_whatever_the_import_order():
    """Loading the library before PyTorch must not map a second HIP runtime
    (two in one process leave the second without a GPU)."""
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_1909_10616_amd import gemmtune as gt\n"
            "gt.lib()\n"
            "import torch\n"
            "m = {l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}\n"
            "print(len(m), sorted(m))\n") % os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.split()[0] == "1", out.stdout
