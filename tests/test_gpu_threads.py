"""gemm_run called from several host threads at once, each on its own stream
(default priority), over every kernel path (direct-load ring, register-staged,
generic, split-K with its clear and atomics): each thread's outputs equal the
single-threaded outputs bit for bit on small-integer inputs, where every
partial sum is exact in fp32 whatever the order of the adds."""
import sys
import threading

import numpy as np
import pytest
import torch

from workloads import make_inputs, raw_bytes

pytestmark = pytest.mark.gpu

M, N, K = 64, 256, 1024
CASES = [
    # (dtype, configuration) at 64x256x1024
    ("bf16", ((1, 1, 2, 32), (4, 8, 2, 16), (4, 2, 1, 32), 32)),   # direct-load, split K
    ("bf16", ((1, 2, 2, 16), (8, 1, 4, 32), (4, 2, 2, 16), 16)),   # direct-load
    ("f32", ((2, 2, 1, 16), (4, 4, 8, 8), (4, 2, 2, 16), 0)),      # register-staged, split K
    ("f32", ((2, 2, 1, 16), (16, 1, 8, 8), (4, 2, 2, 16), 0)),     # register-staged
    ("bf16", ((2, 1, 2, 16), (16, 4, 4, 4), (2, 2, 2, 32), 16)),   # generic, split K
    ("f32", ((64, 1, 1, 1), (64, 1, 4, 4), (4, 2, 2, 16), 0)),     # generic
]


@pytest.fixture(scope="module")
def gt():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_1909_10616_amd import gemmtune
    gemmtune.lib()
    return gemmtune


def test_concurrent_gemm_run_matches_serial(gt, orc):
    dev = torch.device("cuda:0")
    ops = {}
    for dt in ("bf16", "f32"):
        A, B = make_inputs(M, N, K, dt, 21, "smallint")
        ops[dt] = (A.to(dev), B.to(dev), orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, dt))
    for dt, cfg in CASES:
        info = gt.lower(cfg, M, N, K, dt)
        print(f"{dt} {gt.fmt_cfg(cfg)} fast={info['fast']} dl={info['dl']} "
              f"split={info['grid_y']}", flush=True)
        Ad, Bd, ref = ops[dt]
        C = torch.full((M, N), float("nan"), device=dev)
        gt.gemm_run(cfg, Ad, Bd, C)
        torch.cuda.synchronize()
        assert np.array_equal(C.cpu().numpy().astype(np.float64), ref), cfg
    sys.stdout.flush()

    n_threads, rounds = 4, 25
    outs = [[torch.full((M, N), float("nan"), device=dev) for _ in CASES] for _ in range(n_threads)]
    errors = []

    def worker(t):
        try:
            s = torch.cuda.Stream(device=dev)
            for r in range(rounds):
                n = (t + r) % len(CASES)           # each thread and round its own order
                for k in list(range(n, len(CASES))) + list(range(n)):
                    dt, cfg = CASES[k]
                    Ad, Bd, _ = ops[dt]
                    gt.gemm_run(cfg, Ad, Bd, outs[t][k], stream=s)
            s.synchronize()
        except Exception as e:   # reported below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(n_threads)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for t in range(n_threads):
        for k, (dt, cfg) in enumerate(CASES):
            got = outs[t][k].cpu().numpy().astype(np.float64)
            assert np.array_equal(got, ops[dt][2]), (t, cfg)


def test_concurrent_compare_returns_each_callers_result(gt):
    """gt_compare from several threads on their own streams: the per-GPU
    result buffer is taken in turn, so every call returns its own pair's
    error (the pairs differ in one element by a different amount each)."""
    dev = torch.device("cuda:0")
    n_threads, calls, n = 6, 60, 1 << 16
    g = torch.Generator(device="cpu").manual_seed(5)
    R = (torch.rand(n, generator=g) + 0.5).to(dev)
    pairs, expect = [], []
    for t in range(n_threads):
        C = R.clone()
        C[1000 * t + 7] += 0.125 * (t + 1)
        pairs.append(C)
        expect.append(gt.gt_compare(C, R))
    torch.cuda.synchronize()
    assert len(set(expect)) == n_threads and all(e > 0 for e in expect)
    got, errors = [[] for _ in range(n_threads)], []

    def worker(t):
        try:
            s = torch.cuda.Stream(device=dev)
            for _ in range(calls):
                got[t].append(gt.gt_compare(pairs[t], R, stream=s))
        except Exception as e:   # reported below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(n_threads)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for t in range(n_threads):
        assert got[t] == [expect[t]] * calls, (t, set(got[t]))


def test_concurrent_timings_take_turns(gt):
    """gt_measure from two threads on their own streams, on the 4096³ bf16
    headline kernel (one workgroup per CU, so two launches in flight at once
    would each run about twice as long): timings take turns per GPU, and
    each thread's median stays at the single-threaded median."""
    import statistics
    dev = torch.device("cuda:0")
    cfg = ((16, 2, 8, 16), (128, 1, 1, 32), (16, 4, 2, 32), 16)
    g = torch.Generator(device="cpu").manual_seed(3)
    A = torch.randn(4096, 4096, generator=g).to(torch.bfloat16).to(dev)
    B = torch.randn(4096, 4096, generator=g).to(torch.bfloat16).to(dev)
    Cs = [torch.empty(4096, 4096, device=dev) for _ in range(2)]
    def solo_median():
        return statistics.median(gt.gt_measure(cfg, A, B, Cs[0], warmup=2, runs=10)["mean_ms"]
                                 for _ in range(9))

    before = solo_median()
    got, errors = [[], []], []

    def worker(t):
        try:
            s = torch.cuda.Stream(device=dev)
            for _ in range(15):
                got[t].append(gt.gt_measure(cfg, A, B, Cs[t], warmup=2, runs=10, stream=s)["mean_ms"])
        except Exception as e:   # reported below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    # the single-threaded median before and after, the larger as the reference
    # (the board's clock can drift between the phases)
    solo = max(before, solo_median())
    print(f"solo median {solo * 1e3:.1f} us", flush=True)
    for t in range(2):
        med = statistics.median(got[t])
        print(f"thread {t} median {med * 1e3:.1f} us", flush=True)
        assert med < 1.3 * solo, (t, med, solo)
