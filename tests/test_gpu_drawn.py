"""GPU parity of the kernel family on a seeded list of drawn cases: odd
shapes, one to four levels per dimension, both dtypes, A row-major and
K-major, configurations drawn by rank or by a short neighbour walk from the
hand-made start (every kernel path, split-K included). The same list passes
the CPU kernel model first. Alternate cases use small-integer inputs, where
every partial sum is exact in fp32 and the output must equal the fp64
oracle bit for bit; the others use the workloads' value distributions,
within the tolerances of the other parity tests (fp32 ≤ 1e-5·√K, bf16
inputs with fp32 accumulation ≤ 2e-3, normwise)."""
import sys

import numpy as np
import pytest
import torch

from drawn_cases import cases_with_env_seeds
from workloads import make_inputs, make_perceptron_inputs, raw_bytes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gt():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_1909_10616_amd import gemmtune
    gemmtune.lib()
    return gemmtune


def test_drawn_cases_match_oracle(gt, orc):
    dev = torch.device("cuda:0")
    paths = {"dl": 0, "fast": 0, "generic": 0}
    for i, (M, N, K, d, dt, mc, akm, cfg) in enumerate(cases_with_env_seeds(gt)):
        smallint = i % 2 == 0
        dist = "smallint" if smallint else ("normal" if dt == "bf16" else "uniform")
        code = gt.dtype_code(dt) | (gt.A_KMAJOR if akm else 0)
        info = gt.lower(cfg, M, N, K, code)
        path = "dl" if info["dl"] else ("fast" if info["fast"] else "generic")
        paths[path] += 1
        print(f"case {i}: {M}x{N}x{K} d={d} {dt} {'K-major' if akm else 'row-major'} {dist} "
              f"{gt.fmt_cfg(cfg)} {path} grid={info['grid_x']}x{info['grid_y']}", flush=True)
        sys.stdout.flush()
        if akm:
            A, B = make_perceptron_inputs(M, N, K, dt, 100 + i, dist)
            ref = orc.gemm_tn(raw_bytes(A), raw_bytes(B), M, N, K, dt)
        else:
            A, B = make_inputs(M, N, K, dt, 100 + i, dist)
            ref = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, dt)
        C = torch.full((M, N), float("nan"), device=dev, dtype=torch.float32)
        gt.gemm_run(cfg, A.to(dev), B.to(dev), C, a_kmajor=akm)
        torch.cuda.synchronize()
        C = C.cpu().numpy().astype(np.float64)
        if smallint:
            assert np.array_equal(C, ref), (i, cfg)
        else:
            e = float(np.abs(C - ref).max() / max(np.abs(ref).max(), 1e-300))
            assert e <= (1e-5 * K ** 0.5 if dt == "f32" else 2e-3), (i, cfg, e)
    assert paths["dl"] >= 5 and paths["fast"] >= 10 and paths["generic"] >= 40, paths
