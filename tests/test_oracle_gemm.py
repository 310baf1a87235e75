"""Pins for the oracle GEMM (§3.2 three-loop product) — CPU only.

Each test checks the oracle against a fact fixed by mathematics, not against
a retyped copy of its own loop: identities, permutations, exact small-integer
products (numpy int64 matmul is exact), closed forms that expose a transposed
operand or a dropped term, and the bf16 bit-level widening.
"""
import json
import os

import numpy as np
import pytest
import torch

from workloads import make_inputs, raw_bytes

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")


def _f32_bytes(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint8).ravel()


def _bf16_bytes(a):
    return raw_bytes(torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16))


def test_identity_right_and_left(orc):
    rng = np.random.default_rng(5)
    A = rng.uniform(-1, 1, size=(37, 29)).astype(np.float32)
    I29 = np.eye(29, dtype=np.float32)
    I37 = np.eye(37, dtype=np.float32)
    C = orc.gemm(_f32_bytes(A), _f32_bytes(I29), 37, 29, 29, "f32")
    assert np.array_equal(C, A.astype(np.float64))
    C = orc.gemm(_f32_bytes(I37), _f32_bytes(A), 37, 29, 37, "f32")
    assert np.array_equal(C, A.astype(np.float64))


def test_permutations_move_rows_and_columns(orc):
    rng = np.random.default_rng(6)
    A = rng.uniform(-1, 1, size=(16, 24)).astype(np.float32)
    p = rng.permutation(16)
    P = np.zeros((16, 16), np.float32)
    P[np.arange(16), p] = 1.0            # (P·A)[i] = A[p[i]]
    C = orc.gemm(_f32_bytes(P), _f32_bytes(A), 16, 24, 16, "f32")
    assert np.array_equal(C, A[p].astype(np.float64))
    q = rng.permutation(24)
    Q = np.zeros((24, 24), np.float32)
    Q[q, np.arange(24)] = 1.0            # (A·Q)[:, j] = A[:, q[j]]
    C = orc.gemm(_f32_bytes(A), _f32_bytes(Q), 16, 24, 24, "f32")
    assert np.array_equal(C, A[:, q].astype(np.float64))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 1, 1), (7, 5, 3), (33, 65, 129), (64, 48, 256)])
def test_small_integers_exact(orc, dtype, shape):
    M, N, K = shape
    A, B = make_inputs(M, N, K, dtype, 11, "smallint")
    exact = A.to(torch.int64).numpy() @ B.to(torch.int64).numpy()
    C = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, dtype)
    assert np.array_equal(C, exact.astype(np.float64))


def test_all_ones_gives_k(orc):
    M, N, K = 9, 13, 300
    C = orc.gemm(_f32_bytes(np.ones((M, K))), _f32_bytes(np.ones((K, N))), M, N, K, "f32")
    assert np.all(C == K)


def test_closed_form_detects_transpose_and_dropped_terms(orc):
    # A[i][l] = (i+1)(l+1), B[l][j] = j+1  =>  C[i][j] = (i+1)(j+1) K(K+1)/2
    M, N, K = 5, 7, 11
    i = np.arange(M)[:, None] + 1.0
    l = np.arange(K)[None, :] + 1.0
    A = i * l
    B = np.tile(np.arange(N)[None, :] + 1.0, (K, 1))
    C = orc.gemm(_f32_bytes(A), _f32_bytes(B), M, N, K, "f32")
    expect = (np.arange(M)[:, None] + 1.0) * (np.arange(N)[None, :] + 1.0) * K * (K + 1) / 2
    assert np.array_equal(C, expect)


def test_bf16_widening_bit_patterns(orc):
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0001, 0x7F7F, 0x8000], dtype=np.uint16)
    got = orc.widen(bits.view(np.uint8), "bf16")
    expect = [1.0, -2.0, 1.0 + 2.0 ** -7, 2.0 ** -133, (2 - 2.0 ** -7) * 2.0 ** 127, -0.0]
    assert list(got) == expect
    assert np.signbit(got[-1])


def test_entries_match_full_product(orc):
    M, N, K = 40, 24, 96
    A, B = make_inputs(M, N, K, "bf16", 3, "normal")
    full = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, "bf16")
    rows = np.array([0, 39, 17, 5])
    cols = np.array([23, 0, 11, 5])
    ent = orc.gemm_entries(raw_bytes(A), raw_bytes(B), M, N, K, "bf16", rows, cols)
    assert np.array_equal(ent, full[rows, cols])


def test_threads_do_not_change_result(orc):
    M, N, K = 31, 17, 64
    A, B = make_inputs(M, N, K, "f32", 2, "normal")
    c1 = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, "f32", nthreads=1)
    c7 = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, "f32", nthreads=7)
    assert np.array_equal(c1, c7)


def test_fp64_exact_within_rounding_bound(orc):
    # |fl(sum) - sum| <= K * 2^-53 * sum|a||b| (Higham); check against exact rationals
    from fractions import Fraction
    M, N, K = 3, 4, 50
    A, B = make_inputs(M, N, K, "f32", 9, "uniform")
    C = orc.gemm(raw_bytes(A), raw_bytes(B), M, N, K, "f32")
    a, b = A.numpy().astype(np.float64), B.numpy().astype(np.float64)
    for i in range(M):
        for j in range(N):
            exact = sum(Fraction(a[i, l]) * Fraction(b[l, j]) for l in range(K))
            bound = K * 2.0 ** -53 * float(sum(abs(a[i, l] * b[l, j]) for l in range(K)))
            assert abs(Fraction(C[i, j]) - exact) <= Fraction(bound)


def test_paper_mac_example():
    g = json.load(open(GOLD))["mac_example"]
    macs = g["M"] * g["K"] * g["N"]
    assert macs == 33554432
    assert round(macs / 1e6) == g["ops_millions_rounded"]
