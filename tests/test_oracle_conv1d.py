"""Pins for the oracle's 1D convolution (the paper's second listing, Section 2).

Each pin is fixed by mathematics or an independent library, not by re-running the
oracle's own formula: a shifted identity filter, an all-ones closed form, exact
rational brute force, one-tap reduction to a matrix product (torch float64), the
library special case torch.nn.functional.conv1d in float64, and a hand-checked
golden example.
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth


def _rand(shape, stream, lo=-1.0, hi=1.0):
    return synth.uniform(11, stream, shape, lo, hi)


def test_shifted_identity_filter():
    # B[d][ki][ko] = [d == d0][ki == ko]  =>  C[i][x][k] = A[i][x + d0][k]
    nb, L, K, D, d0 = 2, 13, 6, 4, 2
    A = _rand((nb, L, K), 0)
    B = np.zeros((D, K, K), np.float32)
    B[d0] = np.eye(K, dtype=np.float32)
    C, _ = oracle.conv1d(A, B)
    X = L - D + 1
    assert C.shape == (nb, X, K)
    assert np.array_equal(C, A[:, d0:d0 + X, :].astype(np.float64))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_all_ones_closed_form(dt):
    nb, L, Ki, D, Ko = 3, 9, 5, 3, 7
    A = np.ones((nb, L, Ki), np.float32)
    B = np.ones((D, Ki, Ko), np.float32)
    if dt == "bf16":
        A, B = synth.to_bf16_bits(A), synth.to_bf16_bits(B)
    C, S = oracle.conv1d(A, B)
    assert np.all(C == D * Ki) and np.all(S == D * Ki)


def test_bruteforce_exact_rational():
    nb, L, Ki, D, Ko = 2, 6, 3, 3, 2
    A = _rand((nb, L, Ki), 1)
    B = _rand((D, Ki, Ko), 2)
    C, S = oracle.conv1d(A, B)
    X = L - D + 1
    for i in range(nb):
        for x in range(X):
            for ko in range(Ko):
                exact = sum(Fraction(float(A[i, x + d, ki])) * Fraction(float(B[d, ki, ko]))
                            for d in range(D) for ki in range(Ki))
                bound = D * Ki * 2.0 ** -52 * S[i, x, ko]
                assert abs(float(Fraction(C[i, x, ko]) - exact)) <= bound


def test_one_tap_is_matrix_product():
    # D == 1: each sequence is A_i . B[0]
    nb, L, Ki, Ko = 3, 17, 11, 5
    A = _rand((nb, L, Ki), 3)
    B = _rand((1, Ki, Ko), 4)
    C, _ = oracle.conv1d(A, B)
    ref = torch.matmul(torch.from_numpy(A).double(), torch.from_numpy(B[0]).double()).numpy()
    assert np.allclose(C, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("D", [1, 2, 5])
def test_matches_torch_conv1d_float64(D):
    # torch's conv1d is a cross-correlation over [batch][channels][length]:
    # weight[ko][ki][d] = B[d][ki][ko].
    nb, L, Ki, Ko = 2, 23, 7, 9
    A = _rand((nb, L, Ki), 5)
    B = _rand((D, Ki, Ko), 6)
    C, S = oracle.conv1d(A, B)
    a = torch.from_numpy(A).double().permute(0, 2, 1)
    w = torch.from_numpy(B).double().permute(2, 1, 0).contiguous()
    ref = torch.nn.functional.conv1d(a, w).permute(0, 2, 1).numpy()
    assert np.all(np.abs(C - ref) <= 1e-12 * S)


def test_accumulate_and_empty():
    nb, L, Ki, D, Ko = 1, 8, 4, 3, 3
    A = _rand((nb, L, Ki), 7)
    B = _rand((D, Ki, Ko), 8)
    C0, _ = oracle.conv1d(A, B)
    Cin = _rand((nb, L - D + 1, Ko), 9).astype(np.float64)
    C1, _ = oracle.conv1d(A, B, C_in=Cin)
    assert np.allclose(C1, C0 + Cin, rtol=0, atol=1e-15)
    # L < D: no valid position
    Ce, _ = oracle.conv1d(_rand((1, 2, Ki), 10), _rand((3, Ki, Ko), 11))
    assert Ce.shape == (1, 0, Ko)


def test_golden_small_example():
    # tests/golden/conv1d_1x4x2_d2.txt: A, B and C of a hand-checked case
    path = os.path.join(os.path.dirname(__file__), "golden", "conv1d_1x4x2_d2.txt")
    vals = {}
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, *nums = line.split()
        vals[name] = np.array([float(v) for v in nums], np.float32)
    A = vals["A"].reshape(1, 4, 2)
    B = vals["B"].reshape(2, 2, 1)
    C, _ = oracle.conv1d(A, B)
    assert np.array_equal(C.reshape(-1), vals["C"].astype(np.float64))
