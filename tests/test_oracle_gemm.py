"""Pins for the oracle's GEMM (the paper's first listing, Section 2).

Each pin is fixed by mathematics, not by re-running the oracle's own formula:
identity and permutation matrices, a rank-1 closed form, exact rational brute
force, a library special case (torch float64), and normaliser identities.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth


def _rand(shape, stream, lo=-1.0, hi=1.0):
    return synth.uniform(3, stream, shape, lo, hi)


def _golden(name):
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", name)
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    return rows


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_identity_right(dt):
    M, K = 37, 29
    A = _rand((M, K), 0)
    I = np.eye(K, dtype=np.float32)
    if dt == "bf16":
        A = synth.to_bf16_bits(A)
        I = synth.to_bf16_bits(I)
        Aval = synth.bf16_bits_to_f32(A)
    else:
        Aval = A
    C, _ = oracle.gemm(A, I, M, K, K)
    assert np.array_equal(C, Aval.astype(np.float64))


def test_identity_left():
    K, N = 23, 41
    B = _rand((K, N), 1)
    C, _ = oracle.gemm(np.eye(K, dtype=np.float32), B, K, N, K)
    assert np.array_equal(C, B.astype(np.float64))


def test_permutations():
    M, K, N = 19, 13, 17
    A = _rand((M, K), 2)
    B = _rand((K, N), 3)
    pk = np.random.default_rng(0).permutation(K)
    Pc = np.zeros((K, K), np.float32)
    Pc[pk, np.arange(K)] = 1.0          # column j of A.Pc is column pk[j] of A
    C, _ = oracle.gemm(A, Pc, M, K, K)
    assert np.array_equal(C, A[:, pk].astype(np.float64))
    Pr = np.zeros((K, K), np.float32)
    Pr[np.arange(K), pk] = 1.0          # row i of Pr.B is row pk[i] of B
    C2, _ = oracle.gemm(Pr, B, K, N, K)
    assert np.array_equal(C2, B[pk, :].astype(np.float64))


def test_rank1_closed_form():
    # A = u v^T (M x K), B = w z^T (K x N)  =>  A.B = (v . w) u z^T, exact in small integers.
    rng = np.random.default_rng(1)
    M, K, N = 11, 9, 7
    u, v, w, z = (rng.integers(-5, 6, n).astype(np.float32) for n in (M, K, K, N))
    A = np.outer(u, v).astype(np.float32)
    B = np.outer(w, z).astype(np.float32)
    C, S = oracle.gemm(A, B, M, N, K)
    expect = float(np.dot(v.astype(np.int64), w.astype(np.int64))) * np.outer(u, z)
    assert np.array_equal(C, expect)
    assert np.array_equal(S, float(np.dot(np.abs(v), np.abs(w))) * np.outer(np.abs(u), np.abs(z)))


@pytest.mark.parametrize("shape", [(1, 1, 1), (2, 3, 4), (5, 6, 3), (6, 5, 6), (3, 1, 5)])
@pytest.mark.parametrize("ta,tb", [(0, 0), (1, 0), (0, 1), (1, 1)])
def test_bruteforce_exact_rational(shape, ta, tb):
    M, N, K = shape
    Am = _rand((M, K), 4)
    Bm = _rand((K, N), 5)
    A = np.ascontiguousarray(Am.T) if ta else Am
    B = np.ascontiguousarray(Bm.T) if tb else Bm
    C, S = oracle.gemm(A, B, M, N, K, trans_a=ta, trans_b=tb)
    for i in range(M):
        for j in range(N):
            exact = sum((Fraction(float(Am[i, k])) * Fraction(float(Bm[k, j])) for k in range(K)),
                        Fraction(0))
            sabs = sum(abs(Fraction(float(Am[i, k])) * Fraction(float(Bm[k, j]))) for k in range(K))
            assert abs(Fraction(C[i, j]) - exact) <= Fraction(K + 1) * Fraction(2) ** -53 * (sabs + 1e-300)
            assert abs(Fraction(S[i, j]) - sabs) <= Fraction(K + 1) * Fraction(2) ** -53 * sabs


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_matches_torch_float64(dt):
    M, N, K = 70, 45, 133
    A = _rand((M, K), 6)
    B = _rand((K, N), 7)
    if dt == "bf16":
        A, B = synth.to_bf16_bits(A), synth.to_bf16_bits(B)
        Av, Bv = synth.bf16_bits_to_f32(A), synth.bf16_bits_to_f32(B)
    else:
        Av, Bv = A, B
    C, S = oracle.gemm(A, B, M, N, K)
    ref = (torch.from_numpy(Av).double() @ torch.from_numpy(Bv).double()).numpy()
    assert np.max(np.abs(C - ref) / S) < 1e-12


def test_leading_dims_ignore_padding():
    M, N, K = 9, 10, 11
    A = _rand((M, K), 8)
    B = _rand((K, N), 9)
    Ap = np.full((M, K + 5), 1e30, np.float32)
    Ap[:, :K] = A
    Bp = np.full((K, N + 3), -1e30, np.float32)
    Bp[:, :N] = B
    C0, _ = oracle.gemm(A, B, M, N, K)
    C1, _ = oracle.gemm(Ap, Bp, M, N, K, lda=K + 5, ldb=N + 3)
    assert np.array_equal(C0, C1)


def test_transposed_storage_same_result():
    M, N, K = 14, 9, 21
    A = _rand((M, K), 10)
    B = _rand((K, N), 11)
    C0, _ = oracle.gemm(A, B, M, N, K)
    C1, _ = oracle.gemm(np.ascontiguousarray(A.T), np.ascontiguousarray(B.T), M, N, K, 1, 1)
    assert np.array_equal(C0, C1)


def test_accumulate_and_k_zero():
    M, N, K = 5, 6, 7
    A = _rand((M, K), 12)
    B = _rand((K, N), 13)
    Cin = _rand((M, N), 14).astype(np.float64)
    C0, _ = oracle.gemm(A, B, M, N, K)
    C1, S1 = oracle.gemm(A, B, M, N, K, C_in=Cin)
    # accumulation adds C_in first, then the K products: compare within round-off
    assert np.max(np.abs(C1 - (Cin + C0))) <= 1e-14 * np.max(S1)
    Ck, Sk = oracle.gemm(A, B, M, N, 0, C_in=Cin)
    assert np.array_equal(Ck, Cin) and np.array_equal(Sk, np.abs(Cin))
    Cz, _ = oracle.gemm(A, B, M, N, 0)
    assert np.array_equal(Cz, np.zeros((M, N)))


def test_normaliser_equals_result_for_positive_inputs():
    M, N, K = 16, 12, 40
    A = _rand((M, K), 15, 0.0, 1.0)
    B = _rand((K, N), 16, 0.0, 1.0)
    C, S = oracle.gemm(A, B, M, N, K)
    assert np.array_equal(C, S)


def test_golden_integer_example():
    # tests/golden/gemm_int_2x3x4.txt: worked by hand (see its header)
    rows = _golden("gemm_int_2x3x4.txt")
    sec = {}
    cur = None
    for r in rows:
        if r[0] in ("A", "B", "C"):
            cur = r[0]
            sec[cur] = []
        else:
            sec[cur].append([float(v) for v in r])
    A = np.array(sec["A"], np.float32)
    B = np.array(sec["B"], np.float32)
    C, _ = oracle.gemm(A, B, 2, 4, 3)
    assert np.array_equal(C, np.array(sec["C"]))
