"""Input recipes for the benchmark workloads (seed 0, one stream per tensor).

Each builder returns host numpy arrays: fp32 values and, where the workload is
bf16, the bf16 bit patterns (uint16) obtained by RNE from those fp32 values.
The shapes and distributions stand in for the paper's DeepBench-sized and
internal GEMM / GRU workloads and for a MobileNet-style separable layer; none
of those suites' own items are used.
"""
from __future__ import annotations

import math

import numpy as np

from . import normal, to_bf16_bits, uniform

SEED = 0


def gemm_small_fp32(M=128, N=128, K=128, seed=SEED):
    """fp32 C = A.B, A and B i.i.d. uniform[-1, 1), row-major NN."""
    A = uniform(seed, 0, (M, K), -1.0, 1.0)
    B = uniform(seed, 1, (K, N), -1.0, 1.0)
    return {"A": A, "B": B}


def skinny(M=4096, N=32, K=4096, seed=SEED):
    """RNN-style skinny GEMM: weights A uniform[-1/64, 1/64), activations B normal(0, 1)."""
    A = uniform(seed, 0, (M, K), -1.0 / 64, 1.0 / 64)
    B = normal(seed, 1, (K, N))
    return {"A": A, "B": B, "A_bf16": to_bf16_bits(A), "B_bf16": to_bf16_bits(B)}


def gru(T=64, batch=32, input_size=1024, hidden=1024, seed=SEED):
    """GRU forward: W, U uniform[-1/32, 1/32) (rows stacked r, z, n), bias normal(0, 0.01^2),
    x normal(0, 1) laid out [T][batch][input], h0 = 0."""
    H = hidden
    W = uniform(seed, 0, (3 * H, input_size), -1.0 / 32, 1.0 / 32)
    U = uniform(seed, 1, (3 * H, H), -1.0 / 32, 1.0 / 32)
    b = normal(seed, 2, (3 * H,), scale=0.01)
    x = normal(seed, 3, (T, batch, input_size))
    return {"W": W, "U": U, "bias": b, "x": x,
            "W_bf16": to_bf16_bits(W), "U_bf16": to_bf16_bits(U), "x_bf16": to_bf16_bits(x)}


def dwsep(batch=32, H=56, W=56, C_in=128, C_out=256, depth_mult=1, kh=3, kw=3, seed=SEED):
    """Depthwise-separable layer: X NHWC normal(0, 1); depthwise D [kh][kw][C_in][c]
    uniform[-1/3, 1/3); pointwise P [C_in*c][C_out] uniform[-1/11, 1/11)."""
    X = normal(seed, 0, (batch, H, W, C_in))
    D = uniform(seed, 1, (kh, kw, C_in, depth_mult), -1.0 / 3, 1.0 / 3)
    P = uniform(seed, 2, (C_in * depth_mult, C_out), -1.0 / 11, 1.0 / 11)
    return {"X": X, "D": D, "P": P,
            "X_bf16": to_bf16_bits(X), "D_bf16": to_bf16_bits(D), "P_bf16": to_bf16_bits(P)}


def gemm_large_bf16(M=8192, N=8192, K=8192, streams=(0, 1), seed=SEED):
    """Large bf16 GEMM: A and B normal(0, 1) scaled by 1/sqrt(K), NN, returned as bf16 bits."""
    s = 1.0 / math.sqrt(K)
    A = to_bf16_bits(normal(seed, streams[0], (M, K), scale=s))
    B = to_bf16_bits(normal(seed, streams[1], (K, N), scale=s))
    return {"A_bf16": A, "B_bf16": B}


def gemm_square_bf16(seed=SEED):
    return gemm_large_bf16(8192, 8192, 8192, streams=(0, 1), seed=seed)


def gemm_rect_bf16(seed=SEED):
    return gemm_large_bf16(8192, 1024, 16384, streams=(2, 3), seed=seed)


def conv1d(batch=32, X=1024, Ki=512, D=5, Ko=512, seed=SEED):
    """1D convolution (the paper's second listing) at a speech-model-like size:
    A [batch][X+D-1][Ki] normal(0, 1), B [D][Ki][Ko] uniform[-1/sqrt(D*Ki), +); fp32 and bf16."""
    L = X + D - 1
    A = normal(seed, 0, (batch, L, Ki))
    r = 1.0 / math.sqrt(D * Ki)
    B = uniform(seed, 1, (D, Ki, Ko), -r, r)
    return {"A": A, "B": B, "A_bf16": to_bf16_bits(A), "B_bf16": to_bf16_bits(B)}


def rows_sample(M: int, count: int, seed: int = 1234) -> np.ndarray:
    """Sorted distinct row indices for sampled checks; always includes the first and last row."""
    if count >= M:
        return np.arange(M)
    x = (np.arange(count, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15) + np.uint64(seed))
    idx = (x % np.uint64(M)).astype(np.int64)
    idx = np.unique(np.concatenate([idx, [0, M - 1]]))
    return idx
