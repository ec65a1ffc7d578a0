"""CPU oracle -- test infrastructure only.

Thin ctypes wrapper over ``libisam_ref.so`` (built from ``isam_ref.c`` with gcc,
fp64, no fast-math, no FMA contraction).  Only ``tests/``, the smoke check and
the benchmark's CPU-baseline leg may import this package; the GPU library never
does, and the two share no code.

All functions take numpy arrays.  bf16 tensors are passed as uint16 bit
patterns (``dtype=np.uint16``); fp32 tensors as ``np.float32``.  Results are
fp64 numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "isam_ref.c")
_LIB = os.path.join(_HERE, "libisam_ref.so")

F32, BF16 = 0, 1


_SAN_LIB = os.path.join(_HERE, "libisam_ref_san.so")


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (OpenMP, -O2, no fast-math, no FP contraction); with
    sanitize, a separate copy under AddressSanitizer and UndefinedBehaviorSanitizer (load it
    with gcc's libasan and libubsan preloaded and ISAM_REF_LIB pointing at it)."""
    out = _SAN_LIB if sanitize else _LIB
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        san = ["-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"] if sanitize else []
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", *san,
               "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("ISAM_REF_LIB") or _LIB
        if path == _LIB and not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(path)
        i64, vp, dp, fp = ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p
        ci = ctypes.c_int
        L.isam_ref_gemm.argtypes = [ci, ci, i64, i64, i64, ci, vp, i64, vp, i64, dp, dp, dp, ci]
        L.isam_ref_depthwise.argtypes = [i64] * 9 + [ci, vp, vp, dp, dp, ci]
        L.isam_ref_dwsep.argtypes = [i64] * 10 + [ci, vp, vp, vp, dp, dp, ci]
        L.isam_ref_dwsep_direct.argtypes = [i64] * 10 + [ci, vp, vp, vp, dp]
        L.isam_ref_gru.argtypes = [i64, i64, i64, i64, ci, vp, dp, vp, vp, fp, fp, dp, ci]
        L.isam_ref_conv1d.argtypes = [i64] * 5 + [ci, vp, vp, dp, dp, dp, ci]
        L.isam_ref_max_threads.argtypes = []
        for f in ("isam_ref_gemm", "isam_ref_depthwise", "isam_ref_dwsep",
                  "isam_ref_dwsep_direct", "isam_ref_gru", "isam_ref_conv1d", "isam_ref_max_threads"):
            getattr(L, f).restype = ci
        _lib = L
    return _lib


def max_threads() -> int:
    return lib().isam_ref_max_threads()


def _dtype_of(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"oracle inputs must be float32 or uint16 (bf16 bits), got {a.dtype}")


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, name):
    if rc != 0:
        raise RuntimeError(f"{name} returned {rc}")


def gemm(A, B, M, N, K, trans_a=0, trans_b=0, lda=None, ldb=None, C_in=None,
         with_norm=True, threads=0):
    """C = C_in + op(A) op(B) in fp64 (the paper's first listing).  A and B are flat or
    2-D buffers in the stated layout; returns (C, S) with S = sum |a||b| (+|C_in|)."""
    A = np.ascontiguousarray(A)
    B = np.ascontiguousarray(B)
    dt = _dtype_of(A)
    if _dtype_of(B) != dt:
        raise TypeError("A and B must share one dtype")
    lda = lda if lda is not None else (M if trans_a else K)
    ldb = ldb if ldb is not None else (K if trans_b else N)
    C = np.empty((M, N), np.float64)
    S = np.empty((M, N), np.float64) if with_norm else None
    cin = None if C_in is None else np.ascontiguousarray(C_in, dtype=np.float64).reshape(M, N)
    _check(lib().isam_ref_gemm(trans_a, trans_b, M, N, K, dt, _ptr(A), lda, _ptr(B), ldb,
                               _ptr(cin), _ptr(C), _ptr(S), threads), "isam_ref_gemm")
    return C, S


def conv1d(A, B, C_in=None, with_norm=True, threads=0):
    """1D convolution (the paper's second listing, valid positions, stride 1):
    A [batch][L][Ki], B [D][Ki][Ko] -> (C, S) fp64 [batch][L-D+1][Ko]."""
    A = np.ascontiguousarray(A)
    B = np.ascontiguousarray(B)
    dt = _dtype_of(A)
    if _dtype_of(B) != dt:
        raise TypeError("A and B must share one dtype")
    nb, L, Ki = A.shape
    D, Ki2, Ko = B.shape
    assert Ki2 == Ki
    X = max(L - D + 1, 0)
    C = np.empty((nb, X, Ko), np.float64)
    S = np.empty_like(C) if with_norm else None
    cin = None if C_in is None else np.ascontiguousarray(C_in, dtype=np.float64).reshape(nb, X, Ko)
    _check(lib().isam_ref_conv1d(nb, L, Ki, D, Ko, dt, _ptr(A), _ptr(B), _ptr(cin), _ptr(C), _ptr(S), threads),
           "isam_ref_conv1d")
    return C, S


def _out_hw(H, W, kh, kw, stride, pad):
    return (H + 2 * pad - kh) // stride + 1, (W + 2 * pad - kw) // stride + 1


def depthwise(x, dw, stride=1, pad=1, with_norm=True, threads=0):
    """Depthwise half: x NHWC [b][H][W][C], dw [kh][kw][C][c] -> Y [b][Ho][Wo][C*c] fp64."""
    x = np.ascontiguousarray(x)
    dw = np.ascontiguousarray(dw)
    dt = _dtype_of(x)
    b, H, W, C = x.shape
    kh, kw, C2, cm = dw.shape
    assert C2 == C
    Ho, Wo = _out_hw(H, W, kh, kw, stride, pad)
    Y = np.empty((b, Ho, Wo, C * cm), np.float64)
    SY = np.empty_like(Y) if with_norm else None
    _check(lib().isam_ref_depthwise(b, H, W, C, cm, kh, kw, stride, pad, dt, _ptr(x), _ptr(dw),
                                    _ptr(Y), _ptr(SY), threads), "isam_ref_depthwise")
    return Y, SY


def dwsep(x, dw, pw, stride=1, pad=1, with_norm=True, threads=0):
    """Separable depthwise convolution (third listing), factored: returns (Z, S) fp64 NHWC."""
    x = np.ascontiguousarray(x)
    dw = np.ascontiguousarray(dw)
    pw = np.ascontiguousarray(pw)
    dt = _dtype_of(x)
    b, H, W, C = x.shape
    kh, kw, _, cm = dw.shape
    Cm, Co = pw.shape
    assert Cm == C * cm
    Ho, Wo = _out_hw(H, W, kh, kw, stride, pad)
    Z = np.empty((b, Ho, Wo, Co), np.float64)
    S = np.empty_like(Z) if with_norm else None
    _check(lib().isam_ref_dwsep(b, H, W, C, cm, kh, kw, stride, pad, Co, dt, _ptr(x), _ptr(dw),
                                _ptr(pw), _ptr(Z), _ptr(S), threads), "isam_ref_dwsep")
    return Z, S


def dwsep_direct(x, dw, pw, stride=1, pad=1):
    """The third listing's unfactored 8-index sum (self-test only)."""
    x = np.ascontiguousarray(x)
    dw = np.ascontiguousarray(dw)
    pw = np.ascontiguousarray(pw)
    dt = _dtype_of(x)
    b, H, W, C = x.shape
    kh, kw, _, cm = dw.shape
    Cm, Co = pw.shape
    Ho, Wo = _out_hw(H, W, kh, kw, stride, pad)
    Z = np.empty((b, Ho, Wo, Co), np.float64)
    _check(lib().isam_ref_dwsep_direct(b, H, W, C, cm, kh, kw, stride, pad, Co, dt, _ptr(x),
                                       _ptr(dw), _ptr(pw), _ptr(Z)), "isam_ref_dwsep_direct")
    return Z


def gru(x, W, U, bias=None, bhn=None, h0=None, threads=0):
    """GRU forward: x [T][batch][I], W [3H][I], U [3H][H] (gate rows r, z, n), bias [3H] and
    bhn [H] fp32 or None, h0 [batch][H] or None.  Returns h_seq [T][batch][H] fp64."""
    x = np.ascontiguousarray(x)
    W = np.ascontiguousarray(W)
    U = np.ascontiguousarray(U)
    dt = _dtype_of(x)
    assert _dtype_of(W) == dt and _dtype_of(U) == dt
    T, batch, I = x.shape
    H = U.shape[1]
    assert W.shape == (3 * H, I) and U.shape == (3 * H, H)
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    bn = None if bhn is None else np.ascontiguousarray(bhn, dtype=np.float32)
    h = None if h0 is None else np.ascontiguousarray(h0, dtype=np.float64)
    out = np.empty((T, batch, H), np.float64)
    _check(lib().isam_ref_gru(T, batch, I, H, dt, _ptr(x), _ptr(h), _ptr(W), _ptr(U), _ptr(b),
                              _ptr(bn), _ptr(out), threads), "isam_ref_gru")
    return out
