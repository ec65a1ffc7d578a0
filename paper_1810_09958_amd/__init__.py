"""MI355X (gfx950) hot path of ISA Mapper (arXiv 1810.09958): GEMM, separable depthwise
convolution and GRU forward, as hand-written HIP kernels behind the C ABI in
``include/isam.h``.

This module is argument marshalling only: it checks torch tensors (device, dtype,
contiguity), sizes and allocates the workspace, and calls the C ABI on torch's current
stream.  Every arithmetic step runs in the library's kernels.  If ``libisam.so`` is
missing the calls raise; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

from ._lib import (ISAM_BF16, ISAM_F32, IsamError, lib, lib_path)

__all__ = ["gemm", "conv1d", "dwsep_conv", "gru_forward", "gru_forward_noalloc", "gemm_workspace_size",
           "dwsep_conv_workspace_size", "gru_forward_workspace_size", "IsamError",
           "lib", "lib_path", "ISAM_F32", "ISAM_BF16", "version"]

_DT = {torch.float32: ISAM_F32, torch.bfloat16: ISAM_BF16}


def _dt(t: torch.Tensor) -> int:
    try:
        return _DT[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16") from None


def _ptr(t):
    # plain ints: the ctypes signatures convert them (no per-call c_void_p objects)
    return None if t is None else t.data_ptr()


try:
    _raw_stream = torch._C._cuda_getCurrentRawStream  # current stream handle, no Stream object
except AttributeError:  # pragma: no cover - older torch
    _raw_stream = None


def _stream():
    if _raw_stream is not None:
        return _raw_stream(torch.cuda.current_device())
    return torch.cuda.current_stream().cuda_stream


def _check_dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("tensors must be on the GPU")


def _call(rc, name):
    if rc != 0:
        L = lib()
        raise IsamError(rc, f"{name}: {L.isam_status_string(rc).decode()}: {L.isam_last_error().decode()}")


def version() -> int:
    return lib().isam_version()


def conv1d(A: torch.Tensor, B: torch.Tensor, out: torch.Tensor | None = None, *, accumulate=False,
           out_dtype=None):
    """1D convolution (valid, stride 1): C[i][x][ko] (+)= sum_{d,ki} A[i][x+d][ki] * B[d][ki][ko].
    A is [batch][L][Ki], B is [D][Ki][Ko], both contiguous and of one dtype; returns C
    ([batch][L-D+1][Ko], float32 unless out_dtype / out say otherwise)."""
    _check_dev(A, B, out)
    if A.dim() != 3 or B.dim() != 3:
        raise ValueError("A must be [batch][L][Ki] and B [D][Ki][Ko]")
    if not A.is_contiguous() or not B.is_contiguous():
        raise ValueError("A and B must be contiguous")
    if A.dtype != B.dtype:
        raise TypeError("A and B must share a dtype")
    nb, L, Ki = A.shape
    D, Ki2, Ko = B.shape
    if Ki2 != Ki:
        raise ValueError(f"channel counts differ: {Ki} vs {Ki2}")
    X = max(L - D + 1, 0)
    if out is None:
        if accumulate:
            raise ValueError("accumulate needs out")
        out = torch.empty((nb, X, Ko), device=A.device, dtype=out_dtype or torch.float32)
    elif tuple(out.shape) != (nb, X, Ko) or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous [{nb}][{X}][{Ko}] tensor")
    rc = lib().isam_conv1d(nb, L, Ki, D, Ko, _dt(A), _ptr(A), _ptr(B), int(accumulate), _dt(out), _ptr(out),
                           _stream())
    _call(rc, "isam_conv1d")
    return out


def gemm_workspace_size(M, N, K, ab_type, c_type, trans_a=0, trans_b=0) -> int:
    return lib().isam_gemm_workspace_size(trans_a, trans_b, M, N, K, ab_type, c_type)


def gemm(A: torch.Tensor, B: torch.Tensor, out: torch.Tensor | None = None, *, trans_a=False,
         trans_b=False, accumulate=False, out_dtype=None, workspace: torch.Tensor | None = None):
    """C (+)= op(A) op(B).  A is [M][K] ([K][M] with trans_a); B is [K][N] ([N][K] with
    trans_b).  Row strides may exceed the row length (leading dimensions); the inner stride
    must be 1.  Returns C ([M][N], float32 unless out_dtype / out say otherwise)."""
    _check_dev(A, B, out, workspace)
    if A.dim() != 2 or B.dim() != 2:
        raise ValueError("A and B must be 2-D")
    if A.stride(1) != 1 or B.stride(1) != 1:
        raise ValueError("A and B need unit inner stride")
    M, K = (A.shape[1], A.shape[0]) if trans_a else (A.shape[0], A.shape[1])
    KB, N = (B.shape[1], B.shape[0]) if trans_b else (B.shape[0], B.shape[1])
    if KB != K:
        raise ValueError(f"inner sizes differ: {K} vs {KB}")
    if A.dtype != B.dtype:
        raise TypeError("A and B must share a dtype")
    if out is None:
        if accumulate:
            raise ValueError("accumulate needs out")
        out = torch.empty((M, N), device=A.device, dtype=out_dtype or torch.float32)
    if out.shape != (M, N) or (N > 0 and out.stride(1) != 1):
        raise ValueError("out must be [M][N] with unit inner stride")
    ab, ct = _dt(A), _dt(out)
    if workspace is None:
        need = gemm_workspace_size(M, N, K, ab, ct, int(trans_a), int(trans_b))
        workspace = torch.empty(max(need, 1), device=A.device, dtype=torch.uint8)
    rc = lib().isam_gemm(int(trans_a), int(trans_b), M, N, K, ab, _ptr(A), max(A.stride(0), 1),
                         _ptr(B), max(B.stride(0), 1), int(accumulate), ct, _ptr(out),
                         max(out.stride(0), 1), _ptr(workspace), workspace.numel(), _stream())
    _call(rc, "isam_gemm")
    return out


def dwsep_conv_workspace_size(batch, H, W, C_in, depth_mult, kh, kw, stride, pad, C_out,
                              in_type, out_type) -> int:
    return lib().isam_dwsep_conv_workspace_size(batch, H, W, C_in, depth_mult, kh, kw, stride,
                                                pad, C_out, in_type, out_type)


def dwsep_conv(x: torch.Tensor, dw_filter: torch.Tensor, pw_weight: torch.Tensor, *, stride=1,
               pad=1, out: torch.Tensor | None = None, out_dtype=None,
               workspace: torch.Tensor | None = None):
    """Separable depthwise convolution (depthwise kh x kw, then pointwise 1x1), NHWC.
    x [b][H][W][C_in], dw_filter [kh][kw][C_in][c], pw_weight [C_in*c][C_out]."""
    _check_dev(x, dw_filter, pw_weight, out, workspace)
    for t in (x, dw_filter, pw_weight):
        if not t.is_contiguous():
            raise ValueError("inputs must be contiguous")
    if not (x.dtype == dw_filter.dtype == pw_weight.dtype):
        raise TypeError("x, dw_filter and pw_weight must share a dtype")
    b, H, W, C = x.shape
    kh, kw, C2, cm = dw_filter.shape
    Cm, Co = pw_weight.shape
    if C2 != C or Cm != C * cm:
        raise ValueError("filter shapes do not match x")
    Ho = (H + 2 * pad - kh) // stride + 1
    Wo = (W + 2 * pad - kw) // stride + 1
    if out is None:
        out = torch.empty((b, Ho, Wo, Co), device=x.device, dtype=out_dtype or torch.float32)
    if not out.is_contiguous() or tuple(out.shape) != (b, Ho, Wo, Co):
        raise ValueError("out must be contiguous [b][Ho][Wo][C_out]")
    it, ot = _dt(x), _dt(out)
    if workspace is None:
        need = dwsep_conv_workspace_size(b, H, W, C, cm, kh, kw, stride, pad, Co, it, ot)
        workspace = torch.empty(max(need, 1), device=x.device, dtype=torch.uint8)
    rc = lib().isam_dwsep_conv(b, H, W, C, cm, kh, kw, stride, pad, Co, it, _ptr(x),
                               _ptr(dw_filter), _ptr(pw_weight), ot, _ptr(out), _ptr(workspace),
                               workspace.numel(), _stream())
    _call(rc, "isam_dwsep_conv")
    return out


def gru_forward_workspace_size(T, batch, input_size, hidden, w_type) -> int:
    return lib().isam_gru_forward_workspace_size(T, batch, input_size, hidden, w_type)


def gru_forward(x: torch.Tensor, W: torch.Tensor, U: torch.Tensor, *, bias=None, bias_hn=None,
                h0=None, return_sequence=True, h_seq=None, h_T=None,
                workspace: torch.Tensor | None = None):
    """GRU forward.  x [T][batch][I], W [3H][I], U [3H][H] (gate rows r, z, n; float32 or
    bfloat16), bias [3H], bias_hn [H], h0 [batch][H] float32 or None.  Returns (h_seq, h_T)."""
    _check_dev(x, W, U, bias, bias_hn, h0, h_seq, h_T, workspace)
    for t in (x, W, U, bias, bias_hn, h0):
        if t is not None and not t.is_contiguous():
            raise ValueError("inputs must be contiguous")
    if not (x.dtype == W.dtype == U.dtype):
        raise TypeError("x, W, U must share a dtype")
    for t in (bias, bias_hn, h0):
        if t is not None and t.dtype != torch.float32:
            raise TypeError("bias, bias_hn and h0 are float32")
    T, B, I = x.shape
    H = U.shape[1]
    if tuple(W.shape) != (3 * H, I) or tuple(U.shape) != (3 * H, H):
        raise ValueError("W must be [3H][I] and U [3H][H]")
    dev = x.device
    if h_seq is None and return_sequence:
        h_seq = torch.empty((T, B, H), device=dev, dtype=torch.float32)
    if h_T is None:
        h_T = torch.empty((B, H), device=dev, dtype=torch.float32)
    wt = _dt(W)
    if workspace is None:
        need = gru_forward_workspace_size(T, B, I, H, wt)
        workspace = torch.empty(max(need, 1), device=dev, dtype=torch.uint8)
    rc = lib().isam_gru_forward(T, B, I, H, wt, _ptr(x), _ptr(h0), _ptr(W), _ptr(U), _ptr(bias),
                                _ptr(bias_hn), _ptr(h_seq), _ptr(h_T), _ptr(workspace),
                                workspace.numel(), _stream())
    _call(rc, "isam_gru_forward")
    return h_seq, h_T


def gru_forward_noalloc(x: torch.Tensor, W: torch.Tensor, U: torch.Tensor, h_seq: torch.Tensor,
                        h_T: torch.Tensor, *, bias=None, bias_hn=None, h0=None):
    """GRU forward through isam_gru_forward_noalloc: the library's static device scratch
    serves as workspace and nothing is allocated (h_seq and h_T are caller-provided; either
    may be None, not both).  Calls that overlap in time on one device race."""
    _check_dev(x, W, U, bias, bias_hn, h0, h_seq, h_T)
    for t in (x, W, U, bias, bias_hn, h0, h_seq, h_T):
        if t is not None and not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
    if not (x.dtype == W.dtype == U.dtype):
        raise TypeError("x, W, U must share a dtype")
    T, B, I = x.shape
    H = U.shape[1]
    rc = lib().isam_gru_forward_noalloc(T, B, I, H, _dt(W), _ptr(x), _ptr(h0), _ptr(W), _ptr(U), _ptr(bias),
                                        _ptr(bias_hn), _ptr(h_seq), _ptr(h_T), _stream())
    _call(rc, "isam_gru_forward_noalloc")
    return h_seq, h_T
