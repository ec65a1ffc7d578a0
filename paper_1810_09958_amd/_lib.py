"""Loader for the in-tree ``libisam.so`` and ctypes signatures of the C ABI (include/isam.h)."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
ISAM_F32, ISAM_BF16 = 0, 1

# name -> (restype, argtypes), mirroring include/isam.h
i64, vp, sz, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
SIGNATURES = {
    "isam_gemm": (ci, [ci, ci, i64, i64, i64, ci, vp, i64, vp, i64, ci, ci, vp, i64, vp, sz, vp]),
    "isam_gemm_workspace_size": (sz, [ci, ci, i64, i64, i64, ci, ci]),
    "isam_dwsep_conv": (ci, [i64] * 10 + [ci, vp, vp, vp, ci, vp, vp, sz, vp]),
    "isam_dwsep_conv_workspace_size": (sz, [i64] * 10 + [ci, ci]),
    "isam_gru_forward": (ci, [i64, i64, i64, i64, ci, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
    "isam_gru_forward_workspace_size": (sz, [i64, i64, i64, i64, ci]),
    "isam_gru_forward_noalloc": (ci, [i64, i64, i64, i64, ci, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
    "isam_conv1d": (ci, [i64, i64, i64, i64, i64, ci, vp, vp, ci, ci, vp, vp]),
    "isam_status_string": (ctypes.c_char_p, [ci]),
    "isam_last_error": (ctypes.c_char_p, []),
    "isam_version": (ci, []),
}


class IsamError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


def lib_path() -> str:
    """The in-tree libisam.so, or the file ISAM_LIB names (e.g. the sanitizer build)."""
    return os.environ.get("ISAM_LIB") or os.path.join(HERE, "libisam.so")


_lib = None


def lib():
    """Load libisam.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        path = lib_path()
        if not os.path.exists(path):
            raise ImportError(f"{path} is missing: build it with `python -m paper_1810_09958_amd.build`")
        L = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib
