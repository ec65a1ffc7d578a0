"""Shared helpers for the GPU parity tests (not collected: no test_ prefix)."""
import numpy as np
import torch

import synth

TOL_BF16 = 1e-2   # max |gpu - oracle| / sum|a||b| for bf16 inputs
TOL_F32 = 1e-5    # same, fp32 inputs and outputs


def dev():
    return torch.device("cuda:0")


def to_gpu(a: np.ndarray) -> torch.Tensor:
    """fp32 numpy -> float32 cuda tensor; uint16 numpy (bf16 bits) -> bfloat16 cuda tensor."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(dev())
    if a.dtype == np.float32:
        return torch.from_numpy(a.copy()).to(dev())
    raise TypeError(a.dtype)


def to_host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def norm_err(out: np.ndarray, ref: np.ndarray, S: np.ndarray) -> float:
    """max |out - ref| / S over entries with S > 0; entries with S == 0 must match exactly."""
    out = np.asarray(out, np.float64)
    assert np.all(np.isfinite(out)), "non-finite output"
    zero = S == 0
    if np.any(zero):
        assert np.array_equal(out[zero], ref[zero]), "output differs where the normaliser is 0"
    if np.all(zero):
        return 0.0
    return float(np.max(np.abs(out - ref)[~zero] / S[~zero]))


def bits(a_f32: np.ndarray) -> np.ndarray:
    return synth.to_bf16_bits(a_f32)
