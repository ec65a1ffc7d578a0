"""GPU parity of isam_conv1d against the CPU oracle (the paper's second listing:
a 1D convolution computed as one implicit matrix product per sequence)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import workloads
from tests._util import TOL_BF16, TOL_F32, bits, norm_err, to_gpu, to_host_f64

pytestmark = pytest.mark.gpu

import paper_1810_09958_amd as isam


def _case(nb, L, Ki, D, Ko, dt="f32", ot="f32", accumulate=False, seed=0):
    A = synth.normal(seed, 20, (nb, L, Ki))
    B = synth.uniform(seed, 21, (D, Ki, Ko), -0.5, 0.5)
    if dt == "bf16":
        A, B = bits(A), bits(B)
    X = L - D + 1
    odt = torch.bfloat16 if ot == "bf16" else torch.float32
    Cin = None
    if accumulate:
        Cin = synth.uniform(seed, 22, (nb, X, Ko), -1.0, 1.0)
        out = torch.from_numpy(Cin).to("cuda").to(odt)
        Cin = out.float().cpu().numpy()   # what the kernel adds to (rounded to the output type)
        y = isam.conv1d(to_gpu(A), to_gpu(B), out=out, accumulate=True)
    else:
        y = isam.conv1d(to_gpu(A), to_gpu(B), out_dtype=odt)
    torch.cuda.synchronize()
    C, S = oracle.conv1d(A, B, C_in=Cin)
    err = norm_err(to_host_f64(y), C, S)
    tol = TOL_F32 if (dt == "f32" and ot == "f32") else TOL_BF16
    assert err <= tol, f"nb={nb} L={L} Ki={Ki} D={D} Ko={Ko} {dt}->{ot} acc={accumulate}: {err:.3e}"


@pytest.mark.parametrize("dt,ot", [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16")])
def test_shapes(dt, ot):
    # ragged tiles (X, Ko not multiples of the tile), several taps, one tap,
    # channel counts off the 16-byte vector width (element-wise loader)
    for (nb, L, Ki, D, Ko) in [(2, 70, 64, 3, 48), (3, 130, 32, 5, 256), (1, 9, 16, 1, 8),
                               (2, 33, 12, 4, 20), (4, 300, 128, 7, 96)]:
        _case(nb, L, Ki, D, Ko, dt=dt, ot=ot, seed=L + Ki)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_accumulate(dt):
    _case(2, 40, 64, 3, 64, dt=dt, accumulate=True)


def test_no_valid_position_is_noop():
    A = torch.zeros((2, 3, 8), device="cuda")
    B = torch.zeros((4, 8, 8), device="cuda")
    y = isam.conv1d(A, B)
    assert tuple(y.shape) == (2, 0, 8)


@pytest.mark.parametrize("variant", ["bf16", "f32"])
def test_config_full_size_sampled_sequences(variant):
    w = workloads.conv1d()
    A, B = (w["A_bf16"], w["B_bf16"]) if variant == "bf16" else (w["A"], w["B"])
    y = isam.conv1d(to_gpu(A), to_gpu(B))
    torch.cuda.synchronize()
    seqs = [0, 17, 31]   # sequences are independent: the oracle runs on a subset
    C, S = oracle.conv1d(np.ascontiguousarray(A[seqs]), B)
    got = to_host_f64(y[torch.as_tensor(seqs, device="cuda")])
    assert norm_err(got, C, S) <= (TOL_BF16 if variant == "bf16" else TOL_F32)
