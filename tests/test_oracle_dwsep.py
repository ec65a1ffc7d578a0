"""Pins for the oracle's separable depthwise convolution (the paper's third listing,
Section 2) and its factoring into depthwise then pointwise (Section 2.3)."""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth


def _x(shape, stream):
    return synth.normal(5, stream, shape)


def _u(shape, stream, a):
    return synth.uniform(5, stream, shape, -a, a)


@pytest.mark.parametrize("stride", [1, 2])
@pytest.mark.parametrize("cm", [1, 2])
@pytest.mark.parametrize("pad", [0, 1])
@pytest.mark.parametrize("k", [(3, 3), (1, 1), (3, 2)])
def test_factored_equals_direct_listing(stride, cm, pad, k):
    kh, kw = k
    b, H, W, C, Co = 2, 7, 6, 3, 4
    X = _x((b, H, W, C), 0)
    D = _u((kh, kw, C, cm), 1, 1.0 / 3)
    P = _u((C * cm, Co), 2, 1.0 / 11)
    Z, S = oracle.dwsep(X, D, P, stride=stride, pad=pad)
    Zd = oracle.dwsep_direct(X, D, P, stride=stride, pad=pad)
    assert Z.shape == Zd.shape
    # real-arithmetic identity; the two fp64 evaluations differ only by round-off.
    # Outputs whose every tap lies in the zero padding (S == 0) must be exactly 0 in both.
    zero = S == 0
    assert np.all(Z[zero] == 0) and np.all(Zd[zero] == 0)
    assert np.max(np.abs(Z - Zd)[~zero] / S[~zero]) < 1e-13


def test_padding_closed_form_counts():
    # X = 1, D = 1 (c = 1, 3x3, pad 1, stride 1): Y counts the in-image taps: 4 at corners,
    # 6 on edges, 9 inside.  Fixture tests/golden/dw_ones_5x6.txt lists the map.
    X = np.ones((1, 5, 6, 2), np.float32)
    D = np.ones((3, 3, 2, 1), np.float32)
    Y, _ = oracle.depthwise(X, D, stride=1, pad=1)
    path = os.path.join(os.path.dirname(__file__), "golden", "dw_ones_5x6.txt")
    want = np.array([[float(v) for v in l.split()] for l in open(path)
                     if l.strip() and not l.startswith("#")])
    for c in range(2):
        assert np.array_equal(Y[0, :, :, c], want)


def test_delta_filter_is_identity():
    X = _x((2, 5, 7, 4), 3)
    D = np.zeros((3, 3, 4, 1), np.float32)
    D[1, 1] = 1.0
    Y, _ = oracle.depthwise(X, D, stride=1, pad=1)
    assert np.array_equal(Y, X.astype(np.float64))


def test_shifted_delta_filter_is_shift():
    X = _x((1, 6, 5, 3), 4)
    D = np.zeros((3, 3, 3, 1), np.float32)
    D[0, 2] = 1.0   # tap (di=0, dj=2) reads X[i-1][j+1]
    Y, _ = oracle.depthwise(X, D, stride=1, pad=1)
    want = np.zeros_like(Y)
    want[0, 1:, :-1] = X[0, :-1, 1:]
    assert np.array_equal(Y, want)


def test_pointwise_identity():
    X = _x((2, 4, 4, 5), 5)
    D = _u((3, 3, 5, 1), 6, 1.0 / 3)
    Y, _ = oracle.depthwise(X, D)
    Z, _ = oracle.dwsep(X, D, np.eye(5, dtype=np.float32))
    assert np.array_equal(Z, Y)


@pytest.mark.parametrize("stride,pad,cm", [(1, 1, 1), (2, 1, 1), (1, 0, 2), (2, 0, 2)])
def test_matches_torch_conv2d_float64(stride, pad, cm):
    b, H, W, C, Co = 2, 9, 8, 4, 6
    X = _x((b, H, W, C), 7)
    D = _u((3, 3, C, cm), 8, 1.0 / 3)
    P = _u((C * cm, Co), 9, 1.0 / 11)
    Y, SY = oracle.depthwise(X, D, stride=stride, pad=pad)
    xt = torch.from_numpy(X).double().permute(0, 3, 1, 2)
    # grouped conv weight [C*cm][1][kh][kw]; output channel c*cm + r uses D[:, :, c, r]
    wt = torch.from_numpy(D).double().permute(2, 3, 0, 1).reshape(C * cm, 1, 3, 3)
    yt = F.conv2d(xt, wt, stride=stride, padding=pad, groups=C).permute(0, 2, 3, 1).numpy()
    assert np.max(np.abs(Y - yt) / np.maximum(SY, 1e-300)) < 1e-13
    Z, S = oracle.dwsep(X, D, P, stride=stride, pad=pad)
    pt = torch.from_numpy(P).double().t().reshape(Co, C * cm, 1, 1)
    zt = F.conv2d(torch.from_numpy(yt).permute(0, 3, 1, 2), pt).permute(0, 2, 3, 1).numpy()
    assert np.max(np.abs(Z - zt) / S) < 1e-13


def test_normaliser_positive_inputs():
    X = synth.uniform(5, 10, (1, 5, 5, 3), 0.0, 1.0)
    D = synth.uniform(5, 11, (3, 3, 3, 1), 0.0, 1.0)
    P = synth.uniform(5, 12, (3, 4), 0.0, 1.0)
    Z, S = oracle.dwsep(X, D, P)
    assert np.max(np.abs(Z - S) / S) < 1e-15


def test_bf16_inputs_widen_exactly():
    X = _x((1, 4, 4, 3), 13)
    D = _u((3, 3, 3, 1), 14, 1.0 / 3)
    P = _u((3, 2), 15, 1.0 / 11)
    Xb, Db, Pb = (synth.to_bf16_bits(a) for a in (X, D, P))
    Z1, _ = oracle.dwsep(Xb, Db, Pb)
    Z2, _ = oracle.dwsep(*(synth.bf16_bits_to_f32(a) for a in (Xb, Db, Pb)))
    assert np.array_equal(Z1, Z2)
