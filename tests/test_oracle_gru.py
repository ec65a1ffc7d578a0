"""Pins for the oracle's GRU forward (GRU cells mapped to matmul + element-wise work,
Section 6.1; recurrence scheduled as priming / recursive / finish iterations, Section 3.6)."""
import math
import os

import numpy as np
import pytest
import torch

import oracle
import synth


def _w(shape, stream, a=1.0 / 8):
    return synth.uniform(21, stream, shape, -a, a)


def _setup(T=5, B=3, I=6, H=4):
    x = synth.normal(21, 0, (T, B, I))
    W = _w((3 * H, I), 1)
    U = _w((3 * H, H), 2)
    b = synth.normal(21, 3, (3 * H,), scale=0.3)
    bhn = synth.normal(21, 4, (H,), scale=0.3)
    h0 = synth.normal(21, 5, (B, H), scale=0.5).astype(np.float64)
    return x, W, U, b, bhn, h0


def test_update_gate_one_keeps_state():
    # W_z = U_z = 0, b_z = 40: sigmoid(40) rounds to exactly 1.0 in fp64, so h_t = h_{t-1} = h0.
    x, W, U, b, bhn, h0 = _setup()
    H = U.shape[1]
    W[H:2 * H] = 0
    U[H:2 * H] = 0
    b[H:2 * H] = 40.0
    hs = oracle.gru(x, W, U, b, bhn, h0)
    for t in range(hs.shape[0]):
        assert np.array_equal(hs[t], h0)


def test_zero_weights_closed_form():
    # W = U = 0: r = s(b_r), z = s(b_z), n = tanh(b_n + r b_hn) are constants and
    # h_t = n + z^t (h0 - n).
    x, W, U, b, bhn, h0 = _setup(T=7)
    H = U.shape[1]
    W[:] = 0
    U[:] = 0
    hs = oracle.gru(x, W, U, b, bhn, h0)
    sig = lambda v: 1.0 / (1.0 + math.exp(-v))
    for j in range(H):
        r = sig(float(b[j]))
        z = sig(float(b[H + j]))
        n = math.tanh(float(b[2 * H + j]) + r * float(bhn[j]))
        for t in range(hs.shape[0]):
            want = n + z ** (t + 1) * (h0[:, j] - n)
            assert np.max(np.abs(hs[t, :, j] - want)) < 1e-14


def test_single_step_from_zero_state():
    # T = 1, h0 = 0: U contributes nothing; h_1 = (1 - s(W_z x + b_z)) * tanh(W_n x + b_n + r b_hn)
    x, W, U, b, bhn, _ = _setup(T=1)
    H = U.shape[1]
    hs = oracle.gru(x, W, U, b, bhn, None)
    X = x[0].astype(np.float64)
    gx = X @ W.astype(np.float64).T + b.astype(np.float64)
    r = 1 / (1 + np.exp(-gx[:, :H]))
    z = 1 / (1 + np.exp(-gx[:, H:2 * H]))
    n = np.tanh(gx[:, 2 * H:] + r * bhn.astype(np.float64))
    assert np.max(np.abs(hs[0] - (1 - z) * n)) < 1e-14


@pytest.mark.parametrize("split", [1, 2, 4])
def test_time_split_invariance_bit_exact(split):
    # Priming + recursive + finish over T steps equals two runs chained through h_T.
    x, W, U, b, bhn, h0 = _setup(T=6)
    full = oracle.gru(x, W, U, b, bhn, h0)
    first = oracle.gru(x[:split], W, U, b, bhn, h0)
    second = oracle.gru(x[split:], W, U, b, bhn, first[-1])
    assert np.array_equal(np.concatenate([first, second]), full)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_matches_torch_gru_float64(dt):
    T, B, I, H = 6, 3, 10, 8
    x, W, U, b, bhn, h0 = _setup(T, B, I, H)
    if dt == "bf16":
        x, W, U = (synth.to_bf16_bits(a) for a in (x, W, U))
        xv, Wv, Uv = (synth.bf16_bits_to_f32(a) for a in (x, W, U))
    else:
        xv, Wv, Uv = x, W, U
    hs = oracle.gru(x, W, U, b, bhn, h0)
    g = torch.nn.GRU(I, H, batch_first=False).double()
    with torch.no_grad():
        g.weight_ih_l0.copy_(torch.from_numpy(Wv).double())
        g.weight_hh_l0.copy_(torch.from_numpy(Uv).double())
        g.bias_ih_l0.copy_(torch.from_numpy(b).double())
        bh = torch.zeros(3 * H, dtype=torch.float64)
        bh[2 * H:] = torch.from_numpy(bhn).double()
        g.bias_hh_l0.copy_(bh)
        out, hT = g(torch.from_numpy(xv).double(), torch.from_numpy(h0)[None])
    assert np.max(np.abs(hs - out.numpy())) < 1e-13
    assert np.max(np.abs(hs[-1] - hT[0].numpy())) < 1e-13


def test_gate_order_and_n_gate_reset_inside():
    # b_hn sits inside r * (U_n h + b_hn): with b_r = -200 the reset gate is ~1e-87, so even a
    # b_hn scaled by 1e6 leaves h unchanged, while the unmodified cell differs.  A b_hn added
    # outside the reset product would move h by O(1).
    x, W, U, b, bhn, h0 = _setup(T=1)
    H = U.shape[1]
    h_a = oracle.gru(x, W, U, b, bhn, h0)
    b2 = b.copy()
    b2[:H] = -200.0           # r -> exp(-200)-small; n loses the U_n h + b_hn term
    h_b = oracle.gru(x, W, U, b2, bhn * 1e6, h0)
    h_c = oracle.gru(x, W, U, b2, None, h0)
    assert np.max(np.abs(h_b - h_c)) < 1e-70 * 1e6 + 1e-12
    assert np.max(np.abs(h_a - h_c)) > 1e-3


def test_golden_zero_weight_values():
    # tests/golden/gru_zero_weights.txt: H = 2, W = U = 0, h0 = (0.5, -0.25); values derived by hand.
    path = os.path.join(os.path.dirname(__file__), "golden", "gru_zero_weights.txt")
    want = np.array([[float(v) for v in l.split()] for l in open(path)
                     if l.strip() and not l.startswith("#")])
    H = 2
    x = np.zeros((3, 1, 1), np.float32)
    W = np.zeros((3 * H, 1), np.float32)
    U = np.zeros((3 * H, H), np.float32)
    b = np.array([0.0, 0.0, 0.0, 0.0, 0.0, 0.0], np.float32)
    h0 = np.array([[0.5, -0.25]])
    hs = oracle.gru(x, W, U, b, None, h0)
    assert np.max(np.abs(hs[:, 0, :] - want)) < 1e-15
