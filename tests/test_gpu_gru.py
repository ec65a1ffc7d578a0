"""GPU parity of isam_gru_forward against the CPU oracle (GRU cells as matmul + element-wise
work, Section 6.1; recurrence as priming / recursive / finish iterations, Section 3.6).
The GRU output is a convex blend of tanh values and h0, so |h| <= max(1, |h0|); the check is
the maximum absolute difference, with the same 1e-2 (bf16 weights) / 1e-5 (fp32) split."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import workloads
from tests._util import TOL_BF16, TOL_F32, bits, to_gpu

pytestmark = pytest.mark.gpu

import paper_1810_09958_amd as isam


@pytest.fixture(params=["steps", "persistent", "default"])
def mode(request, monkeypatch):
    """The schedules of the recurrence: one kernel per step, one persistent kernel with a
    grid barrier between steps, and the library's own choice
    (the batch-group persistent kernel for bf16 weights and hidden 256..1024)."""
    if request.param == "default":
        monkeypatch.delenv("ISAM_GRU_MODE", raising=False)
    else:
        monkeypatch.setenv("ISAM_GRU_MODE", request.param)
    return request.param


def _inputs(T, B, I, H, seed=0, scale=1 / 32, with_h0=False, with_bhn=False):
    x = synth.normal(seed, 3, (T, B, I))
    W = synth.uniform(seed, 0, (3 * H, I), -scale, scale)
    U = synth.uniform(seed, 1, (3 * H, H), -scale, scale)
    b = synth.normal(seed, 2, (3 * H,), scale=0.1)
    h0 = synth.normal(seed, 4, (B, H), scale=0.5) if with_h0 else None
    bhn = synth.normal(seed, 5, (H,), scale=0.1) if with_bhn else None
    return x, W, U, b, h0, bhn


def _run(T, B, I, H, dt="bf16", seed=0, with_h0=False, with_bhn=False, scale=1 / 32):
    x, W, U, b, h0, bhn = _inputs(T, B, I, H, seed, scale, with_h0, with_bhn)
    if dt == "bf16":
        x, W, U = bits(x), bits(W), bits(U)
    hs, hT = isam.gru_forward(to_gpu(x), to_gpu(W), to_gpu(U), bias=to_gpu(b),
                              bias_hn=None if bhn is None else to_gpu(bhn),
                              h0=None if h0 is None else to_gpu(h0))
    torch.cuda.synchronize()
    ref = oracle.gru(x, W, U, b, bhn, h0)
    hs = hs.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(hs))
    err = float(np.max(np.abs(hs - ref)))
    tol = TOL_BF16 if dt == "bf16" else TOL_F32
    assert err <= tol, f"T={T} B={B} I={I} H={H} {dt} h0={with_h0} bhn={with_bhn}: {err:.3e}"
    assert np.array_equal(hT.cpu().numpy(), hs[-1].astype(np.float32))
    return err


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("T", [1, 2, 3, 9])
def test_small_steps(dt, T, mode):
    _run(T, 4, 40, 64, dt, seed=T, with_h0=True, with_bhn=True, scale=1 / 4)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("B,H", [(1, 128), (16, 256), (17, 64), (33, 96), (5, 1024)])
def test_shapes(dt, B, H, mode):
    _run(5, B, 72, H, dt, seed=B + H, with_h0=(B % 2 == 1), scale=1 / 8)


def test_h0_null_equals_zeros():
    T, B, I, H = 4, 8, 64, 128
    x, W, U, b, _, _ = _inputs(T, B, I, H)
    args = [to_gpu(bits(a)) for a in (x, W, U)]
    hs1, _ = isam.gru_forward(*args, bias=to_gpu(b))
    hs2, _ = isam.gru_forward(*args, bias=to_gpu(b), h0=torch.zeros(B, H, device="cuda"))
    torch.cuda.synchronize()
    assert torch.equal(hs1, hs2)


def test_time_split_chains_through_h_T():
    # Priming + recursive + finish over T steps == two calls chained through h_T.
    T, B, I, H = 6, 4, 64, 128
    x, W, U, b, _, _ = _inputs(T, B, I, H, seed=9)
    xg, Wg, Ug = (to_gpu(a) for a in (x, W, U))
    hs_full, _ = isam.gru_forward(xg, Wg, Ug, bias=to_gpu(b))
    hs1, hT1 = isam.gru_forward(xg[:2].contiguous(), Wg, Ug, bias=to_gpu(b))
    hs2, _ = isam.gru_forward(xg[2:].contiguous(), Wg, Ug, bias=to_gpu(b), h0=hT1)
    torch.cuda.synchronize()
    assert torch.max(torch.abs(torch.cat([hs1, hs2]) - hs_full)).item() <= 1e-6


def test_t_zero_copies_h0():
    B, H = 3, 64
    h0 = torch.randn(B, H, device="cuda")
    x = torch.empty((0, B, 16), device="cuda")
    W = torch.zeros(3 * H, 16, device="cuda")
    U = torch.zeros(3 * H, H, device="cuda")
    _, hT = isam.gru_forward(x, W, U, h0=h0, return_sequence=False)
    torch.cuda.synchronize()
    assert torch.equal(hT, h0)


def test_deterministic_run_twice():
    T, B, I, H = 8, 32, 256, 256
    x, W, U, b, _, _ = _inputs(T, B, I, H)
    args = [to_gpu(bits(a)) for a in (x, W, U)]
    a1, _ = isam.gru_forward(*args, bias=to_gpu(b))
    a2, _ = isam.gru_forward(*args, bias=to_gpu(b))
    torch.cuda.synchronize()
    assert torch.equal(a1, a2)


_FULL_REF = {}


def _full_ref(variant):
    """Oracle h_seq of the whole GRU workload (all 32 sequences), computed once per module."""
    if variant not in _FULL_REF:
        d = workloads.gru()
        x, W, U = (d["x_bf16"], d["W_bf16"], d["U_bf16"]) if variant == "bf16" else (d["x"], d["W"], d["U"])
        _FULL_REF[variant] = (d, x, W, U, oracle.gru(x, W, U, d["bias"], None, None))
    return _FULL_REF[variant]


@pytest.mark.parametrize("variant", ["bf16", "f32"])
def test_config_full_size_all_sequences(variant, mode):
    # Every step of every one of the 32 sequences against the oracle.
    d, x, W, U, ref = _full_ref(variant)
    hs, hT = isam.gru_forward(to_gpu(x), to_gpu(W), to_gpu(U), bias=to_gpu(d["bias"]))
    torch.cuda.synchronize()
    got = hs.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    err = float(np.max(np.abs(got - ref)))
    assert err <= (TOL_BF16 if variant == "bf16" else TOL_F32), err
    assert np.array_equal(hT.cpu().numpy(), hs[-1].cpu().numpy())


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_paper_step_count_128(dt, mode):
    # 128 recurrent steps (the paper's sequence length): one persistent launch, or
    # 128 step kernels
    _run(128, 8, 128, 256, dt, seed=128, with_h0=True, scale=1 / 8)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_schedules_bit_identical(dt, monkeypatch):
    # Both schedules sum each gate pre-activation in the same order (the K split
    # over waves depends on H only), so their outputs agree bit for bit.
    T, B, I, H = 7, 19, 96, 512
    x, W, U, b, h0, bhn = _inputs(T, B, I, H, seed=77, scale=1 / 8, with_h0=True, with_bhn=True)
    if dt == "bf16":
        x, W, U = bits(x), bits(W), bits(U)
    args = [to_gpu(a) for a in (x, W, U)]
    kw = dict(bias=to_gpu(b), bias_hn=to_gpu(bhn), h0=to_gpu(h0))
    out = {}
    for m in ("steps", "persistent"):
        monkeypatch.setenv("ISAM_GRU_MODE", m)
        out[m] = isam.gru_forward(*args, **kw)
    torch.cuda.synchronize()
    assert torch.equal(out["steps"][0], out["persistent"][0])
    assert torch.equal(out["steps"][1], out["persistent"][1])


def test_repeated_calls_see_new_inputs(mode):
    # Repeated calls on the same buffers: new input values written in place between calls
    # must be used (nothing about a call is kept from one call to the next).
    T, B, I, H = 5, 4, 64, 256
    x1, W, U, b, _, _ = _inputs(T, B, I, H, seed=31, scale=1 / 8)
    x2 = synth.normal(32, 3, (T, B, I))
    xg, Wg, Ug, bg = to_gpu(bits(x1)), to_gpu(bits(W)), to_gpu(bits(U)), to_gpu(b)
    hs = torch.empty((T, B, H), device="cuda")
    hT = torch.empty((B, H), device="cuda")
    ws = torch.empty(isam.gru_forward_workspace_size(T, B, I, H, isam.ISAM_BF16), device="cuda", dtype=torch.uint8)
    for xs in (x1, x2, x1):
        xg.copy_(to_gpu(bits(xs)))
        isam.gru_forward(xg, Wg, Ug, bias=bg, h_seq=hs, h_T=hT, workspace=ws)
        torch.cuda.synchronize()
        ref = oracle.gru(bits(xs), bits(W), bits(U), b, None, None)
        err = float(np.max(np.abs(hs.cpu().numpy().astype(np.float64) - ref)))
        assert err <= TOL_BF16, err


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_hidden_too_large_for_lds_runs_stepwise(dt, monkeypatch):
    # The persistent kernel keeps at least 16 rows of U (three gate rows padded to an
    # MFMA tile) in one CU's LDS: 192 KB at H = 6144 (bf16) / 3072 (fp32), over the
    # 160 KB there is.  The stepwise schedule reads U from global memory and has no
    # such limit, so it is taken even when the persistent one is asked for.
    monkeypatch.setenv("ISAM_GRU_MODE", "persistent")
    H = 6144 if dt == "bf16" else 3072
    _run(3, 2, 64, H, dt, seed=5, with_h0=True, scale=1 / 64)


def test_many_workspaces(monkeypatch):
    # Calls on 38 workspace placements in a row on one stream (so they run one after the
    # other), all queued before one sync: every result matches the oracle.
    monkeypatch.setenv("ISAM_GRU_MODE", "steps")
    T, B, I, H = 3, 2, 32, 64
    x, W, U, b, _, _ = _inputs(T, B, I, H, seed=41, scale=1 / 4)
    args = [to_gpu(bits(a)) for a in (x, W, U)]
    ref = oracle.gru(bits(x), bits(W), bits(U), b, None, None)
    need = isam.gru_forward_workspace_size(T, B, I, H, isam.ISAM_BF16)
    pool = torch.empty(need + 40 * 256, device="cuda", dtype=torch.uint8)
    outs = []
    for i in list(range(36)) + [0, 1]:
        ws = pool[i * 256: i * 256 + need]
        hs, _ = isam.gru_forward(*args, bias=to_gpu(b), workspace=ws)
        outs.append(hs)
    torch.cuda.synchronize()
    for hs in outs:
        err = float(np.max(np.abs(hs.cpu().numpy().astype(np.float64) - ref)))
        assert err <= TOL_BF16, err


def test_long_sequence_stepwise(monkeypatch):
    # T = 4097 steps of the stepwise schedule.
    monkeypatch.setenv("ISAM_GRU_MODE", "steps")
    T, B, I, H = 4097, 1, 16, 64
    x, W, U, b, h0, _ = _inputs(T, B, I, H, seed=23, scale=1 / 4, with_h0=True)
    x, W, U = bits(x), bits(W), bits(U)
    hs, hT = isam.gru_forward(to_gpu(x), to_gpu(W), to_gpu(U), bias=to_gpu(b), h0=to_gpu(h0))
    torch.cuda.synchronize()
    ref = oracle.gru(x, W, U, b, None, h0)
    err = float(np.max(np.abs(hs.cpu().numpy().astype(np.float64) - ref)))
    assert err <= TOL_BF16, err
    assert np.array_equal(hT.cpu().numpy(), hs[-1].cpu().numpy())


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_persistent_exchange_on_poisoned_workspace(dt, monkeypatch):
    # Batch 33 x hidden 96: the per-step state (6336 bytes in bf16, 12672 in fp32) is not a
    # whole number of 128-byte lines, the case in which unpadded ring slots would share a
    # line.  The workspace is filled with NaN patterns before each call, and the second call
    # on the same workspace uses other inputs, so a stale or missing exchange shows up as
    # NaN or as the first call's values.
    monkeypatch.setenv("ISAM_GRU_MODE", "persistent")
    T, B, I, H = 9, 33, 72, 96
    need = isam.gru_forward_workspace_size(T, B, I, H, isam.ISAM_BF16 if dt == "bf16" else isam.ISAM_F32)
    ws = torch.empty(need, device="cuda", dtype=torch.uint8)
    for seed in (3, 4):
        x, W, U, b, h0, bhn = _inputs(T, B, I, H, seed=seed, scale=1 / 8, with_h0=True, with_bhn=True)
        if dt == "bf16":
            x, W, U = bits(x), bits(W), bits(U)
        ws.fill_(0xFF)
        hs, hT = isam.gru_forward(to_gpu(x), to_gpu(W), to_gpu(U), bias=to_gpu(b), bias_hn=to_gpu(bhn),
                                  h0=to_gpu(h0), workspace=ws)
        torch.cuda.synchronize()
        got = hs.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(got)), f"seed {seed}: non-finite h"
        ref = oracle.gru(x, W, U, b, bhn, h0)
        err = float(np.max(np.abs(got - ref)))
        assert err <= (TOL_BF16 if dt == "bf16" else TOL_F32), f"seed {seed}: {err:.3e}"
        assert np.array_equal(hT.cpu().numpy(), hs[-1].cpu().numpy())


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_barrier_timeout_returns_nan(dt, monkeypatch):
    # The host sets a barrier target the grid never reaches and a 100 us bound on each wait:
    # every wait ends at the bound (no kernel hangs), the sticky error word is set, and the
    # finish check fills both outputs with NaN.  The next call on the same workspace starts
    # from a cleared error word and is correct again.
    monkeypatch.setenv("ISAM_GRU_MODE", "persistent")
    T, B, I, H = 4, 4, 32, 64
    x, W, U, b, _, _ = _inputs(T, B, I, H, seed=8, scale=1 / 4)
    if dt == "bf16":
        x, W, U = bits(x), bits(W), bits(U)
    args = [to_gpu(a) for a in (x, W, U)]
    need = isam.gru_forward_workspace_size(T, B, I, H, isam.ISAM_BF16 if dt == "bf16" else isam.ISAM_F32)
    ws = torch.empty(need, device="cuda", dtype=torch.uint8)
    monkeypatch.setenv("ISAM_GRU_TEST_STALL", "1")
    hs, hT = isam.gru_forward(*args, bias=to_gpu(b), workspace=ws)
    torch.cuda.synchronize()
    assert torch.all(torch.isnan(hs)).item() and torch.all(torch.isnan(hT)).item()
    monkeypatch.delenv("ISAM_GRU_TEST_STALL")
    hs, hT = isam.gru_forward(*args, bias=to_gpu(b), workspace=ws)
    torch.cuda.synchronize()
    err = float(np.max(np.abs(hs.cpu().numpy().astype(np.float64) - oracle.gru(x, W, U, b, None, None))))
    assert err <= (TOL_BF16 if dt == "bf16" else TOL_F32), err


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_output_guard_bands(dt, mode):
    # h_seq and h_T placed inside larger buffers filled with a sentinel: nothing outside
    # [T][batch][H] and [batch][H] is written.
    T, B, I, H = 6, 5, 48, 128
    x, W, U, b, h0, _ = _inputs(T, B, I, H, seed=12, scale=1 / 4, with_h0=True)
    if dt == "bf16":
        x, W, U = bits(x), bits(W), bits(U)
    g = 1024
    buf_s = torch.full((T * B * H + 2 * g,), -777.0, device="cuda")
    buf_t = torch.full((B * H + 2 * g,), -777.0, device="cuda")
    hs = buf_s[g: g + T * B * H].view(T, B, H)
    hT = buf_t[g: g + B * H].view(B, H)
    isam.gru_forward(to_gpu(x), to_gpu(W), to_gpu(U), bias=to_gpu(b), h0=to_gpu(h0), h_seq=hs, h_T=hT)
    torch.cuda.synchronize()
    for buf, n in ((buf_s, T * B * H), (buf_t, B * H)):
        h = buf.cpu().numpy()
        assert np.all(h[:g] == -777.0) and np.all(h[g + n:] == -777.0)
    err = float(np.max(np.abs(hs.cpu().numpy().astype(np.float64) - oracle.gru(x, W, U, b, None, h0))))
    assert err <= (TOL_BF16 if dt == "bf16" else TOL_F32), err


# Batch-group schedule (bf16 weights, hidden 256/512/768/1024): independent barrier domains of
# H/32 workgroups, each owning a slice of at most 16 batch columns, U rows in registers.
@pytest.fixture(params=["xcd", "device"])
def group_scope(request, monkeypatch):
    """The two exchanges of the batch-group kernel: through the L2 of the XCD a domain
    sits on (taken when all its workgroups share one), or device scope throughout."""
    if request.param == "device":
        monkeypatch.setenv("ISAM_GRU_GROUP_SCOPE", "device")
    else:
        monkeypatch.delenv("ISAM_GRU_GROUP_SCOPE", raising=False)
    return request.param


@pytest.mark.parametrize("H", [256, 512, 768, 1024])
@pytest.mark.parametrize("B", [1, 3, 4, 17, 32, 33, 128])
def test_group_schedule_shapes(H, B, group_scope, monkeypatch):
    monkeypatch.setenv("ISAM_GRU_MODE", "group")
    _run(5 if B < 100 else 3, B, 72, H, "bf16", seed=B + H, with_h0=True, with_bhn=(B % 2 == 1), scale=1 / 8)


@pytest.mark.parametrize("T", [1, 2, 9])
def test_group_schedule_steps(T, group_scope, monkeypatch):
    monkeypatch.setenv("ISAM_GRU_MODE", "group")
    _run(T, 8, 40, 256, "bf16", seed=50 + T, with_h0=True, with_bhn=True, scale=1 / 4)


def test_group_schedule_poisoned_workspace_and_repeat(group_scope, monkeypatch):
    # NaN-filled workspace before each call, two calls with different inputs on one workspace.
    monkeypatch.setenv("ISAM_GRU_MODE", "group")
    T, B, I, H = 7, 33, 64, 768
    need = isam.gru_forward_workspace_size(T, B, I, H, isam.ISAM_BF16)
    ws = torch.empty(need, device="cuda", dtype=torch.uint8)
    for seed in (61, 62):
        x, W, U, b, h0, bhn = _inputs(T, B, I, H, seed=seed, scale=1 / 8, with_h0=True, with_bhn=True)
        x, W, U = bits(x), bits(W), bits(U)
        ws.fill_(0xFF)
        hs, hT = isam.gru_forward(to_gpu(x), to_gpu(W), to_gpu(U), bias=to_gpu(b), bias_hn=to_gpu(bhn),
                                  h0=to_gpu(h0), workspace=ws)
        torch.cuda.synchronize()
        got = hs.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(got))
        err = float(np.max(np.abs(got - oracle.gru(x, W, U, b, bhn, h0))))
        assert err <= TOL_BF16, f"seed {seed}: {err:.3e}"
        assert np.array_equal(hT.cpu().numpy(), hs[-1].cpu().numpy())


def test_group_schedule_barrier_timeout_returns_nan(group_scope, monkeypatch):
    monkeypatch.setenv("ISAM_GRU_MODE", "group")
    T, B, I, H = 4, 4, 32, 256
    x, W, U, b, _, _ = _inputs(T, B, I, H, seed=63, scale=1 / 4)
    x, W, U = bits(x), bits(W), bits(U)
    args = [to_gpu(a) for a in (x, W, U)]
    need = isam.gru_forward_workspace_size(T, B, I, H, isam.ISAM_BF16)
    ws = torch.empty(need, device="cuda", dtype=torch.uint8)
    monkeypatch.setenv("ISAM_GRU_TEST_STALL", "1")
    hs, hT = isam.gru_forward(*args, bias=to_gpu(b), workspace=ws)
    torch.cuda.synchronize()
    assert torch.all(torch.isnan(hs)).item() and torch.all(torch.isnan(hT)).item()
    monkeypatch.delenv("ISAM_GRU_TEST_STALL")
    hs, hT = isam.gru_forward(*args, bias=to_gpu(b), workspace=ws)
    torch.cuda.synchronize()
    err = float(np.max(np.abs(hs.cpu().numpy().astype(np.float64) - oracle.gru(x, W, U, b, None, None))))
    assert err <= TOL_BF16, err


def test_group_schedule_deterministic_and_guarded(group_scope, monkeypatch):
    monkeypatch.setenv("ISAM_GRU_MODE", "group")
    T, B, I, H = 6, 20, 48, 512
    x, W, U, b, h0, _ = _inputs(T, B, I, H, seed=64, scale=1 / 8, with_h0=True)
    x, W, U = bits(x), bits(W), bits(U)
    args = [to_gpu(a) for a in (x, W, U)]
    g = 1024
    outs = []
    for _ in range(2):
        buf_s = torch.full((T * B * H + 2 * g,), -777.0, device="cuda")
        buf_t = torch.full((B * H + 2 * g,), -777.0, device="cuda")
        hs = buf_s[g: g + T * B * H].view(T, B, H)
        hT = buf_t[g: g + B * H].view(B, H)
        isam.gru_forward(*args, bias=to_gpu(b), h0=to_gpu(h0), h_seq=hs, h_T=hT)
        torch.cuda.synchronize()
        for buf, n in ((buf_s, T * B * H), (buf_t, B * H)):
            h = buf.cpu().numpy()
            assert np.all(h[:g] == -777.0) and np.all(h[g + n:] == -777.0)
        outs.append(hs.clone())
    assert torch.equal(outs[0], outs[1])
    err = float(np.max(np.abs(outs[0].cpu().numpy().astype(np.float64) - oracle.gru(x, W, U, b, None, h0))))
    assert err <= TOL_BF16, err


def test_group_mode_rejects_unsupported(monkeypatch):
    monkeypatch.setenv("ISAM_GRU_MODE", "group")
    x, W, U, b, _, _ = _inputs(3, 2, 16, 96, seed=65)
    with pytest.raises(isam.IsamError):
        isam.gru_forward(to_gpu(bits(x)), to_gpu(bits(W)), to_gpu(bits(U)), bias=to_gpu(b))
