"""GPU parity of isam_dwsep_conv against the CPU oracle (the paper's third listing,
factored into depthwise then pointwise as in Section 2.3)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import workloads
from tests._util import TOL_BF16, TOL_F32, bits, norm_err, to_gpu, to_host_f64

pytestmark = pytest.mark.gpu

import paper_1810_09958_amd as isam


def _case(b, H, W, C, Co, cm=1, k=3, stride=1, pad=1, dt="f32", ot="f32", seed=0):
    X = synth.normal(seed, 0, (b, H, W, C))
    D = synth.uniform(seed, 1, (k, k, C, cm), -1 / 3, 1 / 3)
    P = synth.uniform(seed, 2, (C * cm, Co), -1 / 11, 1 / 11)
    if dt == "bf16":
        X, D, P = bits(X), bits(D), bits(P)
    y = isam.dwsep_conv(to_gpu(X), to_gpu(D), to_gpu(P), stride=stride, pad=pad,
                        out_dtype=torch.bfloat16 if ot == "bf16" else torch.float32)
    torch.cuda.synchronize()
    Z, S = oracle.dwsep(X, D, P, stride=stride, pad=pad)
    err = norm_err(to_host_f64(y), Z, S)
    tol = TOL_F32 if (dt == "f32" and ot == "f32") else TOL_BF16
    assert err <= tol, f"b={b} H={H} W={W} C={C} Co={Co} cm={cm} k={k} s={stride} p={pad} {dt}->{ot}: {err:.3e}"


@pytest.mark.parametrize("dt,ot", [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16")])
def test_small_fast_path(dt, ot):
    _case(2, 9, 11, 16, 24, dt=dt, ot=ot)
    _case(3, 17, 5, 64, 40, dt=dt, ot=ot, seed=1)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("cm,k,stride,pad", [(1, 3, 2, 1), (2, 3, 1, 1), (2, 3, 2, 0), (1, 1, 1, 0),
                                             (1, 5, 1, 2), (3, 3, 1, 0)])
def test_generic_path(dt, cm, k, stride, pad):
    _case(2, 10, 9, 8, 12, cm=cm, k=k, stride=stride, pad=pad, dt=dt)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_channels_not_vector_multiple(dt):
    _case(2, 7, 7, 5, 9, dt=dt)
    _case(1, 6, 8, 12, 3, dt=dt)


def test_one_pixel_image():
    _case(1, 1, 1, 8, 8, pad=1)


# Unfused path (fusion switched off): the standalone 3x3 stride-1 depthwise kernel, then the
# pointwise GEMM.  The LDS-staged kernel owns RS rows x SW columns per workgroup (RS: the
# default per dtype, 8 and 3 rows): ragged last
# row segment and column strip, one channel vector per pixel up to a whole workgroup of them,
# a one-pixel image; more channel vectors than one workgroup holds take the register-window
# kernel, as does every shape with the LDS-staged kernel switched off (ISAM_DW_RS=0).
@pytest.mark.parametrize("dt,ot", [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16")])
@pytest.mark.parametrize("shape", [(2, 9, 11, 16, 24), (3, 17, 5, 64, 40), (1, 19, 57, 128, 16),
                                   (2, 6, 7, 8, 8), (1, 1, 1, 8, 8), (1, 10, 3, 1024, 8),
                                   (1, 5, 4, 4096, 8), (2, 3, 1000, 8, 4), (1, 23, 300, 32, 8)])
@pytest.mark.parametrize("rs", ["default", "8", "3", "0"])
def test_unfused_depthwise_kernel(dt, ot, shape, rs, monkeypatch):
    monkeypatch.setenv("ISAM_DWSEP_FUSED", "0")
    if rs == "default":
        monkeypatch.delenv("ISAM_DW_RS", raising=False)
    else:
        monkeypatch.setenv("ISAM_DW_RS", rs)
    b, H, W, C, Co = shape
    _case(b, H, W, C, Co, dt=dt, ot=ot, seed=H + W + C)


_FULL = {}


def _full_ref(dt):
    """Oracle output of the whole 32-image separable-convolution workload, once per dtype."""
    if dt not in _FULL:
        d = workloads.dwsep()
        X, D, P = (d["X"], d["D"], d["P"]) if dt == "f32" else (d["X_bf16"], d["D_bf16"], d["P_bf16"])
        Z, S = oracle.dwsep(X, D, P)
        _FULL[dt] = (X, D, P, Z, S)
    return _FULL[dt]


def _check_full(variant):
    X, D, P, Z, S = _full_ref("f32" if variant == "f32" else "bf16")
    ot = torch.bfloat16 if variant == "bf16_out_bf16" else torch.float32
    y = isam.dwsep_conv(to_gpu(X), to_gpu(D), to_gpu(P), out_dtype=ot)
    torch.cuda.synchronize()
    tol = TOL_F32 if variant == "f32" else TOL_BF16
    err = norm_err(to_host_f64(y), Z, S)
    assert err <= tol, f"{variant}: {err:.3e}"


@pytest.mark.parametrize("variant", ["f32", "bf16", "bf16_out_bf16"])
def test_config_full_size_all_images(variant):
    # all 32 images, every output element, through the default (fused) path
    _check_full(variant)


@pytest.mark.parametrize("variant", ["f32", "bf16_out_bf16"])
def test_config_full_size_unfused(variant, monkeypatch):
    # the full image batch through the standalone depthwise kernel and the pointwise GEMM
    monkeypatch.setenv("ISAM_DWSEP_FUSED", "0")
    monkeypatch.delenv("ISAM_DW_RS", raising=False)
    _check_full(variant)


@pytest.mark.parametrize("dt,ot", [("bf16", "f32"), ("bf16", "bf16"), ("f32", "f32")])
def test_fused_path_needs_no_workspace(dt, ot):
    # The fused kernels keep the depthwise result on chip: the size query returns 0 and the
    # call runs with no workspace at all.
    b, H, W, C, Co = 2, 6, 56, 128, 256
    it = isam.ISAM_BF16 if dt == "bf16" else isam.ISAM_F32
    otc = isam.ISAM_BF16 if ot == "bf16" else isam.ISAM_F32
    assert isam.dwsep_conv_workspace_size(b, H, W, C, 1, 3, 3, 1, 1, Co, it, otc) == 0
    X = synth.normal(5, 0, (b, H, W, C))
    D = synth.uniform(5, 1, (3, 3, C, 1), -1 / 3, 1 / 3)
    P = synth.uniform(5, 2, (C, Co), -1 / 11, 1 / 11)
    if dt == "bf16":
        X, D, P = bits(X), bits(D), bits(P)
    odt = torch.bfloat16 if ot == "bf16" else torch.float32
    y = torch.empty((b, H, W, Co), device="cuda", dtype=odt)
    Xg, Dg, Pg = to_gpu(X), to_gpu(D), to_gpu(P)   # held until the kernel has run
    rc = isam.lib().isam_dwsep_conv(b, H, W, C, 1, 3, 3, 1, 1, Co, it, Xg.data_ptr(), Dg.data_ptr(),
                                    Pg.data_ptr(), otc, y.data_ptr(), None, 0, isam._stream())
    assert rc == 0, isam.lib().isam_last_error()
    torch.cuda.synchronize()
    Z, S = oracle.dwsep(X, D, P)
    assert norm_err(to_host_f64(y), Z, S) <= (TOL_F32 if ot == "f32" and dt == "f32" else TOL_BF16)


@pytest.mark.parametrize("dt,ot,fused", [("bf16", "f32", "1"), ("bf16", "bf16", "1"), ("f32", "f32", "1"),
                                         ("bf16", "bf16", "0"), ("f32", "f32", "0")])
def test_output_guard_bands(dt, ot, fused, monkeypatch):
    # y placed inside a larger sentinel-filled buffer: the fused bf16 and fp32 kernels and the
    # unfused pair write nothing outside [b][H][W][C_out].
    monkeypatch.setenv("ISAM_DWSEP_FUSED", fused)
    b, H, W, C, Co = 3, 7, 56, 128, 96
    X = synth.normal(6, 0, (b, H, W, C))
    D = synth.uniform(6, 1, (3, 3, C, 1), -1 / 3, 1 / 3)
    P = synth.uniform(6, 2, (C, Co), -1 / 11, 1 / 11)
    if dt == "bf16":
        X, D, P = bits(X), bits(D), bits(P)
    odt = torch.bfloat16 if ot == "bf16" else torch.float32
    g = 4096
    n = b * H * W * Co
    buf = torch.full((n + 2 * g,), -768.0, device="cuda", dtype=odt)
    y = buf[g: g + n].view(b, H, W, Co)
    isam.dwsep_conv(to_gpu(X), to_gpu(D), to_gpu(P), out=y)
    torch.cuda.synchronize()
    h = buf.float().cpu().numpy()
    assert np.all(h[:g] == -768.0) and np.all(h[g + n:] == -768.0)
    Z, S = oracle.dwsep(X, D, P)
    assert norm_err(h[g: g + n].reshape(b, H, W, Co).astype(np.float64), Z, S) <= \
        (TOL_F32 if ot == "f32" and dt == "f32" else TOL_BF16)


@pytest.mark.parametrize("ot", ["f32", "bf16"])
@pytest.mark.parametrize("C,Co", [(64, 8), (64, 40), (128, 256), (128, 96)])
def test_fused_path_shapes(ot, C, Co):
    # bf16 3x3 stride-1 pad-1 shapes taken by the fused depthwise+pointwise kernel:
    # widths for 4, 2 and 1 rows per tile, heights not a multiple of the rows per tile
    for (b, H, W) in [(2, 5, 7), (1, 9, 32), (2, 7, 56), (1, 3, 64), (1, 5, 100)]:
        _case(b, H, W, C, Co, dt="bf16", ot=ot, seed=H * W + C)


@pytest.mark.parametrize("ot", ["f32", "bf16"])
def test_fused_tile_ranges_cross_images(ot):
    # More tiles than CUs: each workgroup walks a contiguous range of tiles that
    # crosses image boundaries (the input-row sequence restarts), and with 8-9
    # two-row tiles per workgroup the 16-row input ring wraps.
    _case(60, 5, 56, 128, 256, dt="bf16", ot=ot, seed=7)
    _case(150, 28, 16, 64, 40, dt="bf16", ot=ot, seed=8)


def test_fused_tiny_images_many_tiles():
    # One- and two-row images: every tile starts a new image (all R+2 input
    # rows new, two of them outside the image), several tiles per workgroup,
    # the input ring wraps; tiny widths leave most MFMA columns unused.
    _case(300, 1, 5, 64, 16, dt="bf16", ot="f32", seed=31)
    _case(1200, 2, 3, 128, 24, dt="bf16", ot="bf16", seed=32)
    _case(40, 3, 1, 128, 256, dt="bf16", ot="f32", seed=33)


@pytest.mark.parametrize("C,Co", [(32, 16), (64, 48), (96, 256), (128, 256), (128, 112)])
def test_fused_f32_path_shapes(C, Co):
    # fp32 3x3 stride-1 pad-1 shapes taken by the fused fp32 kernel (W % 8 == 0,
    # W <= 64): one to eight 16-pixel tiles per 2-row tile, odd heights (a
    # partial last tile), C_out below 256 (idle waves)
    for (b, H, W) in [(2, 5, 8), (1, 9, 16), (2, 7, 56), (1, 3, 64), (1, 4, 24)]:
        _case(b, H, W, C, Co, dt="f32", ot="f32", seed=H * W + C + Co)


def test_fused_f32_row_ranges_cross_images():
    # More rows than CUs: each workgroup takes a contiguous range of rows whose
    # tiles (up to two rows, never crossing an image) include one-row tiles and
    # image boundaries, and its step pipeline spans several tiles.
    _case(40, 9, 16, 64, 48, dt="f32", ot="f32", seed=21)
    _case(20, 30, 8, 32, 16, dt="f32", ot="f32", seed=22)
    _case(6, 56, 56, 128, 256, dt="f32", ot="f32", seed=23)


# Input and output just under the 2^31-byte limit of the 32-bit buffer offsets, on the fused
# kernels (bf16: 2674 images of 56 x 56 x 128; fp32: 1337).  X is a 16-image random block
# repeated along the batch; the oracle checks sampled images, the last ones among them.
@pytest.mark.parametrize("dt,batch", [("bf16", 2674), ("f32", 1337)])
def test_fused_at_the_extent_limit(dt, batch):
    H = W = 56
    C = Co = 128
    es = 2 if dt == "bf16" else 4
    assert batch * H * W * C * es < 2 ** 31 and batch * H * W * C * es > 2 ** 31 - 2 ** 22
    blk = synth.normal(batch, 0, (16, H, W, C))
    D = synth.uniform(batch, 1, (3, 3, C, 1), -1 / 3, 1 / 3)
    P = synth.uniform(batch, 2, (C, Co), -1 / 11, 1 / 11)
    if dt == "bf16":
        blk, D, P = bits(blk), bits(D), bits(P)
    X = to_gpu(blk).repeat(batch // 16 + 1, 1, 1, 1)[:batch].contiguous()
    y = isam.dwsep_conv(X, to_gpu(D), to_gpu(P), out_dtype=torch.bfloat16 if dt == "bf16" else torch.float32)
    torch.cuda.synchronize()
    imgs = [0, 1, batch // 2, batch - 2, batch - 1]
    Z, S = oracle.dwsep(np.ascontiguousarray(blk[[i % 16 for i in imgs]]), D, P)
    got = to_host_f64(y[torch.as_tensor(imgs, device="cuda")])
    assert norm_err(got, Z, S) <= (TOL_BF16 if dt == "bf16" else TOL_F32)
    del X, y
    torch.cuda.empty_cache()
