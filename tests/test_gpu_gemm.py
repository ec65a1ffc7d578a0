"""GPU parity of isam_gemm against the CPU oracle (the paper's first listing)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import workloads
from tests._util import TOL_BF16, TOL_F32, bits, norm_err, to_gpu, to_host_f64

pytestmark = pytest.mark.gpu

import paper_1810_09958_amd as isam


def _run_case(M, N, K, dt, ct, ta=0, tb=0, accumulate=False, seed=0, pad_ld=0):
    Am = synth.uniform(seed, 10, (M, K), -1, 1)
    Bm = synth.uniform(seed, 11, (K, N), -1, 1)
    A_host = np.ascontiguousarray(Am.T) if ta else Am
    B_host = np.ascontiguousarray(Bm.T) if tb else Bm
    if pad_ld:
        A_host = np.pad(A_host, ((0, 0), (0, pad_ld)), constant_values=7.0)
        B_host = np.pad(B_host, ((0, 0), (0, pad_ld)), constant_values=-7.0)
    if dt == "bf16":
        A_host, B_host = bits(A_host), bits(B_host)
    A, B = to_gpu(A_host), to_gpu(B_host)
    if pad_ld:
        A = A[:, : A.shape[1] - pad_ld]
        B = B[:, : B.shape[1] - pad_ld]
    out_dtype = torch.bfloat16 if ct == "bf16" else torch.float32
    C_in = None
    if accumulate:
        c0 = synth.uniform(seed, 12, (M, N), -1, 1)
        C = to_gpu(bits(c0) if ct == "bf16" else c0)
        C_in = to_host_f64(C)
        isam.gemm(A, B, C, trans_a=bool(ta), trans_b=bool(tb), accumulate=True)
    else:
        C = isam.gemm(A, B, trans_a=bool(ta), trans_b=bool(tb), out_dtype=out_dtype)
    torch.cuda.synchronize()
    lda = A_host.shape[1]
    ldb = B_host.shape[1]
    ref, S = oracle.gemm(A_host, B_host, M, N, K, ta, tb, lda=lda, ldb=ldb, C_in=C_in)
    err = norm_err(to_host_f64(C), ref, S)
    tol = TOL_F32 if (dt == "f32" and ct == "f32") else TOL_BF16
    assert err <= tol, f"M={M} N={N} K={K} {dt}->{ct} ta={ta} tb={tb} acc={accumulate}: err {err:.3e}"
    return err


def test_config_fp32_128_cubed():
    d = workloads.gemm_small_fp32()
    A, B = to_gpu(d["A"]), to_gpu(d["B"])
    C = isam.gemm(A, B)
    torch.cuda.synchronize()
    ref, S = oracle.gemm(d["A"], d["B"], 128, 128, 128)
    assert norm_err(to_host_f64(C), ref, S) <= TOL_F32


SIZES = [1, 7, 31, 64, 65, 129]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_shape_sweep_layouts(dt, ta, tb):
    for M in SIZES:
        for N in (1, 33, 64, 200):
            for K in (1, 31, 64, 129):
                _run_case(M, N, K, dt, "f32" if dt == "f32" else "bf16", ta, tb, seed=M * 7 + N + K)


@pytest.mark.parametrize("dt,ct", [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16"), ("f32", "bf16")])
@pytest.mark.parametrize("shape", [(256, 256, 256), (300, 520, 192), (1000, 96, 1000), (520, 700, 64),
                                   (64, 4096, 72), (2048, 40, 2048)])
def test_tiles_and_outputs(dt, ct, shape):
    M, N, K = shape
    _run_case(M, N, K, dt, ct)


@pytest.mark.parametrize("dt,ct", [("f32", "f32"), ("bf16", "bf16")])
def test_accumulate(dt, ct):
    _run_case(129, 65, 257, dt, ct, accumulate=True)
    _run_case(1024, 32, 2048, dt, ct, accumulate=True)   # split-K path with accumulate


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_leading_dimension_padding(dt):
    _run_case(100, 72, 136, dt, "f32", pad_ld=8)
    _run_case(100, 72, 136, dt, "f32", ta=1, tb=1, pad_ld=8)


def test_k_zero():
    A = torch.empty((5, 0), device="cuda", dtype=torch.float32)
    B = torch.empty((0, 6), device="cuda", dtype=torch.float32)
    C = isam.gemm(A, B)
    torch.cuda.synchronize()
    assert torch.count_nonzero(C).item() == 0
    C2 = torch.full((5, 6), 3.0, device="cuda")
    isam.gemm(A, B, C2, accumulate=True)
    torch.cuda.synchronize()
    assert torch.all(C2 == 3.0)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_guard_bands_untouched(dt):
    M, N, K, ldc = 130, 70, 96, 80
    A_h = synth.uniform(1, 0, (M, K), -1, 1)
    B_h = synth.uniform(1, 1, (K, N), -1, 1)
    if dt == "bf16":
        A_h, B_h = bits(A_h), bits(B_h)
    A, B = to_gpu(A_h), to_gpu(B_h)
    buf = torch.full((M * ldc + 4096,), -12345.0, device="cuda")
    C = buf[2048: 2048 + M * ldc].view(M, ldc)[:, :N]
    isam.gemm(A, B, C)
    torch.cuda.synchronize()
    h = buf.cpu().numpy()
    assert np.all(h[:2048] == -12345.0) and np.all(h[2048 + M * ldc:] == -12345.0)
    body = h[2048: 2048 + M * ldc].reshape(M, ldc)
    assert np.all(body[:, N:] == -12345.0)
    ref, S = oracle.gemm(A_h, B_h, M, N, K)
    assert norm_err(body[:, :N].astype(np.float64), ref, S) <= (TOL_F32 if dt == "f32" else TOL_BF16)


def test_deterministic_run_twice():
    for (M, N, K) in [(512, 512, 512), (4096, 32, 4096)]:
        A = to_gpu(bits(synth.uniform(2, 0, (M, K), -1, 1)))
        B = to_gpu(bits(synth.uniform(2, 1, (K, N), -1, 1)))
        c1 = isam.gemm(A, B)
        c2 = isam.gemm(A, B)
        torch.cuda.synchronize()
        assert torch.equal(c1, c2)


@pytest.mark.parametrize("variant", ["bf16", "f32"])
def test_config_skinny_full(variant):
    d = workloads.skinny()
    A_h = d["A_bf16"] if variant == "bf16" else d["A"]
    B_h = d["B_bf16"] if variant == "bf16" else d["B"]
    C = isam.gemm(to_gpu(A_h), to_gpu(B_h))
    torch.cuda.synchronize()
    ref, S = oracle.gemm(A_h, B_h, 4096, 32, 4096)
    err = norm_err(to_host_f64(C), ref, S)
    assert err <= (TOL_BF16 if variant == "bf16" else TOL_F32), err


_LARGE_REF = {}


def _large_ref(which):
    """Oracle result and normaliser of a whole large bf16 product, computed once per module
    (about 20 s for 8192^3 on 16 host cores)."""
    if which not in _LARGE_REF:
        _LARGE_REF.clear()   # hold one (2 x 512 MiB for 8192^2) at a time
        d = workloads.gemm_square_bf16() if which == "square" else workloads.gemm_rect_bf16()
        A_h, B_h = d["A_bf16"], d["B_bf16"]
        M, K = A_h.shape
        N = B_h.shape[1]
        ref, S = oracle.gemm(A_h, B_h, M, N, K)
        _LARGE_REF[which] = (A_h, B_h, ref, S)
    return _LARGE_REF[which]


@pytest.mark.parametrize("which", ["square", "rect"])
def test_config_large_bf16_every_element(which):
    # 8192^3 and 8192 x 1024 x 16384 in the launch configuration the benchmark times, fp32 and
    # bf16 output, every element against the oracle.
    A_h, B_h, ref, S = _large_ref(which)
    A, B = to_gpu(A_h), to_gpu(B_h)
    for out_dtype in (torch.float32, torch.bfloat16):
        C = isam.gemm(A, B, out_dtype=out_dtype)
        torch.cuda.synchronize()
        err = norm_err(to_host_f64(C), ref, S)
        assert err <= TOL_BF16, f"{which} {out_dtype}: {err:.3e}"
        del C


# Every direct-to-LDS kernel instance, forced on small shapes and checked on every element:
# 256x256 tiles with 8 waves (the large-GEMM kernel) and with 4, 256x128 with 8 and 4, and
# 128x128; B K-contiguous (NT) and N-contiguous (NN); K a multiple of the 64-deep tile (copy
# offsets as base + per-tile delta) and with a ragged last tile; fp32 and bf16 output;
# unsplit and split into two K slices (partial sums + fixed-order reduction).
# Two K slices of 256x256 tiles summed inside the kernel (slice 1 adds slice 0's partial
# sums, exchanged through the L2 of the XCD both share): tile counts that are multiples of
# 8 (the condition for the in-kernel sum), ragged M and N, both B layouts, both output
# types, accumulate, repeated calls on one workspace; K with a ragged last tile takes the
# reduction pass instead.  Every element against the oracle.
# Both forms: each slice finishing half of the tile (every workgroup resident: the default
# here) and the one-way form (fixup=1: slice 1 finishes the whole tile).
@pytest.mark.parametrize("shape,in_kernel", [((512, 1024, 1280), True), ((500, 1000, 1280), True),
                                             ((512, 1024, 1200), False)])
@pytest.mark.parametrize("tb", [0, 1])
@pytest.mark.parametrize("form", ["halves", "one_way"])
def test_split_sum_in_kernel_every_element(shape, in_kernel, tb, form, monkeypatch, capfd):
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "tile=0,dma=1,dmaw=8,splits=2" + (",fixup=1" if form == "one_way" else ""))
    monkeypatch.setenv("ISAM_LOG", "1")
    M, N, K = shape
    for rep in range(2):
        for ct in ("f32", "bf16"):
            _run_case(M, N, K, "bf16", ct, tb=tb, seed=M + K + tb + rep)
    _run_case(M, N, K, "bf16", "f32", tb=tb, accumulate=True, seed=M + K + 7)
    log = capfd.readouterr().err
    assert ("two K slices summed in the kernel" in log) == in_kernel
    assert ("each slice finishes half" in log) == (in_kernel and form == "halves")


@pytest.mark.parametrize("form", ["halves", "one_way"])
def test_split_sum_in_kernel_timeout_gives_nan(form, monkeypatch):
    # The slices' waits are bounded; the host forces them to expire (each waits for a flag
    # value that is never written, under a 1 ms bound): every output is NaN, and the next
    # call on the same workspace is correct again.
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "tile=0,dma=1,dmaw=8,splits=2" + (",fixup=1" if form == "one_way" else ""))
    M, N, K = 512, 1024, 1280
    A_h = bits(synth.uniform(3, 10, (M, K), -1, 1))
    B_h = bits(synth.uniform(3, 11, (K, N), -1, 1))
    A, B = to_gpu(A_h), to_gpu(B_h)
    ws = torch.empty(isam.gemm_workspace_size(M, N, K, 1, 0), device="cuda", dtype=torch.uint8)
    monkeypatch.setenv("ISAM_GEMM_TEST_FIXUP_STALL", "1")
    C = isam.gemm(A, B, workspace=ws)
    torch.cuda.synchronize()
    assert torch.all(torch.isnan(C)).item()
    monkeypatch.delenv("ISAM_GEMM_TEST_FIXUP_STALL")
    C = isam.gemm(A, B, workspace=ws)
    torch.cuda.synchronize()
    ref, S = oracle.gemm(A_h, B_h, M, N, K)
    assert norm_err(to_host_f64(C), ref, S) <= TOL_BF16


# Stream-K schedule: a persistent grid in which every workgroup takes an equal share of the
# (output tile, 64-deep K tile) units of its XCD's range of tiles, and a tile's owner starts
# from the partial sums of the later shares of its K range (fixed order).  Forced on each tile
# shape it covers, with a few more tiles than workgroups (shares of 1 to 1.1 tiles, so most
# tiles are split between two workgroups): both B layouts, K a multiple of 64 and ragged,
# ragged M and N with a tile count that is not a multiple of the XCD count, both output
# types, accumulate.  Every element.
SK_CASES = [("0", 4352, 4096), ("1", 4352, 2048), ("1", 4400, 1904), ("2", 2900, 2944)]


@pytest.mark.parametrize("tile,M,N", SK_CASES)
@pytest.mark.parametrize("tb", [0, 1])
@pytest.mark.parametrize("K", [640, 600])
def test_stream_k_every_element(tile, M, N, tb, K, monkeypatch, capfd):
    monkeypatch.setenv("ISAM_GEMM_CONFIG", f"tile={tile},dma=1,sk=1")
    monkeypatch.setenv("ISAM_LOG", "1")
    for ct in ("f32", "bf16"):
        _run_case(M, N, K, "bf16", ct, tb=tb, seed=M + N + K + tb)
    _run_case(M, N, K, "bf16", "f32", tb=tb, accumulate=True, seed=M + K + 5)
    assert "stream-K" in capfd.readouterr().err


# Whole rounds first, then the remaining tiles' units in shares: 4352 x 4352 (289 tiles of
# 256x256, 36-37 per XCD on 32 workgroups) with K deep enough (64 K tiles) that the 4-5
# remaining tiles are shared without the last whole round.  Forced, both output types, K a
# multiple of 64 and ragged; every element.
@pytest.mark.parametrize("K", [4096, 4040])
def test_stream_k_whole_rounds_first_every_element(K, monkeypatch, capfd):
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "tile=0,dma=1,sk=1")
    monkeypatch.setenv("ISAM_LOG", "1")
    for ct in ("f32", "bf16"):
        _run_case(4352, 4352, K, "bf16", ct, seed=K + (ct == "bf16"))
    assert "stream-K" in capfd.readouterr().err


# The planner takes stream-K by itself for 256x256 tiles when at least one whole round exists
# and the last round would keep at most a quarter of the CUs busy: 4352 x 4096 (272 tiles; the
# small remainder joins the last whole round) with K a multiple of 64 and ragged, and
# 4352 x 4352 x 4096 (289 tiles; whole round first).  Every element, and bit-identical on a
# second call.
@pytest.mark.parametrize("shape", [(4352, 4096, 1024), (4352, 4096, 1000), (4352, 4352, 4096)])
def test_stream_k_planned_every_element(shape, monkeypatch, capfd):
    monkeypatch.delenv("ISAM_GEMM_CONFIG", raising=False)
    monkeypatch.setenv("ISAM_LOG", "1")
    M, N, K = shape
    A_h = bits(synth.normal(M, 40, (M, K)) / np.sqrt(K))
    B_h = bits(synth.normal(M, 41, (K, N)) / np.sqrt(K))
    A, B = to_gpu(A_h), to_gpu(B_h)
    C1 = isam.gemm(A, B)
    C2 = isam.gemm(A, B)
    torch.cuda.synchronize()
    assert "stream-K" in capfd.readouterr().err
    assert torch.equal(C1, C2)
    ref, S = oracle.gemm(A_h, B_h, M, N, K)
    assert norm_err(to_host_f64(C1), ref, S) <= TOL_BF16


def test_stream_k_timeout_gives_nan(monkeypatch):
    # An owner's wait for the partial sums of its tile is bounded; the host forces it to expire
    # (the flag value waited for is never written, 1 ms bound): the tiles shared between
    # workgroups come back NaN, the others are still right, and the next call on the same
    # workspace is correct everywhere.
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "tile=0,dma=1,sk=1")
    M, N, K = 4352, 4096, 640
    A_h = bits(synth.uniform(5, 10, (M, K), -1, 1))
    B_h = bits(synth.uniform(5, 11, (K, N), -1, 1))
    A, B = to_gpu(A_h), to_gpu(B_h)
    ws = torch.empty(isam.gemm_workspace_size(M, N, K, 1, 0), device="cuda", dtype=torch.uint8)
    monkeypatch.setenv("ISAM_GEMM_TEST_FIXUP_STALL", "1")
    C = isam.gemm(A, B, workspace=ws)
    torch.cuda.synchronize()
    ref, S = oracle.gemm(A_h, B_h, M, N, K)
    tiles = to_host_f64(C).reshape(M // 256, 256, N // 256, 256).transpose(0, 2, 1, 3)
    nan_tile = np.isnan(tiles).any(axis=(2, 3))
    assert nan_tile.any() and not nan_tile.all()
    assert np.isnan(tiles[nan_tile]).all(), "a tile is partly NaN"
    good = ~np.repeat(np.repeat(nan_tile, 256, axis=0), 256, axis=1)
    assert norm_err(np.where(good, to_host_f64(C), ref), ref, S) <= TOL_BF16
    monkeypatch.delenv("ISAM_GEMM_TEST_FIXUP_STALL")
    C = isam.gemm(A, B, workspace=ws)
    torch.cuda.synchronize()
    assert norm_err(to_host_f64(C), ref, S) <= TOL_BF16


DMA_INSTANCES = [("0", "8"), ("0", "4"), ("1", "8"), ("1", "4"), ("2", "4")]


@pytest.mark.parametrize("tile,waves", DMA_INSTANCES)
@pytest.mark.parametrize("tb", [0, 1])
@pytest.mark.parametrize("K", [640, 600])
@pytest.mark.parametrize("splits", [1, 2])
def test_dma_instances_every_element(tile, waves, tb, K, splits, monkeypatch):
    monkeypatch.setenv("ISAM_GEMM_CONFIG", f"tile={tile},dma=1,dmaw={waves},splits={splits}")
    for ct in ("f32", "bf16"):
        _run_case(512, 768, K, "bf16", ct, tb=tb, seed=K + splits + int(tile))
    _run_case(512, 768, K, "bf16", "f32", tb=tb, accumulate=True, seed=K + 7)


# The direct-to-LDS kernels' two-A / three-B-stage ring (the last K tile without copies) on K
# slices of one, two and three tiles, and a ragged one: unsplit, split with a reduction pass and,
# for 256x256 tiles with 8 waves over 8 tiles, split with the in-kernel sum; every element.
@pytest.mark.parametrize("K,splits,N", [(64, 1, 768), (128, 1, 768), (192, 1, 768), (128, 2, 768), (640, 3, 768),
                                        (100, 1, 768), (128, 2, 1024), (256, 2, 1024), (384, 2, 1024)])
@pytest.mark.parametrize("tb", [0, 1])
@pytest.mark.parametrize("tile,waves", DMA_INSTANCES)
def test_dma_ring_short_slices(K, splits, N, tb, tile, waves, monkeypatch):
    monkeypatch.setenv("ISAM_GEMM_CONFIG", f"tile={tile},dma=1,dmaw={waves},splits={splits}")
    for ct in ("f32", "bf16"):
        _run_case(512, N, K, "bf16", ct, tb=tb, seed=K + splits + N)
    _run_case(512, N, K, "bf16", "f32", tb=tb, accumulate=True, seed=K + 3)


def _guarded_gemm(M, N, K, dt, ct, pad_cols, seed, tb=0, env=None, monkeypatch=None):
    """C written into a [M][N + pad_cols] window of a larger sentinel-filled buffer: checks
    that nothing outside the M x N block changes and that the block matches the oracle."""
    if env is not None:
        monkeypatch.setenv("ISAM_GEMM_CONFIG", env)
    Am = synth.uniform(seed, 30, (M, K), -1, 1)
    Bm = synth.uniform(seed, 31, (K, N), -1, 1)
    B_host = np.ascontiguousarray(Bm.T) if tb else Bm
    if dt == "bf16":
        Am, B_host = bits(Am), bits(B_host)
        Bm = bits(Bm)
    A, B = to_gpu(Am), to_gpu(B_host)
    ldc = N + pad_cols
    g = 4096
    tdt = torch.bfloat16 if ct == "bf16" else torch.float32
    sentinel = -12345.0
    buf = torch.full((M * ldc + 2 * g,), sentinel, device="cuda", dtype=tdt)
    C = buf[g: g + M * ldc].view(M, ldc)[:, :N]
    isam.gemm(A, B, C, trans_b=bool(tb))
    torch.cuda.synchronize()
    h = buf.float().cpu().numpy()
    sv = float(torch.tensor(sentinel, dtype=tdt).float())
    assert np.all(h[:g] == sv) and np.all(h[g + M * ldc:] == sv), "write before or after C"
    body = h[g: g + M * ldc].reshape(M, ldc)
    assert np.all(body[:, N:] == sv), "write into the row padding of C"
    ref, S = oracle.gemm(Am, Bm, M, N, K)
    tol = TOL_F32 if (dt == "f32" and ct == "f32") else TOL_BF16
    assert norm_err(body[:, :N].astype(np.float64), ref, S) <= tol


GUARD_CASES = ["dma256", "dma256_split", "dma256_split_sum", "dma128", "dma_sk", "skinny_rows", "skinny_split",
               "narrow", "stream", "tile_f32", "small", "packed", "f32_split"]


@pytest.mark.parametrize("ct", ["f32", "bf16"])
@pytest.mark.parametrize("case", GUARD_CASES)
def test_guard_bands_every_kernel(ct, case, monkeypatch):
    # Each GEMM kernel writes exactly its M x N block: the direct-to-LDS kernels (256x256
    # whole and split along K, 128x128, the stream-K schedule), the skinny kernels (one pass
    # and split-K), the narrow dot-product kernel, the streaming kernel, the fp32 tile kernel,
    # the small-product kernel, and the products on operands packed or split into bf16 terms
    # in the workspace, with C rows padded (ldc > N).
    cases = {
        "dma256": dict(M=520, N=776, K=640, dt="bf16", env="tile=0,dma=1,dmaw=8"),
        "dma256_split": dict(M=520, N=776, K=640, dt="bf16", env="tile=0,dma=1,dmaw=8,splits=2"),
        "dma256_split_sum": dict(M=500, N=1000, K=1280, dt="bf16", env="tile=0,dma=1,dmaw=8,splits=2"),
        "dma128": dict(M=520, N=776, K=600, dt="bf16", env="tile=2,dma=1"),
        "dma_sk": dict(M=4400, N=1904, K=600, dt="bf16", env="tile=1,dma=1,sk=1"),
        "skinny_rows": dict(M=4100, N=32, K=1000, dt="bf16", env=None),
        "skinny_split": dict(M=300, N=24, K=6000, dt="f32", env=None),
        "narrow": dict(M=1000, N=3, K=2000, dt="bf16", env=None),
        "stream": dict(M=300, N=72, K=96, dt="bf16", env="stream=1"),
        "tile_f32": dict(M=300, N=200, K=130, dt="f32", env=None),
        "small": dict(M=100, N=64, K=520, dt="f32", env=None),
        "packed": dict(M=2048, N=2040, K=1001, dt="bf16", env=None),
        "f32_split": dict(M=2048, N=2040, K=1000, dt="f32", env=None),
    }
    c = cases[case]
    _guarded_gemm(c["M"], c["N"], c["K"], c["dt"], ct, pad_cols=8, seed=100 + GUARD_CASES.index(case),
                  env=c["env"], monkeypatch=monkeypatch)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("N", [8, 16, 24, 32])
def test_skinny_shapes(dt, N):
    # streaming kernel for N <= 32: ragged M, K covering partial and multiple K slices
    for M, K in [(1, 8), (33, 1000), (100, 2048), (4097, 4104), (257, 6000)]:
        _run_case(M, N, K, dt, "f32", seed=M + K + N)
    _run_case(300, N, 3000, dt, "bf16", seed=N)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("N", [1, 2, 3, 5, 6, 7])
def test_narrow_shapes(dt, N):
    # dot-product kernel for N < 8: ragged M, K within one and over several
    # LDS slices of B^T, B rows wider than N, bf16 output, accumulate
    for M, K in [(1, 8), (33, 1000), (100, 2048), (4097, 4104), (70, 7168)]:
        _run_case(M, N, K, dt, "f32", seed=M + K + N)
    _run_case(300, N, 3000, dt, "bf16", seed=N, pad_ld=8)
    _run_case(129, N, 520, dt, "f32", accumulate=True, seed=2 * N)
    _run_case(64, N, 333, dt, "f32", seed=3 * N)   # A rows not 16-byte aligned: tile kernel


def test_skinny_accumulate_and_fallback_layouts():
    _run_case(513, 32, 5000, "bf16", "f32", accumulate=True)
    _run_case(513, 32, 5000, "f32", "f32", accumulate=True)
    _run_case(300, 32, 2048, "bf16", "f32", ta=1)      # transposed A: tile kernel
    _run_case(300, 16, 2048, "bf16", "f32", tb=1)      # transposed B: tile kernel


# Small products (at most 64 output tiles of 32x32, K <= 1024, A K-contiguous and aligned):
# one tile per workgroup with the four waves splitting K.  Ragged M and N, K that is not a
# multiple of the MFMA step (only of the 16-byte piece), both B layouts, accumulate and both
# output types; the same shapes through the tile kernels (small=0) agree within the tolerance.
@pytest.mark.parametrize("dt,ct", [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16"), ("f32", "bf16")])
@pytest.mark.parametrize("tb", [0, 1])
@pytest.mark.parametrize("shape", [(128, 128, 128), (33, 250, 24), (256, 256, 1024), (1, 40, 8), (100, 64, 520)])
def test_small_products(dt, ct, tb, shape):
    M, N, K = shape
    _run_case(M, N, K, dt, ct, tb=tb, seed=M + N + K)


@pytest.mark.parametrize("dt,ct", [("f32", "f32"), ("bf16", "bf16")])
def test_small_products_accumulate_and_tile_path(dt, ct, monkeypatch):
    _run_case(96, 160, 200, dt, ct, accumulate=True, seed=5)
    _run_case(96, 160, 200, dt, ct, tb=1, accumulate=True, seed=6)
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "small=0")
    _run_case(96, 160, 200, dt, ct, accumulate=True, seed=5)


# The 256x256 direct-to-LDS kernel in both copy modes: K a multiple of 64 (offsets as base +
# per-tile delta; unsplit at 4096^2, split into K slices at 2048^2) and K with a ragged last tile (range-checked offsets); NN
# and NT; sampled rows (first, last, spread) against the oracle.
@pytest.mark.parametrize("K", [1024, 1000, 4160, 4100])
@pytest.mark.parametrize("tb", [0, 1])
def test_dma_256_tile_copy_modes(K, tb):
    M = N = 4096 if K < 2048 else 2048   # 2048^2: 64 tiles, split along K
    A_h = bits(synth.uniform(K, 20, (M, K), -1, 1))
    Bm = bits(synth.uniform(K, 21, (K, N), -1, 1))
    B_h = np.ascontiguousarray(Bm.T) if tb else Bm
    C = isam.gemm(to_gpu(A_h), to_gpu(B_h), trans_b=bool(tb))
    torch.cuda.synchronize()
    rows = workloads.rows_sample(M, 24)
    ref, S = oracle.gemm(np.ascontiguousarray(A_h[rows]), Bm, len(rows), N, K)
    got = to_host_f64(C[torch.as_tensor(rows, device="cuda")])
    assert norm_err(got, ref, S) <= TOL_BF16


# The 128x128 direct-to-LDS kernel (shallow K, grid covering the CUs) in both copy modes.
@pytest.mark.parametrize("K", [1024, 1000])
@pytest.mark.parametrize("tb", [0, 1])
def test_dma_128_tile_copy_modes(K, tb):
    M, N = 2048, 3072
    A_h = bits(synth.uniform(K, 22, (M, K), -1, 1))
    Bm = bits(synth.uniform(K, 23, (K, N), -1, 1))
    B_h = np.ascontiguousarray(Bm.T) if tb else Bm
    C = isam.gemm(to_gpu(A_h), to_gpu(B_h), trans_b=bool(tb))
    torch.cuda.synchronize()
    rows = workloads.rows_sample(M, 24)
    ref, S = oracle.gemm(np.ascontiguousarray(A_h[rows]), Bm, len(rows), N, K)
    got = to_host_f64(C[torch.as_tensor(rows, device="cuda")])
    assert norm_err(got, ref, S) <= TOL_BF16


# Operands whose rows cannot be copied 16 bytes at a time (K or the contiguous M / N off the
# vector width, a leading dimension or base pointer off 16 bytes) are packed into the
# workspace with zero-padded K and run on the MFMA kernels; every element against the oracle.
def _packed_case(M, N, K, dt, ct, ta, tb, monkeypatch, capfd, a_shift=0, ld_pad=0, accumulate=False,
                 expect_pack=True, workspace=None, seed=0, key="packed operands", env=None):
    if env is None:
        monkeypatch.delenv("ISAM_GEMM_CONFIG", raising=False)
    else:
        monkeypatch.setenv("ISAM_GEMM_CONFIG", env)
    monkeypatch.setenv("ISAM_LOG", "1")
    Am = synth.uniform(seed, 50, (M, K), -1, 1)
    Bm = synth.uniform(seed, 51, (K, N), -1, 1)
    A_host = np.ascontiguousarray(Am.T) if ta else Am
    B_host = np.ascontiguousarray(Bm.T) if tb else Bm
    if ld_pad:
        A_host = np.pad(A_host, ((0, 0), (0, ld_pad)), constant_values=5.0)
        B_host = np.pad(B_host, ((0, 0), (0, ld_pad)), constant_values=-5.0)
    if dt == "bf16":
        A_host, B_host = bits(A_host), bits(B_host)
    A_flat = to_gpu(np.concatenate([np.zeros(a_shift, A_host.dtype), A_host.ravel()]))
    A = A_flat[a_shift:].view(A_host.shape)
    B = to_gpu(B_host)
    if ld_pad:
        A = A[:, : A.shape[1] - ld_pad]
        B = B[:, : B.shape[1] - ld_pad]
    tdt = torch.bfloat16 if ct == "bf16" else torch.float32
    C_in = None
    if accumulate:
        c0 = synth.uniform(seed, 52, (M, N), -1, 1)
        C = to_gpu(bits(c0) if ct == "bf16" else c0)
        C_in = to_host_f64(C)
        isam.gemm(A, B, C, trans_a=bool(ta), trans_b=bool(tb), accumulate=True, workspace=workspace)
    else:
        C = isam.gemm(A, B, trans_a=bool(ta), trans_b=bool(tb), out_dtype=tdt, workspace=workspace)
    torch.cuda.synchronize()
    err_log = capfd.readouterr().err
    assert (key in err_log) == expect_pack, err_log[-2000:]
    ref, S = oracle.gemm(A_host, B_host, M, N, K, ta, tb, lda=A_host.shape[1], ldb=B_host.shape[1], C_in=C_in)
    tol = TOL_F32 if (dt == "f32" and ct == "f32") else TOL_BF16
    err = norm_err(to_host_f64(C), ref, S)
    assert err <= tol, err
    return C


@pytest.mark.parametrize("dt,ct", [("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32")])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_packed_odd_k_every_element(dt, ct, ta, tb, monkeypatch, capfd):
    # K = 1001: both operands padded to K = 1024, A transposed into
    # [M][K] when it is given as [K][M]; 2048^2 takes the 128x128 tiles.  With A [K][M] and
    # B [K][N] no row runs along K: fp32 is then not packed, bf16 only for A's transpose.
    # (fp32 with the bf16-term split switched off: that path is tested below.)
    _packed_case(2048, 2048, 1001, dt, ct, ta, tb, monkeypatch, capfd,
                 expect_pack=not (ta and not tb and dt == "f32"), env="f32split=0" if dt == "f32" else None)


@pytest.mark.parametrize("case", ["n_ragged", "m_ragged_ta", "ta_aligned", "tt_aligned", "a_shift", "ld_odd",
                                  "accumulate", "deep_k", "k_vector_pad", "k3", "k13_nt"])
def test_packed_layouts_every_element(case, monkeypatch, capfd):
    c = {
        # B [K][N] with N off the vector width: packed transposed to [N][K]
        "n_ragged": dict(M=2048, N=2044, K=1024, ta=0, tb=0),
        # A [K][M] with M off the vector width: packed transposed to [M][K]
        "m_ragged_ta": dict(M=2044, N=2048, K=1024, ta=1, tb=0),
        # bf16 A given as [K][M] with aligned rows: copied transposed for the direct-to-LDS kernel
        "ta_aligned": dict(M=2048, N=2048, K=1024, ta=1, tb=0),
        "tt_aligned": dict(M=2048, N=2048, K=1024, ta=1, tb=1),
        # A's base 2 bytes past a 16-byte boundary: only A is copied
        "a_shift": dict(M=2048, N=2048, K=1024, ta=0, tb=1, a_shift=1),
        # leading dimensions K + 1 (rows off 16 bytes) in both operands
        "ld_odd": dict(M=2048, N=2048, K=1024, ta=0, tb=1, ld_pad=1),
        "accumulate": dict(M=2048, N=2048, K=1001, ta=0, tb=0, accumulate=True),
        # deep odd K on 256x256 tiles (split along K after packing)
        "deep_k": dict(M=1024, N=1024, K=4101, ta=0, tb=0),
        # K padded to the vector width only (968; 1024 would add more than 1/16)
        "k_vector_pad": dict(M=2048, N=2048, K=961, ta=0, tb=1),
        # K below one 64-deep tile: padded to 8 / 16, one ragged K tile
        "k3": dict(M=4096, N=4096, K=3, ta=0, tb=0),
        "k13_nt": dict(M=4096, N=4096, K=13, ta=0, tb=1),
    }[case]
    kw = {k: v for k, v in c.items() if k not in ("M", "N", "K", "ta", "tb")}
    if case in ("a_shift", "ld_odd"):
        # the sizes-only workspace query cannot see a pointer or leading dimension: the caller
        # passes room for the copies (here both operands, 2 x 4 MiB)
        kw["workspace"] = torch.empty(8 << 20, device="cuda", dtype=torch.uint8)
    _packed_case(c["M"], c["N"], c["K"], "bf16", "bf16", c["ta"], c["tb"], monkeypatch, capfd, **kw)


def test_packed_needs_workspace_else_tile_kernel(monkeypatch, capfd):
    # Without room for the packed copies the element-wise tile kernel runs; same results to
    # the tolerance, and the sizes-only workspace query covers the packed path.
    M, N, K = 2048, 2048, 1001
    assert isam.gemm_workspace_size(M, N, K, 1, 1) == 2 * (2048 * 1024 * 2)
    tiny = torch.empty(16, device="cuda", dtype=torch.uint8)
    C0 = _packed_case(M, N, K, "bf16", "bf16", 0, 0, monkeypatch, capfd, expect_pack=False, workspace=tiny)
    C1 = _packed_case(M, N, K, "bf16", "bf16", 0, 0, monkeypatch, capfd)
    assert torch.isfinite(C0.float()).all() and torch.isfinite(C1.float()).all()


# Large fp32 products run as one bf16 product over six K blocks of the operands' bf16 terms
# (A (h, h, m, h, l, m), B (h, m, h, l, h, m)): every element against the oracle at the fp32
# tolerance, with the fp32 tile kernel (f32split=0) beside it.
@pytest.mark.parametrize("case", ["nn_ragged_k", "nt", "bf16_out", "accumulate", "a_shift", "nn_4096", "native",
                                  "k5", "n_ragged_nt"])
def test_fp32_split_every_element(case, monkeypatch, capfd):
    c = {
        "nn_ragged_k": dict(M=2048, N=2048, K=1001, tb=0),   # K per block 1024, four K slices after
        "nt": dict(M=2048, N=2048, K=1024, tb=1),
        "bf16_out": dict(M=2048, N=2048, K=1024, tb=0, ct="bf16"),
        "accumulate": dict(M=2048, N=2048, K=1000, tb=1, accumulate=True),
        "a_shift": dict(M=2048, N=2048, K=1024, tb=0, a_shift=1),  # A 4 bytes past 16: element reads
        "nn_4096": dict(M=4096, N=4096, K=4096, tb=0),
        "native": dict(M=2048, N=2048, K=1024, tb=0, env="f32split=0", expect_pack=False),
        # K = 5: six blocks of 8 (bf16 K' = 48, one ragged K tile)
        "k5": dict(M=4096, N=4096, K=5, tb=0),
        # B as [N][K] with N off 8 (allowed: K runs along B's rows)
        "n_ragged_nt": dict(M=2048, N=2044, K=1024, tb=1),
    }[case]
    kw = {k: v for k, v in c.items() if k not in ("M", "N", "K", "tb", "ct")}
    _packed_case(c["M"], c["N"], c["K"], "f32", c.get("ct", "f32"), 0, c["tb"], monkeypatch, capfd,
                 key="fp32 split into bf16 terms", **kw)


# Very shallow bf16 products (K <= 256, N <= 256 with N % 4 == 0, A and B not transposed): the
# streaming kernel (B in registers, A through an LDS ring).  Forced on small shapes with
# stream=1: ragged last 32-row tile, K not a multiple of the 16-deep MFMA step, N not a multiple
# of a wave's 32 columns, padded leading dimensions, fp32 and bf16 output, accumulate; then
# chosen by the planner on its own for a shape with enough row tiles, against the tile path.
@pytest.mark.parametrize("ct", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(33, 8, 8), (100, 40, 72), (257, 256, 128), (64, 100, 200),
                                   (95, 256, 256), (1, 4, 64), (300, 12, 24)])
def test_stream_kernel_forced(ct, shape, monkeypatch):
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "stream=1")
    M, N, K = shape
    _run_case(M, N, K, "bf16", ct, seed=M + N + K)
    _run_case(M, N, K, "bf16", ct, accumulate=True, seed=M + N + K + 1)
    _run_case(M, N, K, "bf16", ct, seed=M + N + K + 2, pad_ld=8)


@pytest.mark.parametrize("shape", [(32768, 64, 64), (40001, 256, 128), (33000, 200, 256)])
def test_stream_kernel_planned(shape, monkeypatch):
    M, N, K = shape
    monkeypatch.delenv("ISAM_GEMM_CONFIG", raising=False)
    e_stream = _run_case(M, N, K, "bf16", "f32", seed=M)
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "stream=0")
    e_tile = _run_case(M, N, K, "bf16", "f32", seed=M)
    assert e_stream <= TOL_BF16 and e_tile <= TOL_BF16


# A operand just under the 2^31-byte limit of the 32-bit buffer offsets: bf16 65536 x 16376
# (direct-to-LDS 256x256 kernel, ragged last K tile) and fp32 65536 x 8188 (fp32 tile kernel:
# its split copies would pass the limit).  A is a 4096-row random block repeated down the
# rows; the oracle checks sampled rows, the last ones (largest offsets) among them.
@pytest.mark.parametrize("dt,K", [("bf16", 16376), ("f32", 8188)])
def test_operand_at_the_extent_limit(dt, K):
    M, N = 65536, 256
    es = 2 if dt == "bf16" else 4
    assert M * K * es < 2 ** 31 and M * K * es > 2 ** 31 - 2 ** 22
    blk = synth.uniform(K, 70, (4096, K), -1, 1)
    Bm = synth.uniform(K, 71, (K, N), -1, 1)
    if dt == "bf16":
        blk, Bm = bits(blk), bits(Bm)
    A = to_gpu(blk).repeat(M // 4096, 1)
    C = isam.gemm(A, to_gpu(Bm))
    torch.cuda.synchronize()
    rows = [0, 1, 4095, 4096, 32767, 40000, 65534, 65535]
    A_rows = np.ascontiguousarray(blk[[r % 4096 for r in rows]])
    ref, S = oracle.gemm(A_rows, Bm, len(rows), N, K)
    got = to_host_f64(C[torch.as_tensor(rows, device="cuda")])
    assert norm_err(got, ref, S) <= (TOL_BF16 if dt == "bf16" else TOL_F32)
    del A, C
    torch.cuda.empty_cache()
