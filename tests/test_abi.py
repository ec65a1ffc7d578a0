"""C-ABI checks that need no GPU: the library loads, exports every function the header
declares, and rejects bad arguments during host-side validation (before any HIP call)."""
import ctypes
import os
import re

import pytest

from paper_1810_09958_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "isam.h")

OK, INVALID, UNSUPPORTED, WORKSPACE, HIPERR = 0, 1, 2, 3, 4
F32, BF16 = 0, 1
FAKE = ctypes.c_void_p(0x10000)      # never dereferenced: validation fails before any launch
FAKE2 = ctypes.c_void_p(0x20000000)


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(isam_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return _lib.lib()


def test_header_declares_expected_entry_points():
    names = header_functions()
    for n in ("isam_gemm", "isam_dwsep_conv", "isam_gru_forward", "isam_gemm_workspace_size",
              "isam_dwsep_conv_workspace_size", "isam_gru_forward_workspace_size",
              "isam_status_string", "isam_last_error", "isam_version"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    for n in header_functions():
        assert hasattr(L, n), f"libisam.so does not export {n}"
    assert set(header_functions()) == set(_lib.SIGNATURES)


def test_binding_has_no_compute_fallback():
    import paper_1810_09958_amd as P
    src = open(P.__file__).read() + open(_lib.__file__).read()
    assert "import oracle" not in src and "from oracle" not in src
    for op in ("torch.matmul", "torch.mm(", "conv2d", "torch.nn.GRU", ".numpy()"):
        assert op not in src


def test_version_and_status_strings(L):
    assert L.isam_version() >= 100
    for s in range(5):
        assert L.isam_status_string(s).startswith(b"ISAM_")
    assert b"unknown" in L.isam_status_string(99)


def gemm(L, ta=0, tb=0, M=4, N=4, K=4, ab=F32, A=FAKE, lda=4, B=FAKE2, ldb=4, acc=0, ct=F32,
         C=ctypes.c_void_p(0x40000000), ldc=4, ws=None, wsb=0):
    return L.isam_gemm(ta, tb, M, N, K, ab, A, lda, B, ldb, acc, ct, C, ldc, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(M=-1), INVALID), (dict(N=-2), INVALID), (dict(K=-3), INVALID),
    (dict(ta=2), INVALID), (dict(tb=-1), INVALID), (dict(acc=3), INVALID),
    (dict(ab=7), INVALID), (dict(ct=5), INVALID),
    (dict(C=None), INVALID), (dict(ldc=3), INVALID),
    (dict(A=None), INVALID), (dict(B=None), INVALID),
    (dict(lda=3), INVALID), (dict(ldb=3), INVALID),
    (dict(ta=1, M=8, lda=4), INVALID), (dict(tb=1, K=8, lda=8, ldb=4), INVALID),
    (dict(M=1 << 20, K=1 << 12, lda=1 << 12, ldc=4), UNSUPPORTED),
    (dict(C=FAKE), INVALID),          # C overlaps A
])
def test_gemm_validation(L, kw, code):
    assert gemm(L, **kw) == code
    assert L.isam_last_error() != b""


def test_gemm_splitk_workspace_must_not_overlap_operands(L):
    # 512 x 32 x 8192 fp32 is planned with split-K partial sums in the workspace: a workspace
    # that overlaps C, A or B is rejected before anything is launched.
    M, N, K = 512, 32, 8192
    need = L.isam_gemm_workspace_size(0, 0, M, N, K, F32, F32)
    assert need > 0
    A, B, C = (ctypes.c_void_p(v) for v in (0x100000000, 0x200000000, 0x300000000))
    for ws in (C, A, B, ctypes.c_void_p(0x300000000 - need + 4)):
        assert gemm(L, M=M, N=N, K=K, A=A, lda=K, B=B, ldb=N, C=C, ldc=N, ws=ws, wsb=need) == INVALID
        assert b"workspace overlaps" in L.isam_last_error()


def test_gemm_workspace_query_covers_packing(L, monkeypatch):
    # A contiguous dimension off the vector width (8 bf16 / 4 fp32 values): room for the
    # packed operands with K rounded up (A as [M][Kp]; B as [Kp][N], or [N][Kp] when N is
    # off the vector width), each a multiple of 256 bytes, plus what the packed product
    # uses itself.  Kp: a multiple of 64 when both are copied and that adds at most K/16.
    # Only B copied, K unchanged (N off the vector width), or A only (A transposed).
    monkeypatch.delenv("ISAM_GEMM_CONFIG", raising=False)
    assert L.isam_gemm_workspace_size(0, 0, 2048, 2048, 1001, BF16, BF16) == 2 * (2048 * 1024 * 2)
    assert L.isam_gemm_workspace_size(1, 1, 2048, 2048, 1001, BF16, F32) == 2 * (2048 * 1024 * 2)
    assert L.isam_gemm_workspace_size(0, 0, 8192, 8192, 8100, BF16, BF16) == 2 * (8192 * 8128 * 2)
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "f32split=0")
    assert L.isam_gemm_workspace_size(0, 0, 2048, 2048, 1001, F32, F32) == 2 * (2048 * 1024 * 4)
    monkeypatch.delenv("ISAM_GEMM_CONFIG")
    # K = 961: a multiple of 64 (1024) would add more than 1/16, so the vector width (968)
    assert L.isam_gemm_workspace_size(0, 0, 2048, 2048, 961, BF16, BF16) == 2 * (2048 * 968 * 2)
    assert L.isam_gemm_workspace_size(0, 0, 2048, 2044, 1024, BF16, BF16) == 2044 * 1024 * 2
    assert L.isam_gemm_workspace_size(1, 0, 2044, 2048, 1024, BF16, BF16) == 2044 * 1024 * 2
    # deep K: the packed product is split along K and its partial sums follow the copies
    assert L.isam_gemm_workspace_size(0, 0, 1024, 1024, 4101, BF16, BF16) == \
        2 * (1024 * 4160 * 2) + 8 * 1024 * 1024 * 4
    # bf16 A given as [K][M] is copied transposed (fp32 is not)
    assert L.isam_gemm_workspace_size(1, 0, 4096, 4096, 4096, BF16, BF16) == 4096 * 4096 * 2
    assert L.isam_gemm_workspace_size(1, 1, 4096, 4096, 4096, BF16, F32) == 4096 * 4096 * 2
    assert L.isam_gemm_workspace_size(1, 0, 4096, 4096, 4096, F32, F32) == 0
    # products too small for the large tiles are not packed
    assert L.isam_gemm_workspace_size(0, 0, 100, 100, 101, BF16, BF16) == 0
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "pack=0")
    assert L.isam_gemm_workspace_size(0, 0, 2048, 2048, 1001, BF16, BF16) == 0


def test_gemm_workspace_query_covers_fp32_split(L, monkeypatch):
    # Large fp32 products with A [M][K] (B either layout, N a multiple of 8 when B is
    # [K][N]) run as one bf16 product over six K blocks of each operand's bf16 terms: room
    # for both split copies (12 bytes per operand value, K per block rounded up to 64 when
    # that adds at most K/16) plus what that bf16 product uses (here four K slices).
    monkeypatch.delenv("ISAM_GEMM_CONFIG", raising=False)
    assert L.isam_gemm_workspace_size(0, 0, 2048, 2048, 1001, F32, F32) == \
        2 * (2048 * 6 * 1024 * 2) + 4 * 2048 * 2048 * 4
    assert L.isam_gemm_workspace_size(0, 1, 4096, 4096, 4096, F32, F32) == 2 * (4096 * 6 * 4096 * 2)
    assert L.isam_gemm_workspace_size(0, 0, 4096, 4096, 4096, F32, BF16) == 2 * (4096 * 6 * 4096 * 2)
    # not split: A transposed, B [K][N] with N off 8, products whose copies would not pay
    assert L.isam_gemm_workspace_size(1, 0, 4096, 4096, 4096, F32, F32) == 0
    assert L.isam_gemm_workspace_size(0, 0, 4096, 4092, 4096, F32, F32) == 0
    small = L.isam_gemm_workspace_size(0, 0, 512, 512, 512, F32, F32)
    monkeypatch.setenv("ISAM_GEMM_CONFIG", "f32split=0")
    assert L.isam_gemm_workspace_size(0, 1, 4096, 4096, 4096, F32, F32) == 0
    assert L.isam_gemm_workspace_size(0, 0, 512, 512, 512, F32, F32) == small


def test_gemm_split_workspace_must_not_overlap_operands(L, monkeypatch):
    monkeypatch.delenv("ISAM_GEMM_CONFIG", raising=False)
    M, N, K = 4096, 4096, 4096
    need = L.isam_gemm_workspace_size(0, 1, M, N, K, F32, F32)
    A, B, C = (ctypes.c_void_p(v) for v in (0x100000000, 0x200000000, 0x300000000))
    for ws in (C, A, B):
        assert gemm(L, tb=1, M=M, N=N, K=K, ab=F32, A=A, lda=K, B=B, ldb=K, ct=F32, C=C, ldc=N,
                    ws=ws, wsb=need) == INVALID
        assert b"workspace overlaps" in L.isam_last_error()


def test_gemm_pack_workspace_must_not_overlap_operands(L, monkeypatch):
    # The packed copies go to the start of the workspace: one that overlaps A, B or C is
    # rejected before anything is launched.
    monkeypatch.delenv("ISAM_GEMM_CONFIG", raising=False)
    M, N, K = 2048, 2048, 1001
    need = L.isam_gemm_workspace_size(0, 0, M, N, K, BF16, BF16)
    A, B, C = (ctypes.c_void_p(v) for v in (0x100000000, 0x200000000, 0x300000000))
    for ws in (C, A, B):
        assert gemm(L, M=M, N=N, K=K, ab=BF16, A=A, lda=K, B=B, ldb=N, ct=BF16, C=C, ldc=N,
                    ws=ws, wsb=need) == INVALID
        assert b"workspace overlaps" in L.isam_last_error()


def test_gemm_empty_is_noop(L):
    assert gemm(L, M=0, A=None, B=None, C=None) == OK
    assert gemm(L, N=0, A=None, B=None, C=None) == OK


def test_gemm_workspace_queries(L):
    # A skinny-N product with enough 16-row blocks to cover the CUs streams each block
    # through one workgroup and needs no workspace (bf16 and fp32); with few rows and deep K
    # it is split along K and needs partial-sum space.
    assert L.isam_gemm_workspace_size(0, 0, 4096, 32, 4096, F32, F32) == 0
    assert L.isam_gemm_workspace_size(0, 0, 4096, 32, 4096, BF16, F32) == 0
    ws = L.isam_gemm_workspace_size(0, 0, 512, 32, 8192, F32, F32)
    assert ws > 0 and ws % (512 * 32 * 4) == 0
    assert L.isam_gemm_workspace_size(0, 0, 8192, 8192, 8192, BF16, BF16) == 0
    assert L.isam_gemm_workspace_size(0, 0, 0, 8, 8, BF16, BF16) == 0


def dw(L, batch=1, H=8, W=8, C=4, cm=1, kh=3, kw=3, s=1, p=1, Co=4, it=F32, x=FAKE,
       dwf=ctypes.c_void_p(0x30000), pw=ctypes.c_void_p(0x50000), ot=F32,
       y=ctypes.c_void_p(0x70000000), ws=ctypes.c_void_p(0x90000000), wsb=1 << 30):
    return L.isam_dwsep_conv(batch, H, W, C, cm, kh, kw, s, p, Co, it, x, dwf, pw, ot, y, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(batch=-1), INVALID), (dict(H=0), INVALID), (dict(C=0), INVALID), (dict(cm=0), INVALID),
    (dict(kh=0), INVALID), (dict(s=0), INVALID), (dict(p=-1), INVALID), (dict(Co=0), INVALID),
    (dict(it=3), INVALID), (dict(ot=9), INVALID), (dict(H=2, p=0), INVALID),
    (dict(x=None), INVALID), (dict(y=None), INVALID), (dict(pw=None), INVALID),
    (dict(ws=None), WORKSPACE), (dict(wsb=16), WORKSPACE),
    (dict(y=FAKE), INVALID),
])
def test_dwsep_validation(L, kw, code):
    assert dw(L, **kw) == code


def test_dwsep_workspace_query(L):
    # The fused kernels (3x3, stride 1, pad 1 at these channel counts) keep the depthwise
    # result on chip and need no workspace; other shapes hold Y in the workspace.
    assert L.isam_dwsep_conv_workspace_size(32, 56, 56, 128, 1, 3, 3, 1, 1, 256, BF16, F32) == 0
    assert L.isam_dwsep_conv_workspace_size(32, 56, 56, 128, 1, 3, 3, 1, 1, 256, BF16, BF16) == 0
    assert L.isam_dwsep_conv_workspace_size(32, 56, 56, 128, 1, 3, 3, 1, 1, 256, F32, F32) == 0
    n = L.isam_dwsep_conv_workspace_size(32, 56, 56, 128, 1, 3, 3, 2, 1, 256, BF16, F32)
    assert n >= 32 * 28 * 28 * 128 * 2
    n = L.isam_dwsep_conv_workspace_size(32, 56, 56, 128, 1, 3, 3, 1, 1, 256, F32, BF16)
    assert n >= 32 * 56 * 56 * 128 * 4
    assert L.isam_dwsep_conv_workspace_size(32, 56, 56, 128, 1, 3, 3, 0, 1, 256, BF16, F32) == 0
    assert dw(L, batch=0, x=None, y=None) == OK


def gru(L, T=4, B=2, I=8, H=8, wt=F32, x=FAKE, h0=None, W=ctypes.c_void_p(0x30000),
        U=ctypes.c_void_p(0x50000), bias=None, bhn=None, hseq=ctypes.c_void_p(0x70000000),
        hT=None, ws=ctypes.c_void_p(0x90000000), wsb=1 << 30):
    return L.isam_gru_forward(T, B, I, H, wt, x, h0, W, U, bias, bhn, hseq, hT, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(T=-1), INVALID), (dict(B=-1), INVALID), (dict(I=0), INVALID), (dict(H=0), INVALID),
    (dict(wt=2), INVALID), (dict(hseq=None), INVALID), (dict(x=None), INVALID),
    (dict(U=None), INVALID), (dict(H=6), UNSUPPORTED), (dict(H=12, wt=BF16), UNSUPPORTED),
    (dict(ws=None), WORKSPACE), (dict(wsb=64), WORKSPACE),
    (dict(hseq=FAKE), INVALID),
])
def test_gru_validation(L, kw, code):
    assert gru(L, **kw) == code


def test_gru_workspace_query(L):
    n = L.isam_gru_forward_workspace_size(64, 32, 1024, 1024, BF16)
    assert n >= 64 * 32 * 3 * 1024 * 4 + 2 * 32 * 1024 * 2
    assert gru(L, B=0) == OK


def conv1d(L, nb=2, Ln=10, Ki=8, D=3, Ko=8, ab=F32, A=FAKE, B=FAKE2, acc=0, ct=F32,
           C=ctypes.c_void_p(0x70000000)):
    return L.isam_conv1d(nb, Ln, Ki, D, Ko, ab, A, B, acc, ct, C, None)


@pytest.mark.parametrize("kw,code", [
    ({"Ki": 0}, INVALID), ({"D": 0}, INVALID), ({"nb": -1}, INVALID), ({"Ko": -1}, INVALID),
    ({"ab": 2}, INVALID), ({"ct": 5}, INVALID), ({"acc": 2}, INVALID),
    ({"A": None}, INVALID), ({"C": None}, INVALID),
    ({"C": FAKE}, INVALID),                           # C overlaps A
    ({"nb": 70000, "Ln": 4, "Ki": 4, "D": 1, "Ko": 4}, UNSUPPORTED),
])
def test_conv1d_validation(L, kw, code):
    assert conv1d(L, **kw) == code


def test_conv1d_noops(L):
    assert conv1d(L, nb=0, A=None, B=None, C=None) == OK
    assert conv1d(L, Ko=0, A=None, B=None, C=None) == OK
    assert conv1d(L, Ln=2, D=3, A=None, B=None, C=None) == OK   # no valid position


def test_gru_noalloc_rejects_sizes_beyond_its_scratch(L):
    # T = 1024, batch 32, hidden 1024 needs ~410 MB of workspace, more than the 64 MiB static
    # scratch of the allocation-free entry point: rejected before any HIP call.
    need = L.isam_gru_forward_workspace_size(1024, 32, 1024, 1024, BF16)
    assert need > 64 << 20
    rc = L.isam_gru_forward_noalloc(1024, 32, 1024, 1024, BF16, FAKE, None, ctypes.c_void_p(0x30000),
                                    ctypes.c_void_p(0x50000), None, None, ctypes.c_void_p(0x700000000),
                                    None, None)
    assert rc == WORKSPACE
    assert b"static scratch" in L.isam_last_error()
    assert L.isam_gru_forward_workspace_size(64, 32, 1024, 1024, BF16) <= 64 << 20
