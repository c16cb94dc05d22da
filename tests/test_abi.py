"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function include/puro.h declares, and rejects invalid arguments with the
documented status before launching anything."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "puro.h")
LIB = os.path.join(ROOT, "paper_2608_27370_amd", "libpuro.so")

OK, ERR_NULL, ERR_SHAPE, ERR_UNSUPPORTED, ERR_ALIGN, ERR_WORKSPACE = 0, 1, 2, 3, 4, 5


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(puro_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def puro():
    if not os.path.exists(LIB):
        from paper_2608_27370_amd import build
        build.build()
    from paper_2608_27370_amd import puro as p
    return p


def test_header_declares_the_path():
    names = _declared()
    for n in ("puro_amax", "puro_quantize_fp8", "puro_fp8_gemm", "puro_linear_fwd", "puro_linear_bwd"):
        assert n in names


def test_library_exports_every_declared_function(puro):
    lib = ctypes.CDLL(puro.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing


def test_binding_covers_every_declared_function(puro):
    assert set(_declared()) == set(puro._SIGS)


def test_status_strings(puro):
    for code in range(7):
        assert puro.status_string(code)
    assert puro.status_string(0) == "ok"


FAKE = 0x10000   # a 16-byte aligned non-NULL address; validation fails before any use


def test_amax_validation(puro):
    L = puro.lib()
    assert L.puro_amax(None, 4, 16, 16, FAKE, FAKE, 1 << 20, None) == ERR_NULL
    assert L.puro_amax(FAKE, 4, 16, 8, FAKE, FAKE, 1 << 20, None) == ERR_SHAPE      # ld < cols
    assert L.puro_amax(FAKE, -1, 16, 16, FAKE, FAKE, 1 << 20, None) == ERR_SHAPE
    assert L.puro_amax(FAKE, 4, 12, 16, FAKE, FAKE, 1 << 20, None) == ERR_ALIGN     # cols % 8
    assert L.puro_amax(FAKE + 2, 4, 16, 16, FAKE, FAKE, 1 << 20, None) == ERR_ALIGN
    assert L.puro_amax(FAKE, 4, 16, 16, None, FAKE, 1 << 20, None) == ERR_NULL
    assert L.puro_amax(FAKE, 4096, 4096, 4096, FAKE, FAKE, 0, None) == ERR_WORKSPACE
    assert L.puro_amax_workspace_size(0, 16) == 0
    assert L.puro_amax_workspace_size(4096, 4096) > 0


def test_quantize_validation(puro):
    L = puro.lib()
    q = lambda *a: L.puro_quantize_fp8(*a)
    big = 1 << 20
    # bad format / rounding / mode
    assert q(FAKE, 128, 128, 128, 7, 0, 0, None, FAKE, FAKE, None, None, FAKE, big, None) == ERR_UNSUPPORTED
    assert q(FAKE, 128, 128, 128, 0, 0, 5, None, FAKE, FAKE, None, None, FAKE, big, None) == ERR_UNSUPPORTED
    assert q(FAKE, 128, 128, 128, 0, 9, 0, None, FAKE, FAKE, None, None, FAKE, big, None) == ERR_UNSUPPORTED
    # grouped modes require power-of-two scales and no supplied amax
    assert q(FAKE, 128, 128, 128, 0, 1, 0, None, FAKE, FAKE, None, None, None, 0, None) == ERR_UNSUPPORTED
    assert q(FAKE, 128, 128, 128, 0, 3, 1, FAKE, FAKE, FAKE, None, None, None, 0, None) == ERR_UNSUPPORTED
    # outputs missing
    assert q(FAKE, 128, 128, 128, 0, 0, 0, None, None, FAKE, None, None, FAKE, big, None) == ERR_NULL
    assert q(FAKE, 128, 128, 128, 0, 0, 0, None, FAKE, None, None, None, FAKE, big, None) == ERR_NULL
    assert q(FAKE, 128, 128, 128, 0, 2, 1, None, None, None, None, None, None, 0, None) == ERR_NULL
    # alignment of grouped dimensions and of the transposed copy
    assert q(FAKE, 128, 136, 136, 0, 1, 1, None, FAKE, FAKE, None, None, None, 0, None) == ERR_ALIGN
    assert q(FAKE, 120, 128, 128, 0, 2, 1, None, None, None, FAKE, FAKE, None, 0, None) == ERR_ALIGN
    assert q(FAKE, 120, 128, 128, 0, 3, 1, None, FAKE, FAKE, None, None, None, 0, None) == ERR_ALIGN
    assert q(FAKE, 24, 128, 128, 0, 0, 0, None, None, FAKE, FAKE, None, FAKE, big, None) == ERR_ALIGN
    assert q(FAKE, 16, 24, 24, 0, 0, 0, None, FAKE, FAKE, None, None, FAKE, big, None) == ERR_ALIGN
    # a row pitch whose 128-row tiles exceed 32-bit buffer offsets
    assert q(FAKE, 16, 128, 1 << 23, 0, 0, 0, None, FAKE, FAKE, None, None, FAKE, big, None) == ERR_SHAPE
    # per-tensor without workspace for the amax pass
    assert q(FAKE, 4096, 4096, 4096, 0, 0, 0, None, FAKE, FAKE, None, None, FAKE, 0, None) == ERR_WORKSPACE
    # the k-major layout flag belongs to the grouped modes
    KM = puro.SCALE_KMAJOR
    assert q(FAKE, 128, 128, 128, 0, 0 | KM, 0, None, FAKE, FAKE, None, None, FAKE, big, None) == ERR_UNSUPPORTED
    assert q(FAKE, 128, 136, 136, 0, 1 | KM, 1, None, FAKE, FAKE, None, None, None, 0, None) == ERR_ALIGN


def test_static_quantize_validation(puro):
    """The allocation-free quantise validates like puro_quantize_fp8 and
    returns before any HIP call (none is possible here: no GPU)."""
    L = puro.lib()
    q = lambda *a: L.puro_quantize_fp8_static(*a)
    assert q(FAKE, 128, 128, 128, 7, 0, 0, None, FAKE, FAKE, None, None, None) == ERR_UNSUPPORTED
    assert q(None, 128, 128, 128, 0, 0, 0, None, FAKE, FAKE, None, None, None) == ERR_NULL
    assert q(FAKE, 128, 128, 128, 0, 0, 0, None, None, None, None, None, None) == ERR_NULL
    assert q(FAKE, 16, 24, 24, 0, 0, 0, None, FAKE, FAKE, None, None, None) == ERR_ALIGN
    assert q(FAKE, 16, 128, 1 << 23, 0, 0, 0, None, FAKE, FAKE, None, None, None) == ERR_SHAPE
    assert q(FAKE, 128, 128, 128, 0, 1, 0, None, FAKE, FAKE, None, None, None) == ERR_UNSUPPORTED


def test_gemm_validation(puro):
    L = puro.lib()
    Op = puro.Operand
    good = Op(FAKE, 256, 0, 0, FAKE)
    byref = ctypes.byref

    def g(M, N, K, A, B, D=FAKE, dt=0, ldd=None, ws=FAKE, wsb=1 << 30):
        return L.puro_fp8_gemm(M, N, K, byref(A), byref(B), D, dt, N if ldd is None else ldd, 0, ws, wsb, None)

    assert g(-1, 16, 256, good, good) == ERR_SHAPE
    assert g(16, 16, 512, good, good) == ERR_SHAPE                      # ld < K
    assert g(16, 16, 250, Op(FAKE, 256, 0, 0, FAKE), good) == ERR_ALIGN  # K % 16
    assert g(16, 16, 256, Op(FAKE, 264, 0, 0, FAKE), good) == ERR_ALIGN  # ld % 16
    assert g(16, 16, 256, Op(FAKE, 256, 3, 0, FAKE), good) == ERR_UNSUPPORTED
    assert g(16, 16, 256, Op(FAKE, 256, 0, 2, FAKE), good) == ERR_UNSUPPORTED  # column mode is not a GEMM operand
    assert g(16, 16, 256, Op(None, 256, 0, 0, FAKE), good) == ERR_NULL
    assert g(16, 16, 256, Op(FAKE, 256, 0, 0, None), good) == ERR_NULL
    assert g(16, 16, 0, Op(FAKE, 0, 0, 0, None), good) == ERR_NULL       # scale is read even for K == 0
    assert g(16, 16, 208, Op(FAKE, 208, 0, 1, FAKE), Op(FAKE, 208, 0, 0, FAKE)) == ERR_ALIGN  # grouped needs K % 128
    KM = puro.SCALE_KMAJOR
    assert g(16, 16, 256, Op(FAKE, 256, 0, KM, FAKE), good) == ERR_UNSUPPORTED      # k-major: grouped modes only
    assert g(16, 16, 256, Op(FAKE, 256, 0, 2 | KM, FAKE), good) == ERR_UNSUPPORTED
    assert g(16, 16, 208, Op(FAKE, 208, 0, 1 | KM, FAKE), Op(FAKE, 208, 0, 3 | KM, FAKE)) == ERR_ALIGN
    assert puro.fp8_gemm_plan(4096, 4096, 4096, 1 | KM, 3 | KM)["launches"] == 1
    assert g(16, 16, 256, good, good, dt=4) == ERR_UNSUPPORTED
    assert g(16, 16, 256, good, good, ldd=8) == ERR_SHAPE
    assert g(16, 18, 256, good, good, ldd=18) == ERR_ALIGN
    assert g(16, 16, 256, good, good, D=None) == ERR_NULL
    assert g(16, 16, 256, good, good, D=FAKE + 4) == ERR_ALIGN
    # a split-K plan needs its workspace
    need = L.puro_fp8_gemm_workspace_size(128, 128, 8192, 1)
    assert need > 0
    big = Op(FAKE, 8192, 0, 0, FAKE)
    assert L.puro_fp8_gemm(128, 128, 8192, byref(big), byref(big), FAKE, 1, 128, 0, FAKE, need - 1, None) \
        == ERR_WORKSPACE
    assert L.puro_fp8_gemm(0, 128, 8192, byref(big), byref(big), FAKE, 1, 128, 0, None, 0, None) == OK


def test_linear_validation(puro):
    L = puro.lib()
    rc = puro.LinearRecipe().c()
    rb = puro.LinearRecipe(blockwise=1).c()
    bad = puro.LinearRecipe(x_fmt=9).c()
    s = puro.Saved(FAKE, FAKE, FAKE, FAKE)
    byref = ctypes.byref
    assert L.puro_linear_fwd(FAKE, FAKE, 256, 256, 256, byref(bad), FAKE, byref(s), FAKE, 1 << 30, None) \
        == ERR_UNSUPPORTED
    assert L.puro_linear_fwd(FAKE, FAKE, 250, 256, 256, byref(rc), FAKE, byref(s), FAKE, 1 << 30, None) \
        == ERR_ALIGN
    assert L.puro_linear_fwd(FAKE, FAKE, 256, 256, 144, byref(rb), FAKE, byref(s), FAKE, 1 << 30, None) \
        == ERR_ALIGN                                                       # blockwise needs 128
    assert L.puro_linear_fwd(None, FAKE, 256, 256, 256, byref(rc), FAKE, byref(s), FAKE, 1 << 30, None) \
        == ERR_NULL
    need = L.puro_linear_fwd_workspace_size(256, 256, 256, byref(rc))
    assert need > 0
    assert L.puro_linear_fwd(FAKE, FAKE, 256, 256, 256, byref(rc), FAKE, byref(s), FAKE, need - 1, None) \
        == ERR_WORKSPACE
    need = L.puro_linear_bwd_workspace_size(256, 256, 256, byref(rb))
    assert L.puro_linear_bwd(FAKE, byref(s), 256, 256, 256, byref(rb), FAKE, FAKE, 0, FAKE, need - 1, None) \
        == ERR_WORKSPACE
    # every dimension is an FP8 operand pitch of one of the GEMMs: above 2^22
    # the call fails before the quantisers run (with the NULL and FAKE buffers
    # here, anything enqueued would fault or fail to launch)
    big = (1 << 22) + 128
    for dims in ((256, 256, big), (256, big, 256), (big, 256, 256)):
        for r in (rc, rb):
            assert L.puro_linear_fwd(FAKE, FAKE, *dims, byref(r), FAKE, byref(s), FAKE, 1 << 62, None) == ERR_SHAPE
            assert L.puro_linear_bwd(FAKE, byref(s), *dims, byref(r), FAKE, FAKE, 0, FAKE, 1 << 62, None) \
                == ERR_SHAPE
            assert L.puro_linear_fwd_workspace_size(*dims, byref(r)) == 0
    sizes = (ctypes.c_size_t * 4)()
    total = L.puro_linear_saved_bytes(256, 512, 384, byref(rb), byref(sizes))
    assert list(sizes) == [384 * 256, 384 * 2 * 4, 384 * 512, 3 * 4 * 4] and total == sum(sizes)
    total = L.puro_linear_saved_bytes(256, 512, 384, byref(rc), byref(sizes))
    assert list(sizes) == [384 * 256, 4, 384 * 512, 4]


# Shapes on which the GEMM planner takes each of its kernel configurations
# (tile, ring depth) and the split-K path; tests/test_gpu_gemm.py runs them.
PLAN_SHAPES = {(256, 256, 2): (3072, 4096, 256), (256, 192, 2): (3072, 3072, 256),
               (128, 128, 4): (1024, 1024, 2048), (128, 128, 2): (1536, 3072, 256)}
SPLIT_SHAPES = [(256, 256, 1024), (768, 768, 4096)]   # split-K with the 2- and the 4-deep 128x128 tiles


@pytest.mark.parametrize("modes", [(0, 0), (1, 3)], ids=["tensor", "row-block"])
def test_gemm_plan_covers_every_configuration(puro, modes):
    for cfg, shape in PLAN_SHAPES.items():
        p = puro.fp8_gemm_plan(*shape, *modes)
        assert (p["tile_m"], p["tile_n"], p["stages"]) == cfg, (shape, p)
        assert p["splits"] == 1 and p["launches"] == 1
    for shape, stages in zip(SPLIT_SHAPES, (2, 4)):
        p = puro.fp8_gemm_plan(*shape, *modes)
        assert p["splits"] > 1 and p["launches"] == 2 and p["stages"] == stages, (shape, p)


def test_gemm_plan_validation(puro):
    L = puro.lib()
    assert L.puro_fp8_gemm_plan(-1, 16, 16, 0, 0, None, None, None, None, None) == ERR_SHAPE
    assert L.puro_fp8_gemm_plan(16, 16, 16, 2, 0, None, None, None, None, None) == ERR_UNSUPPORTED  # 128x1
    assert L.puro_fp8_gemm_plan(16, 16, 16, 0, 0, None, None, None, None, None) == OK
    assert puro.fp8_gemm_plan(0, 16, 16)["launches"] == 0


def test_swiglu_quantize_validation(puro):
    L = puro.lib()
    f = L.puro_swiglu_quantize_fp8
    big = 1 << 20
    # gu NULL, and a row pitch shorter than the two halves
    assert f(None, 16, 128, 256, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_NULL
    assert f(FAKE, 16, 128, 200, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_SHAPE
    assert f(FAKE, 16, -1, 256, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_SHAPE
    # cols % 16, misaligned gu
    assert f(FAKE, 16, 24, 48, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_ALIGN
    assert f(FAKE + 8, 16, 128, 256, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_ALIGN
    # 128x128 blocks are for weights, not for this activation
    assert f(FAKE, 128, 128, 256, 0, 3, 1, FAKE, FAKE, None, None, None, 0, None) == ERR_UNSUPPORTED
    # grouped modes need a power-of-two rule; 1x128 groups need cols % 128
    assert f(FAKE, 128, 128, 256, 0, 1, 0, FAKE, FAKE, None, None, None, 0, None) == ERR_UNSUPPORTED
    assert f(FAKE, 128, 144, 288, 0, 1, 1, FAKE, FAKE, None, None, None, 0, None) == ERR_ALIGN
    # per-tensor without workspace for the amax pass
    assert f(FAKE, 4096, 4096, 8192, 0, 0, 0, FAKE, FAKE, None, None, FAKE, 0, None) == ERR_WORKSPACE
    assert L.puro_swiglu_quantize_workspace_size(4096, 4096) == L.puro_quantize_workspace_size(4096, 4096)


def test_rmsnorm_quantize_validation(puro):
    L = puro.lib()
    f = L.puro_rmsnorm_quantize_fp8
    big = 1 << 20
    # x, gamma, rstd NULL
    assert f(None, FAKE, 16, 128, 128, 1e-6, 0, 0, 0, FAKE, FAKE, None, None, FAKE, FAKE, big, None) == ERR_NULL
    assert f(FAKE, None, 16, 128, 128, 1e-6, 0, 0, 0, FAKE, FAKE, None, None, FAKE, FAKE, big, None) == ERR_NULL
    assert f(FAKE, FAKE, 16, 128, 128, 1e-6, 0, 0, 0, FAKE, FAKE, None, None, None, FAKE, big, None) == ERR_NULL
    # misaligned gamma or rstd; cols % 16
    assert f(FAKE, FAKE + 4, 16, 128, 128, 1e-6, 0, 0, 0, FAKE, FAKE, None, None, FAKE, FAKE, big, None) == ERR_ALIGN
    assert f(FAKE, FAKE, 16, 128, 128, 1e-6, 0, 0, 0, FAKE, FAKE, None, None, FAKE + 4, FAKE, big, None) == ERR_ALIGN
    assert f(FAKE, FAKE, 16, 24, 24, 1e-6, 0, 0, 0, FAKE, FAKE, None, None, FAKE, FAKE, big, None) == ERR_ALIGN
    # eps negative or NaN; 128x128 blocks; a row without columns
    assert f(FAKE, FAKE, 16, 128, 128, -1.0, 0, 0, 0, FAKE, FAKE, None, None, FAKE, FAKE, big, None) == ERR_UNSUPPORTED
    assert f(FAKE, FAKE, 16, 128, 128, float("nan"), 0, 0, 0, FAKE, FAKE, None, None, FAKE, FAKE, big,
             None) == ERR_UNSUPPORTED
    assert f(FAKE, FAKE, 128, 128, 128, 1e-6, 0, 3, 1, FAKE, FAKE, None, None, FAKE, None, 0, None) == ERR_UNSUPPORTED
    assert f(FAKE, FAKE, 16, 0, 0, 1e-6, 0, 0, 0, FAKE, FAKE, None, None, FAKE, FAKE, big, None) == ERR_SHAPE
    # per-tensor without workspace
    assert f(FAKE, FAKE, 4096, 1536, 1536, 1e-6, 0, 0, 0, FAKE, FAKE, None, None, FAKE, FAKE, 0, None) == ERR_WORKSPACE
    assert L.puro_rmsnorm_quantize_workspace_size(8192, 1536) >= 2048 * 4 + 4


def test_swiglu_bwd_quantize_validation(puro):
    L = puro.lib()
    f = L.puro_swiglu_bwd_quantize_fp8
    big = 1 << 20
    # dH or gu NULL; gu's pitch shorter than its two halves
    assert f(None, 128, FAKE, 256, 16, 128, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_NULL
    assert f(FAKE, 128, None, 256, 16, 128, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_NULL
    assert f(FAKE, 128, FAKE, 200, 16, 128, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_SHAPE
    # cols % 8, misaligned gu
    assert f(FAKE, 12, FAKE, 24, 16, 12, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_ALIGN
    assert f(FAKE, 128, FAKE + 8, 256, 16, 128, 0, 0, 0, FAKE, FAKE, None, None, FAKE, big, None) == ERR_ALIGN
    # 128x128 blocks; 1x128 groups need 2 cols % 128
    assert f(FAKE, 128, FAKE, 256, 128, 128, 0, 3, 1, FAKE, FAKE, None, None, None, 0, None) == ERR_UNSUPPORTED
    assert f(FAKE, 96, FAKE, 192, 128, 96, 0, 1, 1, FAKE, FAKE, None, None, None, 0, None) == ERR_ALIGN
    # per-tensor without workspace
    assert f(FAKE, 4096, FAKE, 8192, 4096, 4096, 0, 0, 0, FAKE, FAKE, None, None, FAKE, 0, None) == ERR_WORKSPACE


def test_gemm_epilogue_validation(puro):
    L = puro.lib()
    f = L.puro_fp8_gemm_epilogue
    good = puro.Operand(FAKE, 256, 0, 0, FAKE)
    big = 1 << 30
    g = lambda *a: f(*a)
    # misaligned bias / residual, a residual pitch below N or not a multiple of 4
    assert g(16, 16, 256, good, good, FAKE, 16, FAKE + 2, None, 0, FAKE, big, None) == ERR_ALIGN
    assert g(16, 16, 256, good, good, FAKE, 16, None, FAKE + 0x10000 + 8, 16, FAKE, big, None) == ERR_ALIGN
    assert g(16, 16, 256, good, good, FAKE, 16, None, FAKE + 0x10000, 8, FAKE, big, None) == ERR_SHAPE
    assert g(16, 16, 256, good, good, FAKE, 16, None, FAKE + 0x10000, 18, FAKE, big, None) == ERR_ALIGN
    # a residual pitch beyond the operands' limit, 2^22
    assert g(16, 16, 256, good, good, FAKE, 16, None, FAKE + 0x10000, (1 << 22) + 4, FAKE, big, None) == ERR_SHAPE
    # a residual overlapping D without being D, and D itself with another pitch
    assert g(16, 16, 256, good, good, FAKE, 16, None, FAKE + 64, 16, FAKE, big, None) == ERR_SHAPE
    assert g(16, 16, 256, good, good, FAKE, 16, None, FAKE, 32, FAKE, big, None) == ERR_SHAPE


def test_lm_head_validation(puro):
    L = puro.lib()
    big = 1 << 40
    fwd = lambda M, V, K, r=0, X=FAKE, W=FAKE, t=FAKE, lse=FAKE, loss=FAKE, ws=FAKE, nb=big: L.puro_lm_head_ce_fwd(
        X, W, t, M, V, K, r, lse, loss, ws, nb, None)
    assert fwd(128, 256, 128, r=2) == ERR_UNSUPPORTED
    assert fwd(0, 256, 128) == ERR_SHAPE
    assert fwd(128, (1 << 21) + 128, 128) == ERR_SHAPE
    assert fwd(128, 200, 128) == ERR_ALIGN
    assert fwd(128, 256, 128, X=None) == ERR_NULL
    assert fwd(128, 256, 128, t=FAKE + 2) == ERR_ALIGN
    assert fwd(128, 256, 128, loss=None) == ERR_NULL
    assert fwd(128, 256, 128, nb=16) == ERR_WORKSPACE
    need = L.puro_lm_head_ce_workspace_size(128, 256, 128, 1, 1)
    assert need > L.puro_lm_head_ce_workspace_size(128, 256, 128, 1, 0) > 0
    assert L.puro_lm_head_ce_workspace_size(128, 200, 128, 0, 0) == 0
    bwd = lambda g=1.0, dX=FAKE, nb=big: L.puro_lm_head_ce_bwd(FAKE, FAKE, FAKE, FAKE, 128, 256, 128, 1, g, dX, FAKE,
                                                               FAKE, nb, None)
    assert bwd(g=float("nan")) == ERR_UNSUPPORTED
    assert bwd(g=float("inf")) == ERR_UNSUPPORTED
    assert bwd(dX=None) == ERR_NULL
    assert bwd(nb=need - 1) == ERR_WORKSPACE


def test_muonh_validation(puro):
    L = puro.lib()
    big = 1 << 40
    step = lambda cnt=2, rows=256, cols=384, W=FAKE, wb=None, G=FAKE, buf=FAKE, R=FAKE, mu=0.95, eta=0.01, st=5, \
        u=None, ws=FAKE, nb=big: L.puro_muonh_step(cnt, rows, cols, W, wb, G, buf, R, mu, 1, eta, st, u, ws, nb, None)
    assert step(cnt=0) == ERR_SHAPE
    assert step(cnt=65536) == ERR_SHAPE
    assert step(rows=(1 << 21) + 128) == ERR_SHAPE
    assert step(cols=200) == ERR_ALIGN
    assert step(G=None) == ERR_NULL
    assert step(R=None) == ERR_NULL
    assert step(W=FAKE + 8) == ERR_ALIGN
    assert step(wb=FAKE + 8) == ERR_ALIGN
    assert step(R=FAKE + 2) == ERR_ALIGN
    assert step(mu=float("nan")) == ERR_UNSUPPORTED
    assert step(eta=float("inf")) == ERR_UNSUPPORTED
    assert step(st=-1) == ERR_UNSUPPORTED
    need = L.puro_muonh_workspace_size(2, 256, 384)
    assert need > 0 and L.puro_muonh_workspace_size(2, 384, 256) == need
    assert step(nb=need - 1) == ERR_WORKSPACE
    ns = lambda cnt=1, r=128, c=256, X=FAKE, steps=5, out=FAKE, nb=big: L.puro_newton_schulz_bf16(
        cnt, r, c, X, steps, out, FAKE, nb, None)
    assert ns(r=256, c=128) == ERR_SHAPE
    assert ns(X=None) == ERR_NULL
    assert ns(out=FAKE + 4) == ERR_ALIGN
    assert ns(steps=65) == ERR_UNSUPPORTED
    assert L.puro_newton_schulz_workspace_size(1, 256, 128) == 0
    assert ns(nb=L.puro_newton_schulz_workspace_size(1, 128, 256) - 1) == ERR_WORKSPACE
