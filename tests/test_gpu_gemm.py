"""GPU parity of the scaled FP8 GEMM against the oracle's FP64 GEMM.

Operands are quantised by the oracle from seeded BF16 data and uploaded, so
these tests isolate the GEMM kernels. FP32 outputs must satisfy
|d - ref| <= 1e-5 * sum_k |a_k b_k|; BF16 outputs must be the BF16 rounding
of a value within that tolerance."""

import numpy as np
import pytest

from oracle import bf16, fp8, gemm, quant
from paper_2608_27370_amd import inputs

import mfma_model
from gpu_util import bf16_bits, check_bf16, check_fp32, host, to_dev, to_dev_bf16

pytestmark = pytest.mark.gpu

E4, E5 = 0, 1
OFMT = {E4: fp8.E4M3, E5: fp8.E5M2}
MODE = {"tensor": 0, "row": 1, "block": 3}


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


def _operand_tensor(seed, rows, K, fmt, std=1.0, kind="normal"):
    x = inputs.case(seed, (rows, K), std=std, kind=kind)
    q, _, s, _ = quant.quantize_tensor(x, OFMT[fmt])
    return q, s


def _operand_grouped(seed, rows, K, fmt, mode, std=1.0, kind="normal"):
    x = inputs.case(seed, (rows, K), std=std, kind=kind)
    if mode == "row":
        return quant.quantize_rows_1x128(x, OFMT[fmt])
    pad = (-rows) % 128                            # blocks over a ragged row count
    xp = np.concatenate([x, np.zeros((pad, K), np.uint16)]) if pad else x
    q, s, _, _ = quant.quantize_blocks_128x128(xp, OFMT[fmt])
    return q[:rows], s


def _run(P, a, fa, sa, am, b, fb, sb, bm, out, D0=None, ld_pad=0):
    M, K = a.shape
    N = b.shape[0]
    if ld_pad:
        a = np.concatenate([a, np.full((M, ld_pad), 0x3F, np.uint8)], axis=1)   # junk beyond K
        b = np.concatenate([b, np.full((N, ld_pad), 0x5A, np.uint8)], axis=1)
    da, db = to_dev(a), to_dev(b)
    dsa, dsb = to_dev(np.atleast_1d(np.asarray(sa, np.float32))), to_dev(np.atleast_1d(np.asarray(sb, np.float32)))
    A = P.operand(da[:, :K] if ld_pad else da, fa, MODE[am], dsa)
    B = P.operand(db[:, :K] if ld_pad else db, fb, MODE[bm], dsb)
    D = None if D0 is None else to_dev(D0)
    return P.fp8_gemm(A, M, B, N, K, out, D=D, accumulate=D0 is not None)


def _check(P, out, D, ref, den, what, op):
    """op: the oracle GEMM arguments, for the instruction-truncation allowance."""
    slack = mfma_model.truncation_loss_full(*op)
    if out == P.OUT_FP32:
        check_fp32(host(D), ref, den, what=what, slack=slack)
    else:
        check_bf16(bf16_bits(D), ref, den, what=what, slack=slack)


SHAPES = [(300, 520, 384), (256, 256, 1536), (64, 32, 16), (1, 4, 16), (200, 136, 208), (513, 260, 1040),
          (1024, 2048, 256)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("out", [0, 1], ids=["bf16", "fp32"])
def test_gemm_tensor_scales(P, shape, out):
    M, N, K = shape
    a, sa = _operand_tensor(1, M, K, E4)
    b, sb = _operand_tensor(2, N, K, E4, std=0.02)
    D = _run(P, a, E4, sa, "tensor", b, E4, sb, "tensor", out)
    op = (a, fp8.E4M3, sa, "tensor", b, fp8.E4M3, sb, "tensor")
    ref, den = gemm.gemm(*op)
    _check(P, out, D, ref, den, "tensor %s" % (shape,), op)


@pytest.mark.parametrize("fa,fb", [(E5, E4), (E4, E5), (E5, E5)])
def test_gemm_formats(P, fa, fb):
    M, N, K = 384, 264, 640
    a, sa = _operand_tensor(3, M, K, fa, std=1e-3)
    b, sb = _operand_tensor(4, N, K, fb, kind="student_t")
    for out in (0, 1):
        D = _run(P, a, fa, sa, "tensor", b, fb, sb, "tensor", out)
        op = (a, OFMT[fa], sa, "tensor", b, OFMT[fb], sb, "tensor")
        ref, den = gemm.gemm(*op)
        _check(P, out, D, ref, den, "formats %d %d" % (fa, fb), op)


@pytest.mark.parametrize("shape", [(128, 128, 8192), (64, 2048, 4096), (256, 96, 2048)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("out", [0, 1], ids=["bf16", "fp32"])
def test_gemm_split_k(P, shape, out):
    M, N, K = shape
    assert P.fp8_gemm_workspace_size(M, N, K, out) > 0          # the split path is taken
    a, sa = _operand_tensor(5, M, K, E5, std=1e-3)
    b, sb = _operand_tensor(6, N, K, E4)
    D = _run(P, a, E5, sa, "tensor", b, E4, sb, "tensor", out)
    op = (a, fp8.E5M2, sa, "tensor", b, fp8.E4M3, sb, "tensor")
    ref, den = gemm.gemm(*op)
    _check(P, out, D, ref, den, "split-k %s" % (shape,), op)


@pytest.mark.parametrize("out", [0, 1], ids=["bf16", "fp32"])
@pytest.mark.parametrize("shape", [(256, 384, 512), (96, 64, 4096)], ids=lambda s: "x".join(map(str, s)))
def test_gemm_accumulate(P, out, shape):
    M, N, K = shape
    a, sa = _operand_tensor(7, M, K, E4)
    b, sb = _operand_tensor(8, N, K, E4)
    g = np.random.default_rng(3)
    D0f = g.standard_normal((M, N)).astype(np.float32)
    if out == P.OUT_FP32:
        D0 = D0f
        old = D0f.astype(np.float64)
    else:
        D0 = inputs.bf16_from_f64(D0f).view(np.int16)
        old = bf16.to_f32(D0.view(np.uint16)).astype(np.float64)
    import torch
    D = _run(P, a, E4, sa, "tensor", b, E4, sb, "tensor", out, D0=D0)
    if out == P.OUT_BF16:
        D = D.view(torch.bfloat16) if D.dtype != torch.bfloat16 else D
    op = (a, fp8.E4M3, sa, "tensor", b, fp8.E4M3, sb, "tensor")
    ref, den = gemm.gemm(*op)
    # the old value enters the FP32 sum exactly; its own rounding adds |old| * 2**-24
    _check(P, out, D, ref + old, den + np.abs(old) * 2.0 ** -24 / 1e-5, "accumulate", op)


@pytest.mark.parametrize("am,bm", [("row", "block"), ("row", "row"), ("tensor", "block"), ("row", "tensor")])
@pytest.mark.parametrize("shape", [(256, 384, 512), (300, 260, 384), (128, 128, 128)],
                         ids=lambda s: "x".join(map(str, s)))
def test_gemm_grouped_scales(P, am, bm, shape):
    M, N, K = shape
    if am == "tensor":
        a, sa = _operand_tensor(9, M, K, E4)
    else:
        a, sa = _operand_grouped(9, M, K, E4, am, kind="outliers")
    if bm == "tensor":
        b, sb = _operand_tensor(10, N, K, E4, std=0.02)
    else:
        b, sb = _operand_grouped(10, N, K, E4, bm, std=0.02)
    for out in (0, 1):
        D = _run(P, a, E4, sa, am, b, E4, sb, bm, out)
        op = (a, fp8.E4M3, sa, am, b, fp8.E4M3, sb, bm)
        ref, den = gemm.gemm(*op)
        _check(P, out, D, ref, den, "grouped %s/%s %s" % (am, bm, shape), op)


def test_gemm_grouped_split_k(P):
    """Wgrad form (row scales on both operands) with a long reduction."""
    M, N, K = 128, 256, 8192
    a, sa = _operand_grouped(11, M, K, E5, "row", std=1e-3)
    b, sb = _operand_grouped(12, N, K, E4, "row")
    assert P.fp8_gemm_workspace_size(M, N, K, 1) > 0
    D = _run(P, a, E5, sa, "row", b, E4, sb, "row", 1)
    op = (a, fp8.E5M2, sa, "row", b, fp8.E4M3, sb, "row")
    ref, den = gemm.gemm(*op)
    check_fp32(host(D), ref, den, what="grouped split-k", slack=mfma_model.truncation_loss_full(*op))


def test_gemm_padded_leading_dimension(P):
    M, N, K = 200, 132, 256
    a, sa = _operand_tensor(13, M, K, E4)
    b, sb = _operand_tensor(14, N, K, E4)
    D = _run(P, a, E4, sa, "tensor", b, E4, sb, "tensor", 1, ld_pad=32)
    op = (a, fp8.E4M3, sa, "tensor", b, fp8.E4M3, sb, "tensor")
    ref, den = gemm.gemm(*op)
    check_fp32(host(D), ref, den, what="padded ld", slack=mfma_model.truncation_loss_full(*op))


def test_gemm_empty_reduction(P):
    import torch
    a = np.zeros((64, 0), np.uint8)
    b = np.zeros((32, 0), np.uint8)
    da = torch.empty(64, 16, dtype=torch.uint8, device="cuda")[:, :0]
    db = torch.empty(32, 16, dtype=torch.uint8, device="cuda")[:, :0]
    s = to_dev(np.array([2.0], np.float32))
    A = P.operand(da, E4, 0, s)
    B = P.operand(db, E4, 0, s)
    D = P.fp8_gemm(A, 64, B, 32, 0, P.OUT_FP32)
    assert float(D.abs().max()) == 0.0
    D0 = torch.full((64, 32), 3.0, dtype=torch.float32, device="cuda")
    D = P.fp8_gemm(A, 64, B, 32, 0, P.OUT_FP32, D=D0, accumulate=True)
    assert float((D - 3.0).abs().max()) == 0.0
    del a, b


def test_gemm_is_deterministic(P):
    M, N, K = 128, 256, 8192      # split-K path
    a, sa = _operand_tensor(15, M, K, E4)
    b, sb = _operand_tensor(16, N, K, E4)
    D1 = host(_run(P, a, E4, sa, "tensor", b, E4, sb, "tensor", 1))
    D2 = host(_run(P, a, E4, sa, "tensor", b, E4, sb, "tensor", 1))
    assert np.array_equal(D1.view(np.uint32), D2.view(np.uint32))


# One shape per kernel configuration of the planner (tile, ring depth) and two
# that take the split-K path (with the 2- and the 4-deep 128x128 tiles, the
# latter with producer waves); tests/test_abi.py checks that the planner maps
# them so. Outputs are compared on stratified samples plus the whole first and
# last 256x256 tiles.
PLAN_CASES = [(3072, 4096, 256), (3072, 3072, 256), (1024, 1024, 2048), (1536, 3072, 256), (256, 256, 1024),
              (768, 768, 4096)]


@pytest.mark.parametrize("shape", PLAN_CASES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("scales", ["tensor", "row-block"])
def test_gemm_every_configuration(P, shape, scales):
    from gpu_util import sample_entries
    M, N, K = shape
    if scales == "tensor":
        a, sa = _operand_tensor(21, M, K, E5, std=1e-3)
        b, sb = _operand_tensor(22, N, K, E4, std=0.02)
        am, bm = "tensor", "tensor"
    else:
        a, sa = _operand_grouped(21, M, K, E5, "row", std=1e-3)
        b, sb = _operand_grouped(22, N, K, E4, "block", std=0.02)
        am, bm = "row", "block"
    plan = P.fp8_gemm_plan(M, N, K, MODE[am], MODE[bm])
    op = (a, fp8.E5M2, sa, am, b, fp8.E4M3, sb, bm)
    ms, ns = sample_entries(M, N, np.random.default_rng(M + N + K))
    ref, den = gemm.gemm_entries(ms, ns, *op)
    slack = mfma_model.truncation_loss(ms, ns, *op)
    for out in (0, 1):
        D = _run(P, a, E5, sa, am, b, E4, sb, bm, out)
        what = "%s %s plan %s out %d" % (scales, shape, plan, out)
        if out == 1:
            check_fp32(host(D)[ms, ns], ref, den, what=what, slack=slack)
        else:
            check_bf16(bf16_bits(D)[ms, ns], ref, den, what=what, slack=slack)


@pytest.mark.parametrize("shape", [(3072, 3072, 256), (6144, 1344, 256)], ids=lambda s: "x".join(map(str, s)))
def test_gemm_block_scales_change_between_blocks(P, shape):
    """Block-scaled B whose 128-row blocks all get different power-of-two
    scales (rows of block b scaled by 2^(b mod 7)), on shapes planned with
    192-wide tiles whose rows straddle block boundaries."""
    from gpu_util import sample_entries
    M, N, K = shape
    a, sa = _operand_grouped(23, M, K, E4, "row")
    x = inputs.case(24, (N, K), std=0.02)
    mult = np.repeat(2.0 ** (np.arange((N + 127) // 128) % 7), 128)[:N]
    xb = bf16.from_f64_rne(bf16.to_f32(x).astype(np.float64) * mult[:, None])
    pad = (-N) % 128                               # blocks over a ragged row count
    xp = np.concatenate([xb, np.zeros((pad, K), np.uint16)]) if pad else xb
    b, sb, _, _ = quant.quantize_blocks_128x128(xp, fp8.E4M3)
    b = b[:N]
    assert len(np.unique(sb[:, 0])) > 1
    op = (a, fp8.E4M3, sa, "row", b, fp8.E4M3, sb, "block")
    ms, ns = sample_entries(M, N, np.random.default_rng(5))
    ref, den = gemm.gemm_entries(ms, ns, *op)
    slack = mfma_model.truncation_loss(ms, ns, *op)
    for out in (0, 1):
        D = _run(P, a, E4, sa, "row", b, E4, sb, "block", out)
        what = "block-scale boundaries %s plan %s out %d" % (shape, P.fp8_gemm_plan(M, N, K, 1, 3), out)
        if out == 1:
            check_fp32(host(D)[ms, ns], ref, den, what=what, slack=slack)
        else:
            check_bf16(bf16_bits(D)[ms, ns], ref, den, what=what, slack=slack)


def _epilogue_terms(seed, M, N, bias, residual):
    rng = np.random.default_rng(seed)
    b = inputs.bf16_from_f64(0.5 * rng.standard_normal(N)) if bias else None
    r = inputs.bf16_from_f64(rng.standard_normal((M, N))) if residual else None
    return b, r


def _run_epi(P, a, fa, sa, am, b, fb, sb, bm, bias, resid, ld_pad=0, in_place=False):
    M, K = a.shape
    N = b.shape[0]
    da, db = to_dev(a), to_dev(b)
    dsa, dsb = to_dev(np.atleast_1d(np.asarray(sa, np.float32))), to_dev(np.atleast_1d(np.asarray(sb, np.float32)))
    A = P.operand(da, fa, MODE[am], dsa)
    B = P.operand(db, fb, MODE[bm], dsb)
    import torch
    D = torch.empty(M, N + ld_pad, dtype=torch.bfloat16, device="cuda")[:, :N]
    dbias = to_dev_bf16(bias) if bias is not None else None
    if in_place:
        D.view(torch.int16).copy_(to_dev(resid.view(np.int16)))
        dres = D
    elif resid is not None:
        # the residual with the same row pitch as D
        dres = to_dev_bf16(np.pad(resid, ((0, 0), (0, ld_pad))))[:, :N]
    else:
        dres = None
    return P.fp8_gemm_epilogue(A, M, B, N, K, bias=dbias, residual=dres, D=D)


EPI_SHAPES = [(300, 520, 384), (200, 258, 208), (256, 256, 1024), (513, 260, 1040)]


@pytest.mark.parametrize("shape", EPI_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("terms", ["bias", "residual", "both", "in_place"])
def test_gemm_epilogue(P, shape, terms):
    """D = BF16(A B^T + bias + residual): every entry within the BF16 band
    of the oracle's exact value (oracle/gemm.py's epilogue); ragged N, a
    split-K shape (whose reduction kernel applies the epilogue), and the
    residual being D itself."""
    M, N, K = shape
    a, sa = _operand_tensor(31, M, K, E4)
    b, sb = _operand_tensor(32, N, K, E4, std=0.02)
    bias, resid = _epilogue_terms(M + N, M, N, terms in ("bias", "both", "in_place"), terms != "bias")
    D = _run_epi(P, a, E4, sa, "tensor", b, E4, sb, "tensor", bias, resid, ld_pad=(-N) % 4 + 4 * (N % 4 != 0),
                 in_place=terms == "in_place")
    op = (a, fp8.E4M3, sa, "tensor", b, fp8.E4M3, sb, "tensor")
    ref, den = gemm.gemm(*op)
    ref, den = gemm.epilogue(ref, den, None if bias is None else bf16.to_f32(bias)[None, :],
                             None if resid is None else bf16.to_f32(resid))
    check_bf16(bf16_bits(D), ref, den, what="epilogue %s %s plan %s" % (terms, shape, P.fp8_gemm_plan(M, N, K)),
               slack=mfma_model.truncation_loss_full(*op))


# The epilogue on the tile configurations the shapes above do not reach:
# 256x256 (the one-pass BF16 staging, whose residual block arrives in LDS by
# DMA before the tile's stores: here in place on D), 256x192 (bias repeating
# with period 3 over a lane's store iterations), and 128x128 with a 4-deep
# ring and producer waves, alone and split over K.
EPI_TILE_CASES = [
    # (M, N, K, tile_m, tile_n, stages, splits, in_place, full_tiles)
    (4096, 4096, 512, 256, 256, 2, 1, True, True),
    (8192, 1536, 1536, 256, 192, 2, 1, True, True),
    (2048, 1536, 2048, 128, 128, 4, 1, False, True),
    (1024, 768, 8192, 128, 128, 4, 4, True, False),
]


@pytest.mark.parametrize("case", EPI_TILE_CASES, ids=lambda c: "x".join(map(str, c[:3])))
def test_gemm_epilogue_tile_configs(P, case):
    """Bias plus residual (in place on D where marked) on sampled entries:
    16 in every 256x256 block, plus the whole first and last blocks where
    marked."""
    from gpu_util import sample_entries
    M, N, K, tm, tn, st, sp, in_place, full = case
    plan = P.fp8_gemm_plan(M, N, K)
    assert (plan["tile_m"], plan["tile_n"], plan["stages"], plan["splits"]) == (tm, tn, st, sp), plan
    a, sa = _operand_tensor(41, M, K, E4)
    b, sb = _operand_tensor(42, N, K, E4, std=0.02)
    bias, resid = _epilogue_terms(43, M, N, True, True)
    D = _run_epi(P, a, E4, sa, "tensor", b, E4, sb, "tensor", bias, resid, in_place=in_place)
    ms, ns = sample_entries(M, N, np.random.default_rng(44), per_tile=16 if full else 64, full_tiles=full)
    op = (a, fp8.E4M3, sa, "tensor", b, fp8.E4M3, sb, "tensor")
    ref, den = gemm.gemm_entries(ms, ns, *op)
    ref, den = gemm.epilogue(ref, den, bf16.to_f32(bias)[ns], bf16.to_f32(resid)[ms, ns])
    check_bf16(bf16_bits(D)[ms, ns], ref, den, what="epilogue %s plan %s" % (case[:3], plan),
               slack=mfma_model.truncation_loss(ms, ns, *op))


def test_gemm_epilogue_block_scales(P):
    M, N, K = 256, 384, 512
    a, sa = _operand_grouped(33, M, K, E4, "row")
    b, sb = _operand_grouped(34, N, K, E4, "block", std=0.02)
    bias, resid = _epilogue_terms(5, M, N, True, True)
    D = _run_epi(P, a, E4, sa, "row", b, E4, sb, "block", bias, resid)
    op = (a, fp8.E4M3, sa, "row", b, fp8.E4M3, sb, "block")
    ref, den = gemm.gemm(*op)
    ref, den = gemm.epilogue(ref, den, bf16.to_f32(bias)[None, :], bf16.to_f32(resid))
    check_bf16(bf16_bits(D), ref, den, what="epilogue block scales", slack=mfma_model.truncation_loss_full(*op))


def test_gemm_epilogue_qkv_bias_full_size(P):
    """The Qwen2-1.5B QKV projection with its bias, 8192 x 2048 x 1536, in the
    bench's launch configuration; 16 entries in every 256x256 tile plus the
    whole first and last tiles."""
    from gpu_util import sample_entries
    d = inputs.qkv()
    xq, _, sx, _ = quant.quantize_tensor(d["X"], fp8.E4M3)
    wq, _, sw, _ = quant.quantize_tensor(d["W"], fp8.E4M3)
    M, N, K = 8192, inputs.QKV_OUT, inputs.HIDDEN
    bias, _ = _epilogue_terms(6, M, N, True, False)
    D = _run_epi(P, xq, E4, sx, "tensor", wq, E4, sw, "tensor", bias, None)
    ms, ns = sample_entries(M, N, np.random.default_rng(13))
    op = (xq, fp8.E4M3, sx, "tensor", wq, fp8.E4M3, sw, "tensor")
    ref, den = gemm.gemm_entries(ms, ns, *op)
    ref, den = gemm.epilogue(ref, den, bf16.to_f32(bias)[ns])
    check_bf16(bf16_bits(D)[ms, ns], ref, den, what="QKV + bias", slack=mfma_model.truncation_loss(ms, ns, *op))


@pytest.mark.parametrize("am,bm", [("row", "block"), ("row", "row")])
@pytest.mark.parametrize("shape", [(384, 264, 512), (256, 392, 1024)], ids=lambda s: "x".join(map(str, s)))
def test_gemm_kmajor_scales(P, am, bm, shape):
    """The k-block-major scale layout (PURO_SCALE_KMAJOR) is only a layout:
    the same operands with their scale arrays transposed give bitwise the
    same output, which matches the oracle."""
    import torch
    M, N, K = shape
    a, sa = _operand_grouped(31, M, K, E4, am, kind="outliers")
    b, sb = _operand_grouped(32, N, K, E4, bm, std=0.02)
    da, db = to_dev(a), to_dev(b)
    for out in (0, 1):
        rm = P.fp8_gemm(P.operand(da, E4, MODE[am], to_dev(sa)), M, P.operand(db, E4, MODE[bm], to_dev(sb)), N, K,
                        out)
        km = P.fp8_gemm(P.operand(da, E4, MODE[am] | P.SCALE_KMAJOR, to_dev(np.ascontiguousarray(sa.T))), M,
                        P.operand(db, E4, MODE[bm] | P.SCALE_KMAJOR, to_dev(np.ascontiguousarray(sb.T))), N, K, out)
        torch.cuda.synchronize()
        assert torch.equal(rm.view(torch.int16) if out == 0 else rm.view(torch.int32),
                           km.view(torch.int16) if out == 0 else km.view(torch.int32))
        op = (a, fp8.E4M3, sa, am, b, fp8.E4M3, sb, bm)
        ref, den = gemm.gemm(*op)
        _check(P, out, km, ref, den, "k-major %s/%s %s" % (am, bm, shape), op)
