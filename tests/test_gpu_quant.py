"""GPU parity of amax and the FP8 quantisers against the oracle: bytes and
scales bit-exact (through the C ABI via the ctypes binding)."""

import numpy as np
import pytest

from oracle import bf16, fp8, quant
from paper_2608_27370_amd import inputs

from gpu_util import (assert_bytes_equal, assert_f32_bits_equal, host, to_dev, to_dev_bf16)

pytestmark = pytest.mark.gpu

E4, E5 = 0, 1
OFMT = {E4: fp8.E4M3, E5: fp8.E5M2}
RULE = {0: "fp32", 1: "pow2", 2: "pow2_floor"}      # puro_scale_rounding -> oracle rule


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


def _special_tensor(shape, seed):
    x = inputs.case(seed, shape, kind="student_t")
    return x


@pytest.mark.parametrize("shape", [(1, 8), (300, 400), (4096, 1536), (257, 8), (0, 16)])
def test_amax(P, shape):
    x = inputs.case(10, shape, kind="student_t") if shape[0] else np.zeros(shape, np.uint16)
    got = host(P.amax(to_dev_bf16(x)))[0]
    want = quant.amax(bf16.to_f32(x))
    assert_f32_bits_equal(np.array([got]), np.array([want]), "amax %s" % (shape,))


def test_amax_strided_and_specials(P):
    x = inputs.case(11, (64, 256))
    d = to_dev_bf16(x)[:, 16:144]             # ld 256, 128 columns
    got = host(P.amax(d))[0]
    assert got == quant.amax(bf16.to_f32(x[:, 16:144]))
    y = np.zeros((32, 64), np.uint16) | np.uint16(0x8000)   # all -0
    assert host(P.amax(to_dev_bf16(y)))[0] == 0.0
    y[3, 5] = 0xFF80                                        # -inf
    assert np.isinf(host(P.amax(to_dev_bf16(y)))[0])
    y[7, 9] = 0x7FC1                                        # NaN
    assert np.isnan(host(P.amax(to_dev_bf16(y)))[0])


@pytest.mark.parametrize("fmt", [E4, E5])
@pytest.mark.parametrize("rnd", [0, 1, 2])
@pytest.mark.parametrize("shape", [(304, 400), (16, 16), (128, 1536), (1040, 2064)])
def test_quantize_tensor(P, fmt, rnd, shape):
    x = inputs.case(12, shape, kind="outliers")
    r = P.quantize_fp8(to_dev_bf16(x), fmt, P.SCALE_TENSOR, rnd, want_q=True, want_qT=True)
    q, qT, s, _ = quant.quantize_tensor(x, OFMT[fmt], rule=RULE[rnd])
    assert_f32_bits_equal(host(r["scale"]), np.array([s]), "scale")
    assert_bytes_equal(host(r["q"]), q, "q")
    assert_bytes_equal(host(r["qT"]), qT, "qT")


@pytest.mark.parametrize("fmt", [E4, E5])
@pytest.mark.parametrize("rnd", [0, 1, 2])
@pytest.mark.parametrize("amax_in", [448.0, 1.0, 3.0, 57344.0, 1e-30, 2e-36, 3.0e38, 0.0, 15.0])
def test_quantize_every_bf16_pattern_with_supplied_amax(P, fmt, rnd, amax_in):
    """All 65536 BF16 patterns (NaN, Inf, subnormals included) through the
    saturating path: exercises the whole codec on the device."""
    x = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(256, 256)
    a = to_dev(np.array([amax_in], np.float32))
    r = P.quantize_fp8(to_dev_bf16(x), fmt, P.SCALE_TENSOR, rnd, amax_in=a, want_q=True, want_qT=True)
    q, qT, s, _ = quant.quantize_tensor(x, OFMT[fmt], amax_in=np.float32(amax_in), rule=RULE[rnd])
    assert_f32_bits_equal(host(r["scale"]), np.array([s]), "scale")
    assert_bytes_equal(host(r["q"]), q, "q")
    assert_bytes_equal(host(r["qT"]), qT, "qT")


@pytest.mark.parametrize("fmt", [E4, E5])
def test_quantize_tensor_nonfinite(P, fmt):
    x = inputs.case(13, (64, 128))
    for special in (0x7F80, 0xFF80, 0x7FC0):
        y = x.copy()
        y[5, 7] = special
        for rnd in (0, 1, 2):
            r = P.quantize_fp8(to_dev_bf16(y), fmt, P.SCALE_TENSOR, rnd, want_q=True, want_qT=True)
            q, qT, s, _ = quant.quantize_tensor(y, OFMT[fmt], rule=RULE[rnd])
            assert_f32_bits_equal(host(r["scale"]), np.array([s]), "scale %#x" % special)
            assert_bytes_equal(host(r["q"]), q, "q %#x" % special)
            assert_bytes_equal(host(r["qT"]), qT, "qT %#x" % special)


def test_quantize_tensor_empty(P):
    x = np.zeros((0, 64), np.uint16)
    r = P.quantize_fp8(to_dev_bf16(x), E4, P.SCALE_TENSOR, 0, want_q=True)
    assert host(r["scale"])[0] == 1.0


def _groups_case(shape, seed, kind, specials):
    x = inputs.case(seed, shape, kind=kind)
    if specials:
        x[0, 0:128] = 0                     # an all-zero row group
        x[1, 130] = 0x7F80                  # +inf in row group (1, 1), column 130
        x[2, 260] = 0x7FC0                  # NaN in row group (2, 2), column 260
        x[200, 3] = 0xFF80                  # -inf in column 3, rows 128..255
    return x


@pytest.mark.parametrize("rnd", [1, 2], ids=["pow2", "pow2_floor"])
@pytest.mark.parametrize("fmt", [E4, E5])
@pytest.mark.parametrize("shape,kind,specials", [((256, 384), "normal", False), ((128, 128), "student_t", False),
                                                 ((384, 1024), "outliers", False), ((256, 384), "normal", True)])
def test_quantize_rows_and_columns(P, fmt, shape, kind, specials, rnd):
    x = _groups_case(shape, 14, kind, specials)
    d = to_dev_bf16(x)
    q, s = quant.quantize_rows_1x128(x, OFMT[fmt], RULE[rnd])
    qT, sT = quant.quantize_cols_128x1(x, OFMT[fmt], RULE[rnd])
    if rnd == 2:
        # groups whose amax significand exceeds 1.75 saturate under the floor rule
        assert (q & 0x7F == (0x7E if fmt == E4 else 0x7B)).any()
    r = P.quantize_fp8(d, fmt, P.SCALE_ROW_1x128, rnd, want_q=True, want_qT=True)
    assert_bytes_equal(host(r["q"]), q, "row q")
    assert_f32_bits_equal(host(r["scale"]), s, "row scale")
    assert_bytes_equal(host(r["qT"]), qT, "col qT (dual)")
    assert_f32_bits_equal(host(r["scaleT"]), sT, "col scaleT (dual)")
    r = P.quantize_fp8(d, fmt, P.SCALE_ROW_1x128, rnd, want_q=True, want_qT=False)
    assert_bytes_equal(host(r["q"]), q, "row q only")
    assert_f32_bits_equal(host(r["scale"]), s, "row scale only")
    r = P.quantize_fp8(d, fmt, P.SCALE_COL_128x1, rnd)
    assert_bytes_equal(host(r["qT"]), qT, "col qT")
    assert_f32_bits_equal(host(r["scaleT"]), sT, "col scaleT")
    # the k-block-major layout: the same codes, the scale arrays transposed
    r = P.quantize_fp8(d, fmt, P.SCALE_ROW_1x128 | P.SCALE_KMAJOR, rnd, want_q=True, want_qT=True)
    assert_bytes_equal(host(r["q"]), q, "row q (k-major)")
    assert_f32_bits_equal(host(r["scale"]), s.T, "row scale (k-major)")
    assert_bytes_equal(host(r["qT"]), qT, "col qT (k-major)")
    assert_f32_bits_equal(host(r["scaleT"]), sT.T, "col scaleT (k-major)")
    r = P.quantize_fp8(d, fmt, P.SCALE_COL_128x1 | P.SCALE_KMAJOR, rnd)
    assert_bytes_equal(host(r["qT"]), qT, "col qT only (k-major)")
    assert_f32_bits_equal(host(r["scaleT"]), sT.T, "col scaleT only (k-major)")


@pytest.mark.parametrize("rnd", [1, 2], ids=["pow2", "pow2_floor"])
@pytest.mark.parametrize("fmt", [E4, E5])
@pytest.mark.parametrize("shape,kind,specials", [((256, 384), "normal", False), ((128, 128), "student_t", False),
                                                 ((512, 256), "outliers", False), ((256, 384), "normal", True)])
def test_quantize_blocks(P, fmt, shape, kind, specials, rnd):
    x = _groups_case(shape, 15, kind, specials)
    q, s, qT, sT = quant.quantize_blocks_128x128(x, OFMT[fmt], RULE[rnd])
    r = P.quantize_fp8(to_dev_bf16(x), fmt, P.SCALE_BLOCK_128x128, rnd, want_q=True, want_qT=True)
    assert_bytes_equal(host(r["q"]), q, "block q")
    assert_f32_bits_equal(host(r["scale"]), s, "block scale")
    assert_bytes_equal(host(r["qT"]), qT, "block qT")
    assert_f32_bits_equal(host(r["scaleT"]), sT, "block scaleT")
    r = P.quantize_fp8(to_dev_bf16(x), fmt, P.SCALE_BLOCK_128x128 | P.SCALE_KMAJOR, rnd, want_q=True, want_qT=True)
    assert_bytes_equal(host(r["q"]), q, "block q (k-major)")
    assert_f32_bits_equal(host(r["scale"]), s.T, "block scale (k-major)")
    assert_bytes_equal(host(r["qT"]), qT, "block qT (k-major)")
    assert_f32_bits_equal(host(r["scaleT"]), sT.T, "block scaleT (k-major)")


def test_quantize_is_deterministic(P):
    x = to_dev_bf16(inputs.case(16, (1024, 1536)))
    a = P.quantize_fp8(x, E4, P.SCALE_TENSOR, 0, want_qT=True)
    b = P.quantize_fp8(x, E4, P.SCALE_TENSOR, 0, want_qT=True)
    assert_bytes_equal(host(a["q"]), host(b["q"]))
    assert_bytes_equal(host(a["qT"]), host(b["qT"]))


def test_quantize_largest_row_pitch(P):
    """The largest row pitch the quantisers accept, ld = 2**23 - 8 elements:
    inside a 128-row tile the byte offsets of the buffer loads reach about
    2**31, the edge of their 32-bit arithmetic. Per-tensor (q, qT) and
    1x128 + 128x1 groups on a 256 x 256 window of a 4.3 GB allocation."""
    import torch
    rows, cols, ld = 256, 256, (1 << 23) - 8
    x = inputs.case(15, (rows, cols), kind="outliers")
    big = torch.empty(rows, ld, dtype=torch.int16, device="cuda")
    big[:, :cols].copy_(torch.from_numpy(x.view(np.int16)).cuda())
    d = big.view(torch.bfloat16)[:, :cols]
    assert d.stride(0) == ld
    r = P.quantize_fp8(d, E4, P.SCALE_TENSOR, 0, want_q=True, want_qT=True)
    q, qT, s, _ = quant.quantize_tensor(x, fp8.E4M3, rule=RULE[0])
    assert_f32_bits_equal(host(r["scale"]), np.array([s]), "scale")
    assert_bytes_equal(host(r["q"]), q, "q")
    assert_bytes_equal(host(r["qT"]), qT, "qT")
    r = P.quantize_fp8(d, E4, P.SCALE_ROW_1x128, 1, want_q=True, want_qT=True)
    q, s = quant.quantize_rows_1x128(x, fp8.E4M3, RULE[1])
    qT, sT = quant.quantize_cols_128x1(x, fp8.E4M3, RULE[1])
    assert_bytes_equal(host(r["q"]), q, "row q")
    assert_f32_bits_equal(host(r["scale"]), s, "row scale")
    assert_bytes_equal(host(r["qT"]), qT, "col qT")
    assert_f32_bits_equal(host(r["scaleT"]), sT, "col scaleT")
    del big, d
    torch.cuda.empty_cache()
