"""Pins of the RMSNorm oracle (oracle/rmsnorm.py): numpy's vector norm (with
eps = 0, y = x / (|x|_2 / sqrt(C)) * gamma), the unit mean square of y / gamma,
scale invariance, a constant row, the role of eps, and the band's width."""

import numpy as np
import pytest

from oracle import bf16, quant, rmsnorm, swiglu
from tests import band_check


def bits(x):
    return bf16.from_f64_rne(np.asarray(x, dtype=np.float64))


def _case(R=16, C=256, seed=3):
    rng = np.random.default_rng(seed)
    return bits(rng.standard_normal((R, C))), bits(1.0 + 0.1 * rng.standard_normal(C))


def test_vector_norm_and_unit_mean_square():
    x, g = _case()
    C = x.shape[1]
    xf = bf16.to_f32(x).astype(np.float64)
    gf = bf16.to_f32(g).astype(np.float64)
    y = rmsnorm.rmsnorm_f64(x, g, 0.0)
    want = xf / (np.linalg.norm(xf, axis=1, keepdims=True) / np.sqrt(C)) * gf
    np.testing.assert_allclose(y, want, rtol=1e-14, atol=0)
    np.testing.assert_allclose(np.mean((y / gf) ** 2, axis=1), 1.0, rtol=1e-13)


def test_scale_invariance_and_constant_row():
    x, g = _case()
    x4 = bits(4.0 * bf16.to_f32(x))                 # exact in BF16
    np.testing.assert_array_equal(rmsnorm.rmsnorm_f64(x4, g, 0.0), rmsnorm.rmsnorm_f64(x, g, 0.0))
    c = bits(np.full((1, 64), -3.0))
    ones = bits(np.ones(64))
    np.testing.assert_array_equal(rmsnorm.rmsnorm_f64(c, ones, 0.0), -1.0)
    assert rmsnorm.rstd_f64(c, 0.0)[0] == 1.0 / 3.0


def test_eps():
    # eps enters as its binary32 value and dominates tiny rows
    x = bits(np.full((1, 32), 2.0 ** -20))
    ones = bits(np.ones(32))
    r = rmsnorm.rstd_f64(x, 1e-6)[0]
    assert r == 1.0 / np.sqrt(2.0 ** -40 + float(np.float32(1e-6)))
    assert rmsnorm.rstd_f64(x, 0.0)[0] == 2.0 ** 20
    y = rmsnorm.rmsnorm_f64(x, ones, 1e-6)
    assert np.all(y < 2.0 ** -20 * 1e3) and np.all(y > 0)


def test_band():
    x, g = _case(64, 512)
    mid, lo, hi = rmsnorm.rmsnorm_bf16_band(x, g, 1e-6)
    t = rmsnorm.rmsnorm_f64(x, g, 1e-6)
    lo_f, hi_f, mid_f = (bf16.to_f32(b).astype(np.float64) for b in (lo, hi, mid))
    assert np.all(lo_f <= mid_f) and np.all(mid_f <= hi_f)
    # mid is the BF16 rounding of the float64 value: within half a BF16 step
    assert np.all(np.abs(mid_f - t) <= np.abs(t) * 2.0 ** -8 + 1e-30)
    # the band holds at most the two BF16 neighbours of the value
    step = np.ldexp(1.0, np.frexp(np.abs(t))[1] - 8)
    assert np.all(hi_f - lo_f <= step * 1.0000001)
    amb = np.mean(lo != hi)
    assert 0 < amb < 0.03, amb


@pytest.mark.parametrize("axis,rule", [(None, "fp32"), (1, "pow2"), (0, "pow2")])
def test_band_check_catches_a_dropped_gamma(axis, rule):
    x, g = _case(256, 256)
    mid, lo, hi = rmsnorm.rmsnorm_bf16_band(x, g, 1e-6)
    un = swiglu.unique_mask(lo, hi)
    ones = bits(np.ones(256))
    for gg, ok in ((g, True), (ones, False)):
        m, _, _ = rmsnorm.rmsnorm_bf16_band(x, gg, 1e-6)
        if axis is None:
            q, _, s, _ = quant.quantize_tensor(m, "e4m3", rule=rule)
        elif axis == 1:
            q, s = quant.quantize_rows_1x128(m, "e4m3", rule)
        else:
            qT, s = quant.quantize_cols_128x1(m, "e4m3", rule)
            q = qT.T
        if ok:
            band_check.check(q, s, mid, lo, hi, un, "e4m3", rule, axis, "oracle")
        else:
            with pytest.raises(AssertionError):
                band_check.check(q, s, mid, lo, hi, un, "e4m3", rule, axis, "planted")
