"""Pins of the SwiGLU oracle (oracle/swiglu.py) and of the band check used by
the fused SwiGLU + quantise parity tests (tests/band_check.py).

silu(g) = g / (1 + e^-g) is pinned by the identity silu(g) - silu(-g) = g, by
the library routine scipy.special.expit (silu(g) = g * expit(g)), and by its
limits; the gate/up split and the linearity in u by constructed inputs; the
band by values exactly on and next to BF16 rounding boundaries; the check by
oracle-made results with one planted mistake each.
"""

import numpy as np
import pytest
from scipy.special import expit

from oracle import bf16, quant, swiglu
from tests import band_check


def bits(x):
    return bf16.from_f64_rne(np.asarray(x, dtype=np.float64))


def test_silu_identity_and_library():
    g = np.linspace(-30, 30, 6001)
    s = swiglu.silu_f64(g)
    assert np.all(np.abs(s - swiglu.silu_f64(-g) - g) <= 1e-13 * np.maximum(1, np.abs(g)))
    np.testing.assert_allclose(s, g * expit(g), rtol=1e-15, atol=1e-300)


def test_silu_limits():
    assert swiglu.silu_f64(0.0) == 0.0
    assert swiglu.silu_f64(40.0) == 40.0          # e^-40 vanishes against 1 in float64
    v = swiglu.silu_f64(np.array([-1000.0, -745.0]))
    assert np.all(v == 0) and not np.isnan(v).any()
    # the minimum of silu is at g ~ -1.278 with value ~ -0.2785
    g = np.linspace(-3, 0, 300001)
    assert abs(swiglu.silu_f64(g).min() + 0.27846454) < 1e-7


def test_gate_up_split_and_linearity():
    rng = np.random.default_rng(1)
    C = 32
    g = rng.standard_normal((4, C))
    ones = np.ones((4, C))
    h = swiglu.swiglu_f64(np.concatenate([bits(g), bits(ones)], axis=1), C)
    np.testing.assert_array_equal(h, swiglu.silu_f64(bf16.to_f32(bits(g)).astype(np.float64)))
    u = rng.standard_normal((4, C))
    gu = np.concatenate([bits(g), bits(u)], axis=1)
    gu2 = np.concatenate([bits(g), bits(2.0 * bf16.to_f32(bits(u)))], axis=1)
    np.testing.assert_array_equal(swiglu.swiglu_f64(gu2, C), 2.0 * swiglu.swiglu_f64(gu, C))
    # columns past 2C (a wider row pitch) are ignored
    wide = np.concatenate([gu, bits(np.full((4, 16), 7.0))], axis=1)
    np.testing.assert_array_equal(swiglu.swiglu_f64(wide, C), swiglu.swiglu_f64(gu, C))


def test_band_exact_and_boundary_values():
    # silu(40) = 40 exactly in float64, so H = 40 * u exactly
    C = 4
    u = np.array([[1.0, 1.5, 1.0 + 2.0 ** -5, -3.0]])
    gu = np.concatenate([bits(np.full((1, C), 40.0)), bits(u)], axis=1)
    mid, lo, hi = swiglu.swiglu_bf16_band(gu, C)
    assert swiglu.unique_mask(lo, hi).all()
    np.testing.assert_array_equal(bf16.to_f32(mid), 40.0 * u)
    # silu(48) = 48, and 48 * (1 + 2^-7) = 48.375 lies exactly halfway between
    # the BF16 neighbours 48.25 and 48.5 (spacing 0.25 at 32..64): both are
    # accepted, and mid is the even one
    u = np.array([[1.0 + 2.0 ** -7]])
    gu = np.concatenate([bits([[48.0]]), bits(u)], axis=1)
    assert bf16.to_f32(bits(u))[0, 0] == u[0, 0]
    mid, lo, hi = swiglu.swiglu_bf16_band(gu, 1)
    assert not swiglu.unique_mask(lo, hi)[0, 0]
    assert (bf16.to_f32(lo)[0, 0], bf16.to_f32(hi)[0, 0]) == (48.25, 48.5)
    assert bf16.to_f32(mid)[0, 0] == 48.5          # 48.5 = 1.1000010b * 2^5 has the even last bit
    # signed zeros: silu(+0) * u keeps the sign of u; the band holds only zero
    gu = np.concatenate([bits([[0.0, 0.0]]), bits([[2.0, -2.0]])], axis=1)
    mid, lo, hi = swiglu.swiglu_bf16_band(gu, 2)
    assert swiglu.unique_mask(lo, hi).all()
    assert list(mid[0]) == [0x0000, 0x8000]
    # where e^-g overflows binary32, zero is accepted
    gu = np.concatenate([bits([[-100.0]]), bits([[1.0]])], axis=1)
    mid, lo, hi = swiglu.swiglu_bf16_band(gu, 1)
    assert bf16.to_f32(lo)[0, 0] <= 0.0 <= bf16.to_f32(hi)[0, 0]


@pytest.mark.parametrize("axis,rule", [(None, "fp32"), (None, "pow2"), (1, "pow2"), (0, "pow2"), (1, "pow2_floor")])
def test_band_check_accepts_oracle_and_rejects_mistakes(axis, rule):
    rng = np.random.default_rng(2)
    R, C = 256, 256
    gu = bits(rng.standard_normal((R, 2 * C)))
    mid, lo, hi = swiglu.swiglu_bf16_band(gu, C)
    un = swiglu.unique_mask(lo, hi)
    fmt = "e4m3"
    if axis is None:
        q, _, s, _ = quant.quantize_tensor(mid, fmt, rule=rule)
    elif axis == 1:
        q, s = quant.quantize_rows_1x128(mid, fmt, rule)
    else:
        qT, s = quant.quantize_cols_128x1(mid, fmt, rule)
        q = qT.T
    band_check.check(q, s, mid, lo, hi, un, fmt, rule, axis, "oracle")
    # a wrong code where H is unique
    i = tuple(np.argwhere(un & (q != 0))[0])
    q2 = q.copy()
    q2[i] ^= 0x01
    with pytest.raises(AssertionError):
        band_check.check(q2, s, mid, lo, hi, un, fmt, rule, axis, "planted code")
    # a wrong scale
    s2 = np.array(s, dtype=np.float32).reshape(-1).copy()
    s2[0] *= 2
    with pytest.raises(AssertionError):
        band_check.check(q, s2, mid, lo, hi, un, fmt, rule, axis, "planted scale")
    # H taken without the up half (u = 1) must be caught
    gu1 = np.concatenate([gu[:, :C], bits(np.ones((R, C)))], axis=1)
    m1, _, _ = swiglu.swiglu_bf16_band(gu1, C)
    if axis is None:
        q1, _, s1, _ = quant.quantize_tensor(m1, fmt, rule=rule)
    elif axis == 1:
        q1, s1 = quant.quantize_rows_1x128(m1, fmt, rule)
    else:
        q1T, s1 = quant.quantize_cols_128x1(m1, fmt, rule)
        q1 = q1T.T
    with pytest.raises(AssertionError):
        band_check.check(q1, s1, mid, lo, hi, un, fmt, rule, axis, "planted operand")


def test_dsilu_identities_and_finite_differences():
    g = np.linspace(-30, 30, 6001)
    d = swiglu.dsilu_f64(g)
    # d/dg [silu(g) - silu(-g)] = d/dg g = 1
    assert np.all(np.abs(d + swiglu.dsilu_f64(-g) - 1.0) <= 1e-13)
    assert swiglu.dsilu_f64(0.0) == 0.5
    # central differences of the forward oracle
    h = 1e-5
    fd = (swiglu.silu_f64(g + h) - swiglu.silu_f64(g - h)) / (2 * h)
    assert np.all(np.abs(fd - d) <= 1e-8)
    assert swiglu.dsilu_f64(40.0) == 1.0 and abs(swiglu.dsilu_f64(-40.0)) < 1e-15
    # silu' vanishes at the minimum of silu (g ~ -1.2785)
    gg = np.linspace(-1.3, -1.25, 50001)
    assert abs(gg[np.argmin(np.abs(swiglu.dsilu_f64(gg)))] + 1.27846) < 1e-4


def test_backward_layout_and_band():
    rng = np.random.default_rng(4)
    R, C = 64, 128
    gu = bits(rng.standard_normal((R, 2 * C)) * 1.7)
    dh = bits(rng.standard_normal((R, C)) * 1e-3)
    t = swiglu.swiglu_bwd_f64(dh, gu, C)
    g, u = swiglu.split(gu, C)
    dhf = bf16.to_f32(dh).astype(np.float64)
    np.testing.assert_allclose(t[:, C:], dhf * g * expit(g), rtol=1e-14, atol=1e-300)
    sg = expit(g)
    np.testing.assert_allclose(t[:, :C], dhf * u * (sg + g * sg * (1 - sg)), rtol=1e-12, atol=1e-300)
    mid, lo, hi = swiglu.swiglu_bwd_bf16_band(dh, gu, C)
    assert mid.shape == (R, 2 * C)
    lo_f, hi_f, mid_f = (bf16.to_f32(b) for b in (lo, hi, mid))
    assert np.all(lo_f <= mid_f) and np.all(mid_f <= hi_f)
    un = swiglu.unique_mask(lo, hi)
    assert 0.9 < un.mean() < 1.0
    # at the zero of silu' the absolute allowance covers the error a binary32
    # evaluation makes there (s^2 |g| times a few 2^-24 in 1 - s: about 2^-26)
    gz = bits([[-1.28125]])                       # the BF16 value nearest the zero
    m, l, h = swiglu.swiglu_bwd_bf16_band(bits([[1.0]]), np.concatenate([gz, bits([[1.0]])], axis=1), 1)
    tz = swiglu.dsilu_f64(bf16.to_f32(gz).astype(np.float64))[0, 0]
    assert abs(tz) < 2e-3
    lo_f, hi_f = bf16.to_f32(l)[0, 0], bf16.to_f32(h)[0, 0]
    for e in (-2.0 ** -25, 2.0 ** -25):
        v = bf16.to_f32(bf16.from_f64_rne(np.array([tz + e])))[0]
        assert lo_f <= v <= hi_f


def _every_gate_value():
    """Every finite BF16 pattern as float32 gate values."""
    g = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    g32 = bf16.to_f32(g)
    return g[np.isfinite(g32)], g32[np.isfinite(g32)]


def _in_band(h_bits, lo, hi):
    h, l, u = (bf16.to_f32(b).astype(np.float64) for b in (h_bits, lo, hi))
    return (l <= h) & (h <= u)


@pytest.mark.parametrize("u", [1.0, -3.0, 2.0 ** -10, 300.0])
def test_band_holds_ieee_binary32_evaluation(u):
    """The reading evaluates silu(g) u = g / (1 + e^-g) * u in binary32. numpy's
    float32 arithmetic is IEEE binary32 with gradual underflow, so its result,
    rounded to BF16, must lie in the band for every finite gate value; and
    wherever that BF16 value is non-zero the band must exclude zero. In
    particular zero is accepted only where e^-g overflows binary32 (there the
    binary32 quotient is -0): for g in [-88.72, -64) a binary32 evaluation is
    non-zero and so must a kernel's be."""
    gb, g32 = _every_gate_value()
    C = gb.size
    ub = bits(np.full(C, u))
    with np.errstate(over="ignore", invalid="ignore", under="ignore"):
        u32 = bf16.to_f32(ub)
        h32 = (g32 / (np.float32(1.0) + np.exp(-g32))) * u32
    assert h32.dtype == np.float32
    h = bf16.from_f64_rne(h32.astype(np.float64))
    mid, lo, hi = swiglu.swiglu_bf16_band(np.concatenate([gb, ub])[None, :], C)
    ok = _in_band(h[None, :], lo, hi)
    assert ok.all(), g32[~ok[0]][:8]
    nz = bf16.to_f32(h) != 0
    zero_in = (bf16.to_f32(lo)[0] <= 0) & (0 <= bf16.to_f32(hi)[0])
    assert not (nz & zero_in).any(), g32[nz & zero_in][:8]
    # the tail in question: non-zero below -64 down to the overflow point
    tail = (g32 >= swiglu.G_OVERFLOW) & (g32 < -64)
    assert tail.sum() > 10 and nz[tail].all()
    # where e^-g overflows binary32 the float32 result is a zero, and the bound
    # TINY * max(1, |u|) on the exact value holds
    deep = g32 < swiglu.G_OVERFLOW
    assert (h32[deep] == 0).all()
    assert (np.abs(swiglu.silu_f64(g32[deep].astype(np.float64))) < swiglu.TINY).all()


@pytest.mark.parametrize("dh,u", [(1e-3, 1.0), (1.0, -3.0), (2.0 ** -10, 300.0)])
def test_backward_band_holds_ieee_binary32_evaluation(dh, u):
    """The backward's halves dg = dH u s (1 + g (1 - s)) and du = dH g s with
    s = 1 / (1 + e^-g), evaluated in binary32 by numpy, lie in the band for
    every finite gate value, and the band excludes zero wherever that
    evaluation is non-zero in BF16."""
    gb, g32 = _every_gate_value()
    C = gb.size
    ub, dhb = bits(np.full(C, u)), bits(np.full(C, dh))
    with np.errstate(over="ignore", invalid="ignore", under="ignore"):
        u32, dh32 = bf16.to_f32(ub), bf16.to_f32(dhb)
        s = np.float32(1.0) / (np.float32(1.0) + np.exp(-g32))
        dg = dh32 * u32 * (s * (np.float32(1.0) + g32 * (np.float32(1.0) - s)))
        du = dh32 * (g32 * s)
    h = bf16.from_f64_rne(np.concatenate([dg, du]).astype(np.float64))[None, :]
    mid, lo, hi = swiglu.swiglu_bwd_bf16_band(dhb[None, :], np.concatenate([gb, ub])[None, :], C)
    ok = _in_band(h, lo, hi)
    assert ok.all(), np.concatenate([g32, g32])[~ok[0]][:8]
    nz = bf16.to_f32(h)[0] != 0
    zero_in = (bf16.to_f32(lo)[0] <= 0) & (0 <= bf16.to_f32(hi)[0])
    assert not (nz & zero_in).any()
    tail = np.concatenate([(g32 >= swiglu.G_OVERFLOW) & (g32 < -64)] * 2)
    assert nz[tail].all()
