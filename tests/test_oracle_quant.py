"""Pins of the oracle's amax, scale rules and quantisers (``oracle.quant``):
closed forms of the scale rules, invariances (permutation, sign, powers of
two, transposition), block locality and the encoding error bound."""

import numpy as np
import pytest

from oracle import bf16, fp8, quant
from paper_2608_27370_amd import inputs

FMTS = (fp8.E4M3, fp8.E5M2)


def test_amax_integer_form_and_invariances():
    x = inputs.case(1, (64, 256), kind="student_t")
    xf = bf16.to_f32(x)
    a = quant.amax(xf)
    # integer form: BF16 magnitudes order like their bit patterns without the sign
    mag_bits = (x & 0x7FFF).max()
    assert a == bf16.to_f32(np.array([mag_bits], np.uint16))[0]
    g = np.random.default_rng(5)
    perm = g.permutation(xf.size)
    assert quant.amax(xf.ravel()[perm]) == a
    flips = g.choice([-1.0, 1.0], xf.shape).astype(np.float32)
    assert quant.amax(xf * flips) == a


def test_amax_nan_and_empty_and_negative_zero():
    assert np.isnan(quant.amax(np.array([1.0, np.nan, 3.0], np.float32)))
    assert quant.amax(np.zeros((0, 16), np.float32)) == 0
    assert quant.amax(np.array([-0.0, -0.0], np.float32)) == 0


@pytest.mark.parametrize("fmt", FMTS)
def test_tensor_scale_closed_forms(fmt):
    fm = fp8.fmax(fmt)
    assert quant.tensor_scale(fm, fmt) == (1.0, 1.0)
    assert quant.tensor_scale(2 * fm, fmt) == (2.0, 0.5)
    assert quant.tensor_scale(0.0, fmt) == (1.0, 1.0)
    s, r = quant.tensor_scale(3.0, fmt)
    assert s == np.float32(3.0) / np.float32(fm) and r == np.float32(fm) / np.float32(3.0)


@pytest.mark.parametrize("fmt", FMTS)
def test_pow2_exponent_closed_forms(fmt):
    fm = fp8.fmax(fmt)
    for j in range(-20, 21):
        assert quant.pow2_exponent(fm * 2.0 ** j, fmt) == j
        assert quant.pow2_exponent(fm * 2.0 ** j * (1 + 2.0 ** -7), fmt) == j + 1
        assert quant.pow2_exponent(fm * 2.0 ** j * (1 - 2.0 ** -8), fmt) == j
    assert quant.pow2_exponent(0.0, fmt) == 0
    assert quant.pow2_exponent(np.inf, fmt) == 127
    assert quant.pow2_exponent(np.nan, fmt) is None
    assert quant.pow2_exponent(1e-38, fmt) == -127         # clamped to the E8M0 range
    # 448 * 2**-9 = 0.875 < 1 <= 448 * 2**-8
    if fmt == fp8.E4M3:
        assert quant.pow2_exponent(1.0, fmt) == -8


@pytest.mark.parametrize("fmt", FMTS)
def test_per_tensor_max_element_hits_fmax(fmt):
    x = inputs.case(2, (32, 128))
    q, qT, s, a = quant.quantize_tensor(x, fmt)
    xf = bf16.to_f32(x)
    i = np.argmax(np.abs(xf))
    top = 0x7E if fmt == fp8.E4M3 else 0x7B
    assert (q.ravel()[i] & 0x7F) == top
    assert np.array_equal(qT, q.T)
    assert s == np.float32(a) / np.float32(fp8.fmax(fmt))


@pytest.mark.parametrize("fmt", FMTS)
def test_sign_symmetry(fmt):
    x = inputs.case(3, (16, 256))
    xn = x ^ np.uint16(0x8000)
    q1, _, s1, _ = quant.quantize_tensor(x, fmt)
    q2, _, s2, _ = quant.quantize_tensor(xn, fmt)
    assert s1 == s2 and np.array_equal(q2, q1 ^ 0x80)
    r1, t1 = quant.quantize_rows_1x128(x, fmt)
    r2, t2 = quant.quantize_rows_1x128(xn, fmt)
    assert np.array_equal(t1, t2) and np.array_equal(r2, r1 ^ 0x80)


def _times_pow2(x_bits, j):
    """Multiply BF16 values by 2**j exactly (exponent field shift, no overflow)."""
    f = bf16.to_f32(x_bits).astype(np.float64) * 2.0 ** j
    out = inputs.bf16_from_f64(f)
    assert np.array_equal(bf16.to_f32(out).astype(np.float64), f)
    return out


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("j", [-5, 3])
def test_power_of_two_equivariance(fmt, j):
    x = inputs.case(4, (128, 256), kind="outliers")
    y = _times_pow2(x, j)
    qa, sa = quant.quantize_rows_1x128(x, fmt)
    qb, sb = quant.quantize_rows_1x128(y, fmt)
    assert np.array_equal(qa, qb) and np.array_equal(sb, sa * np.float32(2.0 ** j))
    qa, sa, _, _ = quant.quantize_blocks_128x128(x, fmt)
    qb, sb, _, _ = quant.quantize_blocks_128x128(y, fmt)
    assert np.array_equal(qa, qb) and np.array_equal(sb, sa * np.float32(2.0 ** j))
    # the per-tensor rule with pow2 scales is equivariant as well
    qa, _, sa, _ = quant.quantize_tensor(x, fmt, rule="pow2")
    qb, _, sb, _ = quant.quantize_tensor(y, fmt, rule="pow2")
    assert np.array_equal(qa, qb) and sb == sa * np.float32(2.0 ** j)


@pytest.mark.parametrize("fmt", FMTS)
def test_pow2_scales_never_saturate_and_fill_the_top_binade(fmt):
    x = inputs.case(5, (8, 1024), kind="student_t")
    q, s = quant.quantize_rows_1x128(x, fmt)
    xf = bf16.to_f32(x).reshape(8, 8, 128)
    vals = fp8.decode(q, fmt).reshape(8, 8, 128) * s[:, :, None]
    # exact powers of two
    m, _ = np.frexp(s)
    assert np.all(m == 0.5)
    # the group maximum lands in (FMAX/2, FMAX] after scaling: no saturation,
    # and no wasted binade
    amx = np.abs(xf).max(axis=2)
    scaled = amx / s
    assert np.all(scaled <= fp8.fmax(fmt)) and np.all(scaled > fp8.fmax(fmt) / 2)
    # the dequantised values are within half a grid step of the inputs
    assert np.all(np.abs(vals - xf) <= np.abs(xf) * 2.0 ** -(fp8.mbits(fmt) + 1)
                  + s[:, :, None] * 2.0 ** (fp8.emin(fmt) - fp8.mbits(fmt) - 1))


def test_transposition_rules():
    x = inputs.case(6, (256, 384))
    q, qT, s, _ = quant.quantize_tensor(x, fp8.E4M3)
    q2, _, s2, _ = quant.quantize_tensor(np.ascontiguousarray(x.T), fp8.E4M3)
    assert s == s2 and np.array_equal(q2, q.T) and np.array_equal(qT, q.T)
    a, sa, aT, saT = quant.quantize_blocks_128x128(x, fp8.E4M3)
    b, sb, _, _ = quant.quantize_blocks_128x128(np.ascontiguousarray(x.T), fp8.E4M3)
    assert np.array_equal(b, a.T) and np.array_equal(sb, sa.T)
    assert np.array_equal(aT, a.T) and np.array_equal(saT, sa.T)
    cT, scT = quant.quantize_cols_128x1(x, fp8.E4M3)
    r, sr = quant.quantize_rows_1x128(np.ascontiguousarray(x.T), fp8.E4M3)
    assert np.array_equal(cT, r) and np.array_equal(scT, sr)


def test_block_locality():
    x = inputs.case(7, (256, 384))
    y = x.copy()
    y[130, 200] = inputs.bf16_from_f64(np.array([1000.0]))[0]   # in block (1, 1) only
    qa, sa, _, _ = quant.quantize_blocks_128x128(x, fp8.E4M3)
    qb, sb, _, _ = quant.quantize_blocks_128x128(y, fp8.E4M3)
    changed = np.argwhere(sa != sb)
    assert changed.tolist() == [[1, 1]]
    diff = np.argwhere(qa != qb)
    assert np.all((diff[:, 0] // 128 == 1) & (diff[:, 1] // 128 == 1))
    ra, rsa = quant.quantize_rows_1x128(x, fp8.E4M3)
    rb, rsb = quant.quantize_rows_1x128(y, fp8.E4M3)
    assert np.argwhere(rsa != rsb).tolist() == [[130, 1]]
    d = np.argwhere(ra != rb)
    assert np.all((d[:, 0] == 130) & (d[:, 1] // 128 == 1))


def test_supplied_amax_saturates_large_values():
    x = inputs.case(8, (16, 128))
    xf = bf16.to_f32(x)
    a = quant.amax(xf)
    q, _, s, _ = quant.quantize_tensor(x, fp8.E4M3, amax_in=a / 4)
    # values above a/4 in magnitude saturate to +-448
    big = np.abs(xf) > a / 4 * (1 + 2.0 ** -4)
    assert np.all((q[big] & 0x7F) == 0x7E)


def test_zero_tensor_and_zero_groups():
    x = np.zeros((4, 256), np.uint16)
    x[1, 130] = inputs.bf16_from_f64(np.array([0.5]))[0]
    q, s = quant.quantize_rows_1x128(x, fp8.E4M3)
    assert s[0, 0] == 1.0 and s[1, 0] == 1.0
    assert s[1, 1] == 2.0 ** -9                        # 0.5 / 448 -> ceil(log2) = -9
    assert q[1, 130] == 0x78                           # 0.5 * 2**9 = 256 = 2**8: exponent field 15
    q, _, s, a = quant.quantize_tensor(np.zeros((3, 16), np.uint16), fp8.E5M2)
    assert s == 1.0 and a == 0.0 and not q.any()


# ---- the OCP-MX (floor) power-of-two rule, kept for comparison -------------

@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_pow2_floor_exponent_closed_forms(fmt):
    fm = fp8.fmax(fmt)
    em = quant.emax(fmt)
    assert fm == 1.75 * 2.0 ** em                          # 448 = 1.75 * 2^8, 57344 = 1.75 * 2^15
    for j in range(-20, 20):
        assert quant.pow2_floor_exponent(2.0 ** (em + j), fmt) == j
        assert quant.pow2_floor_exponent(fm * 2.0 ** j, fmt) == j
        # significand above 1.75: the floor rule stays at j, the ceil rule moves to j + 1
        a = fm * 2.0 ** j * (1 + 2.0 ** -7)
        assert quant.pow2_floor_exponent(a, fmt) == j and quant.pow2_exponent(a, fmt) == j + 1
        assert quant.pow2_floor_exponent(2.0 ** (em + j + 1) * (1 - 2.0 ** -8), fmt) == j
    assert quant.pow2_floor_exponent(0.0, fmt) == 0
    assert quant.pow2_floor_exponent(np.inf, fmt) == 127
    assert quant.pow2_floor_exponent(np.nan, fmt) is None
    assert quant.pow2_floor_exponent(1e-38, fmt) == -127
    assert quant.pow2_floor_exponent(3e38, fmt) == 127 - em           # 3e38 = 1.76 * 2^127


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_pow2_floor_matches_log2_on_every_bf16_magnitude(fmt):
    """Brute force over all positive finite BF16 patterns: the floor rule is
    floor(log2 a) - emax, with log2 from the math library (exact here: a
    BF16 value that is not a power of two is at least 2^-8 of an octave away
    from one)."""
    em = quant.emax(fmt)
    bits = np.arange(1, 0x7F80, dtype=np.uint16)
    vals = bf16.to_f32(bits).astype(np.float64)
    got = np.array([quant.pow2_floor_exponent(v, fmt) for v in vals])
    want = np.clip(np.floor(np.log2(vals)).astype(int) - em, -127, 127)
    assert np.array_equal(got, want)
    # and it is the ceil rule's exponent, or one less exactly when the
    # significand exceeds FMAX's 1.75 (outside the clamp)
    ceil = np.array([quant.pow2_exponent(v, fmt) for v in vals])
    sig = vals / 2.0 ** np.floor(np.log2(vals))
    inside = (want > -127) & (want < 127) & (ceil > -127) & (ceil < 127)
    assert np.array_equal((ceil - got)[inside], (sig > 1.75)[inside].astype(int))


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_pow2_floor_saturates_only_above_fmax_significand(fmt):
    fm = fp8.fmax(fmt)
    rng = np.random.default_rng(9)
    for top in (1.5, 1.75, 1.875):
        x = rng.uniform(-1, 1, (4, 128))
        x[:, 7] = top                                  # the block's amax, significand `top`
        xb = bf16.from_f64_rne(x * 2.0 ** 3)
        q, s = quant.quantize_rows_1x128(xb, fmt, "pow2_floor")
        d = fp8.decode(q, fmt).astype(np.float64) * s.repeat(128, axis=1)
        amax_code = q[:, 7]
        if top > 1.75:
            # the top value is clipped to FMAX * s, below the amax
            assert np.all(fp8.decode(amax_code, fmt) == fm)
            assert np.all(d[:, 7] < bf16.to_f32(xb[:, 7]))
        else:
            # nothing saturates: the ceil rule gives the same scales and bytes
            q2, s2 = quant.quantize_rows_1x128(xb, fmt, "pow2")
            assert np.array_equal(q, q2) and np.array_equal(s, s2)
