"""Pins of the oracle's FP8 codec (``oracle.fp8``) against the format
definitions: fixed points, round trips, ties, saturation, underflow, brute
force over the code table and an independent library cast."""

import os

import numpy as np
import pytest

from oracle import fp8

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fp8_format_fixed_points.txt")
FMTS = (fp8.E4M3, fp8.E5M2)


def _golden_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            fmt, name, code, value = line.split()
            rows.append((fmt, name, int(code, 16), value))
    return rows


@pytest.mark.parametrize("row", _golden_rows(), ids=lambda r: "%s-%s" % (r[0], r[1]))
def test_fixed_points_decode(row):
    fmt, name, code, value = row
    got = fp8.decode(np.array([code], np.uint8), fmt)[0]
    if value == "nan":
        assert np.isnan(got)
    else:
        want = float(value)
        assert got == want
        assert np.signbit(got) == value.startswith("-")


@pytest.mark.parametrize("row", [r for r in _golden_rows() if r[3] not in ("nan", "inf", "-inf")],
                         ids=lambda r: "%s-%s" % (r[0], r[1]))
def test_fixed_points_encode(row):
    fmt, name, code, value = row
    assert fp8.encode(np.array([float(value)], np.float32), fmt)[0] == code


def test_nan_codes_complete():
    # E4M3 has exactly two NaN codes and no infinities; E5M2 six NaNs, two infs.
    t = fp8.decode_table(fp8.E4M3)
    assert np.isnan(t).sum() == 2 and np.isinf(t).sum() == 0
    t = fp8.decode_table(fp8.E5M2)
    assert np.isnan(t).sum() == 6 and np.isinf(t).sum() == 2


@pytest.mark.parametrize("fmt", FMTS)
def test_table_monotone_and_sign_symmetric(fmt):
    t = fp8.decode_table(fmt)
    pos = t[:128][np.isfinite(t[:128])]
    assert np.all(np.diff(pos) > 0)            # codes 0..max are increasing
    fin = np.isfinite(t[:128])
    assert np.array_equal(t[128:][fin], -t[:128][fin])


@pytest.mark.parametrize("fmt", FMTS)
def test_every_finite_code_round_trips(fmt):
    codes = np.arange(256, dtype=np.uint8)
    vals = fp8.decode(codes, fmt)
    back = fp8.encode(vals.astype(np.float32), fmt)
    for c, v, b in zip(codes, vals, back):
        if np.isnan(v):
            assert b == 0x7F                     # the canonical NaN code
        elif np.isinf(v):
            assert b == (0x7B | (c & 0x80))     # E5M2 infinities saturate
        else:
            assert b == c


@pytest.mark.parametrize("fmt", FMTS)
def test_midpoints_tie_to_even_and_nudges(fmt):
    t = fp8.decode_table(fmt)
    codes = [c for c in range(128) if np.isfinite(t[c])]
    for lo, hi in zip(codes[:-1], codes[1:]):
        mid = np.float32((t[lo] + t[hi]) / 2)   # exact: FP8 values have <= 4 significant bits
        assert float(mid) == (t[lo] + t[hi]) / 2
        even = lo if lo % 2 == 0 else hi
        for sgn in (1, -1):
            got = fp8.encode(np.array([sgn * mid], np.float32), fmt)[0]
            assert got == (even | (0x80 if sgn < 0 else 0))
        below = np.nextafter(mid, np.float32(0))
        above = np.nextafter(mid, np.float32(np.inf))
        assert fp8.encode(np.array([below], np.float32), fmt)[0] == lo
        assert fp8.encode(np.array([above], np.float32), fmt)[0] == hi


def test_saturation():
    big = [464.0, 470.0, 1e30, float(np.finfo(np.float32).max), np.inf]
    q = fp8.encode(np.array(big, np.float32), fp8.E4M3)
    assert list(q) == [0x7E] * 5
    q = fp8.encode(-np.array(big, np.float32), fp8.E4M3)
    assert list(q) == [0xFE] * 5
    big = [59392.0, 61440.0, 1e30, np.inf]
    q = fp8.encode(np.array(big, np.float32), fp8.E5M2)
    assert list(q) == [0x7B] * 4


def test_every_nan_maps_to_the_canonical_code():
    pats = np.array([0x7FC00000, 0xFFC00000, 0x7F800001, 0xFFBFFFFF], np.uint32)
    for fmt in FMTS:
        assert list(fp8.encode(pats.view(np.float32), fmt)) == [0x7F] * 4


def test_underflow_and_signed_zero():
    one_ulp = 1 + 2.0 ** -23
    q = fp8.encode(np.array([2.0 ** -10, 2.0 ** -10 * one_ulp, -2.0 ** -10, -0.0, 1e-30],
                            np.float32), fp8.E4M3)
    assert list(q) == [0x00, 0x01, 0x80, 0x80, 0x00]
    q = fp8.encode(np.array([2.0 ** -17, 2.0 ** -17 * one_ulp, -2.0 ** -17], np.float32), fp8.E5M2)
    assert list(q) == [0x00, 0x01, 0x80]


def _brute_force_encode(v, fmt):
    """Nearest finite code by scanning the whole table; ties -> even mantissa;
    |v| >= FMAX saturates; NaN -> 0x7F."""
    t = fp8.decode_table(fmt)
    pos_codes = np.array([c for c in range(128) if np.isfinite(t[c])])
    pos_vals = t[pos_codes]
    fm = fp8.fmax(fmt)
    v = np.asarray(v, np.float32)
    sign = (v.view(np.uint32) >> 31).astype(np.uint8) << 7
    a = np.abs(v.astype(np.float64))
    out = np.zeros(v.shape, np.uint8)
    nan = np.isnan(a)
    sat = ~nan & (a >= fm)
    reg = ~nan & ~sat
    d = np.abs(a[reg][:, None] - pos_vals[None, :])
    best = d.min(axis=1, keepdims=True)
    cand = d == best
    # among tied candidates prefer the even code
    even = (pos_codes % 2 == 0)[None, :]
    pick = np.where((cand & even).any(axis=1), np.argmax(cand & even, axis=1), np.argmax(cand, axis=1))
    out[reg] = pos_codes[pick]
    out[sat] = pos_codes[np.argmax(pos_vals)]
    out |= sign
    out[nan] = 0x7F
    return out


@pytest.mark.parametrize("fmt", FMTS)
def test_brute_force_all_bf16_patterns(fmt):
    bits = np.arange(65536, dtype=np.uint32) << 16
    x = bits.view(np.float32)
    rs = [1.0, 448.0 / 3.140625, 2.0 ** 7, 2.0 ** -3, 57344.0 / 1000.0, 0.3359375]
    for r in rs:
        with np.errstate(over="ignore", invalid="ignore"):
            v = (x * np.float32(r)).astype(np.float32)
        assert np.array_equal(fp8.encode(v, fmt), _brute_force_encode(v, fmt)), r


@pytest.mark.parametrize("fmt", FMTS)
def test_brute_force_random_binary32(fmt):
    g = np.random.default_rng(1234)
    # random bit patterns concentrated on the format's range
    e = g.integers(-20, 18, 200000)
    m = g.random(200000) + 1.0
    v = (np.ldexp(m, e) * g.choice([-1, 1], 200000)).astype(np.float32)
    assert np.array_equal(fp8.encode(v, fmt), _brute_force_encode(v, fmt))


@pytest.mark.parametrize("fmt,tdt", [(fp8.E4M3, "float8_e4m3fn"), (fp8.E5M2, "float8_e5m2")])
def test_matches_torch_cpu_cast_in_range(fmt, tdt):
    torch = pytest.importorskip("torch")
    bits = np.arange(65536, dtype=np.uint32) << 16
    x = bits.view(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) <= fp8.fmax(fmt))]
    for r in (1.0, 3.0, 0.0078125):
        v = (x * np.float32(r)).astype(np.float32)
        v = v[np.abs(v) <= fp8.fmax(fmt)]
        t = torch.from_numpy(v).to(getattr(torch, tdt)).view(torch.uint8).numpy()
        assert np.array_equal(fp8.encode(v, fmt), t)
