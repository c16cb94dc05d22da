"""OCP FP8 codecs: E4M3 ("E4M3FN") and E5M2.

Section 3.2 of the paper runs the linear-layer GEMM operands in E4M3 and names
E5M2 as the format with the wider range but fewer mantissa bits; both are the
formats of the FP8-formats proposal the paper cites (OCP 8-bit floating point).

Field layout (sign, exponent, mantissa) and special values:

* E4M3: 1.4.3, bias 7, no infinities, the only NaN pattern is S.1111.111,
  largest finite 1.75 * 2**8 = 448, smallest normal 2**-6, smallest
  subnormal 2**-9.
* E5M2: 1.5.2, bias 15, IEEE-like: S.11111.00 is +-Inf, S.11111.{01,10,11}
  are NaN, largest finite 1.75 * 2**15 = 57344, smallest normal 2**-14,
  smallest subnormal 2**-16.

Encoding (a reading; the paper does not spell out rounding): a binary32 value
``v`` is rounded to the nearest representable value with ties to the code
whose mantissa is even; magnitudes at or above the largest finite value
(including infinities) saturate to +-FMAX; every NaN maps to the one code 0x7F
(IEEE 754 leaves the sign of a NaN produced by arithmetic unspecified, so the
sign of a NaN carries no information); the sign of zero is kept.
"""

import functools

import numpy as np

E4M3 = "e4m3"
E5M2 = "e5m2"

# exponent bits, mantissa bits, exponent bias, largest finite value
_SPEC = {
    E4M3: dict(ebits=4, mbits=3, bias=7, fmax=448.0),
    E5M2: dict(ebits=5, mbits=2, bias=15, fmax=57344.0),
}


def fmax(fmt):
    """Largest finite magnitude of the format (448 or 57344)."""
    return _SPEC[fmt]["fmax"]


def emin(fmt):
    """Exponent of the smallest normal value (-6 or -14)."""
    return 1 - _SPEC[fmt]["bias"]


def mbits(fmt):
    return _SPEC[fmt]["mbits"]


def decode_code(code, fmt):
    """Value of one FP8 byte, written out from its sign/exponent/mantissa fields."""
    sp = _SPEC[fmt]
    eb, mb, bias = sp["ebits"], sp["mbits"], sp["bias"]
    sign = -1.0 if (code >> 7) & 1 else 1.0
    e = (code >> mb) & ((1 << eb) - 1)
    m = code & ((1 << mb) - 1)
    emax_field = (1 << eb) - 1
    if fmt == E4M3:
        if e == emax_field and m == (1 << mb) - 1:
            return float("nan")
    else:
        if e == emax_field:
            return sign * float("inf") if m == 0 else float("nan")
    if e == 0:
        return sign * m * 2.0 ** (1 - bias - mb)
    return sign * (1.0 + m / (1 << mb)) * 2.0 ** (e - bias)


@functools.lru_cache(maxsize=None)
def _table(fmt):
    t = np.array([decode_code(c, fmt) for c in range(256)], dtype=np.float64)
    t.setflags(write=False)
    return t


def decode_table(fmt):
    """float64[256]: the value of every byte (NaN for NaN codes)."""
    return _table(fmt).copy()


def _positive_value_to_code(fmt):
    tab = decode_table(fmt)
    out = {}
    for c in range(128):
        v = tab[c]
        if np.isfinite(v):
            out[float(v)] = c
    return out


_V2C = {E4M3: _positive_value_to_code(E4M3), E5M2: _positive_value_to_code(E5M2)}


def _round_to_grid(a, fmt):
    """Round finite magnitudes ``a`` (< FMAX, float64 holding binary32 values)
    to the format's grid, ties to even.

    The grid spacing at ``a`` is 2**(max(floor(log2 a), emin) - mbits); ``a``
    divided by the spacing is exact in float64, and ``np.rint`` rounds half to
    even, which picks the even mantissa because the spacing is one unit of the
    last mantissa place.
    """
    a = np.asarray(a, dtype=np.float64)
    out = np.zeros_like(a)
    nz = a > 0
    _, ex = np.frexp(a[nz])           # a = f * 2**ex, f in [0.5, 1)
    e = np.maximum(ex - 1, emin(fmt))  # floor(log2 a), clamped to the subnormal range
    quantum = np.ldexp(1.0, e - mbits(fmt))
    out[nz] = np.rint(a[nz] / quantum) * quantum
    return out


def encode(v, fmt):
    """binary32 array -> uint8 FP8 codes (RNE, saturating, NaN -> 0x7F)."""
    v = np.asarray(v, dtype=np.float32)
    bits = v.view(np.uint32)
    sign = ((bits >> 31) & 1).astype(np.uint8) << 7
    a = np.abs(v.astype(np.float64))
    out = np.zeros(v.shape, dtype=np.uint8)
    isnan = np.isnan(a)
    sat = (~isnan) & (a >= fmax(fmt))
    reg = (~isnan) & (~sat)
    fm = fmax(fmt)
    out[isnan] = 0x7F
    out[sat] = _V2C[fmt][fm]
    r = _round_to_grid(a[reg], fmt)
    out[reg] = _lookup(r, fmt)
    out[~isnan] |= sign[~isnan]
    return out


def _lookup(r, fmt):
    """Code of each grid value in ``r`` (non-negative), by search in the
    sorted table of the non-negative finite codes."""
    tab = _table(fmt)[:128]
    finite = np.isfinite(tab)
    vals = tab[finite]
    codes = np.arange(128)[finite]
    order = np.argsort(vals)
    vals, codes = vals[order], codes[order]
    idx = np.searchsorted(vals, r)
    if not np.all(vals[np.minimum(idx, len(vals) - 1)] == r):
        raise AssertionError("rounded value not on the format grid")
    return codes[idx].astype(np.uint8)


def decode(codes, fmt):
    """uint8 codes -> float64 values through the 256-entry table."""
    return _table(fmt)[np.asarray(codes, dtype=np.uint8)]
