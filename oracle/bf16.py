"""BF16 helpers for the oracle.

The linear layer takes BF16 inputs and weights and materialises a BF16 output
(Section 3.2; Appendix C, precision flow). BF16 is the upper half of a binary32
word (1 sign, 8 exponent, 7 mantissa bits), so widening to binary32 is exact.
"""

import numpy as np


def to_f32(bits):
    """uint16 BF16 bit patterns -> float32 values (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def from_f64_rne(x):
    """float64 values -> uint16 BF16 bit patterns, one round-to-nearest-even
    step from the float64 value (no intermediate binary32 rounding).

    Finite values are rounded onto the BF16 grid, whose spacing at |x| is
    2**(max(floor(log2|x|), -126) - 7); results above the largest finite BF16
    value (or exactly at the midpoint beyond it, which rounds to even) become
    infinity, as IEEE rounding does; NaN becomes the quiet NaN 0x7FC0.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    sign = np.signbit(x)
    a = np.abs(x)
    nan = np.isnan(x)
    inf = np.isinf(x)
    fin = ~(nan | inf)
    r = np.zeros_like(a)
    nz = fin & (a > 0)
    _, ex = np.frexp(a[nz])
    e = np.maximum(ex - 1, -126)
    q = np.ldexp(1.0, e - 7)
    r[nz] = np.rint(a[nz] / q) * q
    # every finite r is a binary32 value; values beyond BF16's range overflow
    maxbf = float(np.uint32(0x7F7F0000).view(np.float32))
    over = fin & (r > maxbf)
    with np.errstate(over="ignore"):
        f32 = r.astype(np.float32)
    bits = (f32.view(np.uint32) >> 16).astype(np.uint16)
    bits[over] = 0x7F80
    bits[inf] = 0x7F80
    bits = np.where(sign, bits | np.uint16(0x8000), bits)
    bits[nan] = 0x7FC0
    out[...] = bits
    return out
