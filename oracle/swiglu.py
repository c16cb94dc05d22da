"""SwiGLU of the MLP's fused gate/up output, quantised for the down projection.

Test infrastructure only (see the package docstring).

The model follows the Qwen3-1.7B architecture (Section 2, model architecture
and pretraining system), whose MLP computes down(silu(gate(x)) * up(x)). The
precision flow of Appendix C keeps the hidden flow in BF16 and quantises each
linear layer's input right before its GEMM (Section 3.2). Fusing the SwiGLU
with the down projection's input quantisation must therefore give the codes
and scales that quantising the BF16 tensor H = silu(g) * u gives.

Readings where the paper is silent (each restated in the design notes):

* The fused gate/up GEMM output gu is [R, 2C]: the gate half is columns
  [0, C) and the up half columns [C, 2C).
* silu(g) = g / (1 + exp(-g)) and H = silu(g) * u are evaluated in binary32
  from the BF16 inputs, then rounded to BF16 (round to nearest even).
* The binary32 evaluation of exp is not correctly rounded on either side, so
  H is not unique in its last BF16 bit: any BF16 value that an evaluation
  with relative error at most EPS = 2**-20 (plus 2**-148 absolute, for
  results in binary32's subnormal range) could round to is accepted; where
  e^-g overflows binary32 (g < -ln(FLT_MAX) = -88.72), a binary32
  evaluation of g / (1 + e^-g) is -0, so zero is accepted as well (the exact
  H is then below TINY * max(1, |u|), TINY = 2**-120). Above that point every
  step of a binary32 evaluation stays finite and, with gradual underflow,
  non-zero, and so must H. Where exactly one BF16
  value is accepted (almost everywhere) H is that value, rounded once from
  the float64 evaluation; the quantisation of every accepted H is the
  quantisers' (``oracle.quant``).

The backward (the gate/up projection's dY, quantised inside the op that
produces it) follows below with readings of its own.

Parity unpinned by the paper (it prints no SwiGLU values); pinned by the
closed forms and library special cases in tests/test_oracle_swiglu.py.
"""

import numpy as np

from . import bf16

EPS = 2.0 ** -20
TINY = 2.0 ** -120
# e^-g overflows binary32 for g below -ln(FLT_MAX)
G_OVERFLOW = -float(np.log(np.float64(np.finfo(np.float32).max)))


def split(gu_bits, cols):
    """Gate and up halves of gu [R, 2*cols] as float64 (exact from BF16)."""
    gu = np.asarray(gu_bits, dtype=np.uint16)
    assert gu.ndim == 2 and gu.shape[1] >= 2 * cols
    with np.errstate(invalid="ignore"):
        g = bf16.to_f32(gu[:, :cols]).astype(np.float64)
        u = bf16.to_f32(gu[:, cols:2 * cols]).astype(np.float64)
    return g, u


def silu_f64(g):
    """silu(g) = g / (1 + e^-g) in float64; -0 or 0 where e^-g overflows."""
    g = np.asarray(g, dtype=np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        return g / (1.0 + np.exp(-g))


def swiglu_f64(gu_bits, cols):
    """H = silu(g) * u in float64 (relative error a few 2**-53)."""
    g, u = split(gu_bits, cols)
    with np.errstate(over="ignore", invalid="ignore"):
        return silu_f64(g) * u


def swiglu_bf16_band(gu_bits, cols):
    """H rounded to BF16 from float64, and the band of accepted BF16 values.

    Returns (mid, lo, hi) BF16 bit patterns [R, cols]: mid is the rounding of
    the float64 value; since rounding is monotone the accepted values are
    those between lo and hi (as real numbers). In almost every element lo and
    hi are the same number, and H = mid is unique. NaN inputs give NaN.
    """
    g, u = split(gu_bits, cols)
    with np.errstate(over="ignore", invalid="ignore"):
        t = silu_f64(g) * u
        d = EPS * np.abs(t) + 2.0 ** -148 + np.where(g < G_OVERFLOW, TINY * np.maximum(1.0, np.abs(u)), 0.0)
        d = np.where(np.isfinite(t), d, 0.0)        # infinities are exact
        mid = bf16.from_f64_rne(t)
        lo = bf16.from_f64_rne(t - d)
        hi = bf16.from_f64_rne(t + d)
    return mid, lo, hi


# ---- backward: the gate/up projection's output gradient --------------------
#
# Readings (the paper states no SwiGLU detail; Section 3.2 quantises each
# GEMM's dY right before Dgrad and Wgrad):
#
# * From dH [R, C] and the saved gate/up output gu [R, 2C], the gradient of
#   the gate/up output is dgu [R, 2C] = [dg | du] with
#   dg = dH * u * silu'(g), du = dH * silu(g), silu'(g) = s (1 + g (1 - s)),
#   s = 1 / (1 + e^-g); each evaluated in binary32 and rounded once to BF16.
# * Accepted values: relative EPS as in the forward, plus for dg an absolute
#   2**-20 * |dH * u| * s**2 * |g| * min(1, 2**21 (1 - s)): silu' =
#   s (1 + g (1 - s)) is a difference near its zero (g ~ -1.28). In a binary32
#   evaluation every rounding is a few ulps of the result (covered by EPS)
#   except the error of 1 - s, which reaches silu' multiplied by s |g| and is
#   a few ulps of s (s * 2**-22 at most) or, where s rounds to 1, 1 - s
#   itself; the allowance covers s**2 |g| min(2**-22, 2 (1 - s)) four times;
#   plus the forward's allowances (2**-148 absolute, and
#   zero where e^-g overflows binary32, g < G_OVERFLOW: there s = 0 in
#   binary32 and both halves vanish; |dH| * max(1, |u|) * TINY bounds them).
BWD_ABS = 2.0 ** -20


def dsilu_f64(g):
    """silu'(g) = s (1 + g (1 - s)) with s = 1 / (1 + e^-g), float64."""
    g = np.asarray(g, dtype=np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        sg = 1.0 / (1.0 + np.exp(-g))
        return sg * (1.0 + g * (1.0 - sg))


def swiglu_bwd_f64(dh_bits, gu_bits, cols):
    """[dg | du] [R, 2 cols] in float64."""
    g, u = split(gu_bits, cols)
    with np.errstate(invalid="ignore"):
        dh = bf16.to_f32(np.asarray(dh_bits, dtype=np.uint16)[:, :cols]).astype(np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        return np.concatenate([dh * u * dsilu_f64(g), dh * silu_f64(g)], axis=1)


def swiglu_bwd_bf16_band(dh_bits, gu_bits, cols):
    """(mid, lo, hi) BF16 bit patterns of [dg | du] [R, 2 cols], as
    ``swiglu_bf16_band`` states them for H."""
    g, u = split(gu_bits, cols)
    with np.errstate(invalid="ignore"):
        dh = bf16.to_f32(np.asarray(dh_bits, dtype=np.uint16)[:, :cols]).astype(np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        t = swiglu_bwd_f64(dh_bits, gu_bits, cols)
        deep = np.where(g < G_OVERFLOW, TINY * np.abs(dh) * np.maximum(1.0, np.abs(u)), 0.0)
        sg = 1.0 / (1.0 + np.exp(-g))
        near_zero = np.where(np.isfinite(g),
                             BWD_ABS * np.abs(dh * u) * sg * sg * np.abs(g) * np.minimum(1.0, 2.0 ** 21 * (1.0 - sg)),
                             0.0)
        extra = np.concatenate([near_zero + deep, deep], axis=1)
        d = EPS * np.abs(t) + 2.0 ** -148 + extra
        d = np.where(np.isfinite(t), d, 0.0)
        return bf16.from_f64_rne(t), bf16.from_f64_rne(t - d), bf16.from_f64_rne(t + d)


def unique_mask(lo_bits, hi_bits):
    """Elements whose band holds one value (-0 and +0 count as one value,
    the sign then being mid's; NaN as one value)."""
    lo = bf16.to_f32(lo_bits)
    hi = bf16.to_f32(hi_bits)
    with np.errstate(invalid="ignore"):
        return (lo == hi) | (np.isnan(lo) & np.isnan(hi))
