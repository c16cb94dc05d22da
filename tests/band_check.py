"""Checks of a fused op + quantise result (SwiGLU, RMSNorm) against the
oracle's band of accepted BF16 values of the op's output (oracle/swiglu.py,
oracle/rmsnorm.py). No arithmetic of the method here: scales and codes come
from oracle.quant and oracle.fp8.

For every group (the whole tensor, 128 consecutive values along a row, or 128
down a column) the accepted amax values are those of the band; the result's
scale must be the scale of one of them (almost always there is one; a
group whose largest values all sit in a band around zero has many). With
that scale's multiplier, elements whose value is unique must carry exactly
the oracle's code, and every other element a code whose value lies between
the codes of the band's ends (codes are monotone in the value they encode).
"""

import numpy as np

from oracle import bf16, fp8, quant


def _groups(a, axis, size):
    """[R, C] -> [n_groups, size]: the whole tensor (axis None), runs of
    `size` along each row (axis 1) or down each column (axis 0)."""
    if axis is None:
        return a.reshape(1, -1)
    if axis == 0:
        a = a.T
    return a.reshape(a.shape[0], a.shape[1] // size, size).reshape(-1, size)


def _exponent(a, fmt, rule):
    return quant.pow2_exponent(a, fmt) if rule == "pow2" else quant.pow2_floor_exponent(a, fmt)


def _multiplier(s, a_lo, a_hi, fmt, rule):
    """The multiplier r of a group whose scale is s, if s is the scale of
    some amax in [a_lo, a_hi] (BF16 values); None if it is not."""
    s = np.float32(s)
    if np.isnan(a_lo) or np.isnan(a_hi):
        return np.float32(np.nan) if np.isnan(s) else None
    if rule != "fp32":
        if not np.isfinite(s) or s <= 0:
            return None
        e = int(np.frexp(float(s))[1]) - 1
        if float(s) != 2.0 ** e:
            return None
        ok = (a_lo == 0 and e == 0)
        if a_hi > 0:
            tiny = float(np.uint32(0x00010000).view(np.float32))     # the least positive BF16
            ok = ok or _exponent(max(float(a_lo), tiny), fmt, rule) <= e <= _exponent(float(a_hi), fmt, rule)
        return np.float32(2.0 ** -e) if ok else None
    if a_lo == 0 and s == 1:
        return np.float32(1.0)              # amax 0 (r = 1), or FMAX itself (r = 1 too)
    # the BF16 amax values whose scale is s: next to s * FMAX
    near = bf16.from_f64_rne(np.array([float(s) * fp8.fmax(fmt)]))[0]
    for b in (near, near - 1, near + 1):
        a = bf16.to_f32(np.array([b], np.uint16))[0]
        if a_lo <= a <= a_hi and a > 0:
            sa, ra = quant.tensor_scale(a, fmt)
            if np.float32(sa).view(np.uint32) == s.view(np.uint32):
                return ra
    return None


def amax_band(lo, hi):
    """The lowest and highest amax a tensor with these bands can have."""
    xl, xh = bf16.to_f32(lo), bf16.to_f32(hi)
    if np.isnan(xl).any() or np.isnan(xh).any():
        return np.float32(np.nan), np.float32(np.nan)
    least = np.where((xl <= 0) & (xh >= 0), np.float32(0), np.minimum(np.abs(xl), np.abs(xh)))
    return np.float32(least.max(initial=0)), np.float32(np.maximum(np.abs(xl), np.abs(xh)).max(initial=0))


def check(q, s, mid, lo, hi, unique, fmt, rule, axis=None, what="", tensor_amax=None):
    """q: codes [R, C] (or the transposed copy [C, R] when axis == 0, given
    here transposed back to [R, C]); s: scales, one per group in group order
    (row-major over the quantised copy). ``tensor_amax``: for a per-tensor
    check of a subset of the tensor, the whole tensor's (lowest, highest)
    accepted amax (``amax_band``). Raises AssertionError on a mismatch;
    returns the number of elements checked by membership rather than
    equality."""
    G = quant.GROUP
    xm, xl, xh = (_groups(bf16.to_f32(b), axis, G) for b in (mid, lo, hi))
    un = _groups(unique, axis, G)
    qc = _groups(np.asarray(q, dtype=np.uint8), axis, G)
    s = np.asarray(s, dtype=np.float32).reshape(-1)
    assert s.size == xm.shape[0], "%s: %d scales for %d groups" % (what, s.size, xm.shape[0])
    with np.errstate(invalid="ignore"):
        # the least magnitude in [lo, hi] (zero where the band spans it) and the greatest
        lo_mag = np.where((xl <= 0) & (xh >= 0), np.float32(0), np.minimum(np.abs(xl), np.abs(xh)))
        hi_mag = np.maximum(np.abs(xl), np.abs(xh))
    nan = np.isnan(xm).any(axis=1)
    a_lo = np.where(nan, np.float32(np.nan), lo_mag.max(axis=1))
    a_hi = np.where(nan, np.float32(np.nan), hi_mag.max(axis=1))
    if tensor_amax is not None:
        assert axis is None
        a_lo, a_hi = np.array([tensor_amax[0]], np.float32), np.array([tensor_amax[1]], np.float32)
    r = np.empty(xm.shape[0], dtype=np.float32)
    memo = {}
    for i in range(xm.shape[0]):
        key = (s[i].view(np.uint32).item(), float(a_lo[i]), float(a_hi[i]))
        if key not in memo:
            memo[key] = _multiplier(s[i], a_lo[i], a_hi[i], fmt, rule)
        if memo[key] is None:
            raise AssertionError("%s: group %d scale %r is not the scale of any amax in %r..%r" % (
                what, i, s[i], a_lo[i], a_hi[i]))
        r[i] = memo[key]
    rr = r[:, None]
    exp_mid = quant.encode_scaled(xm, rr, fmt)
    dec = fp8.decode(qc, fmt)
    dlo = fp8.decode(quant.encode_scaled(xl, rr, fmt), fmt)
    dhi = fp8.decode(quant.encode_scaled(xh, rr, fmt), fmt)
    bad_u = un & (qc != exp_mid)
    with np.errstate(invalid="ignore"):
        # (with a NaN scale every value encodes to NaN's code)
        inside = ((dlo <= dec) & (dec <= dhi)) | (np.isnan(dlo) & np.isnan(dhi) & np.isnan(dec))
    bad_b = ~un & ~inside
    if bad_u.any() or bad_b.any():
        i = np.argwhere(bad_u | bad_b)[0]
        idx = tuple(i)
        raise AssertionError("%s: %d unique and %d banded codes off; first at group %d elem %d: got 0x%02x "
                             "expected 0x%02x (H %r, band %r..%r)" % (
                                 what, bad_u.sum(), bad_b.sum(), idx[0], idx[1], qc[idx], exp_mid[idx],
                                 xm[idx], xl[idx], xh[idx]))
    return int((~un).sum())
