"""Checks of a fused SwiGLU + quantise result against the oracle's band of
accepted BF16 H values (oracle/swiglu.py). No arithmetic of the method here:
scales and codes come from oracle.quant and oracle.fp8.

For every group (the whole tensor, 128 consecutive values along a row, or 128
down a column) the accepted amax values are those of the band; the result's
scale must be the scale of one of them (almost always there is one). With
that scale's multiplier, elements whose H is unique must carry exactly the
oracle's code, and every other element a code whose value lies between the
codes of the band's ends (codes are monotone in the value they encode).
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


def _scale(a, fmt, rule):
    if rule == "fp32":
        return quant.tensor_scale(a, fmt)
    return quant.pow2_scale(a, fmt, rule)


def check(q, s, mid, lo, hi, unique, fmt, rule, axis=None, what=""):
    """q: codes [R, C] (or the transposed copy [C, R] when axis == 0, given
    here transposed back to [R, C]); s: scales, one per group in group order
    (row-major over the quantised copy). Raises AssertionError on a mismatch;
    returns the number of elements checked by membership rather than
    equality."""
    G = quant.GROUP
    xm, xl, xh = (_groups(bf16.to_f32(b), axis, G) for b in (mid, lo, hi))
    un = _groups(unique, axis, G)
    qc = _groups(np.asarray(q, dtype=np.uint8), axis, G)
    s = np.asarray(s, dtype=np.float32).reshape(-1)
    assert s.size == xm.shape[0], "%s: %d scales for %d groups" % (what, s.size, xm.shape[0])
    with np.errstate(invalid="ignore"):
        lo_mag = np.minimum(np.abs(xl), np.abs(xh))
        hi_mag = np.maximum(np.abs(xl), np.abs(xh))
    nan = np.isnan(xm).any(axis=1)
    a_lo = np.where(nan, np.float32(np.nan), lo_mag.max(axis=1))
    a_hi = np.where(nan, np.float32(np.nan), hi_mag.max(axis=1))
    r = np.empty(xm.shape[0], dtype=np.float32)
    for i in range(xm.shape[0]):
        cands = {}
        for a in (a_lo[i], a_hi[i]):
            si, ri = _scale(np.float32(a), fmt, rule)
            cands[np.float32(si).view(np.uint32).item()] = ri
        got = s[i].view(np.uint32).item()
        if got not in cands:
            raise AssertionError("%s: group %d scale %r not among %r (amax %r..%r)" % (
                what, i, s[i], [np.uint32(k).view(np.float32) for k in cands], a_lo[i], a_hi[i]))
        r[i] = cands[got]
    rr = r[:, None]
    exp_mid = quant.encode_scaled(xm, rr, fmt)
    dec = fp8.decode(qc, fmt)
    dlo = fp8.decode(quant.encode_scaled(xl, rr, fmt), fmt)
    dhi = fp8.decode(quant.encode_scaled(xh, rr, fmt), fmt)
    bad_u = un & (qc != exp_mid)
    with np.errstate(invalid="ignore"):
        inside = (dlo <= dec) & (dec <= dhi)
    bad_b = ~un & ~inside
    if bad_u.any() or bad_b.any():
        i = np.argwhere(bad_u | bad_b)[0]
        idx = tuple(i)
        raise AssertionError("%s: %d unique and %d banded codes off; first at group %d elem %d: got 0x%02x "
                             "expected 0x%02x (H %r, band %r..%r)" % (
                                 what, bad_u.sum(), bad_b.sum(), idx[0], idx[1], qc[idx], exp_mid[idx],
                                 xm[idx], xl[idx], xh[idx]))
    return int((~un).sum())
