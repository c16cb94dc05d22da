"""Summation behaviour of the gfx950 FP8 matrix instructions, as measured.

Neither the paper nor the method fixes how a matrix unit adds FP8 products;
this module states the behaviour of v_mfma_scale_f32_32x32x64_f8f6f4 (and
16x16x128) that the probes under tests/test_gpu_mfma_model.py pin on the
hardware:

* the products of each aligned run of GROUP = 8 consecutive k (in the order
  the GEMM kernel feeds the instruction, which is ascending k) are added as a
  group;
* inside a group every product a_k * b_k is truncated toward zero to a
  multiple of u = 2**(E - WINDOW), WINDOW = 13, where E is the largest
  exponent sum e(a_k) + e(b_k) in the group (the exponents of the operands,
  not of the product: a significand product of 2 or more does not move the
  window); the truncated products then add exactly. For subnormal operands
  e is taken as the format's smallest normal exponent, which can only make
  the modelled grid coarser than the hardware's, so the loss computed below
  stays an upper bound;
* group sums and the FP32 accumulator combine with ordinary FP32 rounding.

The GEMM tests compare the GPU result with the oracle's exact FP64 sum and
allow, per output entry, the tolerance 1e-5 * sum_k |a_k b_k| (FP32
accumulation and rounding of the result) plus the exact amount the truncation
above removes for that entry's data (``truncation_loss``).
"""

import numpy as np

from oracle import fp8

GROUP = 8
WINDOW = 13


def exponents(fmt):
    """float64[256]: the exponent e(code) the instruction aligns by (unbiased
    exponent of normal codes, the smallest normal exponent for subnormals,
    -inf for zero; NaN/Inf codes get +inf and never occur in the tests)."""
    v = fp8.decode(np.arange(256, dtype=np.uint8), fmt)
    out = np.full(256, np.inf)
    fin = np.isfinite(v)
    a = np.abs(v[fin])
    _, ex = np.frexp(np.where(a > 0, a, 1.0))
    e = np.maximum(ex - 1, fp8.emin(fmt)).astype(np.float64)
    out[fin] = np.where(a > 0, e, -np.inf)
    return out


def truncate_groups(p, e):
    """p [..., K] float64 products and e [..., K] their operand exponent sums
    (-inf for zero products; K % GROUP == 0) -> the products after the
    in-group truncation."""
    shp = p.shape
    g = p.reshape(shp[:-1] + (shp[-1] // GROUP, GROUP))
    emax = np.asarray(e, dtype=np.float64).reshape(g.shape).max(axis=-1, keepdims=True)
    live = np.isfinite(emax)
    u = np.ldexp(1.0, np.where(live, emax, 0).astype(np.int64) - WINDOW)
    t = np.trunc(g / u) * u
    return np.where(live, t, 0.0).reshape(shp)


def _scale_rows(scale, mode, rows, nkb):
    """Per-row, per-128-k-block scale factors [len(rows), nkb] (float64)."""
    s = np.asarray(scale, dtype=np.float64)
    if mode == "tensor":
        return np.full((len(rows), nkb), float(s.reshape(-1)[0]))
    if mode == "row":
        return s[rows][:, :nkb]
    return s[np.asarray(rows) // 128][:, :nkb]


def truncation_loss(ms, ns, a, a_fmt, a_scale, a_mode, b, b_fmt, b_scale, b_mode, chunk=4096):
    """For each entry (ms[i], ns[i]) of D = A B^T: sum over k of |p_k - t_k| with
    p the scaled product and t its truncated value (float64, exact)."""
    a = np.asarray(a, dtype=np.uint8)
    b = np.asarray(b, dtype=np.uint8)
    va, vb = fp8.decode(a, a_fmt), fp8.decode(b, b_fmt)
    xa, xb = exponents(a_fmt)[a], exponents(b_fmt)[b]
    ms = np.asarray(ms, dtype=np.int64)
    ns = np.asarray(ns, dtype=np.int64)
    K = va.shape[1]
    Kp = (K + 127) // 128 * 128
    out = np.zeros(ms.shape, dtype=np.float64)
    for c0 in range(0, ms.size, chunk):
        mm, nn = ms[c0:c0 + chunk], ns[c0:c0 + chunk]
        p = np.zeros((mm.size, Kp))
        p[:, :K] = va[mm] * vb[nn]
        e = np.full((mm.size, Kp), -np.inf)
        e[:, :K] = xa[mm] + xb[nn]
        loss = np.abs(p - truncate_groups(p, e)).reshape(mm.size, Kp // 128, 128).sum(axis=-1)
        sa = _scale_rows(a_scale, a_mode, mm, Kp // 128)
        sb = _scale_rows(b_scale, b_mode, nn, Kp // 128)
        out[c0:c0 + chunk] = (loss * np.abs(sa * sb)).sum(axis=-1)
    return out


def truncation_loss_full(a, a_fmt, a_scale, a_mode, b, b_fmt, b_scale, b_mode):
    M, N = np.asarray(a).shape[0], np.asarray(b).shape[0]
    mm, nn = np.meshgrid(np.arange(M), np.arange(N), indexing="ij")
    return truncation_loss(mm.ravel(), nn.ravel(), a, a_fmt, a_scale, a_mode, b, b_fmt, b_scale,
                           b_mode).reshape(M, N)
