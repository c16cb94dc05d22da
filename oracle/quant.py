"""amax, scale rules and quantisers of the FP8 linear layer.

Section 3.2 of the paper: a linear layer quantises its BF16 inputs and weights
immediately before each GEMM, with scales computed online from the data. With
one scale for a whole tensor a few outliers widen the quantisation interval;
the production recipe therefore groups activations and activation gradients
in runs of 128 consecutive values along the GEMM's reduction dimension and
weights in 128x128 blocks, and each block scale is a power of two (the
exponent-only E8M0 representation of MXFP8).

Readings where the paper is silent (each restated in the design notes):

* Per-tensor scale: s = fl32(amax / FMAX) is the stored dequantisation scale
  and the values are multiplied by r = fl32(FMAX / amax) before encoding;
  amax = 0 gives s = r = 1.
* Power-of-two scale: s = 2**e with e the smallest integer such that
  amax <= FMAX * 2**e (so no value saturates), clamped to the E8M0 range
  [-127, 127]; amax = 0 gives e = 0; a NaN amax gives s = r = NaN.
* The alternative power-of-two rule of the OCP Microscaling (MX) formats,
  kept for comparison: e = floor(log2 amax) - emax, emax the exponent of the
  format's largest normal value (8 for E4M3, 15 for E5M2), with the same
  clamp and special cases. It keeps one more bit of the block's range in the
  top binade but saturates the largest values of a block whose amax has a
  significand above FMAX's (1.75).
* Encoding of a value x: FP8-encode fl32(x * r) (round to nearest even,
  saturating; see ``oracle.fp8``).
* The 128x1 (column) groups used by Wgrad are quantised from the BF16 data,
  not from the row-grouped bytes, and are stored transposed so that the
  reduction dimension is contiguous.
"""

import numpy as np

from . import bf16, fp8

GROUP = 128


def amax(x_f32):
    """max |x| over all elements; NaN if any element is NaN; 0 for empty."""
    x = np.asarray(x_f32, dtype=np.float32)
    if x.size == 0:
        return np.float32(0.0)
    return np.float32(np.max(np.abs(x)))


def tensor_scale(a, fmt):
    """Per-tensor rule: (s, r) = (amax / FMAX, FMAX / amax) in binary32."""
    a = np.float32(a)
    fm = np.float32(fp8.fmax(fmt))
    if a == 0:
        return np.float32(1.0), np.float32(1.0)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        return np.float32(a / fm), np.float32(fm / a)


def pow2_exponent(a, fmt):
    """Smallest integer e with a <= FMAX * 2**e, clamped to [-127, 127].

    Found by exact comparisons in float64 (FMAX * 2**e is exact there, and so
    is every binary32 amax). amax = 0 gives 0; NaN gives None.
    """
    a = float(np.float32(a))
    if np.isnan(a):
        return None
    if a == 0.0:
        return 0
    fm = fp8.fmax(fmt)
    e = -127
    while e < 127 and a > fm * 2.0 ** e:
        e += 1
    return e


def emax(fmt):
    """Exponent of the format's largest normal value (FMAX = 1.75 * 2**emax)."""
    return int(np.frexp(fp8.fmax(fmt))[1]) - 1


def pow2_floor_exponent(a, fmt):
    """OCP-MX rule: floor(log2 a) - emax, clamped to [-127, 127].

    floor(log2 a) is read exactly from the binary exponent (frexp gives
    a = m * 2**x with m in [0.5, 1), so floor(log2 a) = x - 1). amax = 0
    gives 0, an infinite amax 127, NaN None.
    """
    a = float(np.float32(a))
    if np.isnan(a):
        return None
    if a == 0.0:
        return 0
    if np.isinf(a):
        return 127
    e = int(np.frexp(a)[1]) - 1 - emax(fmt)
    return max(-127, min(127, e))


def pow2_scale(a, fmt, rule="pow2"):
    """Power-of-two rule: (s, r) = (2**e, 2**-e) as binary32 (NaN for NaN);
    e from ``pow2_exponent`` ("pow2") or ``pow2_floor_exponent``
    ("pow2_floor")."""
    e = pow2_exponent(a, fmt) if rule == "pow2" else pow2_floor_exponent(a, fmt)
    if e is None:
        return np.float32(np.nan), np.float32(np.nan)
    return np.float32(2.0 ** e), np.float32(2.0 ** (-e))


def encode_scaled(x_f32, r, fmt):
    """FP8 codes of fl32(x * r)."""
    with np.errstate(over="ignore", invalid="ignore"):
        v = (np.asarray(x_f32, dtype=np.float32) * np.float32(r)).astype(np.float32)
    return fp8.encode(v, fmt)


def quantize_tensor(x_bits, fmt, amax_in=None, rule="fp32"):
    """One scale for the whole [R, C] BF16 tensor.

    Returns (q [R, C] uint8, qT [C, R] uint8, s float32, amax float32).
    ``amax_in`` replaces the tensor's own amax when given. ``rule`` is "fp32"
    (amax / FMAX), "pow2" or "pow2_floor".
    """
    x = bf16.to_f32(x_bits)
    a = amax(x) if amax_in is None else np.float32(amax_in)
    s, r = tensor_scale(a, fmt) if rule == "fp32" else pow2_scale(a, fmt, rule)
    q = encode_scaled(x, r, fmt)
    return q, np.ascontiguousarray(q.T), s, a


def quantize_rows_1x128(x_bits, fmt, rule="pow2"):
    """Groups of 128 consecutive values along each row (the reduction
    dimension of the GEMM that consumes the [R, C] tensor); ``rule`` is the
    power-of-two rule ("pow2" or "pow2_floor").

    Returns (q [R, C] uint8, s [R, C/128] float32).
    """
    x = bf16.to_f32(x_bits)
    R, C = x.shape
    assert C % GROUP == 0
    q = np.empty((R, C), dtype=np.uint8)
    s = np.empty((R, C // GROUP), dtype=np.float32)
    for i in range(R):
        for g in range(C // GROUP):
            blk = x[i, g * GROUP:(g + 1) * GROUP]
            si, ri = pow2_scale(amax(blk), fmt, rule)
            s[i, g] = si
            q[i, g * GROUP:(g + 1) * GROUP] = encode_scaled(blk, ri, fmt)
    return q, s


def quantize_cols_128x1(x_bits, fmt, rule="pow2"):
    """Groups of 128 consecutive values down each column of the [R, C]
    tensor (the reduction dimension of Wgrad), stored transposed.

    Returns (qT [C, R] uint8, sT [C, R/128] float32).
    """
    xT = np.ascontiguousarray(np.asarray(x_bits, dtype=np.uint16).T)
    return quantize_rows_1x128(xT, fmt, rule)


def quantize_blocks_128x128(x_bits, fmt, rule="pow2"):
    """One power-of-two scale per 128x128 block of the [R, C] tensor.

    Returns (q [R, C], s [R/128, C/128], qT [C, R], sT [C/128, R/128]); the
    transposed pair holds the same bytes and scales, transposed.
    """
    x = bf16.to_f32(x_bits)
    R, C = x.shape
    assert R % GROUP == 0 and C % GROUP == 0
    q = np.empty((R, C), dtype=np.uint8)
    s = np.empty((R // GROUP, C // GROUP), dtype=np.float32)
    for bi in range(R // GROUP):
        for bj in range(C // GROUP):
            blk = x[bi * GROUP:(bi + 1) * GROUP, bj * GROUP:(bj + 1) * GROUP]
            sb, rb = pow2_scale(amax(blk), fmt, rule)
            s[bi, bj] = sb
            q[bi * GROUP:(bi + 1) * GROUP, bj * GROUP:(bj + 1) * GROUP] = encode_scaled(blk, rb, fmt)
    return q, s, np.ascontiguousarray(q.T), np.ascontiguousarray(s.T)
