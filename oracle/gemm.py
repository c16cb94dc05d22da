"""Scaled FP8 GEMM of the oracle (FP64), and an exact-rational version.

D[m, n] = sum_k A[m, k] * B[n, k] with both operands stored reduction-index
contiguous; Fprop, Dgrad and Wgrad of Section 3.2 are all of this form once
their operands are laid out that way (the linear composition in
``oracle.linear`` does so).

Accuracy: E4M3 values are integer multiples of 2**-9 and below 2**9, so an
E4M3 x E4M3 product is a multiple of 2**-18 below 2**18 and every partial sum
over k < 2**17 terms stays an integer multiple of 2**-18 below 2**53 of those
units: the FP64 sum is exact. With E5M2 operands or longer sums the FP64
rounding error is at most about K * 2**-53 of sum |a*b|, far below the 1e-5
relative tolerance the GPU results are held to. Power-of-two block scales keep
exactness; per-tensor binary32 scales are applied once to the exact sum.

The C loop lives in ``gemm_fp64.c`` and is compiled by ``build_oracle.py``.
"""

import ctypes
import os
from fractions import Fraction

import numpy as np

from . import fp8

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle_gemm.so")

MODES = {"tensor": 0, "row": 1, "block": 2}

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build_oracle
            build_oracle.build()
        lib = ctypes.CDLL(LIB_PATH)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        common = [i64, p, i64, p, p, ctypes.c_int, i64, p, i64, p, p, ctypes.c_int, i64, p, p]
        lib.oracle_gemm_fp64.argtypes = [i64, i64, i64] + common
        lib.oracle_gemm_fp64.restype = None
        lib.oracle_gemm_fp64_entries.argtypes = [i64, p, p, i64] + common
        lib.oracle_gemm_fp64_entries.restype = None
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _operand(codes, fmt, scale, mode):
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    scale = np.ascontiguousarray(np.atleast_1d(np.asarray(scale, dtype=np.float32)))
    lut = np.ascontiguousarray(fp8.decode_table(fmt))
    ld_s = scale.shape[-1] if (mode != "tensor" and scale.ndim == 2) else 1
    return codes, lut, scale, MODES[mode], ld_s


def _kblock(K, a_mode, b_mode):
    if a_mode == "tensor" and b_mode == "tensor":
        return max(K, 1)
    return 128


def gemm(a, a_fmt, a_scale, a_mode, b, b_fmt, b_scale, b_mode):
    """Full FP64 product: returns (ref [M, N], den [M, N]) as float64.

    a: [M, K] codes; b: [N, K] codes; scales per ``MODES`` (a scalar for
    "tensor", [rows, K/128] for "row", [rows/128, K/128] for "block").
    """
    ac, alut, asc, am, ald = _operand(a, a_fmt, a_scale, a_mode)
    bc, blut, bsc, bm, bld = _operand(b, b_fmt, b_scale, b_mode)
    M, K = ac.shape
    N = bc.shape[0]
    assert bc.shape[1] == K
    ref = np.zeros((M, N), dtype=np.float64)
    den = np.zeros((M, N), dtype=np.float64)
    _load().oracle_gemm_fp64(M, N, K, _kblock(K, a_mode, b_mode),
                             _ptr(ac), K, _ptr(alut), _ptr(asc), am, ald,
                             _ptr(bc), K, _ptr(blut), _ptr(bsc), bm, bld,
                             _ptr(ref), _ptr(den))
    return ref, den


def gemm_entries(ms, ns, a, a_fmt, a_scale, a_mode, b, b_fmt, b_scale, b_mode):
    """Selected entries (ms[i], ns[i]) of the same product: (ref, den) [count]."""
    ac, alut, asc, am, ald = _operand(a, a_fmt, a_scale, a_mode)
    bc, blut, bsc, bm, bld = _operand(b, b_fmt, b_scale, b_mode)
    K = ac.shape[1]
    assert bc.shape[1] == K
    ms = np.ascontiguousarray(ms, dtype=np.int64)
    ns = np.ascontiguousarray(ns, dtype=np.int64)
    assert ms.shape == ns.shape
    assert ms.size == 0 or (ms.min() >= 0 and ms.max() < ac.shape[0])
    assert ns.size == 0 or (ns.min() >= 0 and ns.max() < bc.shape[0])
    ref = np.zeros(ms.shape, dtype=np.float64)
    den = np.zeros(ms.shape, dtype=np.float64)
    _load().oracle_gemm_fp64_entries(ms.size, _ptr(ms), _ptr(ns), K, _kblock(K, a_mode, b_mode),
                                     _ptr(ac), K, _ptr(alut), _ptr(asc), am, ald,
                                     _ptr(bc), K, _ptr(blut), _ptr(bsc), bm, bld,
                                     _ptr(ref), _ptr(den))
    return ref, den


def epilogue(ref, den, bias=None, residual=None):
    """The BF16 bias / residual epilogue of a linear layer's GEMM (the bias
    of Qwen2's QKV projection; the residual stream the attention output and
    MLP down projections add into, BF16 per the Appendix C precision flow):
    the exact value ref + bias + residual, and its tolerance scale
    den + |bias| + |residual| (every binary32 addition of the epilogue rounds
    by at most 2**-24 of the magnitudes summed). bias and residual are
    float64 values broadcast against ref (None: absent)."""
    ref = np.asarray(ref, dtype=np.float64)
    den = np.asarray(den, dtype=np.float64)
    for t in (bias, residual):
        if t is not None:
            t = np.asarray(t, dtype=np.float64)
            ref = ref + t
            den = den + np.abs(t)
    return ref, den


def _scale_of(scale, mode, i, kb):
    s = np.asarray(scale, dtype=np.float32)
    if mode == "tensor":
        return Fraction(float(s.reshape(-1)[0]))
    if mode == "row":
        return Fraction(float(s[i, kb]))
    return Fraction(float(s[i // 128, kb]))


def gemm_exact(a, a_fmt, a_scale, a_mode, b, b_fmt, b_scale, b_mode):
    """The same product in exact rational arithmetic (tiny inputs only).

    Returns a nested list of ``fractions.Fraction`` [M][N].
    """
    a = np.asarray(a, dtype=np.uint8)
    b = np.asarray(b, dtype=np.uint8)
    M, K = a.shape
    N = b.shape[0]
    va = [[Fraction(float(fp8.decode_code(int(c), a_fmt))) for c in row] for row in a]
    vb = [[Fraction(float(fp8.decode_code(int(c), b_fmt))) for c in row] for row in b]
    out = []
    for m in range(M):
        row = []
        for n in range(N):
            acc = Fraction(0)
            for k in range(K):
                kb = k // 128
                acc += (_scale_of(a_scale, a_mode, m, kb) * va[m][k]
                        * _scale_of(b_scale, b_mode, n, kb) * vb[n][k])
            row.append(acc)
        out.append(row)
    return out
