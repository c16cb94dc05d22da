"""RMSNorm ahead of a linear layer's input quantisation.

Test infrastructure only (see the package docstring).

The model follows the Qwen3-1.7B architecture (Section 2, Pipeline at a
Glance): every attention and MLP block starts with an RMSNorm whose output is
the input X of the next linear layer (QKV, gate/up). The precision flow of
Appendix C keeps the norm in BF16 and quantises each linear layer's input
right before its GEMM (Section 3.2). Fusing the norm with the quantisation
must therefore give the codes and scales that quantising the BF16 norm output
gives, and the per-row reciprocal RMS that the norm's backward reuses.

Readings where the paper is silent (each restated in the design notes):

* y = x * rstd * gamma with rstd = 1 / sqrt(mean(x^2) + eps) over the row,
  evaluated in binary32 from the BF16 x and gamma, rounded once to BF16 (as
  the Transformer Engine norm the paper's Megatron stack runs does); eps is
  an argument (1e-6 in Qwen3).
* The binary32 sum of squares depends on its order, so y is not unique in its
  last BF16 bit: any BF16 value within relative EPS = 2**-16 of the float64 y
  is accepted (a binary32 sum of d terms in a tree of chunk sums is within
  about (chunk + log2 d) * 2**-24 of the exact sum; rsqrt and two products
  add a few ulp). The accepted rstd is likewise within EPS of the float64
  value. The quantisation of every accepted y is the quantisers'.
* Rows whose sum of squares overflows binary32 (|x| near 2**63 and above)
  are outside this statement: binary32 gives rstd = 0 there.

Parity unpinned by the paper (it prints no norm values); pinned by closed
forms and numpy's vector norm in tests/test_oracle_rmsnorm.py.
"""

import numpy as np

from . import bf16

EPS = 2.0 ** -16


def rstd_f64(x_bits, eps):
    """1 / sqrt(mean(x^2) + eps) per row, float64."""
    x = bf16.to_f32(x_bits).astype(np.float64)
    return 1.0 / np.sqrt(np.mean(x * x, axis=1) + float(np.float32(eps)))


def rmsnorm_f64(x_bits, gamma_bits, eps):
    """y = x * rstd * gamma in float64 [R, C]."""
    x = bf16.to_f32(x_bits).astype(np.float64)
    g = bf16.to_f32(gamma_bits).astype(np.float64)
    return x * rstd_f64(x_bits, eps)[:, None] * g[None, :]


def rmsnorm_bf16_band(x_bits, gamma_bits, eps):
    """y rounded to BF16 from float64, and the band of accepted BF16 values:
    (mid, lo, hi) BF16 bit patterns [R, C], as in ``oracle.swiglu``."""
    t = rmsnorm_f64(x_bits, gamma_bits, eps)
    d = EPS * np.abs(t)
    return bf16.from_f64_rne(t), bf16.from_f64_rne(t - d), bf16.from_f64_rne(t + d)
