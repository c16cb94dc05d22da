"""The language-model head with its cross-entropy loss, forward and backward.

Test infrastructure only (see the package docstring).

Section 3.1.3 of the paper names the LM head as the layer whose cost sets the
pipeline's last stage apart, and the precision flow of Appendix C keeps it in
BF16 while the transformer blocks' linear layers run in FP8. The operation:
for hidden states X [M, K] (BF16), the output embedding W [V, K] (BF16) and a
target token t_m per row,

    z = X W^T                                   logits [M, V]
    lse_m = log sum_v exp(z_mv)                 (log-sum-exp per row)
    loss_m = lse_m - z_{m, t_m}                 (cross-entropy per token)
    dz_mv = g (exp(z_mv - lse_m) - [v == t_m])  (gradient of g * loss_m)
    dX = dz W,  dW = dz^T X.

Here it is stated in float64, which is exact for the BF16 products; the sums
over K and V round at a few 2**-53. Two recipes (the readings, each restated in
the design notes):

* BF16 (as the paper runs the LM head): the GEMMs take the BF16 operands and
  accumulate in binary32; the logits stay binary32 inside the fused operation
  (they are never stored); dz is rounded to BF16, the operand precision of the
  backward GEMMs; dX is BF16, dW binary32.
* FP8 (the blockwise recipe of Section 3.2 applied to this layer): X in 1x128
  row groups for the logits GEMM and 128x1 column groups for dW, W in 128x128
  blocks, dz rounded to BF16 and then quantised in 1x128 row groups (along V,
  for dX) and 128x1 column groups (along M, for dW); E4M3 with power-of-two
  scales throughout. The GEMMs take the dequantised codes.

Which values a binary32 evaluation may give is stated as a band around the
float64 value: the logits within TOL_Z of sum_k |x_k w_k| (the GEMMs' binary32
accumulation) plus what the matrix instruction's truncation may remove (a
caller-supplied allowance), lse within the largest logit allowance of its row
plus LSE_ABS, and dz within the resulting relative error of exp(z - lse).

Parity unpinned by the paper (it prints no LM-head values); pinned by the
library routine scipy.special.logsumexp, the identities sum_v dz_mv = 0 and
dz = d(g loss)/dz (finite differences), and closed forms (two classes,
uniform logits) in tests/test_oracle_lm_head.py.
"""

import numpy as np

from . import bf16

TOL_Z = 1e-5           # binary32 accumulation of a logit, relative to sum_k |x_k w_k|
LSE_ABS = 2.0 ** -16   # binary32 evaluation of log(sum exp) over up to 2^18 terms
EXP_REL = 2.0 ** -20   # binary32 exp and its argument's rounding, relative


def to_f64(bits):
    return bf16.to_f32(np.asarray(bits, dtype=np.uint16)).astype(np.float64)


def logits(X_bits, W_bits):
    """z = X W^T and S = |X| |W|^T (float64, [M, V]) from BF16 operands."""
    x, w = to_f64(X_bits), to_f64(W_bits)
    return x @ w.T, np.abs(x) @ np.abs(w).T


def log_sum_exp(z):
    """log sum_v exp(z_v) per row, shifted by the row maximum (float64)."""
    z = np.asarray(z, dtype=np.float64)
    m = np.max(z, axis=1, keepdims=True)
    return (m + np.log(np.sum(np.exp(z - m), axis=1, keepdims=True)))[:, 0]


def forward(z, targets):
    """(lse [M], loss [M]) with loss_m = lse_m - z_{m, t_m}."""
    lse = log_sum_exp(z)
    zt = np.asarray(z, dtype=np.float64)[np.arange(z.shape[0]), np.asarray(targets)]
    return lse, lse - zt


def dlogits(z, lse, targets, g=1.0):
    """dz = g (softmax(z) - onehot(t)) [M, V] in float64."""
    p = np.exp(np.asarray(z, dtype=np.float64) - np.asarray(lse, dtype=np.float64)[:, None])
    p[np.arange(p.shape[0]), np.asarray(targets)] -= 1.0
    return g * p


def tolerances(z, S, targets, slack=0.0):
    """Allowances of a binary32 evaluation: per logit za[m, v] = TOL_Z *
    S[m, v] + slack (lse is 1-Lipschitz in the largest logit error); per row
    lse_tol[m] = max_v za[m, v] + LSE_ABS (1 + |lse_m|); and the loss's
    loss_tol[m] = lse_tol[m] + za[m, t_m]."""
    za = TOL_Z * np.asarray(S, dtype=np.float64) + slack
    lse = log_sum_exp(z)
    lse_tol = np.max(za, axis=1) + LSE_ABS * (1.0 + np.abs(lse))
    zt_tol = za[np.arange(za.shape[0]), np.asarray(targets)]
    return za, lse_tol, lse_tol + zt_tol


def dlogits_band(z, S, targets, g=1.0, slack=0.0):
    """(mid, lo, hi) BF16 bit patterns of dz: mid is the rounding of the float64
    value; lo and hi the roundings of its ends under the allowances above
    (exp(z - lse) moves by at most |d(z - lse)| + EXP_REL relative). As in
    the other bands, rounding is monotone, so the accepted values are those
    between lo and hi."""
    za, lse_tol, _ = tolerances(z, S, targets, slack)
    lse = log_sum_exp(z)
    p = np.exp(np.asarray(z, dtype=np.float64) - lse[:, None])
    t = dlogits(z, lse, targets, g)
    d = abs(g) * p * np.expm1(za + lse_tol[:, None] + EXP_REL) + 2.0 ** -140
    return bf16.from_f64_rne(t), bf16.from_f64_rne(t - d), bf16.from_f64_rne(t + d)
