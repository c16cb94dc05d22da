"""The FP8 linear layer, forward and backward, composed from the oracle parts.

Section 3.2 and Appendix C (precision flow) of the paper: Y = X W^T with X
[M, K] and W [N, K] in BF16. The layer quantises X and W immediately before
the Fprop GEMM and writes Y in BF16; it keeps the quantised input for Wgrad;
the backward pass quantises dY and runs Dgrad (dX = dY W, BF16) and Wgrad
(dW = dY^T X, accumulated in FP32) in FP8 as well.

Two recipes:

* "tensor": one scale per tensor (X and W in E4M3, dY in ``dy_fmt``).
* "block": X and dY in 1x128 groups along each GEMM's reduction dimension
  (row groups for Fprop/Dgrad, column groups stored transposed for Wgrad),
  W in 128x128 blocks, power-of-two scales; the 128x128 W blocks serve
  Dgrad unchanged, transposed.

Every GEMM is posed with both operands reduction-contiguous:
Fprop A = Xq [M, K], B = Wq [N, K]; Dgrad A = dYq [M, N], B = WqT [K, N];
Wgrad A = dYqT [N, M], B = XqT [K, M].
"""

from . import bf16, gemm, quant  # noqa: F401

E4M3 = "e4m3"
E5M2 = "e5m2"


def recipe(mode="tensor", x_fmt=E4M3, w_fmt=E4M3, dy_fmt=E5M2, rule=None):
    """``rule``: the scale rule ("fp32", "pow2" or "pow2_floor"); by default
    "fp32" for one scale per tensor and "pow2" for block scales."""
    assert mode in ("tensor", "block")
    if rule is None:
        rule = "fp32" if mode == "tensor" else "pow2"
    assert rule in (("fp32", "pow2", "pow2_floor") if mode == "tensor" else ("pow2", "pow2_floor"))
    return dict(mode=mode, x_fmt=x_fmt, w_fmt=w_fmt, dy_fmt=dy_fmt, rule=rule)


def fwd_operands(X, W, rc):
    """Quantise X [M, K] and W [N, K] (BF16 bits).

    Returns (fprop, saved): ``fprop`` is the GEMM argument tuple
    (a, a_fmt, a_scale, a_mode, b, b_fmt, b_scale, b_mode); ``saved`` holds
    what the backward pass reuses plus the forward's quantised bytes.
    """
    if rc["mode"] == "tensor":
        xq, xqT, sx, ax = quant.quantize_tensor(X, rc["x_fmt"], rule=rc["rule"])
        wq, wqT, sw, aw = quant.quantize_tensor(W, rc["w_fmt"], rule=rc["rule"])
        fprop = (xq, rc["x_fmt"], sx, "tensor", wq, rc["w_fmt"], sw, "tensor")
        saved = dict(xq=xq, xq_t=xqT, x_scale=sx, x_amax=ax,
                     wq=wq, wq_t=wqT, w_scale=sw, w_amax=aw)
    else:
        xq, sx = quant.quantize_rows_1x128(X, rc["x_fmt"], rc["rule"])
        xqT, sxT = quant.quantize_cols_128x1(X, rc["x_fmt"], rc["rule"])
        wq, sw, wqT, swT = quant.quantize_blocks_128x128(W, rc["w_fmt"], rc["rule"])
        fprop = (xq, rc["x_fmt"], sx, "row", wq, rc["w_fmt"], sw, "block")
        saved = dict(xq=xq, x_scale=sx, xq_t=xqT, x_scale_t=sxT,
                     wq=wq, w_scale=sw, wq_t=wqT, w_scale_t=swT)
    return fprop, saved


def bwd_operands(dY, saved, rc):
    """Quantise dY [M, N] and pose Dgrad and Wgrad.

    Returns (dgrad, wgrad, dq): GEMM argument tuples and dY's quantised bytes.
    """
    if rc["mode"] == "tensor":
        dyq, dyqT, sdy, ady = quant.quantize_tensor(dY, rc["dy_fmt"], rule=rc["rule"])
        dgrad = (dyq, rc["dy_fmt"], sdy, "tensor",
                 saved["wq_t"], rc["w_fmt"], saved["w_scale"], "tensor")
        wgrad = (dyqT, rc["dy_fmt"], sdy, "tensor",
                 saved["xq_t"], rc["x_fmt"], saved["x_scale"], "tensor")
        dq = dict(dyq=dyq, dyq_t=dyqT, dy_scale=sdy, dy_amax=ady)
    else:
        dyq, sdy = quant.quantize_rows_1x128(dY, rc["dy_fmt"], rc["rule"])
        dyqT, sdyT = quant.quantize_cols_128x1(dY, rc["dy_fmt"], rc["rule"])
        dgrad = (dyq, rc["dy_fmt"], sdy, "row",
                 saved["wq_t"], rc["w_fmt"], saved["w_scale_t"], "block")
        wgrad = (dyqT, rc["dy_fmt"], sdyT, "row",
                 saved["xq_t"], rc["x_fmt"], saved["x_scale_t"], "row")
        dq = dict(dyq=dyq, dy_scale=sdy, dyq_t=dyqT, dy_scale_t=sdyT)
    return dgrad, wgrad, dq


def linear_fwd(X, W, rc):
    """Y reference in FP64 with its magnitude sum: (y_ref, y_den, saved)."""
    fprop, saved = fwd_operands(X, W, rc)
    y_ref, y_den = gemm.gemm(*fprop)
    return y_ref, y_den, saved


def linear_bwd(dY, saved, rc):
    """(dx_ref, dx_den, dw_ref, dw_den, dq) in FP64."""
    dgrad, wgrad, dq = bwd_operands(dY, saved, rc)
    dx_ref, dx_den = gemm.gemm(*dgrad)
    dw_ref, dw_den = gemm.gemm(*wgrad)
    return dx_ref, dx_den, dw_ref, dw_den, dq
