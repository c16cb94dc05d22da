"""GPU parity of the FP8 linear layer (puro_linear_fwd / puro_linear_bwd)
against the oracle's composition: saved FP8 bytes and scales bit-exact, Y and
dX within the BF16 band, dW within the FP32 tolerance."""

import numpy as np
import pytest

from oracle import gemm, linear
from paper_2608_27370_amd import inputs

import mfma_model
from gpu_util import (assert_bytes_equal, assert_f32_bits_equal, bf16_bits, check_bf16, check_fp32, host,
                      to_dev_bf16)


def _ref(op):
    """Exact oracle GEMM, its magnitude sum and the instruction-truncation allowance."""
    ref, den = gemm.gemm(*op)
    return ref, den, mfma_model.truncation_loss_full(*op)

pytestmark = pytest.mark.gpu

E4, E5 = 0, 1
ONAME = {E4: "e4m3", E5: "e5m2"}


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


CASES = [
    # (M, N, K, blockwise, dy_fmt, rounding: 0 FP32 / 1 POW2 / 2 POW2_FLOOR)
    (256, 384, 512, 0, E5, 0),
    (304, 400, 160, 0, E5, 0),
    (512, 256, 1024, 0, E4, 0),
    (256, 384, 512, 0, E5, 2),
    (256, 384, 512, 1, E4, 1),
    (384, 256, 128, 1, E4, 1),
    (256, 512, 384, 1, E5, 1),
    (256, 384, 512, 1, E4, 2),
]
RULE = {0: "fp32", 1: "pow2", 2: "pow2_floor"}


@pytest.mark.parametrize("case", CASES, ids=lambda c: "M%d_N%d_K%d_%s_%s_%s" % (
    c[0], c[1], c[2], "block" if c[3] else "tensor", ONAME[c[4]], RULE[c[5]]))
def test_linear_fwd_bwd(P, case):
    M, N, K, blockwise, dyf, rnd = case
    X = inputs.case(40, (M, K), kind="outliers")
    W = inputs.case(41, (N, K), std=0.02)
    dY = inputs.case(42, (M, N), std=1e-3)
    rc = P.LinearRecipe(E4, E4, dyf, blockwise, rnd)
    orc = linear.recipe("block" if blockwise else "tensor", dy_fmt=ONAME[dyf],
                        rule=None if (rnd == 0 and blockwise) else RULE[rnd])

    Y, saved = P.linear_fwd(to_dev_bf16(X), to_dev_bf16(W), rc)
    fprop, osaved = linear.fwd_operands(X, W, orc)
    y_ref, y_den, y_sl = _ref(fprop)
    assert_bytes_equal(host(saved["xq_t"]), osaved["xq_t"], "saved xq_t")
    assert_bytes_equal(host(saved["wq_t"]), osaved["wq_t"], "saved wq_t")
    if blockwise:
        # the saved blockwise scales are k-block-major: transposed views of the oracle's
        assert_f32_bits_equal(host(saved["x_scale"]).T, osaved["x_scale_t"], "saved x scales")
        assert_f32_bits_equal(host(saved["w_scale"]).T, osaved["w_scale_t"], "saved w scales")
    else:
        assert_f32_bits_equal(host(saved["x_scale"]), np.array([osaved["x_scale"]]), "x scale")
        assert_f32_bits_equal(host(saved["w_scale"]), np.array([osaved["w_scale"]]), "w scale")
    check_bf16(bf16_bits(Y), y_ref, y_den, what="Y", slack=y_sl)

    dX, dW = P.linear_bwd(to_dev_bf16(dY), saved, rc, K)
    dgrad, wgrad, _ = linear.bwd_operands(dY, osaved, orc)
    dx_ref, dx_den, dx_sl = _ref(dgrad)
    dw_ref, dw_den, dw_sl = _ref(wgrad)
    check_bf16(bf16_bits(dX), dx_ref, dx_den, what="dX", slack=dx_sl)
    check_fp32(host(dW), dw_ref, dw_den, what="dW", slack=dw_sl)

    # dW accumulation and the single-output variants
    _, dW2 = P.linear_bwd(to_dev_bf16(dY), saved, rc, K, want_dx=False, dW=dW.clone(), accumulate_dw=True)
    check_fp32(host(dW2), 2 * dw_ref, 2 * dw_den, what="dW accumulated", slack=2 * dw_sl)
    dX3, none = P.linear_bwd(to_dev_bf16(dY), saved, rc, K, want_dw=False)
    assert none is None
    assert np.array_equal(bf16_bits(dX3), bf16_bits(dX))


def test_linear_pow2_per_tensor(P):
    M, N, K = 256, 256, 256
    X = inputs.case(43, (M, K))
    W = inputs.case(44, (N, K), std=0.02)
    rc = P.LinearRecipe(E4, E4, E5, 0, P.SCALE_POW2)
    Y, saved = P.linear_fwd(to_dev_bf16(X), to_dev_bf16(W), rc)
    from oracle import quant
    xq, xqT, sx, _ = quant.quantize_tensor(X, "e4m3", rule="pow2")
    wq, wqT, sw, _ = quant.quantize_tensor(W, "e4m3", rule="pow2")
    assert_bytes_equal(host(saved["xq_t"]), xqT, "xq_t")
    assert_f32_bits_equal(host(saved["x_scale"]), np.array([sx]), "x scale")
    ref, den, sl = _ref((xq, "e4m3", sx, "tensor", wq, "e4m3", sw, "tensor"))
    check_bf16(bf16_bits(Y), ref, den, what="Y pow2", slack=sl)


def test_linear_is_deterministic(P):
    M, N, K = 512, 384, 1024
    X = to_dev_bf16(inputs.case(45, (M, K)))
    W = to_dev_bf16(inputs.case(46, (N, K), std=0.02))
    dY = to_dev_bf16(inputs.case(47, (M, N), std=1e-3))
    for blockwise in (0, 1):
        rc = P.LinearRecipe(E4, E4, E4 if blockwise else E5, blockwise, P.SCALE_FP32)
        outs = []
        for _ in range(2):
            Y, saved = P.linear_fwd(X, W, rc)
            dX, dW = P.linear_bwd(dY, saved, rc, K)
            outs.append((bf16_bits(Y), bf16_bits(dX), host(dW).view(np.uint32)))
        for a, b in zip(*outs):
            assert np.array_equal(a, b)
