"""GPU parity at the full sizes of the Qwen2-1.5B-shaped workloads, in the
launch configuration bench.py times: quantised bytes and scales compared in
full (or on sampled rows/columns where the oracle would take minutes), GEMM
outputs on stratified samples (16 random entries in every 256x256 output
tile plus the whole first and last tiles), each entry a full-length FP64 dot
product of the oracle."""

import numpy as np
import pytest

from oracle import fp8, gemm, linear, quant
from paper_2608_27370_amd import inputs

import mfma_model
from gpu_util import (assert_bytes_equal, assert_f32_bits_equal, bf16_bits, check_bf16, check_fp32, host,
                      sample_entries, to_dev_bf16)

pytestmark = pytest.mark.gpu

E4, E5 = 0, 1


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


def test_single_forward_256x1536x1536(P):
    """X [256,1536] ~ N(0,1), W [1536,1536] ~ N(0,0.02^2), seed 0; per-tensor
    E4M3; the whole Y compared."""
    d = inputs.single_fwd()
    rc = P.LinearRecipe(E4, E4, E5, 0, P.SCALE_FP32)
    Y, saved = P.linear_fwd(to_dev_bf16(d["X"]), to_dev_bf16(d["W"]), rc)
    fprop, osaved = linear.fwd_operands(d["X"], d["W"], linear.recipe("tensor"))
    y_ref, y_den = gemm.gemm(*fprop)
    assert_bytes_equal(host(saved["xq_t"]), osaved["xq_t"], "xq_t")
    assert_bytes_equal(host(saved["wq_t"]), osaved["wq_t"], "wq_t")
    assert_f32_bits_equal(host(saved["x_scale"]), np.array([osaved["x_scale"]]), "x scale")
    # the plain bound max|err| / sum|ab| <= 1e-5 holds here and is asserted
    check_bf16(bf16_bits(Y), y_ref, y_den, what="single forward Y", slack=mfma_model.truncation_loss_full(*fprop),
               strict=True)


def _entries_check(P, D, out, ms, ns, op, what, strict=False):
    ref, den = gemm.gemm_entries(ms, ns, *op)
    slack = mfma_model.truncation_loss(ms, ns, *op)
    if out == 1:
        check_fp32(host(D)[ms, ns], ref, den, what=what, slack=slack, strict=strict)
    else:
        check_bf16(bf16_bits(D)[ms, ns], ref, den, what=what, slack=slack, strict=strict)


def test_qkv_projection_fwd_dgrad_wgrad(P):
    """M 8192, K 1536, N 2048; X ~ N(0,1), W ~ N(0,0.02^2), dY ~ N(0,1e-6);
    X, W in E4M3 and dY in E5M2 with per-tensor scales."""
    d = inputs.qkv()
    M, K, N = 8192, 1536, 2048
    rc = P.LinearRecipe(E4, E4, E5, 0, P.SCALE_FP32)
    Y, saved = P.linear_fwd(to_dev_bf16(d["X"]), to_dev_bf16(d["W"]), rc)
    dX, dW = P.linear_bwd(to_dev_bf16(d["dY"]), saved, rc, K)
    orc = linear.recipe("tensor")
    fprop, osaved = linear.fwd_operands(d["X"], d["W"], orc)
    dgrad, wgrad, dq = linear.bwd_operands(d["dY"], osaved, orc)
    assert_bytes_equal(host(saved["xq_t"]), osaved["xq_t"], "xq_t")
    assert_bytes_equal(host(saved["wq_t"]), osaved["wq_t"], "wq_t")
    assert_f32_bits_equal(host(saved["x_scale"]), np.array([osaved["x_scale"]]), "x scale")
    assert_f32_bits_equal(host(saved["w_scale"]), np.array([osaved["w_scale"]]), "w scale")
    # the plain bound max|err| / sum|ab| <= 1e-5 holds on all three and is asserted
    g = np.random.default_rng(2)
    ms, ns = sample_entries(M, N, g)
    _entries_check(P, Y, 0, ms, ns, fprop, "qkv Y", strict=True)
    ms, ns = sample_entries(M, K, g)
    _entries_check(P, dX, 0, ms, ns, dgrad, "qkv dX", strict=True)
    ms, ns = sample_entries(N, K, g)
    _entries_check(P, dW, 1, ms, ns, wgrad, "qkv dW", strict=True)
