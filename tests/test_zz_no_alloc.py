"""GPU check of the allocation-free quantise entry point
(puro_quantize_fp8_static) through the C ABI: bitwise the same codes and
scales as puro_quantize_fp8 with a caller workspace, on two calls in a row
that share the library's scratch, the second with a smaller input. The first
input is large enough that its amax pass takes the one-block reduction,
whose result also lives in the scratch."""

import numpy as np
import pytest

from paper_2608_27370_amd import inputs

from gpu_util import assert_bytes_equal, assert_f32_bits_equal, host, to_dev_bf16

pytestmark = pytest.mark.gpu

E4, E5 = 0, 1


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


def _same(P, x, fmt, mode, rnd, what):
    import torch
    ref = P.quantize_fp8(x, fmt, mode, rnd, want_q=True, want_qT=True)
    got = P.quantize_fp8_static(x, fmt, mode, rnd, want_q=True, want_qT=True)
    torch.cuda.synchronize()
    for k in ("q", "qT"):
        assert_bytes_equal(host(got[k]), host(ref[k]), "%s %s" % (what, k))
    for k in ("scale", "scaleT"):
        if ref[k] is not None:
            assert_f32_bits_equal(host(got[k]), host(ref[k]), "%s %s" % (what, k))


def test_static_scratch_matches_workspace_calls(P):
    # 8192 x 8192: 4096 partial maxima, reduced by the one-block kernel into
    # the scratch's amax slot; then a smaller per-tensor call (128 partials,
    # reduced inside the quantise blocks) over the same scratch
    big = to_dev_bf16(inputs.case(71, (8192, 8192), kind="student_t"))
    assert P.lib().puro_quantize_workspace_size(8192, 8192) <= 32768
    _same(P, big, E4, P.SCALE_TENSOR, P.SCALE_FP32, "8192x8192 tensor")
    del big
    small = to_dev_bf16(inputs.case(72, (1024, 1536)))
    _same(P, small, E5, P.SCALE_TENSOR, P.SCALE_FP32, "1024x1536 tensor")
    # a grouped mode takes no scratch and gives the workspace call's result too
    _same(P, small, E4, P.SCALE_ROW_1x128, P.SCALE_POW2, "1024x1536 groups")
    # and a per-tensor call after the grouped one still matches (scratch reused)
    tiny = to_dev_bf16(inputs.case(73, (256, 384), std=1e-3))
    _same(P, tiny, E4, P.SCALE_TENSOR, P.SCALE_POW2, "256x384 tensor pow2")
