"""Pins of the oracle's scaled FP8 GEMM (``oracle.gemm``) and of the linear
composition (``oracle.linear``): exact rationals on tiny inputs, closed forms,
the adjoint identity tying Fprop, Dgrad and Wgrad together, and agreement of
the sampled-entry and full versions."""

import math

import numpy as np
import pytest

from oracle import bf16, fp8, gemm, linear, quant
from paper_2608_27370_amd import inputs

E4, E5 = fp8.E4M3, fp8.E5M2


def _finite_codes(g, shape, fmt, lo_exp_field=None):
    """Random finite, non-NaN codes of a format."""
    t = fp8.decode_table(fmt)
    ok = np.array([c for c in range(256) if np.isfinite(t[c])], np.uint8)
    return g.choice(ok, size=shape)


@pytest.mark.parametrize("afmt,bfmt", [(E4, E4), (E5, E4), (E5, E5)])
def test_exact_rationals_tensor_scales(afmt, bfmt):
    g = np.random.default_rng(11)
    for (M, N, K) in [(1, 1, 1), (3, 5, 7), (16, 9, 16), (4, 4, 33)]:
        a = _finite_codes(g, (M, K), afmt)
        b = _finite_codes(g, (N, K), bfmt)
        sa, sb = np.float32(0.0137), np.float32(3.5e-4)
        ref, den = gemm.gemm(a, afmt, sa, "tensor", b, bfmt, sb, "tensor")
        ex = gemm.gemm_exact(a, afmt, sa, "tensor", b, bfmt, sb, "tensor")
        for m in range(M):
            for n in range(N):
                if afmt == bfmt == E4:
                    # E4M3 x E4M3 sums are exact in FP64 (multiples of 2**-18 below 2**53 units)
                    assert ref[m, n] == float(ex[m][n])
                else:
                    # wider products: FP64 rounding of at most K * 2**-53 of the magnitude sum
                    assert abs(ref[m, n] - float(ex[m][n])) <= (K + 1) * 2.0 ** -53 * den[m, n]
                assert den[m, n] >= abs(ref[m, n])


def test_exact_rationals_block_scales():
    """Two k-blocks, row scales on A, 128x128 block scales on B with a row of
    B in the second block row (exercises i // 128 and the k-block index)."""
    g = np.random.default_rng(12)
    M, N, K = 2, 129, 256
    a = _finite_codes(g, (M, K), E4)
    b = _finite_codes(g, (N, K), E4)
    sa = np.ldexp(1.0, g.integers(-10, 10, (M, 2))).astype(np.float32)
    sb = np.ldexp(1.0, g.integers(-10, 10, (2, 2))).astype(np.float32)
    ref, _ = gemm.gemm(a, E4, sa, "row", b, E4, sb, "block")
    ex = gemm.gemm_exact(a, E4, sa, "row", b, E4, sb, "block")
    for m in range(M):
        for n in (0, 1, 64, 127, 128):
            assert ref[m, n] == float(ex[m][n])
    # row scales on both operands (the Wgrad form)
    sb2 = np.ldexp(1.0, g.integers(-10, 10, (N, 2))).astype(np.float32)
    ref, _ = gemm.gemm(a, E4, sa, "row", b, E4, sb2, "row")
    ex = gemm.gemm_exact(a, E4, sa, "row", b, E4, sb2, "row")
    for m in range(M):
        for n in (0, 5, 128):
            assert ref[m, n] == float(ex[m][n])


def test_closed_forms():
    K = 384
    a = np.full((4, K), 0x3A, np.uint8)          # E4M3 1.25
    b = np.full((3, K), 0xC2, np.uint8)          # E4M3 -2.5 (sign, exp field 8 -> 2**1, m 2 -> 1.25)
    assert fp8.decode_code(0x3A, E4) == 1.25 and fp8.decode_code(0xC2, E4) == -2.5
    ref, den = gemm.gemm(a, E4, 0.5, "tensor", b, E4, 4.0, "tensor")
    assert np.all(ref == K * 1.25 * -2.5 * 2.0) and np.all(den == K * 1.25 * 2.5 * 2.0)
    # identity B: D = dequant(A) * sa * sb
    g = np.random.default_rng(3)
    A = _finite_codes(g, (5, 64), E4)
    I = np.zeros((64, 64), np.uint8)
    np.fill_diagonal(I, 0x38)                    # E4M3 1.0
    ref, _ = gemm.gemm(A, E4, 0.25, "tensor", I, E4, 8.0, "tensor")
    assert np.array_equal(ref, fp8.decode(A, E4) * 2.0)


def test_entries_match_full():
    g = np.random.default_rng(4)
    a = _finite_codes(g, (70, 256), E5)
    b = _finite_codes(g, (90, 256), E4)
    sa = np.ldexp(1.0, g.integers(-4, 4, (70, 2))).astype(np.float32)
    sb = np.ldexp(1.0, g.integers(-4, 4, (1, 2))).astype(np.float32)
    ref, den = gemm.gemm(a, E5, sa, "row", b, E4, sb, "block")
    ms = g.integers(0, 70, 500)
    ns = g.integers(0, 90, 500)
    r2, d2 = gemm.gemm_entries(ms, ns, a, E5, sa, "row", b, E4, sb, "block")
    assert np.array_equal(r2, ref[ms, ns]) and np.array_equal(d2, den[ms, ns])


def _fsum_inner(u, v):
    return math.fsum((u * v).ravel().tolist())


@pytest.mark.parametrize("dy_fmt", [E5, E4])
def test_adjoint_identity_ties_the_three_gemms(dy_fmt):
    """<Xq Wq^T, dYq> = <Xq, dYq Wq> = <Wq, dYq^T Xq> with the layer's own
    per-tensor scales: pins the operand orientations of Fprop, Dgrad and
    Wgrad against each other (the block recipe is pinned below)."""
    M, N, K = 256, 128, 256
    X = inputs.case(20, (M, K))
    W = inputs.case(21, (N, K), std=0.02)
    dY = inputs.case(22, (M, N), std=1e-3)
    rc = linear.recipe("tensor", dy_fmt=dy_fmt)
    y_ref, _, saved = linear.linear_fwd(X, W, rc)
    dx_ref, _, dw_ref, _, dq = linear.linear_bwd(dY, saved, rc)
    xq = fp8.decode(saved["xq"], rc["x_fmt"]) * float(saved["x_scale"])
    wq = fp8.decode(saved["wq"], rc["w_fmt"]) * float(saved["w_scale"])
    dyq = fp8.decode(dq["dyq"], rc["dy_fmt"]) * float(dq["dy_scale"])
    lhs = _fsum_inner(y_ref, dyq)
    mid = _fsum_inner(xq, dx_ref)
    rhs = _fsum_inner(wq, dw_ref)
    assert math.isclose(lhs, mid, rel_tol=1e-12) and math.isclose(lhs, rhs, rel_tol=1e-12)
    # the orientation of each result, against numpy's float64 products
    assert np.allclose(y_ref, xq @ wq.T, rtol=1e-12, atol=1e-12)
    assert np.allclose(dx_ref, dyq @ wq, rtol=1e-12, atol=1e-12)
    assert np.allclose(dw_ref, dyq.T @ xq, rtol=1e-12, atol=1e-12)


def test_block_recipe_layout_against_dequantised_products():
    """Block recipe: each GEMM equals the float64 product of the dequantised
    operands, with every operand expanded to its own per-element scales."""
    M, N, K = 256, 256, 384
    X = inputs.case(30, (M, K), kind="outliers")
    W = inputs.case(31, (N, K), std=0.02)
    dY = inputs.case(32, (M, N), std=1e-3)
    rc = linear.recipe("block", dy_fmt=E4)
    y_ref, _, saved = linear.linear_fwd(X, W, rc)
    dx_ref, _, dw_ref, _, dq = linear.linear_bwd(dY, saved, rc)

    def deq_rows(q, s, fmt):           # s: [rows, cols/128]
        return fp8.decode(q, fmt) * np.repeat(s.astype(np.float64), 128, axis=1)

    def deq_blocks(q, s, fmt):         # s: [rows/128, cols/128]
        e = np.repeat(np.repeat(s.astype(np.float64), 128, axis=0), 128, axis=1)
        return fp8.decode(q, fmt) * e

    xr = deq_rows(saved["xq"], saved["x_scale"], E4)
    xc = deq_rows(saved["xq_t"], saved["x_scale_t"], E4)           # [K, M]
    w = deq_blocks(saved["wq"], saved["w_scale"], E4)
    wt = deq_blocks(saved["wq_t"], saved["w_scale_t"], E4)         # [K, N]
    dyr = deq_rows(dq["dyq"], dq["dy_scale"], E4)
    dyc = deq_rows(dq["dyq_t"], dq["dy_scale_t"], E4)              # [N, M]
    assert np.array_equal(wt, w.T)
    assert np.allclose(y_ref, xr @ w.T, rtol=1e-12, atol=1e-14)
    assert np.allclose(dx_ref, dyr @ wt.T, rtol=1e-12, atol=1e-14)
    assert np.allclose(dw_ref, dyc @ xc.T, rtol=1e-12, atol=1e-14)
    # and the quantised layer is close to the BF16 layer (a few FP8 ulps)
    xf = bf16.to_f32(X).astype(np.float64)
    wf = bf16.to_f32(W).astype(np.float64)
    exact = xf @ wf.T
    err = np.abs(y_ref - exact) / (np.abs(xf) @ np.abs(wf).T)
    assert err.max() < 2 * 2.0 ** -4


def test_per_tensor_scale_applied_once():
    """Per-tensor GEMM equals (sa * sb) times the unscaled exact sum."""
    g = np.random.default_rng(9)
    a = _finite_codes(g, (8, 96), E4)
    b = _finite_codes(g, (6, 96), E4)
    sa, sb = np.float32(1.0 / 3), np.float32(7.0 / 11)
    r1, _ = gemm.gemm(a, E4, sa, "tensor", b, E4, sb, "tensor")
    r0, _ = gemm.gemm(a, E4, 1.0, "tensor", b, E4, 1.0, "tensor")
    assert np.array_equal(r1, r0 * (float(sa) * float(sb)))


def test_bf16_rounding_helper():
    vals = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -40,
                     -0.0, 3.0e38, 3.4e38, np.inf, np.nan, 2.0 ** -133, 2.0 ** -134])
    bits = bf16.from_f64_rne(vals)
    assert list(bits[:4]) == [0x3F80, 0x3F80, 0x3F82, 0x3F81]
    assert bits[4] == 0x8000
    assert bits[5] == 0x7F62 and bits[6] == 0x7F80 and bits[7] == 0x7F80
    assert bits[8] == 0x7FC0
    assert bits[9] == 0x0001 and bits[10] == 0x0000    # tie at half the smallest subnormal -> even


def test_epilogue_closed_forms():
    """A zero product leaves bias + residual; the tolerance scale grows by
    their magnitudes; absent terms change nothing."""
    rng = np.random.default_rng(12)
    b = bf16.to_f32(bf16.from_f64_rne(rng.standard_normal(8))).astype(np.float64)
    r = bf16.to_f32(bf16.from_f64_rne(rng.standard_normal((4, 8)))).astype(np.float64)
    ref, den = gemm.epilogue(np.zeros((4, 8)), np.zeros((4, 8)), b, r)
    np.testing.assert_array_equal(ref, b[None, :] + r)
    np.testing.assert_array_equal(den, np.abs(b)[None, :] + np.abs(r))
    x = rng.standard_normal((4, 8))
    ref, den = gemm.epilogue(x, np.abs(x))
    np.testing.assert_array_equal(ref, x)
    np.testing.assert_array_equal(den, np.abs(x))
