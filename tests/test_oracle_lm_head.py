"""Pins of the LM-head cross-entropy oracle (oracle/lm_head.py).

log-sum-exp is pinned by the library routine scipy.special.logsumexp, by
uniform logits (lse = log V) and by the shift identity; the loss by the
two-class closed form log(1 + e^(z_o - z_t)) and by being >= 0; the gradient
by sum_v dz = 0, by central differences of g * loss and by the closed form
of the two-class case; the logits by brute force on tiny BF16 inputs; and the
bands by the values they must hold and planted mistakes they must reject.
"""

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import bf16, lm_head


def bits(x):
    return bf16.from_f64_rne(np.asarray(x, dtype=np.float64))


def test_log_sum_exp_matches_scipy_and_closed_forms():
    rng = np.random.default_rng(1)
    z = rng.standard_normal((6, 1000)) * 5
    np.testing.assert_allclose(lm_head.log_sum_exp(z), logsumexp(z, axis=1), rtol=1e-14)
    # uniform logits: lse = c + log V
    for V in (1, 2, 151936):
        assert abs(lm_head.log_sum_exp(np.full((1, V), 3.5))[0] - (3.5 + np.log(V))) < 1e-12
    # shift invariance without overflow
    big = z + 700.0
    np.testing.assert_allclose(lm_head.log_sum_exp(big), lm_head.log_sum_exp(z) + 700.0, rtol=1e-14)


def test_loss_two_classes_and_sign():
    z = np.array([[2.0, -1.0], [0.5, 0.5], [-30.0, 10.0]])
    t = np.array([0, 1, 0])
    _, loss = lm_head.forward(z, t)
    want = np.log1p(np.exp(np.array([-3.0, 0.0, 40.0])))
    np.testing.assert_allclose(loss, want, rtol=1e-14)
    rng = np.random.default_rng(2)
    z = rng.standard_normal((50, 300)) * 3
    t = rng.integers(0, 300, 50)
    _, loss = lm_head.forward(z, t)
    assert (loss >= 0).all()


def test_gradient_identities_and_finite_differences():
    rng = np.random.default_rng(3)
    M, V = 4, 37
    z = rng.standard_normal((M, V)) * 2
    t = rng.integers(0, V, M)
    lse, loss = lm_head.forward(z, t)
    for g in (1.0, 1.0 / M, -2.0):
        dz = lm_head.dlogits(z, lse, t, g)
        assert np.abs(dz.sum(axis=1)).max() < 1e-14
        h = 1e-6
        for (m, v) in ((0, 0), (1, int(t[1])), (3, 20)):
            zp, zm = z.copy(), z.copy()
            zp[m, v] += h
            zm[m, v] -= h
            fd = g * (lm_head.forward(zp, t)[1][m] - lm_head.forward(zm, t)[1][m]) / (2 * h)
            assert abs(fd - dz[m, v]) < 1e-8
    # two classes: dz_t = -(1 - p_t) with p_t = 1 / (1 + e^(z_o - z_t))
    z2 = np.array([[1.0, 3.0]])
    dz = lm_head.dlogits(z2, lm_head.forward(z2, [0])[0], [0])
    pt = 1.0 / (1.0 + np.exp(2.0))
    np.testing.assert_allclose(dz[0], [pt - 1.0, 1.0 - pt], rtol=1e-14)


def test_logits_brute_force():
    rng = np.random.default_rng(4)
    X = bits(rng.standard_normal((3, 5)))
    W = bits(rng.standard_normal((4, 5)) * 0.02)
    z, S = lm_head.logits(X, W)
    x, w = bf16.to_f32(X).astype(np.float64), bf16.to_f32(W).astype(np.float64)
    for m in range(3):
        for v in range(4):
            assert z[m, v] == sum(x[m, k] * w[v, k] for k in range(5))
            assert S[m, v] == sum(abs(x[m, k] * w[v, k]) for k in range(5))


def test_bands_hold_the_value_and_reject_mistakes():
    rng = np.random.default_rng(5)
    M, V, K = 8, 512, 64
    X = bits(rng.standard_normal((M, K)))
    W = bits(rng.standard_normal((V, K)) * 0.3)
    t = rng.integers(0, V, M)
    z, S = lm_head.logits(X, W)
    mid, lo, hi = lm_head.dlogits_band(z, S, t)
    f = lambda b: bf16.to_f32(b).astype(np.float64)
    assert (f(lo) <= f(mid)).all() and (f(mid) <= f(hi)).all()
    # most elements have a single accepted BF16 value (here the logit
    # allowance, 1e-5 sum|x w| ~ 1e-4, moves p by ~3e-4 of a 2^-8 BF16 step)
    assert np.mean(f(lo) == f(hi)) > 0.75
    # a binary32 evaluation (numpy float32 throughout) lies in the bands
    z32 = (X.astype(np.uint32) << 16).view(np.float32) @ ((W.astype(np.uint32) << 16).view(np.float32)).T
    m32 = z32.max(axis=1, keepdims=True)
    lse32 = m32[:, 0] + np.log(np.exp(z32 - m32).sum(axis=1, dtype=np.float32))
    p32 = np.exp(z32 - lse32[:, None])
    p32[np.arange(M), t] -= np.float32(1.0)
    d32 = f(bits(p32.astype(np.float64)))
    assert ((f(lo) <= d32) & (d32 <= f(hi))).all()
    _, lse_tol, loss_tol = lm_head.tolerances(z, S, t)
    lse, loss = lm_head.forward(z, t)
    assert (np.abs(lse32 - lse) <= lse_tol).all()
    assert (np.abs((lse32 - z32[np.arange(M), t]) - loss) <= loss_tol).all()
    # a gradient without the onehot, or scaled by 2, falls outside
    wrong = f(bits(lm_head.dlogits(z, lse, t) + np.eye(V)[t]))
    assert not ((f(lo) <= wrong) & (wrong <= f(hi))).all()
    wrong = f(bits(2 * lm_head.dlogits(z, lse, t)))
    assert not ((f(lo) <= wrong) & (wrong <= f(hi))).all()
    # a loss against the wrong target falls outside its tolerance
    _, bad = lm_head.forward(z, (t + 1) % V)
    assert (np.abs(bad - loss) > loss_tol).any()
