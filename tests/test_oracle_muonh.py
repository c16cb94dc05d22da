"""Pins of the MuonH oracle (oracle/muonh.py) against what the mathematics
fixes: Newton-Schulz acts on singular values alone (closed form through
numpy's SVD), the hyperball step's geometry (Section 3.3, equation
hyperball-update: radius R, displacement eta R, effective learning rate
eta), and the momentum's closed form under a constant gradient."""

import numpy as np
import pytest

from oracle import bf16, muonh


def _rand(seed, shape, std=1.0):
    return np.random.default_rng(seed).normal(0.0, std, shape)


@pytest.mark.parametrize("shape", [(48, 80), (80, 48), (64, 64)])
def test_newton_schulz_is_the_polynomial_of_the_singular_values(shape):
    V = _rand(1, shape)
    u = muonh.newton_schulz(V)
    U, S, Vt = np.linalg.svd(V, full_matrices=False)
    ref = (U * muonh.polynomial(S / (np.linalg.norm(V) + muonh.EPS))) @ Vt
    assert u.shape == V.shape
    assert np.max(np.abs(u - ref)) < 1e-12


def test_newton_schulz_of_a_scaled_orthogonal_matrix():
    """Rows of Q orthonormal: X_0 = 3 Q / (3 sqrt(r) + EPS), and every
    singular value follows the scalar map from 3 / (3 sqrt(r) + EPS)."""
    r, c = 32, 96
    Q = np.linalg.qr(_rand(2, (c, r)))[0].T          # [r, c], Q Q^T = I
    u = muonh.newton_schulz(3.0 * Q)
    s = 3.0 / (3.0 * np.sqrt(r) + muonh.EPS)
    a, b, cc = muonh.COEFFS
    for _ in range(muonh.STEPS):
        s = a * s + b * s ** 3 + cc * s ** 5
    assert np.max(np.abs(u - s * Q)) < 1e-12
    # the published coefficients leave singular values near (not at) one
    assert 0.6 < s < 1.25


def test_newton_schulz_commutes_with_transposition():
    V = _rand(3, (40, 72))
    assert np.max(np.abs(muonh.newton_schulz(V.T) - muonh.newton_schulz(V).T)) < 1e-13


def test_hyperball_geometry():
    """W on the sphere of radius R and u orthogonal to W (Frobenius inner
    product): the displacement eta R u_hat has norm eta R, so ||W~|| =
    R sqrt(1 + eta^2), and the projected W' makes <W', W> = R^2 / sqrt(1 +
    eta^2) and <W', u_hat> = -eta R / sqrt(1 + eta^2)."""
    R, eta = 3.7, 0.05
    W = _rand(4, (24, 40))
    W *= R / np.linalg.norm(W)
    u = _rand(5, (24, 40))
    u -= np.sum(u * W) / np.sum(W * W) * W
    uh = u / np.linalg.norm(u)
    Wn = muonh.hyperball(W, u, eta, R)
    k = np.sqrt(1.0 + eta * eta)
    assert abs(np.linalg.norm(Wn) - R) < 1e-12
    assert abs(np.sum(Wn * W) - R * R / k) < 1e-11
    assert abs(np.sum(Wn * uh) + eta * R / k) < 1e-12
    # the update's own scale drops out
    assert np.max(np.abs(muonh.hyperball(W, 7.0 * u, eta, R) - Wn)) < 1e-14


def test_hyperball_keeps_the_radius_off_the_sphere():
    """A W of any norm comes back to radius R."""
    W = _rand(6, (16, 48), std=0.3)
    Wn = muonh.hyperball(W, _rand(7, (16, 48)), 0.01, 2.5)
    assert abs(np.linalg.norm(Wn) - 2.5) < 1e-12


def test_zero_update_only_projects():
    W = _rand(13, (16, 32))
    V = np.zeros((16, 32), dtype=np.float32)
    u = muonh.to_f64(muonh.newton_schulz_bf16(V))
    assert not np.any(u)
    assert np.max(np.abs(muonh.hyperball(W, u, 0.1, 2.0) - 2.0 * W / np.linalg.norm(W))) < 1e-15


def test_momentum_under_a_constant_gradient():
    """From a zero buffer and a constant G: buf_k = (1 - mu^k) G and the
    Nesterov input V_k = (1 - mu^(k+1)) G, up to binary32 rounding."""
    mu = 0.95
    G = _rand(8, (8, 128)).astype(np.float32)
    buf = np.zeros_like(G)
    for k in range(1, 21):
        buf, V = muonh.momentum(buf, G, mu)
        assert buf.dtype == np.float32 and V.dtype == np.float32
        tol = 4e-7 * (k + 2) * np.abs(G)
        assert np.all(np.abs(buf - (1.0 - mu ** k) * G) <= tol)
        assert np.all(np.abs(V - (1.0 - mu ** (k + 1)) * G) <= tol)
    nb, V = muonh.momentum(buf, G, mu, nesterov=False)
    assert np.array_equal(nb, V)


def test_bf16_newton_schulz_within_bf16_noise():
    """The BF16 rounding points keep the result within a few BF16 steps of
    the float64 definition (relative Frobenius error well under 2^-4), and
    with no steps it is X_0 rounded."""
    V = _rand(9, (64, 192)).astype(np.float32)
    u64 = muonh.newton_schulz(V)
    ub = muonh.to_f64(muonh.newton_schulz_bf16(V))
    assert np.linalg.norm(ub - u64) / np.linalg.norm(u64) < 2.0 ** -4
    x0 = muonh.newton_schulz_bf16(V, steps=0)
    ref = bf16.from_f64_rne(V.astype(np.float64) / (np.linalg.norm(V.astype(np.float64)) + muonh.EPS))
    assert np.array_equal(x0, ref)
    Vt = np.ascontiguousarray(V.T)
    assert np.array_equal(muonh.newton_schulz_bf16(Vt), np.ascontiguousarray(muonh.newton_schulz_bf16(V).T))


def test_step_composes_momentum_newton_schulz_and_hyperball():
    W = _rand(10, (32, 64), std=0.02)
    R = np.linalg.norm(W)
    G = _rand(11, (32, 64), std=1e-3).astype(np.float32)
    buf = _rand(12, (32, 64), std=1e-3).astype(np.float32)
    Wn, nb, u = muonh.step(W, G, buf, 0.95, 0.01, R)
    assert abs(np.linalg.norm(Wn) - R) < 1e-12 * R
    assert np.array_equal(nb, muonh.momentum(buf, G, 0.95)[0])
    # the displacement before projection is eta R along u_hat
    uh = muonh.to_f64(u) / np.linalg.norm(muonh.to_f64(u))
    Wt = W - 0.01 * R * uh
    assert np.max(np.abs(Wn - R * Wt / np.linalg.norm(Wt))) < 1e-15
