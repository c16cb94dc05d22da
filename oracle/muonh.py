"""MuonH: the Muon update under the hyperball wrapper, for one weight matrix.

Test infrastructure only (see the package docstring).

Section 3.3 (Hyperball Optimization), equation (hyperball-update): each
wrapped matrix keeps the Frobenius radius R = ||W_0||_F it started with. With
the Muon update u_t and the weight learning rate eta_t, one step is

    u_hat = u / ||u||_F
    W~    = W - eta R u_hat
    W'    = R W~ / ||W~||_F.

The displacement eta R u_hat has norm eta R against ||W|| = R, which is why the
section calls eta the effective learning rate.

The paper takes Muon itself from its training framework and states nothing of
its internals. The readings below follow the published Muon method (momentum
with a Nesterov look-ahead, then a quintic Newton-Schulz orthogonalisation):

* momentum (FP32 state, as the paper keeps optimiser state):
      buf' = mu buf + (1 - mu) G
      V    = (1 - mu) G + mu buf'    (Nesterov; V = buf' without it)
  each product and sum rounded to binary32 in that order, with (1 - mu)
  rounded to binary32 first;
* Newton-Schulz: X_0 = V / (||V||_F + EPS), transposed when the matrix has more
  rows than columns (so that the Gram matrix is the smaller one), then
      A_k = X_k X_k^T,   B_k = b A_k + c A_k A_k,   X_{k+1} = a X_k + B_k X_k
  for STEPS steps with (a, b, c) = COEFFS, and u = X_STEPS (transposed back).
  The polynomial a s + b s^3 + c s^5 acts on every singular value of X alone,
  so u = U f(S / ||V||) V^T for V = U S V^T and f that polynomial applied
  STEPS times (the pin of this module);
* Muon's own rescaling of u (by a shape factor) is dropped: u_hat divides it
  out;
* a zero u (all of V zero, so X_0 = 0) displaces nothing: W' = R W / ||W||.

Two evaluations: ``newton_schulz`` in float64 (the definition), and
``newton_schulz_bf16``, the rounding points of the BF16 implementation: X_0,
each A_k, B_k and X_{k+1} rounded once to BF16 from the float64 value of
its expression (products of BF16 values summed exactly up to float64
rounding). The hyperball step is float64 from the FP32 W and the BF16 u.

Parity pins (tests/test_oracle_muonh.py): the singular-value closed form
through numpy's SVD, the transposition symmetry, a scaled orthogonal input
whose iterates follow the scalar polynomial, the radius and effective-LR
identities of the hyperball step, the momentum's closed form under a constant
gradient, and the BF16 evaluation staying within BF16 noise of the float64 one.
"""

import numpy as np

from . import bf16

COEFFS = (3.4445, -4.7750, 2.0315)
STEPS = 5
EPS = 1e-7


def momentum(buf, G, mu, nesterov=True):
    """(buf', V) from FP32 buf and G, binary32 arithmetic in the stated order."""
    buf = np.asarray(buf, dtype=np.float32)
    G = np.asarray(G, dtype=np.float32)
    m = np.float32(mu)
    om = np.float32(np.float32(1.0) - m)
    nb = (m * buf + om * G).astype(np.float32)
    v = (om * G + m * nb).astype(np.float32) if nesterov else nb
    return nb, v


def frobenius(x):
    return float(np.sqrt(np.sum(np.square(np.asarray(x, dtype=np.float64)))))


def _oriented(V):
    V = np.asarray(V, dtype=np.float64)
    return (V.T, True) if V.shape[0] > V.shape[1] else (V, False)


def newton_schulz(V, steps=STEPS, coeffs=COEFFS, eps=EPS):
    """u = NS(V) in float64."""
    a, b, c = coeffs
    X, tr = _oriented(V)
    X = X / (frobenius(X) + eps)
    for _ in range(steps):
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    return X.T if tr else X


def polynomial(s, steps=STEPS, coeffs=COEFFS):
    """The scalar map NS applies to each singular value of X_0."""
    a, b, c = coeffs
    s = np.asarray(s, dtype=np.float64)
    for _ in range(steps):
        s = a * s + b * s ** 3 + c * s ** 5
    return s


def to_f64(bits):
    return bf16.to_f32(np.asarray(bits, dtype=np.uint16)).astype(np.float64)


def ns_start_bf16(V, eps=EPS):
    """X_0 (BF16 bits, oriented so that rows <= columns) of an FP32 V."""
    X, _ = _oriented(V)
    return bf16.from_f64_rne(X / (frobenius(X) + eps))


def ns_step_bf16(X_bits, coeffs=COEFFS):
    """One Newton-Schulz step at the BF16 rounding points: returns the BF16
    bits of (A, B, X')."""
    a, b, c = coeffs
    X = to_f64(X_bits)
    A_bits = bf16.from_f64_rne(X @ X.T)
    A = to_f64(A_bits)
    B_bits = bf16.from_f64_rne(b * A + c * (A @ A))
    B = to_f64(B_bits)
    Xn_bits = bf16.from_f64_rne(a * X + B @ X)
    return A_bits, B_bits, Xn_bits


def newton_schulz_bf16(V, steps=STEPS, coeffs=COEFFS, eps=EPS):
    """u (BF16 bits, in V's orientation) with the BF16 rounding points."""
    tr = np.asarray(V).shape[0] > np.asarray(V).shape[1]
    X = ns_start_bf16(V, eps)
    for _ in range(steps):
        X = ns_step_bf16(X, coeffs)[2]
    return np.ascontiguousarray(X.T) if tr else X


def hyperball(W, u, eta, R):
    """W' (float64) from W, the update u (float64 values), eta and R. A zero
    u (all of V zero) has no direction: W' is W projected (reading)."""
    W = np.asarray(W, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    nu = frobenius(u)
    Wt = W - eta * R * (u / nu) if nu > 0 else W
    return R * Wt / frobenius(Wt)


def step(W, G, buf, mu, eta, R, nesterov=True, steps=STEPS, coeffs=COEFFS, eps=EPS):
    """One MuonH step of one matrix with the BF16 Newton-Schulz: returns
    (W' float64, buf' float32, u BF16 bits)."""
    nb, V = momentum(buf, G, mu, nesterov)
    u = newton_schulz_bf16(V, steps, coeffs, eps)
    return hyperball(W, to_f64(u), eta, R), nb, u
