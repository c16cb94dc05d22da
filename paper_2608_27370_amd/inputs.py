"""Seeded synthetic inputs for the FP8 linear layer (no arithmetic of the method).

The paper trains on its own corpus, which is not available here; these
generators stand in for its activations, weights and gradients with the shapes
of a Qwen2-1.5B-sized transformer (hidden 1536, QKV 2048 = 12 query + 2 key +
2 value heads of 128, MLP 8960 with fused gate/up 17920, vocabulary 151936)
and with the value distributions stated per workload below. Values are drawn
in float64 from numpy's PCG64, rounded to binary32 and then to BF16 (both
round-to-nearest-even), and returned as uint16 BF16 bit patterns; the same
bytes are handed to the HIP library and to the oracle.

Workloads (M tokens, K input features, N output features):

* ``single_fwd``  -- X [256, 1536] ~ N(0, 1), W [1536, 1536] ~ N(0, 0.02^2);
  ``default_rng(0)``, X drawn first.
* ``qkv``         -- M 8192, K 1536, N 2048: X ~ N(0,1), W ~ N(0, 0.02^2),
  dY ~ N(0, (1e-3)^2); ``SeedSequence([0, 2, t])`` with t = 0, 1, 2.
* ``mlp``         -- gate/up M 8192, K 1536, N 17920 and down M 8192,
  K 8960, N 1536; activations N(0,1) with 1% of the input channels scaled by
  20 (outlier channels), weights N(0, 0.02^2), gradients N(0, (1e-3)^2);
  ``SeedSequence([0, 3, t])``, t = 0..5.
* ``layers``      -- per layer l < 28 and linear j (qkv 2048x1536, o
  1536x1536, gate/up 17920x1536, down 1536x8960) at M 16384:
  ``SeedSequence([0, 4, l, j, t])``.
* ``lm_head``     -- M 8192, K 1536, N 151936: X ~ Student-t(3), W ~
  N(0, 0.02^2), targets uniform over the vocabulary, dY = softmax(X W^T) -
  onehot(target) per row (no 1/M factor); ``SeedSequence([0, 5, t])``.
* ``paper_linear`` -- the paper's 1.7B ladder model (d 2048, 16 query and 8
  key/value heads of 128, d_ff 6144) at M 8192: qkv 4096x2048, o 2048x2048,
  fused gate/up 12288x2048, down 2048x6144; X ~ N(0,1) with 1% outlier
  channels scaled by 20, W ~ N(0, 0.02^2), dY ~ N(0, (1e-3)^2);
  ``SeedSequence([0, 6, j, t])``.
* ``muonh_matrix`` -- one MuonH-wrapped matrix [rows, cols] in binary32
  (FP32 master weights and optimiser state): W ~ N(0, 0.02^2), the gradient
  G ~ N(0, (1e-3)^2) and the momentum buffer ~ N(0, (1e-3)^2) (a state some
  steps in); ``SeedSequence([0, 7, key, t])``. The wrapped matrices of a layer
  are those of ``LAYER_LINEARS`` (the MLP's gate/up as one [17920, 1536]
  matrix).
"""

import numpy as np

HIDDEN = 1536
QKV_OUT = 2048
MLP = 8960
VOCAB = 151936
LAYERS = 28

LAYER_LINEARS = (("qkv", QKV_OUT, HIDDEN), ("o", HIDDEN, HIDDEN),
                 ("gate_up", 2 * MLP, HIDDEN), ("down", HIDDEN, MLP))
# the paper's 1.7B model: (name, N out, K in)
PAPER_D, PAPER_QKV, PAPER_FF = 2048, 4096, 6144
PAPER_LINEARS = (("qkv", PAPER_QKV, PAPER_D), ("o", PAPER_D, PAPER_D),
                 ("gate_up", 2 * PAPER_FF, PAPER_D), ("down", PAPER_D, PAPER_FF))


def bf16_from_f64(x):
    """float64 -> binary32 (RNE) -> BF16 bits (RNE on the binary32 word)."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def bf16_to_f32(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def normal(g, shape, std=1.0):
    return bf16_from_f64(std * g.standard_normal(shape))


def with_outlier_columns(g, shape, frac=0.01, factor=20.0):
    """N(0,1) with round(frac * C) distinct columns multiplied by ``factor``
    (before the BF16 rounding); the columns are drawn after the values."""
    x = g.standard_normal(shape)
    C = shape[1]
    cols = g.choice(C, size=int(round(frac * C)), replace=False)
    x[:, cols] *= factor
    return bf16_from_f64(x)


def student_t(g, shape, nu=3.0):
    return bf16_from_f64(g.standard_t(nu, shape))


# ---- workloads ---------------------------------------------------------------

def single_fwd():
    g = np.random.default_rng(0)
    X = bf16_from_f64(g.standard_normal((256, HIDDEN)))
    W = bf16_from_f64(0.02 * g.standard_normal((HIDDEN, HIDDEN)))
    return dict(X=X, W=W)


def qkv(M=8192):
    return dict(X=normal(rng(0, 2, 0), (M, HIDDEN)),
                W=normal(rng(0, 2, 1), (QKV_OUT, HIDDEN), 0.02),
                dY=normal(rng(0, 2, 2), (M, QKV_OUT), 1e-3))


def mlp(M=8192):
    return dict(X=with_outlier_columns(rng(0, 3, 0), (M, HIDDEN)),
                W_gu=normal(rng(0, 3, 1), (2 * MLP, HIDDEN), 0.02),
                dY_gu=normal(rng(0, 3, 2), (M, 2 * MLP), 1e-3),
                H=with_outlier_columns(rng(0, 3, 3), (M, MLP)),
                W_dn=normal(rng(0, 3, 4), (HIDDEN, MLP), 0.02),
                dY_dn=normal(rng(0, 3, 5), (M, HIDDEN), 1e-3))


def mlp_gate_up(M=8192):
    """A stand-in for the fused gate/up GEMM output [M, 2 * MLP] that the
    SwiGLU consumes: normal with the spread that X W_gu^T has for the MLP
    inputs above (rows of 1536 N(0,1) values, 1% of them x20, against
    N(0, 0.02^2) weights: variance 0.02^2 * (1521 + 15 * 400) ~ 1.7^2)."""
    return normal(rng(0, 3, 6), (M, 2 * MLP), 1.7)


def norm_input(M=8192, d=HIDDEN):
    """The residual stream an RMSNorm reads before the QKV projection
    [M, d] (N(0,1) with 1% of the channels x20, like the MLP inputs) and the
    norm's weight [d] ~ N(1, 0.1^2)."""
    return dict(x=with_outlier_columns(rng(0, 7, 0), (M, d)),
                gamma=bf16_from_f64(1.0 + 0.1 * rng(0, 7, 1).standard_normal(d)))


def layer_linear(layer, j, M=16384):
    name, N, K = LAYER_LINEARS[j]
    return dict(name=name,
                X=normal(rng(0, 4, layer, j, 0), (M, K)),
                W=normal(rng(0, 4, layer, j, 1), (N, K), 0.02),
                dY=normal(rng(0, 4, layer, j, 2), (M, N), 1e-3))


def paper_linear(j, M=8192):
    name, N, K = PAPER_LINEARS[j]
    return dict(name=name,
                X=with_outlier_columns(rng(0, 6, j, 0), (M, K)),
                W=normal(rng(0, 6, j, 1), (N, K), 0.02),
                dY=normal(rng(0, 6, j, 2), (M, N), 1e-3))


def lm_head_xw(M=8192, V=VOCAB):
    X = student_t(rng(0, 5, 0), (M, HIDDEN))
    W = normal(rng(0, 5, 1), (V, HIDDEN), 0.02)
    t = rng(0, 5, 2).integers(0, V, size=M)
    return dict(X=X, W=W, targets=t)


def softmax_minus_onehot_rows(logits_f32, targets):
    """dY rows from binary32 logits: softmax(z) - onehot(t), in binary32,
    rounded to BF16. Used for the LM-head gradient input."""
    z = np.asarray(logits_f32, dtype=np.float32)
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z, dtype=np.float32)
    p = e / e.sum(axis=1, keepdims=True, dtype=np.float32)
    p[np.arange(p.shape[0]), targets] -= np.float32(1.0)
    return bf16_from_f64(p.astype(np.float64))


def lm_head(M=8192, V=VOCAB, chunk=512):
    """The LM-head workload with dY computed on the host in row chunks."""
    d = lm_head_xw(M, V)
    Xf = bf16_to_f32(d["X"])
    Wf = bf16_to_f32(d["W"])
    dY = np.empty((M, V), dtype=np.uint16)
    for r0 in range(0, M, chunk):
        r1 = min(M, r0 + chunk)
        z = Xf[r0:r1] @ Wf.T
        dY[r0:r1] = softmax_minus_onehot_rows(z, d["targets"][r0:r1])
    d["dY"] = dY
    return d


def muonh_matrix(rows, cols, key=0):
    """(W, G, buf) float32 [rows, cols] for one MuonH matrix."""
    f = lambda t, std: (rng(0, 7, key, t).standard_normal((rows, cols)) * std).astype(np.float32)
    return f(0, 0.02), f(1, 1e-3), f(2, 1e-3)


# ---- small cases for tests -----------------------------------------------------

def case(seed, shape, std=1.0, kind="normal"):
    """A small seeded BF16 tensor: ``normal``, ``outliers`` or ``student_t``."""
    g = rng(0, 99, seed)
    if kind == "normal":
        return normal(g, shape, std)
    if kind == "outliers":
        return with_outlier_columns(g, shape)
    if kind == "student_t":
        return student_t(g, shape)
    raise ValueError(kind)
