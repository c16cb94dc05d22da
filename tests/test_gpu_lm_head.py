"""GPU parity of the fused LM head + cross-entropy (puro_lm_head_ce_fwd /
puro_lm_head_ce_bwd) against the oracle (oracle/lm_head.py with
oracle/quant.py and oracle/gemm.py), through the C ABI.

lse and loss are compared row by row with the oracle's float64 values within
its allowances for a binary32 evaluation. dX and dW are compared with the
float64 products of the oracle's dz: the tolerance is the GEMMs' own
(1e-5 sum|ab| plus the FP8 instruction's truncation) plus, per output,
sum over the reduction of the width of dz's band times |the other operand|
(the kernel may take any BF16 dz in the band; for the FP8 recipe any code that
quantising a value of the band can give). The small cases check everything;
the full-size case (M 8192, V 151936, K 1536) checks every row's loss and
sampled rows of dX and rows of dW.
"""

import numpy as np
import pytest

from oracle import bf16, fp8, lm_head, quant
from paper_2608_27370_amd import inputs

import mfma_model
from gpu_util import bf16_bits, check_bf16, check_fp32, host, to_dev, to_dev_bf16

pytestmark = pytest.mark.gpu

BF16, FP8 = 0, 1


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


def f64(b):
    return bf16.to_f32(np.asarray(b, dtype=np.uint16)).astype(np.float64)


class Operands:
    """The oracle's view of the GEMM operands of a recipe, as float64 values:
    x and w as the logits GEMM reads them (dequantised FP8 codes for the FP8
    recipe), wt as dX reads W and xt as dW reads X (the 128x1 column groups
    for the FP8 recipe), with the codes and scales the truncation allowance
    needs."""

    def __init__(self, X, W, recipe):
        self.recipe = recipe
        if recipe == BF16:
            self.x, self.w = f64(X), f64(W)
            self.wt, self.xt = self.w, self.x
            return
        deq = lambda q, s, ax0, ax1: fp8.decode(q, fp8.E4M3) * np.repeat(np.repeat(s, ax0, axis=0), ax1, axis=1)
        self.xq, self.xs = quant.quantize_rows_1x128(X, fp8.E4M3)
        self.x = deq(self.xq, self.xs, 1, 128)
        self.wq, self.ws, self.wqT, self.wsT = quant.quantize_blocks_128x128(W, fp8.E4M3)
        self.w = deq(self.wq, self.ws, 128, 128)
        self.wt = self.w                                    # same codes and scales, transposed
        self.xqT, self.xsT = quant.quantize_cols_128x1(X, fp8.E4M3)
        self.xt = deq(self.xqT, self.xsT, 1, 128).T         # [M, K] as dW reads X

    def truncation(self, ms, ns):
        """FP8 recipe: the instruction's truncation allowance of logits (ms[i], ns[i])."""
        return mfma_model.truncation_loss(ms, ns, self.xq, fp8.E4M3, self.xs, "row", self.wq, fp8.E4M3, self.ws,
                                          "block")

    def logits(self):
        """z, S = |x| |w|^T and the truncation allowance of every logit."""
        z, S = self.x @ self.w.T, np.abs(self.x) @ np.abs(self.w).T
        if self.recipe == BF16:
            return z, S, 0.0
        mm, nn = np.meshgrid(np.arange(self.x.shape[0]), np.arange(self.w.shape[0]), indexing="ij")
        return z, S, self.truncation(mm.ravel(), nn.ravel()).reshape(mm.shape)


def dz_operand(dz_mid, lo, hi, recipe, axis):
    """The dz operand the backward GEMMs read, as float64 values, the
    per-element width of what the kernel may have used instead, and (FP8) the
    (codes, group scales) pairs that the truncation allowance is taken over.
    BF16 recipe: the band [lo, hi]. FP8 recipe: the codes of the oracle's
    quantisation of dz_mid (groups along `axis`: 1 = rows, for dX; 0 =
    columns, for dW, returned transposed as [V, M]); the kernel may have
    quantised any value of the band, under any power-of-two group scale that
    a group maximum within the band gives (the scale rule is monotone in the
    maximum, so these lie between the scales of the smallest and the largest
    magnitudes the band allows), and each element's code under a fixed scale
    lies between those of the band's ends."""
    mid, l, h = f64(dz_mid), f64(lo), f64(hi)
    tr = (lambda v: v) if axis == 1 else (lambda v: np.ascontiguousarray(v.T))
    if recipe == BF16:
        return tr(mid), tr(np.maximum(mid - l, h - mid)), []
    grp = quant.quantize_rows_1x128 if axis == 1 else quant.quantize_cols_128x1
    q, s = grp(dz_mid, fp8.E4M3)
    mid, l, h = tr(mid), tr(l), tr(h)
    val = fp8.decode(q, fp8.E4M3) * np.repeat(s.astype(np.float64), 128, axis=1)
    lb, hb = np.asarray(lo, dtype=np.uint16), np.asarray(hi, dtype=np.uint16)
    mag_lo = np.where((lb >> 15) == (hb >> 15), np.minimum(lb & 0x7FFF, hb & 0x7FFF), 0).astype(np.uint16)
    mag_hi = np.maximum(lb & 0x7FFF, hb & 0x7FFF).astype(np.uint16)
    s_lo, s_hi = grp(mag_lo, fp8.E4M3)[1], grp(mag_hi, fp8.E4M3)[1]
    steps = int(np.max(np.log2(s_hi.astype(np.float64) / s_lo)))
    assert 0 <= steps <= 2, "the band spans %d group-scale steps" % steps
    width, cands = np.zeros_like(val), []
    for j in range(steps + 1):
        sc = np.minimum(s_lo * np.float32(2.0 ** j), s_hi).astype(np.float32)
        srep = np.repeat(sc.astype(np.float64), 128, axis=1)
        r = (1.0 / srep).astype(np.float32)
        enc = lambda v: fp8.decode(quant.encode_scaled(v.astype(np.float32), r, fp8.E4M3), fp8.E4M3) * srep
        width = np.maximum(width, np.maximum(np.abs(enc(l) - val), np.abs(enc(h) - val)))
        cands.append((quant.encode_scaled(mid.astype(np.float32), r, fp8.E4M3), sc))
    return val, width, cands


def truncation_max(cands, loss):
    """The largest truncation allowance over the candidate dz quantisations."""
    out = 0.0
    for q, s in cands:
        out = np.maximum(out, loss(q, s))
    return out


def run(P, X, W, t, recipe, g=1.0, lse_in=None):
    """Forward, then backward from the forward's lse (or from lse_in)."""
    Xd, Wd, td = to_dev_bf16(X), to_dev_bf16(W), to_dev(np.asarray(t, dtype=np.int32))
    lse, loss = P.lm_head_ce_fwd(Xd, Wd, td, recipe)
    lse_b = lse if lse_in is None else to_dev(np.asarray(lse_in, dtype=np.float32))
    dX, dW = P.lm_head_ce_bwd(Xd, Wd, td, lse_b, recipe, grad_scale=g)
    return host(lse), host(loss), dX, dW


def check_small(P, X, W, t, recipe, g):
    """lse and loss of every row, and every entry of dX and dW, against the
    oracle's float64 values within the allowances of a binary32 evaluation."""
    lse_k, loss_k, dX, dW = run(P, X, W, t, recipe, g)
    ops = Operands(X, W, recipe)
    z, S, slack = ops.logits()
    lse, loss = lm_head.forward(z, t)
    _, lse_tol, loss_tol = lm_head.tolerances(z, S, t, slack)
    assert np.all(np.abs(lse_k - lse) <= lse_tol), np.max(np.abs(lse_k - lse) / lse_tol)
    assert np.all(np.abs(loss_k - loss) <= loss_tol), np.max(np.abs(loss_k - loss) / loss_tol)
    mid, lo, hi = lm_head.dlogits_band(z, S, t, g, slack)
    name = "fp8" if recipe == FP8 else "bf16"
    # dX = dz W: reduction over V
    dzx, wx, cx = dz_operand(mid, lo, hi, recipe, 1)
    ref, den = dzx @ ops.wt, np.abs(dzx) @ np.abs(ops.wt)
    extra = wx @ np.abs(ops.wt) + truncation_max(cx, lambda q, s: mfma_model.truncation_loss_full(
        q, fp8.E4M3, s, "row", ops.wqT, fp8.E4M3, ops.wsT, "block"))
    check_bf16(bf16_bits(dX), ref, den, what="lm_head %s dX" % name, slack=extra)
    # dW = dz^T X: reduction over M
    dzw, ww, cw = dz_operand(mid, lo, hi, recipe, 0)      # [V, M]
    ref, den = dzw @ ops.xt, np.abs(dzw) @ np.abs(ops.xt)
    extra = ww @ np.abs(ops.xt) + truncation_max(cw, lambda q, s: mfma_model.truncation_loss_full(
        q, fp8.E4M3, s, "row", ops.xqT, fp8.E4M3, ops.xsT, "row"))
    check_fp32(host(dW), ref, den, what="lm_head %s dW" % name, slack=extra)


@pytest.mark.parametrize("recipe", [BF16, FP8], ids=["bf16", "fp8"])
@pytest.mark.parametrize("M,V,K", [(256, 1152, 256), (128, 256, 384)])
def test_lm_head_small(P, recipe, M, V, K):
    """Every output of a small case; V = 1152 leaves the last 256-wide tile
    half empty."""
    X = inputs.case(81, (M, K), kind="student_t")
    W = inputs.case(82, (V, K), std=0.05)
    t = inputs.rng(0, 99, 83).integers(0, V, M)
    check_small(P, X, W, t, recipe, 1.0 / M)


@pytest.mark.parametrize("recipe", [BF16, FP8], ids=["bf16", "fp8"])
def test_lm_head_target_positions(P, recipe):
    """Targets placed at every kind of column position rather than at random:
    in each 8-column group the first and last column of both 4-column halves
    (the two lanes that hold a row's columns), the first and last column of a
    128-column block, of a 256-column tile and of the vocabulary, and every
    column of one 8-column group. Rows 0-127 spread their targets over all
    blocks; rows 128-255 put the targets of a whole 32-row fragment into one
    block (so several rows of a fragment meet their target in the same place)
    and leave other fragments with none in most blocks."""
    M, V, K = 256, 640, 128
    X = inputs.case(86, (M, K), kind="student_t")
    W = inputs.case(87, (V, K), std=0.05)
    pos = [0, 3, 4, 7, 8, 11, 12, 15, 120, 123, 124, 127, 128, 131, 132, 255, 256, 259, 260, 383, 384,
           511, 512, 636, 637, 638, 639] + list(range(136, 144))
    t = np.empty(M, np.int64)
    t[:128] = [pos[i % len(pos)] for i in range(128)]
    for f in range(4):                       # rows 128 + 32 f .. : one block per fragment
        base = (f % 5) * 128
        t[128 + 32 * f: 160 + 32 * f] = base + (np.arange(32) * 5) % 128
    check_small(P, X, W, t, recipe, 1.0 / M)


def test_lm_head_targets_outside_give_nan(P):
    M, V, K = 128, 256, 128
    X = inputs.case(84, (M, K))
    W = inputs.case(85, (V, K), std=0.05)
    t = np.arange(M) % V
    t[3] = V + 5
    t[7] = -1
    lse_k, loss_k, _, _ = run(P, X, W, t, BF16)
    assert np.isnan(loss_k[3]) and np.isnan(loss_k[7])
    assert np.isfinite(np.delete(loss_k, [3, 7])).all() and np.isfinite(lse_k).all()


@pytest.mark.timeout(1500)
@pytest.mark.parametrize("recipe", [BF16, FP8], ids=["bf16", "fp8"])
def test_lm_head_full_size(P, recipe):
    """M 8192 tokens, V 151936, K 1536 (the vocabulary walked in 18 full
    chunks and a narrower last one): X Student-t(3), W ~ N(0, 0.02^2),
    uniform targets, grad_scale 1 (the sum over tokens).

    Forward: every row's lse and loss. The oracle's logits come from float64
    products in row chunks; the allowance of a row's largest logit error,
    rel * max_v sum_k |x_k w_vk|, is bounded by rel |x|_2 max_v |w_v|_2
    (Cauchy-Schwarz), with rel = 1e-5, plus 2^-10 for the FP8 recipe's
    truncation (a group of 8 products loses less than 8 2^(E-13), and its
    largest product is at least 2^E); the target logits' allowance is exact.
    Backward from the oracle's lse (rounded to binary32, the value both sides
    take): dX on sampled rows and dW on sampled vocabulary rows (targets
    among them, and the last one), full-length float64 reductions, with the
    exact truncation allowance of every logit they depend on."""
    d = inputs.lm_head_xw()
    X, W, t = d["X"], d["W"], d["targets"]
    M, K = X.shape
    V = W.shape[0]
    name = "fp8" if recipe == FP8 else "bf16"
    print("lm_head full %s: oracle operands and lse" % name, flush=True)
    ops = Operands(X, W, recipe)
    lse = np.concatenate([lm_head.log_sum_exp(ops.x[r0:r0 + 512] @ ops.w.T) for r0 in range(0, M, 512)])
    lse32 = lse.astype(np.float32)
    print("lm_head full %s: GPU forward and backward" % name, flush=True)
    lse_k, loss_k, dX, dW = run(P, X, W, t, recipe, 1.0, lse_in=lse32)
    rng = np.random.default_rng(17)
    rows = np.unique(np.concatenate([[0, M - 1], rng.choice(M, 2, replace=False)]))
    cols = np.unique(np.concatenate([[V - 1], t[rng.choice(M, 2, replace=False)], rng.choice(V, 2, replace=False)]))
    dX_rows, dW_rows = bf16_bits(dX)[rows], host(dW[cols])
    del dX, dW
    print("lm_head full %s: forward check" % name, flush=True)
    rel = 1e-5 + (2.0 ** -10 if recipe == FP8 else 0.0)
    lse_tol = rel * np.linalg.norm(ops.x, axis=1) * np.linalg.norm(ops.w, axis=1).max() \
        + lm_head.LSE_ABS * (1.0 + np.abs(lse))
    zt = np.einsum("mk,mk->m", ops.x, ops.w[t])
    zt_tol = 1e-5 * np.einsum("mk,mk->m", np.abs(ops.x), np.abs(ops.w[t]))
    if recipe == FP8:
        zt_tol = zt_tol + ops.truncation(np.arange(M), t)
    assert np.all(np.abs(lse_k - lse) <= lse_tol), np.max(np.abs(lse_k - lse) / lse_tol)
    assert np.all(np.abs(loss_k - (lse - zt)) <= lse_tol + zt_tol), \
        np.max(np.abs(loss_k - (lse - zt)) / (lse_tol + zt_tol))

    def band(ri, ci, tt):
        """BF16 (mid, lo, hi) of dz over logits rows ri x columns ci."""
        z = ops.x[ri] @ ops.w[ci].T
        za = 1e-5 * (np.abs(ops.x[ri]) @ np.abs(ops.w[ci]).T)
        if recipe == FP8:
            mm, nn = np.meshgrid(ri, ci, indexing="ij")
            za = za + ops.truncation(mm.ravel(), nn.ravel()).reshape(mm.shape)
        p = np.exp(z - lse32[ri].astype(np.float64)[:, None])
        dzv = p - tt
        dd = p * np.expm1(za + lm_head.EXP_REL) + 2.0 ** -140
        return bf16.from_f64_rne(dzv), bf16.from_f64_rne(dzv - dd), bf16.from_f64_rne(dzv + dd)

    print("lm_head full %s: dX rows" % name, flush=True)
    allv = np.arange(V)
    mid, lo, hi = band(rows, allv, (t[rows][:, None] == allv[None, :]).astype(np.float64))
    dzx, wx, cx = dz_operand(mid, lo, hi, recipe, 1)
    ref, den = dzx @ ops.wt, np.abs(dzx) @ np.abs(ops.wt)
    mm, kk = np.meshgrid(np.arange(rows.size), np.arange(K), indexing="ij")
    extra = wx @ np.abs(ops.wt) + truncation_max(cx, lambda q, s: mfma_model.truncation_loss(
        mm.ravel(), kk.ravel(), q, fp8.E4M3, s, "row", ops.wqT, fp8.E4M3, ops.wsT, "block",
        chunk=16).reshape(mm.shape))
    check_bf16(dX_rows, ref, den, what="lm_head full %s dX rows" % name, slack=extra)
    print("lm_head full %s: dW rows" % name, flush=True)
    mid, lo, hi = band(np.arange(M), cols, (t[:, None] == cols[None, :]).astype(np.float64))
    dzw, ww, cw = dz_operand(mid, lo, hi, recipe, 0)          # [cols, M]
    ref, den = dzw @ ops.xt, np.abs(dzw) @ np.abs(ops.xt)
    extra = ww @ np.abs(ops.xt) + truncation_max(cw, lambda q, s: mfma_model.truncation_loss_full(
        q, fp8.E4M3, s, "row", ops.xqT, fp8.E4M3, ops.xsT, "row"))
    check_fp32(dW_rows, ref, den, what="lm_head full %s dW rows" % name, slack=extra)
