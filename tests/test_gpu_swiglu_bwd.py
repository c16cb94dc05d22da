"""GPU parity of the fused SwiGLU backward + quantise call
(puro_swiglu_bwd_quantize_fp8) against the oracle (oracle/swiglu.py's
backward with oracle/quant.py), through the C ABI: codes and scales equal to
the oracle's wherever the gradient is unique, valid for the band of accepted
values elsewhere (tests/band_check.py)."""

import numpy as np
import pytest

from oracle import fp8, swiglu
from paper_2608_27370_amd import inputs

import band_check
from gpu_util import host, to_dev_bf16

pytestmark = pytest.mark.gpu

E4, E5 = 0, 1
OFMT = {E4: fp8.E4M3, E5: fp8.E5M2}
RULE = {0: "fp32", 1: "pow2", 2: "pow2_floor"}
TENSOR, ROW, COL = 0, 1, 2


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


def _inputs(seed, rows, cols, pad=0):
    """dH [rows, cols] ~ N(0, (1e-3)^2) and gu [rows, 2 cols + pad] ~ N(0,
    1.7^2); the pad columns of gu hold huge values that must not be read."""
    dh = inputs.case(seed, (rows, cols), std=1e-3)
    gu = inputs.case(seed + 1, (rows, 2 * cols + pad), std=1.7)
    if pad:
        gu[:, 2 * cols:] = 0x7F00
    return dh, gu


def _run(P, dh, gu, fmt, mode, rnd, want_q=True, want_qT=False):
    r = P.swiglu_bwd_quantize_fp8(to_dev_bf16(dh), to_dev_bf16(gu), fmt, mode=mode, rnd=rnd, want_q=want_q,
                                  want_qT=want_qT)
    return {k: (host(v) if v is not None else None) for k, v in r.items()}


def _check_all(r, dh, gu, fmt, mode, rnd, what):
    cols = dh.shape[1]
    mid, lo, hi = swiglu.swiglu_bwd_bf16_band(dh, gu, cols)
    un = swiglu.unique_mask(lo, hi)
    f, rule = OFMT[fmt], RULE[rnd]
    if mode == TENSOR:
        if r["q"] is not None:
            band_check.check(r["q"], r["scale"], mid, lo, hi, un, f, rule, None, what + " q")
        if r["qT"] is not None:
            band_check.check(r["qT"].T, r["scale"], mid, lo, hi, un, f, rule, None, what + " qT")
    if mode == ROW:
        band_check.check(r["q"], r["scale"], mid, lo, hi, un, f, rule, 1, what + " q")
    if (mode == ROW and r["qT"] is not None) or mode == COL:
        band_check.check(r["qT"].T, r["scaleT"], mid, lo, hi, un, f, rule, 0, what + " qT")


@pytest.mark.parametrize("rows,cols,pad", [(128, 64, 0), (208, 72, 48), (256, 192, 16), (16, 8, 0)])
@pytest.mark.parametrize("fmt,rnd", [(E5, 0), (E4, 0), (E4, 1)])
def test_tensor(P, rows, cols, pad, fmt, rnd):
    dh, gu = _inputs(100 + rows + cols, rows, cols, pad)
    r = _run(P, dh, gu, fmt, TENSOR, rnd, want_q=True, want_qT=True)
    _check_all(r, dh, gu, fmt, TENSOR, rnd, "tensor %dx%d" % (rows, cols))


@pytest.mark.parametrize("rows,cols,pad", [(128, 64, 0), (256, 192, 32), (384, 128, 0)])
@pytest.mark.parametrize("fmt,rnd", [(E4, 1), (E5, 1), (E4, 2)])
def test_groups(P, rows, cols, pad, fmt, rnd):
    dh, gu = _inputs(110 + rows + cols, rows, cols, pad)
    r = _run(P, dh, gu, fmt, ROW, rnd, want_q=True, want_qT=True)
    _check_all(r, dh, gu, fmt, ROW, rnd, "1x128+128x1 %dx%d" % (rows, cols))
    r = _run(P, dh, gu, fmt, COL, rnd)
    _check_all(r, dh, gu, fmt, COL, rnd, "128x1 %dx%d" % (rows, cols))


@pytest.mark.parametrize("u", [1.0, -0.75])
def test_every_gate_value(P, u):
    """Every BF16 pattern as a gate value (finite ones; infinities and NaN
    make the whole tensor NaN), a constant up value and dH = 1, in 1x128
    groups: both halves of the gradient over the whole range of g."""
    cols = 128
    g = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(512, cols)
    g[(g & 0x7F80) == 0x7F80] = 0                     # drop infinities and NaN
    gu = np.concatenate([g, np.full((512, cols), inputs.bf16_from_f64(np.array([u]))[0], np.uint16)], axis=1)
    dh = np.full((512, cols), inputs.bf16_from_f64(np.array([1.0]))[0], np.uint16)
    r = _run(P, dh, gu, E4, ROW, 1, want_q=True, want_qT=True)
    _check_all(r, dh, gu, E4, ROW, 1, "every gate value, u = %g" % u)


def test_empty(P):
    dh = np.zeros((0, 64), np.uint16)
    gu = np.zeros((0, 128), np.uint16)
    r = _run(P, dh, gu, E5, TENSOR, 0)
    assert r["scale"][0] == 1.0


@pytest.mark.parametrize("mode,fmt,rnd", [(TENSOR, E5, 0), (ROW, E4, 1)])
def test_mlp_full_size(P, mode, fmt, rnd):
    """The 8192-token MLP: dgu [8192, 17920] from dH [8192, 8960] and the
    gate/up output, per-tensor E5M2 (the per-tensor recipe's gradient format)
    and 1x128 + 128x1 E4M3 (the paper's blockwise recipe), on sampled rows
    and columns (exact subsets since no group crosses a row or a column;
    per-tensor with the whole tensor's accepted amax)."""
    M, F = 8192, inputs.MLP
    gu = inputs.mlp_gate_up(M)
    dh = inputs.normal(inputs.rng(0, 3, 7), (M, F), 1e-3)
    r = _run(P, dh, gu, fmt, mode, rnd, want_q=True, want_qT=True)
    rng = np.random.default_rng(9)
    rws = np.sort(rng.choice(M, 32, replace=False))
    f, rule = OFMT[fmt], RULE[rnd]
    # columns: blocks from both halves, the last block of each
    cls = np.concatenate([np.sort(rng.choice(F // 128, 2, replace=False)) * 128, [F - 128]])
    cls = np.concatenate([cls, F + cls])
    cols_idx = np.concatenate([np.arange(c, c + 128) for c in cls])
    if mode == TENSOR:
        mid, lo, hi = swiglu.swiglu_bwd_bf16_band(dh, gu, F)
        un = swiglu.unique_mask(lo, hi)
        ta = band_check.amax_band(lo, hi)
        band_check.check(r["q"][rws], r["scale"], mid[rws], lo[rws], hi[rws], un[rws], f, rule, None,
                         "full q rows", tensor_amax=ta)
        band_check.check(r["qT"][cols_idx].T, r["scale"], mid[:, cols_idx], lo[:, cols_idx], hi[:, cols_idx],
                         un[:, cols_idx], f, rule, None, "full qT cols", tensor_amax=ta)
        return
    mid, lo, hi = swiglu.swiglu_bwd_bf16_band(dh[rws], gu[rws], F)
    band_check.check(r["q"][rws], r["scale"][rws], mid, lo, hi, swiglu.unique_mask(lo, hi), f, rule, 1,
                     "full 1x128 rows")
    src = np.unique(cols_idx % F)
    mid, lo, hi = swiglu.swiglu_bwd_bf16_band(dh[:, src], np.concatenate([gu[:, src], gu[:, F + src]], axis=1),
                                              src.size)
    # columns of the band: [dg of src | du of src]; the quantised copy's rows cols_idx map onto them
    pos = {c: i for i, c in enumerate(src)}
    sel = np.array([pos[c % F] + (src.size if c >= F else 0) for c in cols_idx])
    band_check.check(r["qT"][cols_idx].T, r["scaleT"][cols_idx], mid[:, sel], lo[:, sel], hi[:, sel],
                     swiglu.unique_mask(lo, hi)[:, sel], f, rule, 0, "full 128x1 cols")
