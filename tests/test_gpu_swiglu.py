"""GPU parity of the fused SwiGLU + quantise call (puro_swiglu_quantize_fp8)
against the oracle (oracle/swiglu.py with oracle/quant.py), through the C
ABI: codes and scales equal to the oracle's wherever H is unique, and valid
for the band of accepted H elsewhere (tests/band_check.py)."""

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


def _gu(seed, rows, cols, pad=0, std=1.7):
    """gu [rows, 2 cols + pad] with the pad columns filled with huge values
    that must not enter H."""
    gu = inputs.case(seed, (rows, 2 * cols + pad), std=std)
    if pad:
        gu[:, 2 * cols:] = 0x7F00          # 1.7e38: would dominate any amax it entered
    return gu


def _run(P, gu, cols, fmt, mode, rnd, want_q=True, want_qT=False):
    r = P.swiglu_quantize_fp8(to_dev_bf16(gu), cols, fmt, mode=mode, rnd=rnd, want_q=want_q, want_qT=want_qT)
    return {k: (host(v) if v is not None else None) for k, v in r.items()}


def _check_all(r, gu, cols, fmt, mode, rnd, what):
    mid, lo, hi = swiglu.swiglu_bf16_band(gu, cols)
    un = swiglu.unique_mask(lo, hi)
    f, rule = OFMT[fmt], RULE[rnd]
    n = 0
    if mode == TENSOR:
        if r["q"] is not None:
            n += band_check.check(r["q"], r["scale"], mid, lo, hi, un, f, rule, None, what + " q")
        if r["qT"] is not None:
            n += band_check.check(r["qT"].T, r["scale"], mid, lo, hi, un, f, rule, None, what + " qT")
    if mode == ROW:
        n += band_check.check(r["q"], r["scale"], mid, lo, hi, un, f, rule, 1, what + " q")
    if (mode == ROW and r["qT"] is not None) or mode == COL:
        n += band_check.check(r["qT"].T, r["scaleT"], mid, lo, hi, un, f, rule, 0, what + " qT")
    return n


@pytest.mark.parametrize("rows,cols,pad", [(128, 128, 0), (208, 144, 64), (256, 384, 16), (16, 16, 0)])
@pytest.mark.parametrize("fmt,rnd", [(E4, 0), (E5, 0), (E4, 1)])
def test_tensor(P, rows, cols, pad, fmt, rnd):
    gu = _gu(40 + rows + cols, rows, cols, pad)
    r = _run(P, gu, cols, fmt, TENSOR, rnd, want_q=True, want_qT=True)
    _check_all(r, gu, cols, fmt, TENSOR, rnd, "tensor %dx%d" % (rows, cols))


@pytest.mark.parametrize("rows,cols,pad", [(128, 128, 0), (256, 384, 32), (384, 256, 0)])
@pytest.mark.parametrize("fmt,rnd", [(E4, 1), (E5, 1), (E4, 2)])
def test_groups(P, rows, cols, pad, fmt, rnd):
    gu = _gu(50 + rows + cols, rows, cols, pad)
    r = _run(P, gu, cols, fmt, ROW, rnd, want_q=True, want_qT=True)
    _check_all(r, gu, cols, fmt, ROW, rnd, "1x128+128x1 %dx%d" % (rows, cols))
    r = _run(P, gu, cols, fmt, ROW, rnd, want_q=True, want_qT=False)
    _check_all(r, gu, cols, fmt, ROW, rnd, "1x128 %dx%d" % (rows, cols))
    r = _run(P, gu, cols, fmt, COL, rnd)
    _check_all(r, gu, cols, fmt, COL, rnd, "128x1 %dx%d" % (rows, cols))


def test_extremes(P):
    """Gate values deep in silu's tails (e^-g overflowing binary32, and silu
    equal to g), zeros of both signs, and a group of zeros."""
    rows, cols = 128, 256
    gu = _gu(60, rows, cols)
    g = np.array([-200.0, -100.0, -88.5, -30.0, 0.0, -0.0, 30.0, 90.0])
    gu[0, :8] = inputs.bf16_from_f64(g)
    gu[1, :cols] = 0
    gu[2, cols:2 * cols] = 0x8000       # up = -0
    for mode, rnd in ((TENSOR, 0), (ROW, 1)):
        r = _run(P, gu, cols, E4, mode, rnd, want_q=True, want_qT=True)
        _check_all(r, gu, cols, E4, mode, rnd, "extremes mode %d" % mode)


@pytest.mark.parametrize("u", [1.0, -3.0])
def test_every_gate_value(P, u):
    """Every BF16 pattern as a gate value (infinities and NaN included),
    against a constant up value, in 1x128 power-of-two groups (whose scales
    make the codes sensitive to H's low bits) and per-tensor."""
    cols = 128
    g = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(512, cols)
    gu = np.concatenate([g, np.full((512, cols), inputs.bf16_from_f64(np.array([u]))[0], np.uint16)], axis=1)
    for mode, rnd in ((ROW, 1), (TENSOR, 0)):
        r = _run(P, gu, cols, E4, mode, rnd, want_q=True, want_qT=True)
        if mode == TENSOR:
            # the NaN gate values make the tensor's scale NaN: every code is NaN's
            assert np.isnan(r["scale"][0]) and (r["q"] == 0x7F).all()
            continue
        _check_all(r, gu, cols, E4, mode, rnd, "every gate value, u = %g" % u)


def test_empty(P):
    gu = np.zeros((0, 256), np.uint16)
    r = _run(P, gu, 128, E4, TENSOR, 0)
    assert r["scale"][0] == 1.0


@pytest.mark.parametrize("mode,rnd", [(TENSOR, 0), (ROW, 1)])
def test_mlp_full_size(P, mode, rnd):
    """The 8192-token MLP: H [8192, 8960] from the gate/up output [8192,
    17920], in the launch configuration the bench times. Per-tensor: the
    scale (whole tensor) and the codes of sampled rows and columns; groups:
    sampled rows (1x128) and sampled columns (128x1), which are exact
    subsets since no group crosses a row or a column."""
    M, F = 8192, inputs.MLP
    gu = inputs.mlp_gate_up(M)
    r = _run(P, gu, F, E4, mode, rnd, want_q=True, want_qT=True)
    rng = np.random.default_rng(7)
    rws = np.sort(rng.choice(M, 48, replace=False))
    cls = np.sort(rng.choice(F // 128, 6, replace=False)) * 128
    cls = np.concatenate([cls, [F - 128]])
    f, rule = OFMT[E4], RULE[rnd]
    if mode == TENSOR:
        # the scale from the whole tensor's band of accepted amax values, the
        # codes of sampled rows and of sampled columns (qT rows)
        mid, lo, hi = swiglu.swiglu_bf16_band(gu, F)
        un = swiglu.unique_mask(lo, hi)
        ta = band_check.amax_band(lo, hi)
        band_check.check(r["q"][rws], r["scale"], mid[rws], lo[rws], hi[rws], un[rws], f, rule, None,
                           "full q rows", tensor_amax=ta)
        cols_idx = np.concatenate([np.arange(c, c + 128) for c in cls])
        band_check.check(r["qT"][cols_idx].T, r["scale"], mid[:, cols_idx], lo[:, cols_idx], hi[:, cols_idx],
                           un[:, cols_idx], f, rule, None, "full qT cols", tensor_amax=ta)
        return
    gr = np.ascontiguousarray(np.concatenate([gu[rws, :F], gu[rws, F:2 * F]], axis=1))
    mid, lo, hi = swiglu.swiglu_bf16_band(gr, F)
    band_check.check(r["q"][rws], r["scale"][rws], mid, lo, hi, swiglu.unique_mask(lo, hi), f, rule, 1,
                       "full 1x128 rows")
    cols_idx = np.concatenate([np.arange(c, c + 128) for c in cls])
    gc = np.ascontiguousarray(np.concatenate([gu[:, cols_idx], gu[:, F + cols_idx]], axis=1))
    mid, lo, hi = swiglu.swiglu_bf16_band(gc, cols_idx.size)
    band_check.check(r["qT"][cols_idx].T, r["scaleT"][cols_idx], mid, lo, hi, swiglu.unique_mask(lo, hi), f,
                       rule, 0, "full 128x1 cols")
