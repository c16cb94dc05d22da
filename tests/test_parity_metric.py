"""Host logic of the GEMM parity metric (tests/gpu_util.py): the rounding
interval of a BF16 value and the least tolerance with which a BF16 output
passes, pinned against round-to-nearest-even itself."""

import numpy as np

from oracle import bf16
from gpu_util import bf16_interval, plain_ratio_bf16, plain_ratio_fp32


def test_bf16_interval_is_the_rounding_preimage():
    b = np.arange(0, 0x7F7F, 7, dtype=np.uint32).astype(np.uint16)
    b = np.concatenate([b, b | 0x8000])
    lo, hi = bf16_interval(b)
    v = bf16.to_f32(b).astype(np.float64)
    assert np.all(lo <= v) and np.all(v <= hi)
    # just inside each end rounds to the value, just outside does not
    eps = np.maximum(np.abs(v), 2.0 ** -133) * 2.0 ** -20
    same = lambda x: bf16.to_f32(bf16.from_f64_rne(x)).astype(np.float64) == v
    assert same(lo + eps).all() and same(hi - eps).all()
    nz = (b & 0x7FFF) != 0
    assert not same(lo - eps)[nz].any() and not same(hi + eps)[nz].any()


def test_plain_ratio_bf16():
    ref = np.array([1.0, 1.0, 1.0, 0.0])
    den = np.array([1.0, 1.0, 100.0, 0.0])
    # 1 + 2^-7 is the next BF16 above 1: its interval starts at 1 + 2^-8
    d = bf16.from_f64_rne(np.array([1.0, 1.0 + 2.0 ** -7, 1.0 + 2.0 ** -7, 0.0]))
    r = plain_ratio_bf16(d, ref, den)
    np.testing.assert_allclose(r, [0.0, 2.0 ** -8, 2.0 ** -8 / 100, 0.0])


def test_plain_ratio_fp32():
    r = plain_ratio_fp32(np.array([1.0, 2.0, 0.0, 1.0]), np.array([1.0, 1.5, 0.0, 0.0]), np.array([1, 10, 0, 0.0]))
    assert list(r[:3]) == [0.0, 0.05, 0.0] and np.isinf(r[3])
