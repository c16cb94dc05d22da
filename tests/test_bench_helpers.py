"""Host-side helpers of bench.py: the mixed-precision effective peak against
the values the paper prints (tests/golden/mixed_precision_peak.txt)."""

import os

import bench

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "mixed_precision_peak.txt")


def _golden():
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    return [tuple(float(v) for v in r) for r in rows]


def test_p_eff_reproduces_the_paper():
    (share, fp8, bf16, printed, thr, mfu), = _golden()
    p = bench.p_eff(share, fp8, bf16)
    assert abs(p - printed) < 0.5                      # printed as "approximately 327"
    assert abs(p - 327.34375) < 1e-9                    # (0.72/419 + 0.28/209.5)^-1 exactly
    assert abs(thr / p - mfu) < 0.005                   # 238 / 327.3 = 0.727 ~ "approximately 73%"


def test_p_eff_limits():
    assert bench.p_eff(1.0, 5000.0, 2500.0) == 5000.0
    assert bench.p_eff(0.0, 5000.0, 2500.0) == 2500.0
    # the harmonic mix lies between the two peaks and below their weighted mean
    p = bench.p_eff(0.72, 5000.0, 2500.0)
    assert 2500.0 < p < 0.72 * 5000 + 0.28 * 2500
