"""Helpers shared by the GPU parity tests (no arithmetic of the method)."""

import numpy as np

from oracle import bf16

TOL = 1e-5   # max |d - ref| / sum_k |a_k b_k| for GEMM outputs

# One record per GEMM check: the plain metric of the acceptance criterion
# (max over the checked entries of the least tolerance t with which the entry
# passes, without the matrix instruction's truncation allowance) and the
# fraction of entries above TOL. Written out at the end of the session.
REPORT = []


def torch_mod():
    import torch
    return torch


def to_dev_bf16(bits):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def to_dev(a):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def bf16_bits(t):
    """BF16 device tensor -> numpy uint16 bit patterns."""
    torch = torch_mod()
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def host(t):
    return t.cpu().numpy()


def _record(what, ratio, strict, kind):
    """Record (and with ``strict`` assert) the plain metric of a check."""
    ratio = np.asarray(ratio, dtype=np.float64)
    mx = float(ratio.max()) if ratio.size else 0.0
    rec = {"what": what, "kind": kind, "entries": int(ratio.size), "max_rel": mx,
           "plain_excess": float(np.mean(ratio > TOL)) if ratio.size else 0.0, "strict": bool(strict)}
    REPORT.append(rec)
    if strict and mx > TOL:
        i = int(np.argmax(ratio))
        raise AssertionError("%s: the plain bound max|err|/sum|ab| <= %g fails: %d of %d entries above it, max %.3g "
                             "(entry %d)" % (what, TOL, int((ratio > TOL).sum()), ratio.size, mx, i))
    return rec


def plain_ratio_fp32(d, ref, den):
    """|d - ref| / den per entry (0 where both vanish, inf where only den does)."""
    d = np.asarray(d, dtype=np.float64)
    err = np.abs(d - ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.where(den > 0, err / np.where(den > 0, den, 1), np.where(err > 0, np.inf, 0.0))


def bf16_interval(d_bits):
    """The real interval [lo, hi] of values that round (RNE) to each BF16
    value: half-way to each neighbour (for +-0, half the smallest subnormal)."""
    b = np.asarray(d_bits, dtype=np.uint16).astype(np.int64)
    sign = np.where(b & 0x8000, -1.0, 1.0)
    m = b & 0x7FFF
    val = lambda k: bf16.to_f32(np.clip(k, 0, 0x7F7F).astype(np.uint16)).astype(np.float64)
    v = val(m)
    below = np.where(m > 0, (v + val(m - 1)) / 2, -val(np.ones_like(m)) / 2)
    above = (v + val(m + 1)) / 2
    lo = np.where(sign > 0, below, -above)
    hi = np.where(sign > 0, above, -below)
    return lo, hi


def plain_ratio_bf16(d_bits, ref, den):
    """The least t with RNE_bf16(ref - t den) <= d <= RNE_bf16(ref + t den):
    the distance from ref to d's rounding interval over den."""
    lo, hi = bf16_interval(d_bits)
    dist = np.maximum(0.0, np.maximum(lo - ref, ref - hi))
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.where(den > 0, dist / np.where(den > 0, den, 1), np.where(dist > 0, np.inf, 0.0))


def check_fp32(d, ref, den, tol=TOL, what="", slack=0.0, strict=False):
    """FP32 outputs: |d - ref| <= tol * den + slack elementwise (d == 0 where
    den == 0). ``slack`` is the per-entry amount the matrix instruction's
    in-group truncation removes (tests/mfma_model.py); with ``strict`` the
    plain bound (no slack) is asserted as well. The plain metric is recorded."""
    d = np.asarray(d, dtype=np.float64)
    _record(what, plain_ratio_fp32(d, ref, den), strict, "fp32")
    err = np.abs(d - ref)
    bad = err > tol * den + slack
    if bad.any():
        i = np.argwhere(bad)[0]
        idx = tuple(i)
        raise AssertionError("%s: %d of %d entries off; first at %s: got %r ref %r den %r (rel %.3g)" % (
            what, bad.sum(), bad.size, idx, d[idx], ref[idx], den[idx],
            err[idx] / den[idx] if den[idx] else np.inf))
    return float(np.max(np.where(den > 0, err / np.where(den > 0, den, 1), 0))) if d.size else 0.0


def check_bf16(d_bits, ref, den, tol=TOL, what="", slack=0.0, strict=False):
    """BF16 outputs: d must lie between the BF16 roundings (RNE) of
    ref - (tol * den + slack) and ref + (tol * den + slack), i.e. d is the BF16
    rounding of some value within the FP32 tolerance of the exact result.
    With ``strict`` the plain band (no slack) is asserted as well. The plain
    metric is recorded."""
    _record(what, plain_ratio_bf16(d_bits, ref, den), strict, "bf16")
    d = bf16.to_f32(d_bits).astype(np.float64)
    allow = tol * den + slack
    lo = bf16.to_f32(bf16.from_f64_rne(ref - allow)).astype(np.float64)
    hi = bf16.to_f32(bf16.from_f64_rne(ref + allow)).astype(np.float64)
    bad = ~((lo <= d) & (d <= hi))
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError("%s: %d of %d BF16 entries outside the band; first at %s: got %r band [%r, %r] "
                             "ref %r" % (what, bad.sum(), bad.size, i, d[i], lo[i], hi[i], ref[i]))


def assert_bytes_equal(got, want, what=""):
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        i = tuple(bad[0])
        raise AssertionError("%s: %d of %d bytes differ; first at %s: got %#x want %#x" % (
            what, len(bad), got.size, i, got[i], want[i]))


def assert_f32_bits_equal(got, want, what=""):
    got = np.ascontiguousarray(got, dtype=np.float32).view(np.uint32)
    want = np.ascontiguousarray(want, dtype=np.float32).view(np.uint32)
    # all NaN patterns count as the same value
    gn = (got & 0x7FFFFFFF) > 0x7F800000
    wn = (want & 0x7FFFFFFF) > 0x7F800000
    same = (got == want) | (gn & wn)
    if not same.all():
        i = tuple(np.argwhere(~same)[0])
        raise AssertionError("%s: scales differ at %s: got %#x want %#x" % (what, i, got[i], want[i]))


def sample_entries(M, N, rng, per_tile=16, tile=256, full_tiles=True):
    """Stratified sample of output entries: ``per_tile`` random entries in every
    tile x tile block, plus every entry of the first and last blocks (the last
    is the ragged corner when M or N is not a multiple of the tile)."""
    ms, ns = [], []
    for t0 in range(0, M, tile):
        for u0 in range(0, N, tile):
            h, w = min(tile, M - t0), min(tile, N - u0)
            ms.append(t0 + rng.integers(0, h, per_tile))
            ns.append(u0 + rng.integers(0, w, per_tile))
    if full_tiles:
        for (t0, u0) in ((0, 0), ((M - 1) // tile * tile, (N - 1) // tile * tile)):
            h, w = min(tile, M - t0), min(tile, N - u0)
            mm, nn = np.meshgrid(np.arange(t0, t0 + h), np.arange(u0, u0 + w), indexing="ij")
            ms.append(mm.ravel())
            ns.append(nn.ravel())
    return np.concatenate(ms).astype(np.int64), np.concatenate(ns).astype(np.int64)
