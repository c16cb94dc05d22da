"""Helpers shared by the GPU parity tests (no arithmetic of the method)."""

import numpy as np

from oracle import bf16

TOL = 1e-5   # max |d - ref| / sum_k |a_k b_k| for GEMM outputs


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


def check_fp32(d, ref, den, tol=TOL, what="", slack=0.0):
    """FP32 outputs: |d - ref| <= tol * den + slack elementwise (d == 0 where
    den == 0). ``slack`` is the per-entry amount the matrix instruction's
    in-group truncation removes (tests/mfma_model.py)."""
    d = np.asarray(d, dtype=np.float64)
    err = np.abs(d - ref)
    bad = err > tol * den + slack
    if bad.any():
        i = np.argwhere(bad)[0]
        idx = tuple(i)
        raise AssertionError("%s: %d of %d entries off; first at %s: got %r ref %r den %r (rel %.3g)" % (
            what, bad.sum(), bad.size, idx, d[idx], ref[idx], den[idx],
            err[idx] / den[idx] if den[idx] else np.inf))
    return float(np.max(np.where(den > 0, err / np.where(den > 0, den, 1), 0))) if d.size else 0.0


def check_bf16(d_bits, ref, den, tol=TOL, what="", slack=0.0):
    """BF16 outputs: d must lie between the BF16 roundings (RNE) of
    ref - (tol * den + slack) and ref + (tol * den + slack), i.e. d is the BF16
    rounding of some value within the FP32 tolerance of the exact result."""
    d = bf16.to_f32(d_bits).astype(np.float64)
    allow = tol * den + slack
    lo = bf16.to_f32(bf16.from_f64_rne(ref - allow)).astype(np.float64)
    hi = bf16.to_f32(bf16.from_f64_rne(ref + allow)).astype(np.float64)
    bad = ~((lo <= d) & (d <= hi))
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError("%s: %d of %d BF16 entries outside the band; first at %s: got %r band [%r, %r] "
                             "ref %r" % (what, bad.sum(), bad.size, i, d[i], lo[i], hi[i], ref[i]))


def plain_excess(d, ref, den, tol=TOL):
    """Fraction of entries whose error exceeds tol * den without the
    instruction-truncation allowance (reported, not asserted)."""
    d = np.asarray(d, dtype=np.float64)
    return float(np.mean(np.abs(d - ref) > tol * den)) if d.size else 0.0


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
