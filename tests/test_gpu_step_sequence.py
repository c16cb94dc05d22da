"""The 28-layer blockwise step as one sequence of calls, as bench.py runs it:
puro_linear_fwd for the 112 linears in layer order, then puro_linear_bwd for
them in reverse, one forward and one backward workspace shared by every call.

Layers 0 and 27 take the seeded workload inputs (inputs.layer_linear) and are
checked against the oracle after the whole sequence. Their saved FP8 state
(XqT, WqT and scales) must survive the other calls in between, and their
outputs must match the oracle on sampled entries: the first and last tiles
of every output, and 256 random entries. The other 26 layers' tensors come
from torch's generator on the device (their values reach no checked output).
Y and dX of the checked layers get buffers of their own. The other layers
share one per kind, as in the bench.
"""

import numpy as np
import pytest

from oracle import gemm, quant
from paper_2608_27370_amd import inputs

import mfma_model
from gpu_util import assert_bytes_equal, assert_f32_bits_equal, bf16_bits, check_bf16, check_fp32, host, to_dev_bf16

pytestmark = pytest.mark.gpu

E4 = 0
M = 16384
CHECKED = (0, inputs.LAYERS - 1)


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


def entries(R, C, rng, n=256):
    """The first and last 16 x 16 corner of the output and n random entries."""
    r0, c0 = np.meshgrid(np.arange(16), np.arange(16), indexing="ij")
    ms = np.concatenate([r0.ravel(), R - 16 + r0.ravel(), rng.integers(0, R, n)])
    ns = np.concatenate([c0.ravel(), C - 16 + c0.ravel(), rng.integers(0, C, n)])
    return ms, ns


def check(D, out, ms, ns, A_bits, A_rule, B, what, b_rows=None):
    """Entries (ms, ns) of D against the oracle; A's rows quantised in 1x128
    groups from A_bits (rows ms), B = (codes, fmt, scales, mode) whole or,
    with b_rows, holding only those rows of the operand."""
    rows = np.unique(ms)
    qa, sa = quant.quantize_rows_1x128(np.ascontiguousarray(A_bits[rows]), "e4m3", A_rule)
    am = np.searchsorted(rows, ms)
    bn = ns if b_rows is None else np.searchsorted(b_rows, ns)
    op = (qa, "e4m3", sa, "row") + B
    ref, den = gemm.gemm_entries(am, bn, *op)
    slack = mfma_model.truncation_loss(am, bn, *op, chunk=64)
    if out == "fp32":
        check_fp32(host(D)[ms, ns], ref, den, what=what, slack=slack, strict=True)
    else:
        check_bf16(bf16_bits(D)[ms, ns], ref, den, what=what, slack=slack, strict=True)


@pytest.mark.timeout(1200)
def test_28_layer_step_sequence(P):
    import torch
    dev = torch.device("cuda", 0)
    rc = P.LinearRecipe(E4, E4, E4, 1, P.SCALE_POW2)
    kinds = inputs.LAYER_LINEARS
    gen = torch.Generator(device=dev)
    gen.manual_seed(28)

    def normal(shape, std):
        return (torch.randn(shape, generator=gen, device=dev) * std).to(torch.bfloat16)
    host_in, layers = {}, []
    print("step sequence: inputs", flush=True)
    for li in range(inputs.LAYERS):
        row = []
        for j, (name, N, K) in enumerate(kinds):
            if li in CHECKED:
                d = inputs.layer_linear(li, j, M=M)
                host_in[(li, j)] = d
                X, W, dY = to_dev_bf16(d["X"]), to_dev_bf16(d["W"]), to_dev_bf16(d["dY"])
            else:
                X, W, dY = normal((M, K), 1.0), normal((N, K), 0.02), normal((M, N), 1e-3)
            row.append(dict(X=X, W=W, dY=dY, saved=P.linear_saved(M, N, K, rc, dev)))
        layers.append(row)
    shared = [dict(Y=torch.empty(M, N, dtype=torch.bfloat16, device=dev),
                   dX=torch.empty(M, K, dtype=torch.bfloat16, device=dev),
                   dW=torch.empty(N, K, dtype=torch.float32, device=dev)) for _, N, K in kinds]
    own = {(li, j): dict(Y=torch.empty(M, N, dtype=torch.bfloat16, device=dev),
                         dX=torch.empty(M, K, dtype=torch.bfloat16, device=dev),
                         dW=torch.empty(N, K, dtype=torch.float32, device=dev))
           for li in CHECKED for j, (_, N, K) in enumerate(kinds)}
    wsf = torch.empty(max(P.linear_fwd_workspace_size(M, N, K, rc) for _, N, K in kinds), dtype=torch.uint8,
                      device=dev)
    wsb = torch.empty(max(P.linear_bwd_workspace_size(M, N, K, rc) for _, N, K in kinds), dtype=torch.uint8,
                      device=dev)
    print("step sequence: forward and backward of 112 linears", flush=True)
    for li, row in enumerate(layers):
        for j, lin in enumerate(row):
            o = own.get((li, j), shared[j])
            P.linear_fwd(lin["X"], lin["W"], rc, Y=o["Y"], saved=lin["saved"], ws=wsf)
    for li in reversed(range(inputs.LAYERS)):
        for j in reversed(range(len(kinds))):
            lin, o = layers[li][j], own.get((li, j), shared[j])
            P.linear_bwd(lin["dY"], lin["saved"], rc, kinds[j][2], dX=o["dX"], dW=o["dW"], ws=wsb)
    torch.cuda.synchronize()
    g = np.random.default_rng(29)
    for li in CHECKED:
        for j, (name, N, K) in enumerate(kinds):
            print("step sequence: check layer %d %s" % (li, name), flush=True)
            d, sv, o = host_in[(li, j)], layers[li][j]["saved"], own[(li, j)]
            X, W, dY = d["X"], d["W"], d["dY"]
            what = "sequence layer %d %s" % (li, name)
            # the saved state after the whole sequence: W's blocks whole, X's column groups on sampled rows
            wq, ws, wqT, wsT = quant.quantize_blocks_128x128(W, "e4m3", "pow2")
            assert_bytes_equal(host(sv["wq_t"]), wqT, what + " wq_t")
            assert_f32_bits_equal(host(sv["w_scale"]).T, wsT, what + " w scales")
            kr = np.unique(g.choice(K, 16, replace=False))
            q, s = quant.quantize_cols_128x1(np.ascontiguousarray(X[:, kr]), "e4m3", "pow2")
            assert_bytes_equal(host(sv["xq_t"])[kr], q, what + " xq_t rows")
            assert_f32_bits_equal(host(sv["x_scale"])[:, kr].T, s, what + " x column-group scales")
            ms, ns = entries(M, N, g)
            check(o["Y"], "bf16", ms, ns, X, "pow2", (wq, "e4m3", ws, "block"), what + " Y")
            ms, ks = entries(M, K, g)
            check(o["dX"], "bf16", ms, ks, dY, "pow2", (wqT, "e4m3", wsT, "block"), what + " dX")
            # Wgrad: dY's and X's 128x1 column groups, as the transposed operands
            ns, ks = entries(N, K, g)
            dyT = np.ascontiguousarray(dY.T)
            kcols = np.unique(ks)
            qx, sx = quant.quantize_cols_128x1(np.ascontiguousarray(X[:, kcols]), "e4m3", "pow2")
            check(o["dW"], "fp32", ns, ks, dyT, "pow2", (qx, "e4m3", sx, "row"), what + " dW", b_rows=kcols)
