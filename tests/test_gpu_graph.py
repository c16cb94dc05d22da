"""The linear layer's fwd + bwd captured in a HIP graph: every replay must
give the bytes the eager calls give (all kernels are deterministic), with
eager work and synchronisations between replays."""

import numpy as np
import pytest

from paper_2608_27370_amd import inputs

from gpu_util import to_dev_bf16

pytestmark = pytest.mark.gpu

E4, E5 = 0, 1


@pytest.mark.parametrize("blockwise", [0, 1], ids=["tensor", "blockwise"])
def test_linear_step_graph_replays_match_eager(blockwise):
    import torch
    from paper_2608_27370_amd import puro
    M, N, K = 1024, 768, 512
    X = to_dev_bf16(inputs.case(31, (M, K), kind="outliers"))
    W = to_dev_bf16(inputs.case(32, (N, K), std=0.02))
    dY = to_dev_bf16(inputs.case(33, (M, N), std=1e-3))
    rc = puro.LinearRecipe(E4, E4, E4 if blockwise else E5, blockwise, puro.SCALE_FP32)
    dev = X.device
    saved = puro.linear_saved(M, N, K, rc, dev)
    Y = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
    dX = torch.empty(M, K, dtype=torch.bfloat16, device=dev)
    dW = torch.empty(N, K, dtype=torch.float32, device=dev)
    wsf = torch.empty(max(1, puro.linear_fwd_workspace_size(M, N, K, rc)), dtype=torch.uint8, device=dev)
    wsb = torch.empty(max(1, puro.linear_bwd_workspace_size(M, N, K, rc)), dtype=torch.uint8, device=dev)

    def step():
        puro.linear_fwd(X, W, rc, Y=Y, saved=saved, ws=wsf)
        puro.linear_bwd(dY, saved, rc, K, dX=dX, dW=dW, ws=wsb)

    def snapshot():
        torch.cuda.synchronize()
        return [t.clone() for t in (Y, dX, dW, saved["xq_t"], saved["x_scale"], saved["wq_t"], saved["w_scale"])]

    step()
    want = snapshot()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                      # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(3):
        for t in (Y, dX, dW, saved["xq_t"], saved["wq_t"]):
            t.zero_()               # eager work between replays; the replay must rewrite everything
        g.replay()
        got = snapshot()
        for i, (a, b) in enumerate(zip(got, want)):
            assert torch.equal(a.view(torch.uint8) if a.dtype != torch.uint8 else a,
                               b.view(torch.uint8) if b.dtype != torch.uint8 else b), (r, i)
    del g
