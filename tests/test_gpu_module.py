"""The autograd wrapper (puro.linear / puro.Linear) runs the same kernels as
the C ABI calls: its forward, dX and dW equal puro_linear_fwd / _bwd bit for
bit, dW accumulates into the FP32 main_grad, and leading dimensions flatten."""

import pytest

from paper_2608_27370_amd import inputs

from gpu_util import to_dev_bf16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    from paper_2608_27370_amd import puro
    puro.lib()
    return puro


def test_linear_module_matches_the_abi_calls(P):
    import torch
    M, K, N = 512, 384, 256
    X = to_dev_bf16(inputs.case(61, (2, M // 2, K)))
    W0 = to_dev_bf16(inputs.case(62, (N, K), std=0.02))
    dY = to_dev_bf16(inputs.case(63, (2, M // 2, N), std=1e-3))
    lin = P.Linear(K, N, device="cuda")
    with torch.no_grad():
        lin.weight.copy_(W0)
    x = X.clone().requires_grad_(True)
    y = lin(x)
    assert y.shape == (2, M // 2, N) and y.dtype == torch.bfloat16
    y.backward(dY)
    Yr, saved = P.linear_fwd(X.reshape(M, K), W0, lin.recipe)
    dXr, dWr = P.linear_bwd(dY.reshape(M, N), saved, lin.recipe, K)
    assert torch.equal(y.reshape(M, N).view(torch.int16), Yr.view(torch.int16))
    assert torch.equal(x.grad.reshape(M, K).view(torch.int16), dXr.view(torch.int16))
    assert lin.weight.grad is None
    assert torch.equal(lin.weight.main_grad, dWr)
    # a second backward accumulates in FP32, in the kernel
    y2 = lin(x)
    y2.backward(dY)
    assert torch.equal(lin.weight.main_grad, (dWr + dWr))


def test_linear_function_without_main_grad(P):
    import torch
    M, K, N = 256, 256, 384
    X = to_dev_bf16(inputs.case(64, (M, K)))
    W = to_dev_bf16(inputs.case(65, (N, K), std=0.02)).requires_grad_(True)
    dY = to_dev_bf16(inputs.case(66, (M, N), std=1e-3))
    rc = P.LinearRecipe(P.E4M3, P.E4M3, P.E5M2, 0, P.SCALE_FP32)
    y = P.linear(X, W, rc)
    y.backward(dY)
    _, saved = P.linear_fwd(X, W.detach(), rc)
    _, dWr = P.linear_bwd(dY, saved, rc, K, want_dx=False)
    assert W.grad.dtype == torch.bfloat16
    assert torch.equal(W.grad.view(torch.int16), dWr.to(torch.bfloat16).view(torch.int16))
