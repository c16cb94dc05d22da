"""Thin ctypes binding of libpuro (include/puro.h): argument marshalling only.

Every operation runs in the HIP kernels of ``libpuro.so``; torch supplies
device memory and the current stream. There is no fallback: if the library
is missing or a call fails, an exception is raised.

Tensors: BF16 data as ``torch.bfloat16`` (or int16/uint16 holding the bit
patterns), FP8 codes as ``torch.uint8``, scales as ``torch.float32``, all on
the GPU; 2-D with unit stride along rows.
"""

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpuro.so")

E4M3, E5M2 = 0, 1
SCALE_TENSOR, SCALE_ROW_1x128, SCALE_COL_128x1, SCALE_BLOCK_128x128 = 0, 1, 2, 3
SCALE_KMAJOR = 0x100    # OR-ed into a grouped mode: k-block-major scale arrays
SCALE_FP32, SCALE_POW2, SCALE_POW2_FLOOR = 0, 1, 2
OUT_BF16, OUT_FP32 = 0, 1

_i64, _sz, _p, _i = ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int


class PuroError(RuntimeError):
    def __init__(self, fn, code, msg):
        super().__init__("%s failed: %s (status %d)" % (fn, msg, code))
        self.code = code


class Operand(ctypes.Structure):
    """puro_fp8_operand: FP8 codes [rows, K] (row pitch ld bytes) and scales."""
    _fields_ = [("data", _p), ("ld", _i64), ("fmt", _i), ("mode", _i), ("scale", _p)]


class Recipe(ctypes.Structure):
    """puro_linear_recipe."""
    _fields_ = [("x_fmt", _i), ("w_fmt", _i), ("dy_fmt", _i), ("blockwise", _i), ("rnd", _i)]


class Saved(ctypes.Structure):
    """puro_linear_saved."""
    _fields_ = [("xq_t", _p), ("x_scale", _p), ("wq_t", _p), ("w_scale", _p)]


_SIGS = {
    "puro_status_string": (ctypes.c_char_p, [_i]),
    "puro_amax_workspace_size": (_sz, [_i64, _i64]),
    "puro_amax": (_i, [_p, _i64, _i64, _i64, _p, _p, _sz, _p]),
    "puro_quantize_workspace_size": (_sz, [_i64, _i64]),
    "puro_quantize_fp8": (_i, [_p, _i64, _i64, _i64, _i, _i, _i, _p, _p, _p, _p, _p, _p, _sz, _p]),
    "puro_quantize_fp8_static": (_i, [_p, _i64, _i64, _i64, _i, _i, _i, _p, _p, _p, _p, _p, _p]),
    "puro_swiglu_quantize_workspace_size": (_sz, [_i64, _i64]),
    "puro_swiglu_quantize_fp8": (_i, [_p, _i64, _i64, _i64, _i, _i, _i, _p, _p, _p, _p, _p, _sz, _p]),
    "puro_swiglu_bwd_quantize_workspace_size": (_sz, [_i64, _i64]),
    "puro_swiglu_bwd_quantize_fp8": (_i, [_p, _i64, _p, _i64, _i64, _i64, _i, _i, _i, _p, _p, _p, _p, _p, _sz, _p]),
    "puro_rmsnorm_quantize_workspace_size": (_sz, [_i64, _i64]),
    "puro_rmsnorm_quantize_fp8": (_i, [_p, _p, _i64, _i64, _i64, ctypes.c_float, _i, _i, _i, _p, _p, _p, _p, _p,
                                       _p, _sz, _p]),
    "puro_fp8_gemm_workspace_size": (_sz, [_i64, _i64, _i64, _i]),
    "puro_fp8_gemm_plan": (_i, [_i64, _i64, _i64, _i, _i, ctypes.POINTER(_i), ctypes.POINTER(_i),
                                ctypes.POINTER(_i), ctypes.POINTER(_i), ctypes.POINTER(_i)]),
    "puro_fp8_gemm": (_i, [_i64, _i64, _i64, ctypes.POINTER(Operand), ctypes.POINTER(Operand),
                           _p, _i, _i64, _i, _p, _sz, _p]),
    "puro_fp8_gemm_epilogue": (_i, [_i64, _i64, _i64, ctypes.POINTER(Operand), ctypes.POINTER(Operand),
                                    _p, _i64, _p, _p, _i64, _p, _sz, _p]),
    "puro_linear_saved_bytes": (_sz, [_i64, _i64, _i64, ctypes.POINTER(Recipe), ctypes.POINTER(_sz * 4)]),
    "puro_linear_fwd_workspace_size": (_sz, [_i64, _i64, _i64, ctypes.POINTER(Recipe)]),
    "puro_linear_bwd_workspace_size": (_sz, [_i64, _i64, _i64, ctypes.POINTER(Recipe)]),
    "puro_linear_fwd": (_i, [_p, _p, _i64, _i64, _i64, ctypes.POINTER(Recipe), _p, ctypes.POINTER(Saved),
                             _p, _sz, _p]),
    "puro_linear_bwd": (_i, [_p, ctypes.POINTER(Saved), _i64, _i64, _i64, ctypes.POINTER(Recipe), _p, _p,
                             _i, _p, _sz, _p]),
    "puro_lm_head_ce_workspace_size": (_sz, [_i64, _i64, _i64, _i, _i]),
    "puro_lm_head_ce_fwd": (_i, [_p, _p, _p, _i64, _i64, _i64, _i, _p, _p, _p, _sz, _p]),
    "puro_lm_head_ce_bwd": (_i, [_p, _p, _p, _p, _i64, _i64, _i64, _i, ctypes.c_float, _p, _p, _p, _sz, _p]),
    "puro_muonh_workspace_size": (_sz, [_i64, _i64, _i64]),
    "puro_muonh_step": (_i, [_i64, _i64, _i64, _p, _p, _p, _p, _p, ctypes.c_float, _i, ctypes.c_float, _i, _p,
                             _p, _sz, _p]),
    "puro_newton_schulz_workspace_size": (_sz, [_i64, _i64, _i64]),
    "puro_newton_schulz_bf16": (_i, [_i64, _i64, _i64, _p, _i, _p, _p, _sz, _p]),
}

_lib = None


def lib():
    """The loaded libpuro (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libpuro.so is not built (run paper_2608_27370_amd/build.py or "
                              "__graft_entry__.build()); there is no fallback path")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def status_string(code):
    return lib().puro_status_string(code).decode()


def _check(fn, code):
    if code != 0:
        raise PuroError(fn, code, status_string(code))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ld(t):
    assert t.dim() == 2, "2-D tensors"
    if t.numel() == 0:
        return t.shape[1]          # torch gives empty tensors zero strides
    assert t.stride(1) == 1, "2-D tensors with unit column stride"
    return t.stride(0)


def _ws(nbytes, ws, device):
    if nbytes == 0:
        return None, 0
    if ws is None:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    assert ws.numel() * ws.element_size() >= nbytes
    return ws, ws.numel() * ws.element_size()


# ------------------------------------------------------------------- amax
def amax(x, out=None, ws=None):
    """max |x| of a 2-D BF16 tensor as a one-element float32 device tensor."""
    rows, cols = x.shape
    if out is None:
        out = torch.empty(1, dtype=torch.float32, device=x.device)
    w, nb = _ws(lib().puro_amax_workspace_size(rows, cols), ws, x.device)
    _check("puro_amax", lib().puro_amax(_ptr(x), rows, cols, _ld(x), _ptr(out), _ptr(w), nb, _stream()))
    return out


# --------------------------------------------------------------- quantise
def quantize_fp8(x, fmt, mode=SCALE_TENSOR, rnd=SCALE_FP32, amax_in=None, want_q=True, want_qT=False,
                 out=None, ws=None):
    """Quantise a 2-D BF16 tensor; returns dict(q, scale, qT, scaleT) (absent
    outputs are None). ``out`` may supply preallocated outputs."""
    rows, cols = x.shape
    dev = x.device
    q, scale, qT, scaleT = _quant_outputs(rows, cols, mode, want_q, want_qT, out, dev)
    w, nb = _ws(lib().puro_quantize_workspace_size(rows, cols), ws, dev)
    _check("puro_quantize_fp8", lib().puro_quantize_fp8(
        _ptr(x), rows, cols, _ld(x), fmt, mode, rnd, _ptr(amax_in), _ptr(q), _ptr(scale), _ptr(qT),
        _ptr(scaleT), _ptr(w), nb, _stream()))
    return dict(q=q, scale=scale, qT=qT, scaleT=scaleT)


def quantize_fp8_static(x, fmt, mode=SCALE_TENSOR, rnd=SCALE_FP32, amax_in=None, want_q=True, want_qT=False,
                        out=None):
    """quantize_fp8 through the allocation-free entry point (the library's
    own per-GPU scratch instead of a workspace); pass preallocated ``out``
    tensors to allocate nothing at all."""
    rows, cols = x.shape
    q, scale, qT, scaleT = _quant_outputs(rows, cols, mode, want_q, want_qT, out, x.device)
    _check("puro_quantize_fp8_static", lib().puro_quantize_fp8_static(
        _ptr(x), rows, cols, _ld(x), fmt, mode, rnd, _ptr(amax_in), _ptr(q), _ptr(scale), _ptr(qT),
        _ptr(scaleT), _stream()))
    return dict(q=q, scale=scale, qT=qT, scaleT=scaleT)


def _quant_outputs(rows, cols, mode, want_q, want_qT, out, dev):
    """Output tensors of a quantisation (supplied ones from `out` kept), in the
    scale layout the mode's SCALE_KMAJOR flag selects."""
    out = dict(out or {})
    G = 128
    km = bool(mode & SCALE_KMAJOR)
    base = mode & ~SCALE_KMAJOR
    if base == SCALE_COL_128x1:
        want_q, want_qT = False, True
    q = out.get("q") if want_q else None
    if want_q and q is None:
        q = torch.empty(rows, cols, dtype=torch.uint8, device=dev)
    qT = out.get("qT") if want_qT else None
    if want_qT and qT is None:
        qT = torch.empty(cols, rows, dtype=torch.uint8, device=dev)
    scale, scaleT = out.get("scale"), out.get("scaleT")

    def new(shape):
        return torch.empty(*(shape[::-1] if km else shape), dtype=torch.float32, device=dev)
    if base == SCALE_TENSOR:
        scale = scale if scale is not None else torch.empty(1, dtype=torch.float32, device=dev)
        scaleT = None
    elif base == SCALE_ROW_1x128:
        scale = scale if scale is not None else new((rows, cols // G))
        if want_qT and scaleT is None:
            scaleT = new((cols, rows // G))
    elif base == SCALE_COL_128x1:
        scale = None
        scaleT = scaleT if scaleT is not None else new((cols, rows // G))
    elif base == SCALE_BLOCK_128x128:
        scale = scale if scale is not None else new((rows // G, cols // G))
        if want_qT and scaleT is None:
            scaleT = new((cols // G, rows // G))
    if not want_qT:
        scaleT = None
    return q, scale, qT, scaleT


# -------------------------------------------- SwiGLU backward + quantise
def swiglu_bwd_quantize_fp8(dh, gu, fmt, mode=SCALE_TENSOR, rnd=SCALE_FP32, want_q=True, want_qT=False,
                            out=None, ws=None):
    """Quantise dgu = [dH u silu'(g) | dH silu(g)] [rows, 2 cols] from dH
    [rows, cols] and the saved gate/up output gu [rows, 2 cols] without
    writing dgu; returns dict(q, scale, qT, scaleT)."""
    rows, cols = dh.shape
    assert gu.shape[0] == rows and gu.shape[1] >= 2 * cols
    dev = dh.device
    q, scale, qT, scaleT = _quant_outputs(rows, 2 * cols, mode, want_q, want_qT, out, dev)
    w, nb = _ws(lib().puro_swiglu_bwd_quantize_workspace_size(rows, cols), ws, dev)
    _check("puro_swiglu_bwd_quantize_fp8", lib().puro_swiglu_bwd_quantize_fp8(
        _ptr(dh), _ld(dh), _ptr(gu), _ld(gu), rows, cols, fmt, mode, rnd, _ptr(q), _ptr(scale), _ptr(qT),
        _ptr(scaleT), _ptr(w), nb, _stream()))
    return dict(q=q, scale=scale, qT=qT, scaleT=scaleT)


# ---------------------------------------------------- RMSNorm + quantise
def rmsnorm_quantize_fp8(x, gamma, eps, fmt, mode=SCALE_TENSOR, rnd=SCALE_FP32, want_q=True, want_qT=False,
                         out=None, ws=None):
    """Quantise y = BF16(x * rstd * gamma) (RMSNorm of each row of x) without
    writing y; returns dict(q, scale, qT, scaleT, rstd) with rstd [rows]
    float32 (out may also supply "rstd")."""
    rows, cols = x.shape
    dev = x.device
    q, scale, qT, scaleT = _quant_outputs(rows, cols, mode, want_q, want_qT, out, dev)
    rstd = (out or {}).get("rstd")
    if rstd is None:
        rstd = torch.empty(rows, dtype=torch.float32, device=dev)
    w, nb = _ws(lib().puro_rmsnorm_quantize_workspace_size(rows, cols), ws, dev)
    _check("puro_rmsnorm_quantize_fp8", lib().puro_rmsnorm_quantize_fp8(
        _ptr(x), _ptr(gamma), rows, cols, _ld(x), float(eps), fmt, mode, rnd, _ptr(q), _ptr(scale), _ptr(qT),
        _ptr(scaleT), _ptr(rstd), _ptr(w), nb, _stream()))
    return dict(q=q, scale=scale, qT=qT, scaleT=scaleT, rstd=rstd)


# ----------------------------------------------------- SwiGLU + quantise
def swiglu_quantize_fp8(gu, cols, fmt, mode=SCALE_TENSOR, rnd=SCALE_FP32, want_q=True, want_qT=False,
                        out=None, ws=None):
    """Quantise H = BF16(silu(gate) * up) of a fused gate/up output gu
    [rows, 2 cols] (gate = gu[:, :cols], up = gu[:, cols:2 cols]) without
    writing H; returns dict(q, scale, qT, scaleT) as quantize_fp8 does."""
    rows = gu.shape[0]
    assert gu.shape[1] >= 2 * cols
    dev = gu.device
    q, scale, qT, scaleT = _quant_outputs(rows, cols, mode, want_q, want_qT, out, dev)
    w, nb = _ws(lib().puro_swiglu_quantize_workspace_size(rows, cols), ws, dev)
    _check("puro_swiglu_quantize_fp8", lib().puro_swiglu_quantize_fp8(
        _ptr(gu), rows, cols, _ld(gu), fmt, mode, rnd, _ptr(q), _ptr(scale), _ptr(qT), _ptr(scaleT),
        _ptr(w), nb, _stream()))
    return dict(q=q, scale=scale, qT=qT, scaleT=scaleT)


# ------------------------------------------------------------------- GEMM
def operand(data, fmt, mode, scale):
    """Describe a reduction-contiguous FP8 operand [rows, K]."""
    op = Operand(data.data_ptr(), _ld(data), fmt, mode, scale.data_ptr())
    op._keep = (data, scale)
    return op


def fp8_gemm_workspace_size(M, N, K, out_dtype):
    return lib().puro_fp8_gemm_workspace_size(M, N, K, out_dtype)


def fp8_gemm_plan(M, N, K, a_mode=SCALE_TENSOR, b_mode=SCALE_TENSOR):
    """The plan puro_fp8_gemm takes: dict(tile_m, tile_n, stages, splits, launches)."""
    v = [_i() for _ in range(5)]
    _check("puro_fp8_gemm_plan", lib().puro_fp8_gemm_plan(M, N, K, a_mode, b_mode, *[ctypes.byref(x) for x in v]))
    return dict(zip(("tile_m", "tile_n", "stages", "splits", "launches"), (x.value for x in v)))


def fp8_gemm(A, a_rows, B, b_rows, K, out_dtype=OUT_BF16, D=None, accumulate=False, ws=None):
    """D[M, N] (+)= sum_k A[m, k] B[n, k] with M = a_rows, N = b_rows."""
    M, N = a_rows, b_rows
    dev = torch.device("cuda", torch.cuda.current_device())
    if D is None:
        dt = torch.bfloat16 if out_dtype == OUT_BF16 else torch.float32
        D = torch.empty(M, N, dtype=dt, device=dev)
    w, nb = _ws(fp8_gemm_workspace_size(M, N, K, out_dtype), ws, dev)
    _check("puro_fp8_gemm", lib().puro_fp8_gemm(M, N, K, ctypes.byref(A), ctypes.byref(B), _ptr(D),
                                                out_dtype, _ld(D), int(bool(accumulate)), _ptr(w), nb,
                                                _stream()))
    return D


def fp8_gemm_epilogue(A, a_rows, B, b_rows, K, bias=None, residual=None, D=None, ws=None):
    """D[M, N] = BF16(sum_k A[m, k] B[n, k] + bias[n] + residual[m, n]) (bias
    and residual BF16, optional; residual may be D itself)."""
    M, N = a_rows, b_rows
    dev = torch.device("cuda", torch.cuda.current_device())
    if D is None:
        D = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
    w, nb = _ws(fp8_gemm_workspace_size(M, N, K, OUT_BF16), ws, dev)
    ldr = _ld(residual) if residual is not None else 0
    _check("puro_fp8_gemm_epilogue", lib().puro_fp8_gemm_epilogue(
        M, N, K, ctypes.byref(A), ctypes.byref(B), _ptr(D), _ld(D), _ptr(bias), _ptr(residual), ldr, _ptr(w), nb,
        _stream()))
    return D


# ----------------------------------------------------------- linear layer
@dataclass
class LinearRecipe:
    x_fmt: int = E4M3
    w_fmt: int = E4M3
    dy_fmt: int = E5M2
    blockwise: int = 0
    rnd: int = SCALE_FP32

    def c(self):
        return Recipe(self.x_fmt, self.w_fmt, self.dy_fmt, self.blockwise, self.rnd)


def linear_saved(M, N, K, recipe, device):
    """Allocate the saved-for-backward buffers of a linear layer."""
    sizes = (_sz * 4)()
    lib().puro_linear_saved_bytes(M, N, K, ctypes.byref(recipe.c()), ctypes.byref(sizes))
    G = 128
    xq_t = torch.empty(K, M, dtype=torch.uint8, device=device)
    wq_t = torch.empty(K, N, dtype=torch.uint8, device=device)
    if recipe.blockwise:
        # k-block-major scale layouts (include/puro.h)
        xs = torch.empty(M // G, K, dtype=torch.float32, device=device)
        wsc = torch.empty(N // G, K // G, dtype=torch.float32, device=device)
    else:
        xs = torch.empty(1, dtype=torch.float32, device=device)
        wsc = torch.empty(1, dtype=torch.float32, device=device)
    assert [xq_t.numel(), xs.numel() * 4, wq_t.numel(), wsc.numel() * 4] == list(sizes)
    return dict(xq_t=xq_t, x_scale=xs, wq_t=wq_t, w_scale=wsc)


def _saved_struct(saved):
    return Saved(saved["xq_t"].data_ptr(), saved["x_scale"].data_ptr(), saved["wq_t"].data_ptr(),
                 saved["w_scale"].data_ptr())


def linear_fwd_workspace_size(M, N, K, recipe):
    return lib().puro_linear_fwd_workspace_size(M, N, K, ctypes.byref(recipe.c()))


def linear_bwd_workspace_size(M, N, K, recipe):
    return lib().puro_linear_bwd_workspace_size(M, N, K, ctypes.byref(recipe.c()))


def linear_fwd(X, W, recipe, Y=None, saved=None, ws=None):
    """Y = X W^T (FP8 Fprop); returns (Y, saved)."""
    M, K = X.shape
    N = W.shape[0]
    dev = X.device
    if Y is None:
        Y = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
    if saved is None:
        saved = linear_saved(M, N, K, recipe, dev)
    w, nb = _ws(linear_fwd_workspace_size(M, N, K, recipe), ws, dev)
    s = _saved_struct(saved)
    _check("puro_linear_fwd", lib().puro_linear_fwd(_ptr(X), _ptr(W), M, N, K, ctypes.byref(recipe.c()),
                                                    _ptr(Y), ctypes.byref(s), _ptr(w), nb, _stream()))
    return Y, saved


def linear_bwd(dY, saved, recipe, K, want_dx=True, want_dw=True, dX=None, dW=None, accumulate_dw=False,
               ws=None):
    """dX = dY W (BF16) and dW = dY^T X (FP32); returns (dX, dW)."""
    M, N = dY.shape
    dev = dY.device
    if want_dx and dX is None:
        dX = torch.empty(M, K, dtype=torch.bfloat16, device=dev)
    if want_dw and dW is None:
        dW = torch.zeros(N, K, dtype=torch.float32, device=dev)
    w, nb = _ws(linear_bwd_workspace_size(M, N, K, recipe), ws, dev)
    s = _saved_struct(saved)
    _check("puro_linear_bwd", lib().puro_linear_bwd(
        _ptr(dY), ctypes.byref(s), M, N, K, ctypes.byref(recipe.c()), _ptr(dX if want_dx else None),
        _ptr(dW if want_dw else None), int(bool(accumulate_dw)), _ptr(w), nb, _stream()))
    return (dX if want_dx else None), (dW if want_dw else None)


class _LinearFn(torch.autograd.Function):
    """Y = X W^T through puro_linear_fwd; the backward runs puro_linear_bwd
    from the FP8 copies the forward saved (the BF16 X is not kept). With a
    ``main_grad`` FP32 buffer on W, dW is accumulated into it by the Wgrad
    GEMM and W gets no .grad; otherwise W's .grad is dW in W's dtype."""

    @staticmethod
    def forward(ctx, X, W, recipe):
        if X.dtype != torch.bfloat16 or W.dtype != torch.bfloat16:
            raise TypeError("the FP8 linear layer takes BF16 X and W")
        Y, saved = linear_fwd(X.contiguous(), W.contiguous(), recipe)
        ctx.saved, ctx.recipe, ctx.K = saved, recipe, X.shape[1]
        ctx.main_grad = getattr(W, "main_grad", None)
        return Y

    @staticmethod
    def backward(ctx, dY):
        want_dx, want_dw = ctx.needs_input_grad[0], ctx.needs_input_grad[1]
        mg = ctx.main_grad if want_dw else None
        dX, dW = linear_bwd(dY.to(torch.bfloat16).contiguous(), ctx.saved, ctx.recipe, ctx.K, want_dx=want_dx,
                            want_dw=want_dw, dW=mg, accumulate_dw=mg is not None)
        ctx.saved = None
        if mg is not None:
            return dX, None, None
        return dX, (dW.to(torch.bfloat16) if dW is not None else None), None


def linear(X, W, recipe):
    """The FP8 linear layer as an autograd operation: X [..., K], W [N, K]
    (BF16); returns Y [..., N] (BF16)."""
    shp = X.shape
    Y = _LinearFn.apply(X.reshape(-1, shp[-1]), W, recipe)
    return Y.reshape(*shp[:-1], Y.shape[-1])


class Linear(torch.nn.Module):
    """A bias-free linear layer whose forward and backward run the FP8 path
    (default: the paper's blockwise recipe, E4M3 with power-of-two scales).
    The weight is BF16, as the model's GEMM operands are (Appendix C); with
    ``main_grad`` (default) its FP32 gradient is accumulated into
    ``weight.main_grad`` across backward passes, for an optimiser that keeps
    FP32 state (zero it after each step)."""

    def __init__(self, in_features, out_features, recipe=None, main_grad=True, device=None):
        super().__init__()
        self.in_features, self.out_features = in_features, out_features
        self.recipe = recipe if recipe is not None else LinearRecipe(E4M3, E4M3, E4M3, 1, SCALE_POW2)
        self.weight = torch.nn.Parameter(torch.empty(out_features, in_features, dtype=torch.bfloat16,
                                                     device=device))
        with torch.no_grad():
            self.weight.normal_(0.0, 0.02)
        if main_grad:
            self.weight.main_grad = torch.zeros(out_features, in_features, dtype=torch.float32,
                                                device=self.weight.device)

    def forward(self, x):
        return linear(x, self.weight, self.recipe)


# ------------------------------------------ LM head with cross-entropy loss
LM_HEAD_BF16, LM_HEAD_FP8 = 0, 1


def lm_head_ce_workspace_size(M, V, K, recipe, backward):
    return lib().puro_lm_head_ce_workspace_size(M, V, K, recipe, int(bool(backward)))


def lm_head_ce_fwd(X, W, targets, recipe=LM_HEAD_BF16, lse=None, loss=None, ws=None):
    """lse [M] and loss [M] = lse - z_target of the logits X W^T (never
    stored); X [M, K], W [V, K] BF16, targets [M] int32; returns (lse, loss)."""
    M, K = X.shape
    V = W.shape[0]
    dev = X.device
    lse = torch.empty(M, dtype=torch.float32, device=dev) if lse is None else lse
    loss = torch.empty(M, dtype=torch.float32, device=dev) if loss is None else loss
    w, nb = _ws(lm_head_ce_workspace_size(M, V, K, recipe, False), ws, dev)
    _check("puro_lm_head_ce_fwd", lib().puro_lm_head_ce_fwd(
        _ptr(X), _ptr(W), _ptr(targets), M, V, K, recipe, _ptr(lse), _ptr(loss), _ptr(w), nb, _stream()))
    return lse, loss


def lm_head_ce_bwd(X, W, targets, lse, recipe=LM_HEAD_BF16, grad_scale=1.0, dX=None, dW=None, ws=None):
    """dX [M, K] (BF16) and dW [V, K] (FP32) of grad_scale * sum of the losses."""
    M, K = X.shape
    V = W.shape[0]
    dev = X.device
    dX = torch.empty(M, K, dtype=torch.bfloat16, device=dev) if dX is None else dX
    dW = torch.empty(V, K, dtype=torch.float32, device=dev) if dW is None else dW
    w, nb = _ws(lm_head_ce_workspace_size(M, V, K, recipe, True), ws, dev)
    _check("puro_lm_head_ce_bwd", lib().puro_lm_head_ce_bwd(
        _ptr(X), _ptr(W), _ptr(targets), _ptr(lse), M, V, K, recipe, float(grad_scale), _ptr(dX), _ptr(dW),
        _ptr(w), nb, _stream()))
    return dX, dW


# ------------------------------------------------------------------- MuonH
def muonh_step(W, G, buf, radius, eta, mu=0.95, nesterov=True, ns_steps=5, w_bf16=None, u_out=None, ws=None):
    """One MuonH step of W [count, rows, cols] (or [rows, cols]) in place,
    with buf (the momentum) updated in place; radius [count] FP32. Returns
    (w_bf16, u_out) when asked for."""
    shp = W.shape
    count, rows, cols = (1,) + tuple(shp) if W.dim() == 2 else tuple(shp)
    w, nb = _ws(lib().puro_muonh_workspace_size(count, rows, cols), ws, W.device)
    _check("puro_muonh_step", lib().puro_muonh_step(
        count, rows, cols, _ptr(W), _ptr(w_bf16), _ptr(G), _ptr(buf), _ptr(radius), float(mu), int(bool(nesterov)),
        float(eta), int(ns_steps), _ptr(u_out), _ptr(w), nb, _stream()))
    return w_bf16, u_out


def newton_schulz_bf16(X, steps=5, out=None, ws=None):
    """steps Newton-Schulz steps on X [count, r, c] (or [r, c]) BF16, r <= c."""
    count, r, c = (1,) + tuple(X.shape) if X.dim() == 2 else tuple(X.shape)
    out = torch.empty_like(X) if out is None else out
    w, nb = _ws(lib().puro_newton_schulz_workspace_size(count, r, c), ws, X.device)
    _check("puro_newton_schulz_bf16", lib().puro_newton_schulz_bf16(
        count, r, c, _ptr(X), int(steps), _ptr(out), _ptr(w), nb, _stream()))
    return out
