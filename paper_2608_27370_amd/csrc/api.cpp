// C ABI of libpuro: argument validation, workspace layout and kernel launches.
// Declarations and their documentation: include/puro.h.

#include "puro.h"

#include <hip/hip_runtime.h>

#include "kernels.h"

using namespace puro;

namespace {

constexpr int64_t kGroup = 128;
constexpr size_t kAlign = 256;
// largest FP8 operand row pitch of the GEMM (bytes): buffer offsets over a
// 256-row tile stay below 2^31
constexpr int64_t kMaxPitch = (int64_t)1 << 22;

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
inline bool fmt_ok(puro_fp8_format f) { return f == PURO_E4M3 || f == PURO_E5M2; }

puro_status launched() {
    return hipGetLastError() == hipSuccess ? PURO_OK : PURO_ERR_HIP;
}

// Byte offsets of named regions carved from a caller workspace.
struct Carver {
    size_t used = 0;
    size_t take(size_t bytes) {
        const size_t at = used;
        used = align_up(used + bytes);
        return at;
    }
};

size_t amax_ws(int64_t rows, int64_t cols) {
    return (size_t)amax_num_partials(rows, cols) * sizeof(uint32_t);
}

puro_status check_bf16_matrix(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld) {
    if (rows < 0 || cols < 0 || ld < cols) return PURO_ERR_SHAPE;
    if (rows > 0 && cols > 0 && !x) return PURO_ERR_NULL;
    if ((cols % 8) != 0 || (ld % 8) != 0 || !aligned16(x)) return PURO_ERR_ALIGN;
    if (rows > (int64_t)65535 * kGroup || cols > ((int64_t)1 << 31)) return PURO_ERR_SHAPE;
    return PURO_OK;
}

}  // namespace

extern "C" {

const char* puro_status_string(puro_status s) {
    switch (s) {
    case PURO_OK: return "ok";
    case PURO_ERR_NULL: return "a required pointer is NULL";
    case PURO_ERR_SHAPE: return "invalid or mismatched sizes";
    case PURO_ERR_UNSUPPORTED: return "unsupported format, scale mode or rounding combination";
    case PURO_ERR_ALIGN: return "size or pointer alignment not supported";
    case PURO_ERR_WORKSPACE: return "workspace too small";
    case PURO_ERR_HIP: return "HIP kernel launch failed";
    }
    return "unknown status";
}

// ------------------------------------------------------------------- amax
size_t puro_amax_workspace_size(int64_t rows, int64_t cols) {
    return amax_ws(rows, cols);
}

puro_status puro_amax(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld, float* amax,
                      void* ws, size_t ws_bytes, hipStream_t stream) {
    puro_status st = check_bf16_matrix(x, rows, cols, ld);
    if (st != PURO_OK) return st;
    if (!amax) return PURO_ERR_NULL;
    const int P = amax_num_partials(rows, cols);
    if (P > 0 && !ws) return PURO_ERR_NULL;
    if (ws_bytes < (size_t)P * sizeof(uint32_t)) return PURO_ERR_WORKSPACE;
    uint32_t* partial = reinterpret_cast<uint32_t*>(ws);
    if (P > 0) launch_amax_partials(x, rows, cols, ld, partial, P, stream);
    launch_amax_finalize(partial, P, amax, stream);
    return launched();
}

// --------------------------------------------------------------- quantise
size_t puro_quantize_workspace_size(int64_t rows, int64_t cols) {
    if (rows < 0 || cols < 0) return 0;
    return quant_tensor_ws_bytes(rows, cols);
}

}  // extern "C"

namespace {

// puro_quantize_fp8 and the fused quantise calls (the mode may carry the
// k-block-major layout flag). The values a quantisation encodes: the BF16 tensor x itself; the SwiGLU
// H = BF16(silu(gate) * up) [rows, cols] of a fused gate/up output x [rows,
// 2 cols]; or the RMSNorm y = BF16(x * rstd * gamma) of x [rows, cols], whose
// per-row rstd is written too.
struct Source {
    enum Kind { kBf16, kSwiglu, kRmsnorm, kSwigluBwd } kind = kBf16;
    const uint16_t* gamma = nullptr;
    float* rstd = nullptr;
    float eps = 0.0f;
    // the SwiGLU backward's saved gate/up output (x is then dH)
    const uint16_t* gu = nullptr;
    int64_t ld_gu = 0;
};

puro_status quantize_impl(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld, puro_fp8_format fmt,
                          puro_scale_mode mode_arg, puro_scale_rounding rnd, const float* amax_in, uint8_t* q,
                          float* scale, uint8_t* qT, float* scaleT, void* ws, size_t ws_bytes,
                          hipStream_t stream, Source src = Source(), bool static_ws = false) {
    // the scale-layout flag of the grouped modes
    const int kmajor = ((int)mode_arg & PURO_SCALE_KMAJOR) != 0;
    const puro_scale_mode mode = (puro_scale_mode)((int)mode_arg & ~(int)PURO_SCALE_KMAJOR);
    if (kmajor && mode == PURO_SCALE_TENSOR) return PURO_ERR_UNSUPPORTED;
    const bool swiglu = src.kind == Source::kSwiglu, rms = src.kind == Source::kRmsnorm;
    const bool bwd = src.kind == Source::kSwigluBwd;
    if (cols < 0) return PURO_ERR_SHAPE;
    // x's columns: 2 cols for the SwiGLU's gate/up input, cols / 2 for the backward's dH
    puro_status st = check_bf16_matrix(x, rows, swiglu ? 2 * cols : (bwd ? cols / 2 : cols), ld);
    if (st != PURO_OK) return st;
    if (bwd) {
        st = check_bf16_matrix(src.gu, rows, cols, src.ld_gu);
        if (st != PURO_OK) return st;
        if (src.ld_gu >= ((int64_t)1 << 23)) return PURO_ERR_SHAPE;
    }
    if ((swiglu || rms || bwd) && (amax_in || mode == PURO_SCALE_BLOCK_128x128)) return PURO_ERR_UNSUPPORTED;
    if (rms) {
        // a row needs its columns (the mean of an empty row is undefined)
        if (rows > 0 && cols == 0) return PURO_ERR_SHAPE;
        if (!(src.eps >= 0.0f) || !(src.eps <= 3.4028235e38f)) return PURO_ERR_UNSUPPORTED;
        if (rows > 0 && (!src.gamma || !src.rstd)) return PURO_ERR_NULL;
        if (rows > 0 && (!aligned16(src.gamma) || (reinterpret_cast<uintptr_t>(src.rstd) & 15) != 0))
            return PURO_ERR_ALIGN;
    }
    if (!fmt_ok(fmt) || (rnd != PURO_SCALE_FP32 && rnd != PURO_SCALE_POW2 && rnd != PURO_SCALE_POW2_FLOOR))
        return PURO_ERR_UNSUPPORTED;
    const bool pow2 = rnd == PURO_SCALE_POW2 || rnd == PURO_SCALE_POW2_FLOOR;
    if ((cols % 16) != 0) return PURO_ERR_ALIGN;
    // a 128-row tile spans less than 2^31 bytes (32-bit buffer offsets)
    if (ld >= ((int64_t)1 << 23)) return PURO_ERR_SHAPE;
    QuantArgs a{};
    a.x = x; a.rows = rows; a.cols = cols; a.ld = ld;
    a.q = q; a.scale = scale; a.qT = qT; a.scaleT = scaleT;
    a.amax = amax_in;
    a.supplied = amax_in != nullptr;
    a.pow2 = rnd == PURO_SCALE_POW2 ? 1 : (rnd == PURO_SCALE_POW2_FLOOR ? 2 : 0);
    a.kmajor = kmajor;
    a.gamma = src.gamma;
    a.rstd = src.rstd;
    a.x2 = src.gu;
    a.ld2 = src.ld_gu;
    // outputs of an empty tensor are never written (torch hands out NULL for them)
    const bool empty = rows == 0 || cols == 0;
    int qmode;
    switch (mode) {
    case PURO_SCALE_TENSOR:
        if (!empty && !q && !qT) return PURO_ERR_NULL;
        if (!scale) return PURO_ERR_NULL;
        if (qT && (rows % 16) != 0) return PURO_ERR_ALIGN;
        qmode = kQTensor;
        break;
    case PURO_SCALE_ROW_1x128:
        if (!empty && (!q || !scale || (qT && !scaleT))) return PURO_ERR_NULL;
        if (!pow2 || amax_in) return PURO_ERR_UNSUPPORTED;
        if ((cols % kGroup) != 0 || (qT && (rows % kGroup) != 0)) return PURO_ERR_ALIGN;
        qmode = kQRow;
        break;
    case PURO_SCALE_COL_128x1:
        if (!empty && (!qT || !scaleT)) return PURO_ERR_NULL;
        if (!pow2 || amax_in) return PURO_ERR_UNSUPPORTED;
        if ((rows % kGroup) != 0) return PURO_ERR_ALIGN;
        a.q = nullptr; a.scale = nullptr;
        qmode = kQCol;
        break;
    case PURO_SCALE_BLOCK_128x128:
        if (!empty && (!q || !scale || (qT && !scaleT))) return PURO_ERR_NULL;
        if (!pow2 || amax_in) return PURO_ERR_UNSUPPORTED;
        if ((rows % kGroup) != 0 || (cols % kGroup) != 0) return PURO_ERR_ALIGN;
        qmode = kQBlock;
        break;
    default:
        return PURO_ERR_UNSUPPORTED;
    }
    if (rms) {
        if (qmode == kQTensor) {
            if (!ws) return PURO_ERR_NULL;
            if (ws_bytes < rmsnorm_ws_bytes(rows)) return PURO_ERR_WORKSPACE;
        } else if (rows == 0) {
            return PURO_OK;
        }
        launch_rmsnorm_quantize(fmt, qmode, a, src.eps, ws, stream);
        return launched();
    }
    if (bwd) {
        if (qmode == kQTensor) {
            if (!ws) return PURO_ERR_NULL;
            if (ws_bytes < swiglu_bwd_ws_bytes(rows, cols)) return PURO_ERR_WORKSPACE;
        } else if (empty) {
            return PURO_OK;
        }
        launch_swiglu_bwd_quantize(fmt, qmode, a, ws, stream);
        return launched();
    }
    if (qmode == kQTensor && !amax_in) {
        if (static_ws) {
            // the library's own scratch (arguments are valid by now)
            if (quant_tensor_ws_bytes(rows, cols) > kStaticScratchBytes) return PURO_ERR_WORKSPACE;
            if (static_scratch(&ws) != hipSuccess) return PURO_ERR_HIP;
            ws_bytes = kStaticScratchBytes;
        }
        if (!ws) return PURO_ERR_NULL;
        if (ws_bytes < quant_tensor_ws_bytes(rows, cols)) return PURO_ERR_WORKSPACE;
        launch_quantize_tensor(fmt, a, ws, stream, swiglu);
        return launched();
    }
    // an empty tensor has no groups
    if ((rows == 0 || cols == 0) && qmode != kQTensor) return PURO_OK;
    launch_quantize(fmt, qmode, a, stream, swiglu);
    return launched();
}

}  // namespace

extern "C" {

puro_status puro_quantize_fp8(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                              puro_fp8_format fmt, puro_scale_mode mode, puro_scale_rounding rnd,
                              const float* amax_in, uint8_t* q, float* scale, uint8_t* qT,
                              float* scaleT, void* ws, size_t ws_bytes, hipStream_t stream) {
    return quantize_impl(x, rows, cols, ld, fmt, mode, rnd, amax_in, q, scale, qT, scaleT, ws, ws_bytes, stream);
}

static_assert(PURO_QUANTIZE_STATIC_SCRATCH_BYTES == kStaticScratchBytes, "scratch size");

puro_status puro_quantize_fp8_static(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                                     puro_fp8_format fmt, puro_scale_mode mode, puro_scale_rounding rnd,
                                     const float* amax_in, uint8_t* q, float* scale, uint8_t* qT, float* scaleT,
                                     hipStream_t stream) {
    return quantize_impl(x, rows, cols, ld, fmt, mode, rnd, amax_in, q, scale, qT, scaleT, nullptr, 0, stream,
                         Source(), true);
}

// ---------------------------------------------------- SwiGLU + quantise
size_t puro_swiglu_quantize_workspace_size(int64_t rows, int64_t cols) {
    if (rows < 0 || cols < 0) return 0;
    return quant_tensor_ws_bytes(rows, cols);
}

puro_status puro_swiglu_quantize_fp8(const uint16_t* gu, int64_t rows, int64_t cols, int64_t ld,
                                     puro_fp8_format fmt, puro_scale_mode mode, puro_scale_rounding rnd,
                                     uint8_t* q, float* scale, uint8_t* qT, float* scaleT, void* ws,
                                     size_t ws_bytes, hipStream_t stream) {
    Source src;
    src.kind = Source::kSwiglu;
    return quantize_impl(gu, rows, cols, ld, fmt, mode, rnd, nullptr, q, scale, qT, scaleT, ws, ws_bytes, stream,
                         src);
}

// ------------------------------------------- SwiGLU backward + quantise
size_t puro_swiglu_bwd_quantize_workspace_size(int64_t rows, int64_t cols) {
    if (rows < 0 || cols < 0) return 0;
    return swiglu_bwd_ws_bytes(rows, 2 * cols);
}

puro_status puro_swiglu_bwd_quantize_fp8(const uint16_t* dh, int64_t ld_dh, const uint16_t* gu, int64_t ld_gu,
                                         int64_t rows, int64_t cols, puro_fp8_format fmt, puro_scale_mode mode,
                                         puro_scale_rounding rnd, uint8_t* q, float* scale, uint8_t* qT,
                                         float* scaleT, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (cols < 0 || cols > ((int64_t)1 << 30)) return PURO_ERR_SHAPE;
    Source src;
    src.kind = Source::kSwigluBwd;
    src.gu = gu;
    src.ld_gu = ld_gu;
    return quantize_impl(dh, rows, 2 * cols, ld_dh, fmt, mode, rnd, nullptr, q, scale, qT, scaleT, ws, ws_bytes,
                         stream, src);
}

// --------------------------------------------------- RMSNorm + quantise
size_t puro_rmsnorm_quantize_workspace_size(int64_t rows, int64_t cols) {
    if (rows < 0 || cols < 0) return 0;
    return rmsnorm_ws_bytes(rows);
}

puro_status puro_rmsnorm_quantize_fp8(const uint16_t* x, const uint16_t* gamma, int64_t rows, int64_t cols,
                                      int64_t ld, float eps, puro_fp8_format fmt, puro_scale_mode mode,
                                      puro_scale_rounding rnd, uint8_t* q, float* scale, uint8_t* qT,
                                      float* scaleT, float* rstd, void* ws, size_t ws_bytes, hipStream_t stream) {
    Source src;
    src.kind = Source::kRmsnorm;
    src.gamma = gamma;
    src.rstd = rstd;
    src.eps = eps;
    return quantize_impl(x, rows, cols, ld, fmt, mode, rnd, nullptr, q, scale, qT, scaleT, ws, ws_bytes, stream,
                         src);
}

// ------------------------------------------------------------------- GEMM
size_t puro_fp8_gemm_workspace_size(int64_t M, int64_t N, int64_t K, puro_out_dtype d_type) {
    if (M <= 0 || N <= 0 || K <= 0) return 0;
    return gemm_workspace_bytes(M, N, K, d_type == PURO_OUT_FP32 ? kOutF32 : kOutBF16);
}

puro_status puro_fp8_gemm_plan(int64_t M, int64_t N, int64_t K, puro_scale_mode a_mode,
                               puro_scale_mode b_mode, int* tile_m, int* tile_n, int* stages, int* splits,
                               int* launches) {
    if (M < 0 || N < 0 || K < 0) return PURO_ERR_SHAPE;
    auto ok = [](puro_scale_mode m) {
        const int g = (int)m & ~(int)PURO_SCALE_KMAJOR;
        return m == PURO_SCALE_TENSOR || g == PURO_SCALE_ROW_1x128 || g == PURO_SCALE_BLOCK_128x128;
    };
    if (!ok(a_mode) || !ok(b_mode)) return PURO_ERR_UNSUPPORTED;
    int tm = 0, tn = 0, ns = 0, s = 1;
    gemm_plan(M, N, K, a_mode != PURO_SCALE_TENSOR || b_mode != PURO_SCALE_TENSOR, &tm, &tn, &ns, &s);
    if (tile_m) *tile_m = tm;
    if (tile_n) *tile_n = tn;
    if (stages) *stages = ns;
    if (splits) *splits = s;
    if (launches) *launches = (M > 0 && N > 0) ? 1 + (s > 1) : 0;
    return PURO_OK;
}

static puro_status check_operand(const puro_fp8_operand* o, int64_t rows, int64_t K, int* smode, int* kmajor) {
    if (!o) return PURO_ERR_NULL;
    // the scale is read whenever the operand has rows (also for K == 0, where
    // the result is a scaled empty sum); the data only when there is a k
    if (rows > 0 && (!o->scale || (K > 0 && !o->data))) return PURO_ERR_NULL;
    if (!fmt_ok(o->fmt)) return PURO_ERR_UNSUPPORTED;
    if (o->ld < K) return PURO_ERR_SHAPE;
    if ((o->ld % 16) != 0 || !aligned16(o->data)) return PURO_ERR_ALIGN;
    // buffer offsets within one tile of 256 rows stay below 2^31
    if (o->ld > kMaxPitch) return PURO_ERR_SHAPE;
    *kmajor = ((int)o->mode & PURO_SCALE_KMAJOR) != 0;
    switch ((int)o->mode & ~(int)PURO_SCALE_KMAJOR) {
    case PURO_SCALE_TENSOR:
        if (*kmajor) return PURO_ERR_UNSUPPORTED;
        *smode = kSTensor;
        break;
    case PURO_SCALE_ROW_1x128: *smode = kSRow; break;
    case PURO_SCALE_BLOCK_128x128: *smode = kSBlock; break;
    default: return PURO_ERR_UNSUPPORTED;
    }
    if (*smode != kSTensor && (K % kGroup) != 0) return PURO_ERR_ALIGN;
    return PURO_OK;
}

}  // extern "C"

namespace {

// puro_fp8_gemm with a choice of grouped-scale layout per operand.
// bias / residual: the BF16 epilogue (both NULL: none).
puro_status gemm_impl(int64_t M, int64_t N, int64_t K, const puro_fp8_operand* A, const puro_fp8_operand* B,
                      void* D, puro_out_dtype d_type, int64_t ldd, int accumulate, void* ws, size_t ws_bytes,
                      hipStream_t stream, const uint16_t* bias = nullptr, const uint16_t* residual = nullptr,
                      int64_t ldr = 0) {
    if (M < 0 || N < 0 || K < 0) return PURO_ERR_SHAPE;
    if (M > INT32_MAX / 2 || N > INT32_MAX / 2 || K > INT32_MAX / 2) return PURO_ERR_SHAPE;
    int sa = 0, sb = 0, a_kmajor = 0, b_kmajor = 0;
    puro_status st = check_operand(A, M, K, &sa, &a_kmajor);
    if (st != PURO_OK) return st;
    st = check_operand(B, N, K, &sb, &b_kmajor);
    if (st != PURO_OK) return st;
    if (d_type != PURO_OUT_BF16 && d_type != PURO_OUT_FP32) return PURO_ERR_UNSUPPORTED;
    if ((K % 16) != 0) return PURO_ERR_ALIGN;
    if (ldd < N) return PURO_ERR_SHAPE;
    if (M == 0 || N == 0) return PURO_OK;
    if (!D) return PURO_ERR_NULL;
    if ((ldd % 4) != 0 || !aligned16(D)) return PURO_ERR_ALIGN;
    const bool epi = bias || residual;
    if (epi) {
        if (d_type != PURO_OUT_BF16 || accumulate) return PURO_ERR_UNSUPPORTED;
        if (bias && !aligned16(bias)) return PURO_ERR_ALIGN;
        // ldr as the operands' pitch: buffer offsets over a tile's rows stay below 2^31
        if (residual && (ldr < N || ldr > kMaxPitch)) return PURO_ERR_SHAPE;
        if (residual && (!aligned16(residual) || (ldr % 4) != 0)) return PURO_ERR_ALIGN;
        // the residual may be D itself (an in-place residual add), but not overlap it otherwise
        if (residual && residual != D) {
            const uintptr_t r0 = (uintptr_t)residual, r1 = r0 + (uintptr_t)(((M - 1) * ldr + N) * 2);
            const uintptr_t d0 = (uintptr_t)D, d1 = d0 + (uintptr_t)(((M - 1) * ldd + N) * 2);
            if (r0 < d1 && d0 < r1) return PURO_ERR_SHAPE;
        }
        if (residual == D && ldr != ldd) return PURO_ERR_SHAPE;
    }
    const int out = d_type == PURO_OUT_FP32 ? kOutF32 : (epi ? kOutBF16Epi : kOutBF16);
    const size_t need = gemm_workspace_bytes(M, N, K, out);
    if (need > 0 && !ws) return PURO_ERR_NULL;
    if (ws_bytes < need) return PURO_ERR_WORKSPACE;
    GemmProblem g{};
    g.M = M; g.N = N; g.K = K;
    g.A = A->data; g.lda = A->ld; g.fa = A->fmt; g.sa_mode = sa; g.sa = A->scale;
    g.B = B->data; g.ldb = B->ld; g.fb = B->fmt; g.sb_mode = sb; g.sb = B->scale;
    g.D = D; g.ldd = ldd; g.out = out; g.accumulate = accumulate != 0;
    g.sa_kmajor = a_kmajor; g.sb_kmajor = b_kmajor;
    g.bias = bias; g.residual = residual; g.ldr = ldr;
    // a linear layer's outputs (Y, dX, dW) are far larger than the L2 and
    // are next read by another kernel: stream them past the caches
    g.nt_out = 1;
    launch_gemm(g, ws, stream);
    return launched();
}

}  // namespace

extern "C" {

puro_status puro_fp8_gemm(int64_t M, int64_t N, int64_t K, const puro_fp8_operand* A,
                          const puro_fp8_operand* B, void* D, puro_out_dtype d_type, int64_t ldd,
                          int accumulate, void* ws, size_t ws_bytes, hipStream_t stream) {
    return gemm_impl(M, N, K, A, B, D, d_type, ldd, accumulate, ws, ws_bytes, stream);
}

puro_status puro_fp8_gemm_epilogue(int64_t M, int64_t N, int64_t K, const puro_fp8_operand* A,
                                   const puro_fp8_operand* B, uint16_t* D, int64_t ldd, const uint16_t* bias,
                                   const uint16_t* residual, int64_t ldr, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
    return gemm_impl(M, N, K, A, B, D, PURO_OUT_BF16, ldd, 0, ws, ws_bytes, stream, bias, residual, ldr);
}

// ----------------------------------------------------------- linear layer
namespace {

// The linear layer keeps its grouped scales k-block-major: the GEMMs load a
// k slice's scales as contiguous runs.
constexpr puro_scale_mode kRowKM = (puro_scale_mode)(PURO_SCALE_ROW_1x128 | PURO_SCALE_KMAJOR);
constexpr puro_scale_mode kBlockKM = (puro_scale_mode)(PURO_SCALE_BLOCK_128x128 | PURO_SCALE_KMAJOR);

// The power-of-two rule of a blockwise recipe.
puro_scale_rounding block_rule(const puro_linear_recipe* r) {
    return r->rnd == PURO_SCALE_POW2_FLOOR ? PURO_SCALE_POW2_FLOOR : PURO_SCALE_POW2;
}

bool recipe_ok(const puro_linear_recipe* r) {
    return r && fmt_ok(r->x_fmt) && fmt_ok(r->w_fmt) && fmt_ok(r->dy_fmt) &&
           (r->blockwise == 0 || r->blockwise == 1) &&
           (r->rnd == PURO_SCALE_FP32 || r->rnd == PURO_SCALE_POW2 || r->rnd == PURO_SCALE_POW2_FLOOR);
}

puro_status check_linear_dims(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* r) {
    if (!recipe_ok(r)) return PURO_ERR_UNSUPPORTED;
    if (M < 0 || N < 0 || K < 0) return PURO_ERR_SHAPE;
    // each of M, N and K is the row pitch of an FP8 operand of one of the
    // three GEMMs (Xq, dYq, the transposed copies), limited to 2^22 bytes;
    // rejected here, before the quantisers write anything
    if (M > kMaxPitch || N > kMaxPitch || K > kMaxPitch) return PURO_ERR_SHAPE;
    const int64_t g = r->blockwise ? kGroup : 16;
    if ((M % g) != 0 || (N % g) != 0 || (K % g) != 0) return PURO_ERR_ALIGN;
    return PURO_OK;
}

struct FwdLayout {
    size_t xq, wq, xs_row, w_blk, part_x, part_w, gemm, total;
};

FwdLayout fwd_layout(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* r) {
    Carver c;
    FwdLayout l{};
    l.xq = c.take((size_t)M * K);
    l.wq = c.take((size_t)N * K);
    if (r->blockwise) {
        l.xs_row = c.take((size_t)M * (K / kGroup) * sizeof(float));
        l.w_blk = c.take((size_t)(N / kGroup) * (K / kGroup) * sizeof(float));
    } else {
        l.part_x = c.take(quant_tensor_ws_bytes(M, K));
        l.part_w = c.take(quant_tensor_ws_bytes(N, K));
    }
    l.gemm = c.take(gemm_workspace_bytes(M, N, K, kOutBF16));
    l.total = c.used;
    return l;
}

struct BwdLayout {
    size_t dyq, dyq_t, dy_scale, dy_scale_t, part, gemm, total;
};

BwdLayout bwd_layout(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* r) {
    Carver c;
    BwdLayout l{};
    l.dyq = c.take((size_t)M * N);
    l.dyq_t = c.take((size_t)N * M);
    if (r->blockwise) {
        l.dy_scale = c.take((size_t)M * (N / kGroup) * sizeof(float));
        l.dy_scale_t = c.take((size_t)N * (M / kGroup) * sizeof(float));
    } else {
        l.dy_scale = c.take(sizeof(float));
        l.part = c.take(quant_tensor_ws_bytes(M, N));
    }
    const size_t g1 = gemm_workspace_bytes(M, K, N, kOutBF16);
    const size_t g2 = gemm_workspace_bytes(N, K, M, kOutF32);
    l.gemm = c.take(g1 > g2 ? g1 : g2);
    l.total = c.used;
    return l;
}

}  // namespace

size_t puro_linear_saved_bytes(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* r,
                               size_t sizes[4]) {
    size_t s[4] = {0, 0, 0, 0};
    if (recipe_ok(r) && M >= 0 && N >= 0 && K >= 0) {
        s[0] = (size_t)K * M;
        s[1] = r->blockwise ? (size_t)K * (M / kGroup) * sizeof(float) : sizeof(float);
        s[2] = (size_t)K * N;
        s[3] = r->blockwise ? (size_t)(K / kGroup) * (N / kGroup) * sizeof(float) : sizeof(float);
    }
    if (sizes)
        for (int i = 0; i < 4; ++i) sizes[i] = s[i];
    return s[0] + s[1] + s[2] + s[3];
}

size_t puro_linear_fwd_workspace_size(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* r) {
    if (check_linear_dims(M, N, K, r) != PURO_OK) return 0;
    return fwd_layout(M, N, K, r).total;
}

size_t puro_linear_bwd_workspace_size(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* r) {
    if (check_linear_dims(M, N, K, r) != PURO_OK) return 0;
    return bwd_layout(M, N, K, r).total;
}

puro_status puro_linear_fwd(const uint16_t* X, const uint16_t* W, int64_t M, int64_t N, int64_t K,
                            const puro_linear_recipe* r, uint16_t* Y, const puro_linear_saved* saved,
                            void* ws, size_t ws_bytes, hipStream_t stream) {
    puro_status st = check_linear_dims(M, N, K, r);
    if (st != PURO_OK) return st;
    if (!saved || !X || !W || !Y || !saved->xq_t || !saved->x_scale || !saved->wq_t || !saved->w_scale)
        return PURO_ERR_NULL;
    if (!aligned16(X) || !aligned16(W) || !aligned16(Y) || !aligned16(saved->xq_t) ||
        !aligned16(saved->wq_t))
        return PURO_ERR_ALIGN;
    const FwdLayout l = fwd_layout(M, N, K, r);
    if (!ws) return PURO_ERR_NULL;
    if (ws_bytes < l.total) return PURO_ERR_WORKSPACE;
    uint8_t* w8 = reinterpret_cast<uint8_t*>(ws);
    uint8_t* xq = w8 + l.xq;
    uint8_t* wq = w8 + l.wq;
    puro_fp8_operand A{}, B{};
    if (!r->blockwise) {
        // X and W with their own amax each: q (Fprop) and qT (kept for Wgrad
        // and Dgrad), in one amax launch and one quantise launch for both
        QuantArgs ax{}, aw{};
        ax.x = X; ax.rows = M; ax.cols = K; ax.ld = K;
        ax.q = xq; ax.scale = saved->x_scale; ax.qT = saved->xq_t;
        ax.pow2 = r->rnd == PURO_SCALE_POW2 ? 1 : (r->rnd == PURO_SCALE_POW2_FLOOR ? 2 : 0);
        aw = ax;
        aw.x = W; aw.rows = N;
        aw.q = wq; aw.scale = saved->w_scale; aw.qT = saved->wq_t;
        if (r->x_fmt == r->w_fmt) {
            launch_quantize_tensor_pair(r->x_fmt, ax, w8 + l.part_x, aw, w8 + l.part_w, stream);
        } else {
            launch_quantize_tensor(r->x_fmt, ax, w8 + l.part_x, stream);
            launch_quantize_tensor(r->w_fmt, aw, w8 + l.part_w, stream);
        }
        if ((st = launched()) != PURO_OK) return st;
        A = puro_fp8_operand{xq, K, r->x_fmt, PURO_SCALE_TENSOR, saved->x_scale};
        B = puro_fp8_operand{wq, K, r->w_fmt, PURO_SCALE_TENSOR, saved->w_scale};
    } else {
        // X: 1x128 row groups for Fprop and, from the same read, the 128x1
        // column-grouped transposed copy kept for Wgrad.
        float* xs_row = reinterpret_cast<float*>(w8 + l.xs_row);
        float* w_blk = reinterpret_cast<float*>(w8 + l.w_blk);
        st = quantize_impl(X, M, K, K, r->x_fmt, kRowKM, block_rule(r), nullptr, xq, xs_row, saved->xq_t,
                           saved->x_scale, nullptr, 0, stream);
        if (st != PURO_OK) return st;
        // W: 128x128 blocks, plus the transposed copy (same blocks) kept for Dgrad.
        st = quantize_impl(W, N, K, K, r->w_fmt, kBlockKM, block_rule(r), nullptr, wq, w_blk, saved->wq_t,
                           saved->w_scale, nullptr, 0, stream);
        if (st != PURO_OK) return st;
        A = puro_fp8_operand{xq, K, r->x_fmt, kRowKM, xs_row};
        B = puro_fp8_operand{wq, K, r->w_fmt, kBlockKM, w_blk};
    }
    return gemm_impl(M, N, K, &A, &B, Y, PURO_OUT_BF16, N, 0, w8 + l.gemm, ws_bytes - l.gemm, stream);
}

puro_status puro_linear_bwd(const uint16_t* dY, const puro_linear_saved* saved, int64_t M, int64_t N,
                            int64_t K, const puro_linear_recipe* r, uint16_t* dX, float* dW,
                            int accumulate_dW, void* ws, size_t ws_bytes, hipStream_t stream) {
    puro_status st = check_linear_dims(M, N, K, r);
    if (st != PURO_OK) return st;
    if (!saved || !dY || !saved->xq_t || !saved->x_scale || !saved->wq_t || !saved->w_scale)
        return PURO_ERR_NULL;
    if (!aligned16(dY) || !aligned16(saved->xq_t) || !aligned16(saved->wq_t) || (dX && !aligned16(dX)) ||
        (dW && !aligned16(dW)))
        return PURO_ERR_ALIGN;
    if (!dX && !dW) return PURO_OK;
    const BwdLayout l = bwd_layout(M, N, K, r);
    if (!ws) return PURO_ERR_NULL;
    if (ws_bytes < l.total) return PURO_ERR_WORKSPACE;
    uint8_t* w8 = reinterpret_cast<uint8_t*>(ws);
    uint8_t* dyq = w8 + l.dyq;
    uint8_t* dyq_t = w8 + l.dyq_t;
    float* dys = reinterpret_cast<float*>(w8 + l.dy_scale);
    float* dys_t = reinterpret_cast<float*>(w8 + l.dy_scale_t);
    void* gws = w8 + l.gemm;
    const size_t gws_bytes = ws_bytes - l.gemm;
    puro_fp8_operand dA{}, dB{}, wA{}, wB{};
    if (!r->blockwise) {
        st = puro_quantize_fp8(dY, M, N, N, r->dy_fmt, PURO_SCALE_TENSOR, r->rnd, nullptr, dyq, dys, dyq_t,
                               nullptr, w8 + l.part, quant_tensor_ws_bytes(M, N), stream);
        if (st != PURO_OK) return st;
        dA = puro_fp8_operand{dyq, N, r->dy_fmt, PURO_SCALE_TENSOR, dys};
        dB = puro_fp8_operand{saved->wq_t, N, r->w_fmt, PURO_SCALE_TENSOR, saved->w_scale};
        wA = puro_fp8_operand{dyq_t, M, r->dy_fmt, PURO_SCALE_TENSOR, dys};
        wB = puro_fp8_operand{saved->xq_t, M, r->x_fmt, PURO_SCALE_TENSOR, saved->x_scale};
    } else {
        st = quantize_impl(dY, M, N, N, r->dy_fmt, kRowKM, block_rule(r), nullptr, dyq, dys, dyq_t, dys_t, nullptr,
                           0, stream);
        if (st != PURO_OK) return st;
        dA = puro_fp8_operand{dyq, N, r->dy_fmt, kRowKM, dys};
        dB = puro_fp8_operand{saved->wq_t, N, r->w_fmt, kBlockKM, saved->w_scale};
        wA = puro_fp8_operand{dyq_t, M, r->dy_fmt, kRowKM, dys_t};
        wB = puro_fp8_operand{saved->xq_t, M, r->x_fmt, kRowKM, saved->x_scale};
    }
    if (dX) {
        st = gemm_impl(M, K, N, &dA, &dB, dX, PURO_OUT_BF16, K, 0, gws, gws_bytes, stream);
        if (st != PURO_OK) return st;
    }
    if (dW) {
        st = gemm_impl(N, K, M, &wA, &wB, dW, PURO_OUT_FP32, K, accumulate_dW, gws, gws_bytes, stream);
        if (st != PURO_OK) return st;
    }
    return PURO_OK;
}

}  // extern "C"

// ------------------------------------------ LM head with cross-entropy loss
namespace {

puro_status check_lm_head(const uint16_t* X, const uint16_t* W, const int32_t* targets, int64_t M, int64_t V,
                          int64_t K, puro_lm_head_recipe r) {
    if (r != PURO_LM_HEAD_BF16 && r != PURO_LM_HEAD_FP8) return PURO_ERR_UNSUPPORTED;
    if (M <= 0 || V <= 0 || K <= 0) return PURO_ERR_SHAPE;
    // BF16 operand pitches (2 M, 2 V, 2 K bytes for the transposed copies) within 2^22
    const int64_t lim = (int64_t)1 << 21;
    if (M > lim || V > lim || K > lim) return PURO_ERR_SHAPE;
    if ((M % kGroup) != 0 || (V % kGroup) != 0 || (K % kGroup) != 0) return PURO_ERR_ALIGN;
    if (!X || !W || !targets) return PURO_ERR_NULL;
    if (!aligned16(X) || !aligned16(W) || ((uintptr_t)targets & 3) != 0) return PURO_ERR_ALIGN;
    return PURO_OK;
}

}  // namespace

extern "C" {

size_t puro_lm_head_ce_workspace_size(int64_t M, int64_t V, int64_t K, puro_lm_head_recipe recipe, int backward) {
    if (check_lm_head(reinterpret_cast<const uint16_t*>(16), reinterpret_cast<const uint16_t*>(16),
                      reinterpret_cast<const int32_t*>(16), M, V, K, recipe) != PURO_OK)
        return 0;
    return lm_head_ws_bytes(M, V, K, recipe == PURO_LM_HEAD_FP8, backward != 0);
}

puro_status puro_lm_head_ce_fwd(const uint16_t* X, const uint16_t* W, const int32_t* targets, int64_t M,
                                int64_t V, int64_t K, puro_lm_head_recipe recipe, float* lse, float* loss,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
    puro_status st = check_lm_head(X, W, targets, M, V, K, recipe);
    if (st != PURO_OK) return st;
    if (!lse || !loss || !ws) return PURO_ERR_NULL;
    if (!aligned16(lse) || !aligned16(loss)) return PURO_ERR_ALIGN;
    if (ws_bytes < lm_head_ws_bytes(M, V, K, recipe == PURO_LM_HEAD_FP8, false)) return PURO_ERR_WORKSPACE;
    launch_lm_head_fwd(X, W, targets, M, V, K, recipe == PURO_LM_HEAD_FP8, lse, loss, ws, stream);
    return launched();
}

puro_status puro_lm_head_ce_bwd(const uint16_t* X, const uint16_t* W, const int32_t* targets, const float* lse,
                                int64_t M, int64_t V, int64_t K, puro_lm_head_recipe recipe, float grad_scale,
                                uint16_t* dX, float* dW, void* ws, size_t ws_bytes, hipStream_t stream) {
    puro_status st = check_lm_head(X, W, targets, M, V, K, recipe);
    if (st != PURO_OK) return st;
    if (!lse || !dX || !dW || !ws) return PURO_ERR_NULL;
    if (!aligned16(lse) || !aligned16(dX) || !aligned16(dW)) return PURO_ERR_ALIGN;
    if (!(grad_scale == grad_scale) || grad_scale > 3.4028235e38f || grad_scale < -3.4028235e38f)
        return PURO_ERR_UNSUPPORTED;
    if (ws_bytes < lm_head_ws_bytes(M, V, K, recipe == PURO_LM_HEAD_FP8, true)) return PURO_ERR_WORKSPACE;
    launch_lm_head_bwd(X, W, targets, lse, M, V, K, recipe == PURO_LM_HEAD_FP8, grad_scale, dX, dW, ws, stream);
    return launched();
}

}  // extern "C"

// ------------------------------------------------------------------- MuonH
namespace {

puro_status check_muonh_shape(int64_t count, int64_t rows, int64_t cols) {
    if (count <= 0 || rows <= 0 || cols <= 0) return PURO_ERR_SHAPE;
    const int64_t lim = (int64_t)1 << 21;
    if (count > 65535 || rows > lim || cols > lim) return PURO_ERR_SHAPE;
    if ((rows % kGroup) != 0 || (cols % kGroup) != 0) return PURO_ERR_ALIGN;
    return PURO_OK;
}

bool finite_f32(float v) { return v == v && v <= 3.4028235e38f && v >= -3.4028235e38f; }

}  // namespace

extern "C" {

size_t puro_muonh_workspace_size(int64_t count, int64_t rows, int64_t cols) {
    if (check_muonh_shape(count, rows, cols) != PURO_OK) return 0;
    return muonh_ws_bytes(count, rows, cols);
}

puro_status puro_muonh_step(int64_t count, int64_t rows, int64_t cols, float* W, uint16_t* w_bf16, const float* G,
                            float* buf, const float* radius, float mu, int nesterov, float eta, int ns_steps,
                            uint16_t* u_out, void* ws, size_t ws_bytes, hipStream_t stream) {
    puro_status st = check_muonh_shape(count, rows, cols);
    if (st != PURO_OK) return st;
    if (!W || !G || !buf || !radius || !ws) return PURO_ERR_NULL;
    if (!aligned16(W) || !aligned16(G) || !aligned16(buf) || ((uintptr_t)radius & 3) != 0 ||
        (w_bf16 && !aligned16(w_bf16)) || (u_out && !aligned16(u_out)))
        return PURO_ERR_ALIGN;
    if (!finite_f32(mu) || !finite_f32(eta) || ns_steps < 0 || ns_steps > 64) return PURO_ERR_UNSUPPORTED;
    if (ws_bytes < muonh_ws_bytes(count, rows, cols)) return PURO_ERR_WORKSPACE;
    launch_muonh_step(count, rows, cols, W, w_bf16, G, buf, radius, mu, nesterov != 0, eta, ns_steps, u_out, ws,
                      stream);
    return launched();
}

size_t puro_newton_schulz_workspace_size(int64_t count, int64_t r, int64_t c) {
    if (check_muonh_shape(count, r, c) != PURO_OK || r > c) return 0;
    return newton_schulz_ws_bytes(count, r, c);
}

puro_status puro_newton_schulz_bf16(int64_t count, int64_t r, int64_t c, const uint16_t* X, int steps,
                                    uint16_t* out, void* ws, size_t ws_bytes, hipStream_t stream) {
    puro_status st = check_muonh_shape(count, r, c);
    if (st != PURO_OK) return st;
    if (r > c) return PURO_ERR_SHAPE;
    if (!X || !out || !ws) return PURO_ERR_NULL;
    if (!aligned16(X) || !aligned16(out)) return PURO_ERR_ALIGN;
    if (steps < 0 || steps > 64) return PURO_ERR_UNSUPPORTED;
    if (ws_bytes < newton_schulz_ws_bytes(count, r, c)) return PURO_ERR_WORKSPACE;
    launch_newton_schulz(X, count, r, c, steps, out, ws, stream);
    return launched();
}

}  // extern "C"
