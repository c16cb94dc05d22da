// Host-side launchers of the HIP kernels (internal to libpuro).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace puro {

// ---- amax / quantisation (quant.hip) ----------------------------------------

// One tensor of an amax pass: P blocks over its rows write partial[0..P).
struct AmaxJob {
    const uint16_t* x;
    int64_t rows, ld;
    uint32_t* partial;
    uint32_t cpr;    // 8-value chunks per row
    int P;
};

// Number of per-block partial maxima the amax pass writes for a tensor.
int amax_num_partials(int64_t rows, int64_t cols);

// Per-block maxima of the BF16 magnitude patterns of x into partial[0..P);
// swiglu: of H = BF16(silu(gate) * up) where x is [rows, 2 cols] (gate =
// columns [0, cols), up = columns [cols, 2 cols)).
void launch_amax_partials(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                          uint32_t* partial, int P, hipStream_t stream, bool swiglu = false);
// amax = max of partial[0..P) as a float (0 when P == 0).
void launch_amax_finalize(const uint32_t* partial, int P, float* amax, hipStream_t stream);

enum QuantMode : int { kQTensor = 0, kQRow = 1, kQCol = 2, kQBlock = 3 };

struct QuantArgs {
    const uint16_t* x;
    int64_t rows, cols, ld;
    uint8_t* q;
    float* scale;
    uint8_t* qT;
    float* scaleT;
    // per-tensor mode: the amax as a device scalar, or (amax NULL) the
    // partial maxima to reduce; supplied: the caller gave the amax (values
    // beyond it saturate) rather than it being computed from x
    const float* amax;
    const uint32_t* partial;
    int npartial;
    int supplied;
    int pow2;
    // grouped modes: scale arrays k-block-major (the group index along the
    // quantised copy's columns outermost) instead of row-major
    int kmajor;
    // RMSNorm source: the per-row reciprocal RMS (written by the row pass)
    // and the norm's weight, BF16 [cols]
    const float* rstd;
    const uint16_t* gamma;
    // SwiGLU backward source: the saved gate/up output [rows, cols] (x is
    // then dH [rows, cols / 2]) and its row pitch
    const uint16_t* x2;
    int64_t ld2;
};

// Workspace of a per-tensor quantisation that computes its own amax.
size_t quant_tensor_ws_bytes(int64_t rows, int64_t cols);

// Size of the library's own per-GPU scratch array (quant.hip), and its
// device address on the current device (looked up once per device).
constexpr size_t kStaticScratchBytes = 32768;
hipError_t static_scratch(void** ptr);
// Per-tensor quantisation with the tensor's own amax: the partial maxima
// pass, then the quantise pass (which reduces them, or reads the amax a
// one-block reduction wrote). ws holds quant_tensor_ws_bytes.
// swiglu: the values are H = BF16(silu(gate) * up) of a.x [rows, 2 cols].
void launch_quantize_tensor(int fmt, QuantArgs a, void* ws, hipStream_t stream, bool swiglu = false);
// The same for two tensors of one format, with one amax launch and one
// quantise launch for both (each tensor with its own workspace).
void launch_quantize_tensor_pair(int fmt, QuantArgs a0, void* ws0, QuantArgs a1, void* ws1,
                                 hipStream_t stream);
// Grouped modes, or per-tensor with a.amax set; swiglu as above (not in
// 128x128 block mode).
void launch_quantize(int fmt, int mode, const QuantArgs& a, hipStream_t stream, bool swiglu = false);

// RMSNorm + quantise: y = BF16(x * rstd * gamma) per row of a.x [rows, cols]
// (rstd = 1 / sqrt(mean(x^2) + eps), written to a.rstd), quantised like a
// BF16 tensor holding y in `mode` (kQTensor, kQRow or kQCol). ws holds
// rmsnorm_ws_bytes(rows) bytes (the per-tensor partial maxima).
size_t rmsnorm_ws_bytes(int64_t rows);
void launch_rmsnorm_quantize(int fmt, int mode, QuantArgs a, float eps, void* ws, hipStream_t stream);

// SwiGLU backward + quantise: the gate/up output's gradient [dg | du]
// [rows, cols] (dg = dH u silu'(g), du = dH silu(g), BF16) from a.x = dH
// [rows, cols / 2] and a.x2 = the gate/up output [rows, cols], quantised in
// `mode` (kQTensor, kQRow or kQCol). ws holds swiglu_bwd_ws_bytes bytes.
size_t swiglu_bwd_ws_bytes(int64_t rows, int64_t cols);
void launch_swiglu_bwd_quantize(int fmt, int mode, QuantArgs a, void* ws, hipStream_t stream);

// ---- GEMM (gemm.hip) ----------------------------------------------------------

// kSNone: an operand without scales (BF16 operands).
enum ScaleMode : int { kSTensor = 0, kSRow = 1, kSBlock = 2, kSNone = 3 };
// kOutBF16Epi: BF16 output with the bias / residual epilogue (the partial
// sums of a split-K plan are kind 2, internal to the GEMM). The LM-head
// kinds replace the output store: kOutLseStats writes per row and 128-column
// block (max, sum of exp(z - max)) and the target's logit; kOutSoftmaxGrad
// writes BF16 dz = g (exp(z - lse) - [column == target]); kOutSoftmaxGradQ
// writes that dz's E4M3 copies instead, in 1x128 row groups and (transposed)
// 128x1 column groups with power-of-two scales, as the quantiser makes them
// from the BF16 dz (E4M3 block-scaled operands). Both dz kinds need M and N
// to be multiples of 128.
enum OutKind : int { kOutBF16 = 0, kOutF32 = 1, kOutBF16Epi = 3, kOutLseStats = 4, kOutSoftmaxGrad = 5,
                     kOutSoftmaxGradQ = 6 };

// K, lda and ldb count operand elements (FP8 codes, or BF16 values when fa
// and fb are kBF16, with scale modes kSNone).
struct GemmProblem {
    int64_t M, N, K;
    const uint8_t* A;
    int64_t lda;
    int fa, sa_mode;
    const float* sa;
    const uint8_t* B;
    int64_t ldb;
    int fb, sb_mode;
    const float* sb;
    void* D;
    int64_t ldd;
    int out;
    int accumulate;
    // grouped scales stored k-block-major ([K/128][rows] or [K/128][rows/128])
    // instead of row-major ([rows][K/128] or [rows/128][K/128])
    int sa_kmajor, sb_kmajor;
    // kOutBF16Epi: D = BF16(alpha * acc + bias[n] + res_scale * residual[m, n]),
    // either term optional (NULL); residual row pitch ldr (residual may be D
    // itself). alpha multiplies the sums of every output kind (with the
    // per-tensor scales).
    const uint16_t* bias;
    const uint16_t* residual;
    int64_t ldr;
    float alpha = 1.0f, res_scale = 1.0f;
    // a symmetric product (M == N, D = D^T): compute only the tiles on or
    // above the diagonal (square tiles); the tiles below are left unwritten
    // (gemm_tile returns the tile edge for filling them in)
    int upper = 0;
    // D is not read back soon: interior tiles store it with non-temporal
    // (streaming) stores, which shorten the output-heavy epilogues
    int nt_out = 0;
    // `batch` independent problems of the same shape and scales: operand,
    // output and residual b start bsa, bsb, bsd, bsr elements after those of
    // problem 0
    int batch = 1;
    int64_t bsa = 0, bsb = 0, bsd = 0, bsr = 0;
    // LM-head output kinds: the target vocabulary id of each row, the
    // vocabulary column of this GEMM's column 0, and stats [M][stats_ld]
    // with zt [M] (kOutLseStats) or lse [M] with the gradient scale
    // (kOutSoftmaxGrad)
    const int32_t* targets;
    int col0;
    float2* stats;
    int64_t stats_ld;
    float* zt;
    const float* lse;
    float grad_scale;
    // kOutSoftmaxGradQ: dz's row-grouped codes [M, N] (ld N) with scales
    // [N / 128][M], and its transposed column-grouped codes [N, M] (ld M)
    // with scales [M / 128][N] (scale arrays k-block-major)
    uint8_t* q8 = nullptr;
    float* q8_scale = nullptr;
    uint8_t* q8t = nullptr;
    float* q8t_scale = nullptr;
};

// Workspace the GEMM needs for split-K partial sums (0 when it runs unsplit);
// K in bytes of an operand row (2 K for BF16 operands).
size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int out, int batch = 1);
// The plan launch_gemm takes: tile, ring depth, k ranges.
void gemm_plan(int64_t M, int64_t N, int64_t K, bool grouped, int* tile_m, int* tile_n, int* stages,
               int* splits);
// Enqueue the GEMM; `ws` must hold gemm_workspace_bytes(...) bytes.
void launch_gemm(const GemmProblem& p, void* ws, hipStream_t stream);
// The output tile edge (rows) of the plan launch_gemm takes for `p`.
int gemm_tile(const GemmProblem& p);

// ---- BF16 transpose (transpose.hip) -------------------------------------------

// dst [C, R] (pitch ldd) = src [R, C] (pitch lds), for `batch` problems whose
// source and destination start bs_src and bs_dst elements after the previous
// one's. R, C, the pitches and the strides are multiples of 8, the pointers
// 16-byte aligned (every caller's shapes are multiples of 128).
void transpose_bf16(const uint16_t* src, int64_t R, int64_t C, int64_t lds, uint16_t* dst, int64_t ldd,
                    hipStream_t stream, int batch = 1, int64_t bs_src = 0, int64_t bs_dst = 0);
// The lower triangle of tiles of a symmetric A [R, R] (pitch ld, R a
// multiple of 64 and of tg) from the upper one: element (i, j) = (j, i)
// wherever i / tg > j / tg; `batch` matrices bs elements apart.
void mirror_lower_bf16(uint16_t* A, int64_t R, int64_t ld, int tg, hipStream_t stream, int batch, int64_t bs);

// ---- LM head with cross-entropy (lm_head.hip) ---------------------------------

// Vocabulary columns per chunk of the backward pass: a chunk's dz copies
// (2 bytes per logit under FP8, at M 8192 128 MB) then stay within the 256 MB
// last-level cache between the epilogue that writes them and the dX and dW
// GEMMs that read them.
constexpr int64_t kLmChunk = 8192;
int64_t lm_head_chunk(int64_t V);
// Workspace of the forward (bwd false) or backward pass; fp8: the blockwise
// FP8 recipe, else BF16 operands. M, V, K multiples of 128.
size_t lm_head_ws_bytes(int64_t M, int64_t V, int64_t K, int fp8, bool bwd);
// lse [M] and loss [M] = lse - z_target from X [M, K], W [V, K] (BF16, dense
// rows) and targets [M].
void launch_lm_head_fwd(const uint16_t* X, const uint16_t* W, const int32_t* targets, int64_t M, int64_t V,
                        int64_t K, int fp8, float* lse, float* loss, void* ws, hipStream_t stream);
// dX [M, K] (BF16) and dW [V, K] (FP32) of grad_scale * loss, from lse.
void launch_lm_head_bwd(const uint16_t* X, const uint16_t* W, const int32_t* targets, const float* lse, int64_t M,
                        int64_t V, int64_t K, int fp8, float grad_scale, uint16_t* dX, float* dW, void* ws,
                        hipStream_t stream);

// ---- MuonH (muonh.hip) ---------------------------------------------------------

// Workspace of one MuonH step of `count` [rows, cols] matrices (rows and cols
// multiples of 128), and of Newton-Schulz on count [r, c] BF16 matrices (r <= c).
size_t muonh_ws_bytes(int64_t count, int64_t rows, int64_t cols);
size_t newton_schulz_ws_bytes(int64_t count, int64_t r, int64_t c);
// out = NS^steps(X), X and out [count][r][c] BF16 (X already normalised).
void launch_newton_schulz(const uint16_t* X, int64_t count, int64_t r, int64_t c, int steps, uint16_t* out,
                          void* ws, hipStream_t stream);
// One MuonH step: buf (FP32) takes the momentum update from G (FP32), W
// (FP32) the hyperball update of radius[b] with the Newton-Schulz direction;
// optional BF16 copies of W' (w_bf16) and of the direction (u_out).
void launch_muonh_step(int64_t count, int64_t rows, int64_t cols, float* W, uint16_t* w_bf16, const float* G,
                       float* buf, const float* radius, float mu, int nesterov, float eta, int steps,
                       uint16_t* u_out, void* ws, hipStream_t stream);

}  // namespace puro
