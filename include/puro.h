/*
 * puro.h -- C ABI of the MI355X (gfx950) FP8 linear-layer library (libpuro.so).
 *
 * The operations are those of an FP8 linear layer as the paper states it
 * (Section 3.2, "FP8 Mixed-Precision Training"; Appendix C, "FP8
 * implementation pipeline" and the precision-flow figure): BF16 inputs and
 * weights are quantised to FP8 immediately before each GEMM, with scales
 * computed online from the data; Fprop (Y = X W^T), Dgrad (dX = dY W) and
 * Wgrad (dW = dY^T X) run on FP8 operands; Y and dX are written in BF16 and
 * dW accumulates in FP32; the quantised input is kept for Wgrad.
 *
 * Conventions for every entry point:
 *  - All tensor pointers are DEVICE pointers owned by the caller. The library
 *    never allocates, frees or synchronises; scratch memory is a caller
 *    workspace (`ws`, `ws_bytes`) sized by the matching *_workspace_size().
 *  - BF16 tensors are passed as their uint16_t bit patterns, FP8 tensors as
 *    uint8_t codes (OCP E4M3 "E4M3FN" or E5M2), scales as float.
 *  - Matrices are row-major; `ld` is the row pitch in elements.
 *  - Arguments are validated on the host before anything is enqueued; an
 *    error status means nothing was launched. On success the work is
 *    enqueued on `stream` and the call returns without waiting.
 *  - Results are deterministic: the same inputs give the same bytes.
 *  - Calls on one stream are ordered; calls that share a workspace must not
 *    run concurrently on different streams.
 *
 * Encoding (readings of the paper, which fixes the formats but not the
 * rounding): a value x is encoded as FP8(fl32(x * r)) with round-to-nearest-
 * even, saturation of finite and infinite magnitudes above the format's
 * largest value (448 for E4M3, 57344 for E5M2) and every NaN mapped to 0x7F.
 * Per-tensor scales: s = fl32(amax / FMAX), r = fl32(FMAX / amax) (s = r = 1
 * when amax = 0). Power-of-two scales: s = 2^e, r = 2^-e with e the smallest
 * integer such that amax <= FMAX * 2^e, clamped to [-127, 127] (e = 0 for
 * amax = 0). The stored scale is always the dequantisation scale s.
 */
#ifndef PURO_H
#define PURO_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PURO_OK = 0,
    PURO_ERR_NULL = 1,        /* a required pointer is NULL                              */
    PURO_ERR_SHAPE = 2,       /* negative size, ld smaller than the row, mismatched dims */
    PURO_ERR_UNSUPPORTED = 3, /* format / mode / rounding combination not provided       */
    PURO_ERR_ALIGN = 4,       /* size or pointer not a multiple the kernels need         */
    PURO_ERR_WORKSPACE = 5,   /* ws_bytes below the matching *_workspace_size()          */
    PURO_ERR_HIP = 6          /* a kernel launch reported an error                       */
} puro_status;

typedef enum { PURO_E4M3 = 0, PURO_E5M2 = 1 } puro_fp8_format;

/* Scale granularity (Section 3.2: one scale per tensor, or groups of 128
 * consecutive values along a GEMM's reduction dimension for activations and
 * gradients, and 128x128 blocks for weights). */
typedef enum {
    PURO_SCALE_TENSOR = 0,        /* one scale                                          */
    PURO_SCALE_ROW_1x128 = 1,     /* one scale per row per 128 consecutive columns      */
    PURO_SCALE_COL_128x1 = 2,     /* one scale per column per 128 consecutive rows      */
    PURO_SCALE_BLOCK_128x128 = 3, /* one scale per 128x128 block                        */
    PURO_SCALE_KMAJOR = 0x100     /* layout flag of the grouped modes (below)           */
} puro_scale_mode;

/* PURO_SCALE_KMAJOR is a layout flag of the grouped modes, OR-ed into a puro_scale_mode argument
 * (the quantise calls) or into puro_fp8_operand.mode (the GEMM): the scale
 * array is stored k-block-major, the index of the 128-wide group along the
 * reduction dimension of the GEMM that reads the codes outermost. Without it
 * grouped scales are row-major. The GEMM then loads each k block's scales as
 * one contiguous run; the linear layer keeps its scales this way. Layouts:
 *   quantise ROW_1x128:     scale  [cols/128][rows], scaleT [rows/128][cols]
 *   quantise COL_128x1:     scaleT [rows/128][cols]
 *   quantise BLOCK_128x128: scale  [cols/128][rows/128], scaleT [rows/128][cols/128]
 *   GEMM operand [rows, K]: ROW_1x128 scale[(k/128) * rows + row],
 *                           BLOCK_128x128 scale[(k/128) * ceil(rows/128) + row/128]
 * With TENSOR it is PURO_ERR_UNSUPPORTED. */

/* Scale value rule. Section 3.2: block scales are powers of two (the
 * exponent-only E8M0 representation of MXFP8). */
typedef enum {
    PURO_SCALE_FP32 = 0, /* s = amax / FMAX in binary32 (per-tensor mode only) */
    PURO_SCALE_POW2 = 1, /* s = 2^e, the smallest power of two that avoids saturation */
    PURO_SCALE_POW2_FLOOR = 2 /* s = 2^(floor(log2 amax) - emax), the OCP-MX rule (emax 8 for
                                 E4M3, 15 for E5M2): the largest values of a group whose amax
                                 has a significand above 1.75 saturate. For comparison. */
} puro_scale_rounding;

typedef enum { PURO_OUT_BF16 = 0, PURO_OUT_FP32 = 1 } puro_out_dtype;

/* Static text for a status code (never NULL). */
const char* puro_status_string(puro_status status);

/* ---------------------------------------------------------------- amax ---
 * amax = max |x| over the [rows, cols] BF16 tensor x (row pitch ld), written
 * as one float to the device scalar `amax`. NaN if any element is NaN; 0 for
 * an empty tensor; -0 counts as 0. Section 3.2 computes scales online from
 * the data; this is the per-tensor statistic they come from.
 * Requirements: cols % 8 == 0, ld % 8 == 0, x 16-byte aligned (rows of whole
 * 16-byte vectors). ws: puro_amax_workspace_size(rows, cols) bytes. */
size_t puro_amax_workspace_size(int64_t rows, int64_t cols);
puro_status puro_amax(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                      float* amax, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------ quantise ---
 * Quantise the [rows, cols] BF16 tensor x (row pitch ld) to FP8 `fmt`.
 * Section 3.2: activations and activation gradients in 1x128 groups along the
 * reduction dimension, weights in 128x128 blocks, or one scale per tensor.
 *
 *  mode TENSOR: q [rows, cols] and/or qT [cols, rows] (the same codes,
 *      transposed); scale[0] = s. rnd FP32, POW2 or POW2_FLOOR. If amax_in is not NULL
 *      the device scalar *amax_in is used instead of the tensor's own amax
 *      (values beyond it saturate).
 *  mode ROW_1x128: q [rows, cols], scale [rows, cols/128]. If qT is not NULL
 *      the same read also writes the column-grouped copy: qT [cols, rows]
 *      with scaleT [cols, rows/128] (128x1 groups down each column, as
 *      Wgrad needs; quantised from the BF16 values, not from q).
 *  mode COL_128x1: only qT [cols, rows] and scaleT [cols, rows/128].
 *  mode BLOCK_128x128: q [rows, cols] with scale [rows/128, cols/128], and
 *      if qT is not NULL also qT [cols, rows] with scaleT [cols/128, rows/128]
 *      (the same codes and scales, transposed).
 *  Grouped modes require rnd == POW2 or POW2_FLOOR, and amax_in == NULL.
 *
 * Requirements: cols % 16 == 0 and ld % 8 == 0 with x 16-byte aligned;
 * ld < 2^23 (else PURO_ERR_SHAPE); rows % 16 == 0 when qT is written; the
 * grouped dimension(s) % 128 == 0.
 * Outputs are dense (row pitch = their column count). ws:
 * puro_quantize_workspace_size(rows, cols) bytes (used in TENSOR mode). */
size_t puro_quantize_workspace_size(int64_t rows, int64_t cols);
puro_status puro_quantize_fp8(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                              puro_fp8_format fmt, puro_scale_mode mode, puro_scale_rounding rnd,
                              const float* amax_in, uint8_t* q, float* scale,
                              uint8_t* qT, float* scaleT, void* ws, size_t ws_bytes,
                              hipStream_t stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): puro_quantize_fp8 without
 * a workspace. The per-tensor mode's amax pass keeps its partial maxima in a
 * library-owned static device array of PURO_QUANTIZE_STATIC_SCRATCH_BYTES
 * (32 KiB) on each GPU it runs on, held until the process ends (its address is
 * looked up on the first such call on a device); nothing is allocated or freed.
 * Every call on one GPU shares that array: calls that overlap on one GPU (on
 * different streams, or from different threads without ordering) race and
 * may give wrong scales; order them on one stream. The partials are written
 * in full by each call, so nothing needs clearing. Sizes whose partials would
 * not fit return PURO_ERR_WORKSPACE (the quantiser uses at most 4096 partials,
 * which always fit). Arguments, outputs and errors otherwise as
 * puro_quantize_fp8; grouped modes and a supplied amax use no scratch. */
#define PURO_QUANTIZE_STATIC_SCRATCH_BYTES 32768
puro_status puro_quantize_fp8_static(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                                     puro_fp8_format fmt, puro_scale_mode mode, puro_scale_rounding rnd,
                                     const float* amax_in, uint8_t* q, float* scale, uint8_t* qT, float* scaleT,
                                     hipStream_t stream);

/* ------------------------------------------------- SwiGLU + quantise ---
 * The MLP of the paper's model (the Qwen3-1.7B architecture, Section 2)
 * computes down(silu(gate(x)) * up(x)); the hidden flow stays BF16 and the
 * down projection quantises its input right before its GEMM (Section 3.2,
 * Appendix C precision flow). This call fuses the two: from the fused
 * gate/up output gu [rows, 2 cols] (gate = columns [0, cols), up = columns
 * [cols, 2 cols), row pitch ld elements) it forms H = silu(gate) * up with
 * silu(g) = g / (1 + e^-g) in binary32, rounds H to BF16 (nearest even) and
 * quantises that H exactly as puro_quantize_fp8 would quantise a BF16 tensor
 * holding it, without writing H. The BF16 value of H can differ in its last
 * bit from another binary32 evaluation of exp; the codes and scales are
 * those of the H this call forms.
 *
 * Modes: TENSOR (q and/or qT; scale[0]; rnd FP32, POW2 or POW2_FLOOR; the
 * tensor's amax comes from a first pass over gu), ROW_1x128 (q, scale and
 * optionally the 128x1 column-grouped qT, scaleT) and COL_128x1 (qT,
 * scaleT), with the layouts of puro_quantize_fp8. BLOCK_128x128 returns
 * PURO_ERR_UNSUPPORTED (weights, not activations, take 128x128 blocks).
 *
 * Requirements: those of puro_quantize_fp8 with the BF16 matrix being gu
 * [rows, 2 cols] (ld >= 2 cols, ld % 8 == 0, ld < 2^23, gu 16-byte aligned)
 * and cols % 16 == 0. ws: puro_swiglu_quantize_workspace_size(rows, cols)
 * bytes (used in TENSOR mode). All pointers are device memory owned by the
 * caller; nothing is allocated or synchronised. */
size_t puro_swiglu_quantize_workspace_size(int64_t rows, int64_t cols);
puro_status puro_swiglu_quantize_fp8(const uint16_t* gu, int64_t rows, int64_t cols, int64_t ld,
                                     puro_fp8_format fmt, puro_scale_mode mode, puro_scale_rounding rnd,
                                     uint8_t* q, float* scale, uint8_t* qT, float* scaleT, void* ws,
                                     size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------- SwiGLU backward + quantise ---
 * The gate/up projection's Dgrad and Wgrad take the gradient of its output
 * quantised (Section 3.2); that gradient is the SwiGLU's backward. From dH
 * [rows, cols] (the down projection's Dgrad output; row pitch ld_dh) and
 * the saved gate/up output gu [rows, 2 cols] (gate = columns [0, cols), up =
 * columns [cols, 2 cols); row pitch ld_gu) this call forms dgu [rows,
 * 2 cols] = [dg | du] with dg = dH * u * silu'(g), silu'(g) = s (1 + g (1 - s)),
 * s = 1 / (1 + e^-g), and du = dH * silu(g), each in binary32 rounded once to
 * BF16, and quantises dgu exactly as puro_quantize_fp8 would quantise a BF16
 * tensor holding it, without writing it: q [rows, 2 cols] for Dgrad and the
 * transposed qT [2 cols, rows] for Wgrad.
 *
 * Modes: TENSOR (q and/or qT; scale[0]; rnd FP32, POW2 or POW2_FLOOR),
 * ROW_1x128 (q, scale [rows, 2 cols / 128] and optionally the 128x1
 * column-grouped qT, scaleT) and COL_128x1 (qT, scaleT); BLOCK_128x128
 * returns PURO_ERR_UNSUPPORTED.
 *
 * Requirements: dH [rows, cols] and gu [rows, 2 cols] meet puro_quantize_fp8's
 * requirements for x; cols % 8 == 0 (2 cols % 16 == 0); the grouped
 * dimension(s) of dgu % 128 == 0. ws: puro_swiglu_bwd_quantize_workspace_size
 * (rows, cols) bytes (used in TENSOR mode). All pointers are device memory
 * owned by the caller; nothing is allocated or synchronised. */
size_t puro_swiglu_bwd_quantize_workspace_size(int64_t rows, int64_t cols);
puro_status puro_swiglu_bwd_quantize_fp8(const uint16_t* dh, int64_t ld_dh, const uint16_t* gu, int64_t ld_gu,
                                         int64_t rows, int64_t cols, puro_fp8_format fmt, puro_scale_mode mode,
                                         puro_scale_rounding rnd, uint8_t* q, float* scale, uint8_t* qT,
                                         float* scaleT, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------ RMSNorm + quantise ---
 * Every attention and MLP block of the paper's model (the Qwen3-1.7B
 * architecture, Section 2) starts with an RMSNorm whose output is the input
 * of the QKV or gate/up projection; the norm stays BF16 and the projection
 * quantises its input right before its GEMM (Section 3.2, Appendix C
 * precision flow). This call fuses the two: for x [rows, cols] (row pitch
 * ld elements) and the norm's weight gamma [cols] (BF16) it computes, per
 * row, rstd = 1 / sqrt(mean(x^2) + eps) in binary32 (written to rstd[rows],
 * float, for the norm's backward), forms y = x * rstd * gamma in binary32,
 * rounds y to BF16 (nearest even) and quantises that y exactly as
 * puro_quantize_fp8 would quantise a BF16 tensor holding it, without
 * writing y. The binary32 sum of squares is taken in this library's order;
 * another order can move rstd, and so y's last BF16 bit, slightly.
 *
 * Modes: TENSOR (q and/or qT; scale[0]; rnd FP32, POW2 or POW2_FLOOR),
 * ROW_1x128 (q, scale and optionally the 128x1 column-grouped qT, scaleT)
 * and COL_128x1 (qT, scaleT), with the layouts of puro_quantize_fp8.
 * BLOCK_128x128 returns PURO_ERR_UNSUPPORTED. eps must be finite and
 * >= 0 (else PURO_ERR_UNSUPPORTED).
 *
 * Requirements: those of puro_quantize_fp8 for x; cols > 0 when rows > 0;
 * gamma and rstd non-NULL and 16-byte aligned when rows > 0. ws:
 * puro_rmsnorm_quantize_workspace_size(rows, cols) bytes (used in TENSOR
 * mode). All pointers are device memory owned by the caller; nothing is
 * allocated or synchronised. */
size_t puro_rmsnorm_quantize_workspace_size(int64_t rows, int64_t cols);
puro_status puro_rmsnorm_quantize_fp8(const uint16_t* x, const uint16_t* gamma, int64_t rows, int64_t cols,
                                      int64_t ld, float eps, puro_fp8_format fmt, puro_scale_mode mode,
                                      puro_scale_rounding rnd, uint8_t* q, float* scale, uint8_t* qT,
                                      float* scaleT, float* rstd, void* ws, size_t ws_bytes,
                                      hipStream_t stream);

/* ---------------------------------------------------------------- GEMM ---
 * D[m, n] = sum_k A[m, k] * B[n, k] with FP32 accumulation (Section 3.2:
 * the Fprop, Dgrad and Wgrad GEMMs of a linear layer run on FP8 operands).
 * Both operands are stored with the reduction index k contiguous: A is
 * [M, K] with row pitch A->ld bytes, B is [N, K] with row pitch B->ld bytes.
 * Fprop is A = Xq, B = Wq; Dgrad A = dYq, B = WqT; Wgrad A = dYqT, B = XqT.
 *
 * Operand scales (device memory, float):
 *   TENSOR:          scale[0]
 *   ROW_1x128:       scale[row * (K/128) + k/128]          ([rows, K/128])
 *   BLOCK_128x128:   scale[(row/128) * (K/128) + k/128]    ([ceil(rows/128), K/128])
 * Grouped scales must be powers of two in [2^-127, 2^127] (as written by
 * puro_quantize_fp8 with POW2); they are applied exactly inside the MFMA.
 * Per-tensor scales are applied once, in FP32, to the accumulated sum.
 *
 * D is BF16 (round-to-nearest-even) or FP32, row pitch ldd elements. With
 * accumulate != 0, D += result (the old value is read in D's type and the sum
 * formed in FP32). Requirements: K % 16 == 0 (K % 128 == 0 with grouped
 * scales), lda and ldb multiples of 16, operand pointers 16-byte aligned,
 * ldd >= N. ws: puro_fp8_gemm_workspace_size(M, N, K, d_type) bytes. */
typedef struct {
    const uint8_t* data;
    int64_t ld;
    puro_fp8_format fmt;
    puro_scale_mode mode;   /* TENSOR, ROW_1x128 or BLOCK_128x128; grouped ones may carry PURO_SCALE_KMAJOR */
    const float* scale;
} puro_fp8_operand;

size_t puro_fp8_gemm_workspace_size(int64_t M, int64_t N, int64_t K, puro_out_dtype d_type);
/* The execution plan puro_fp8_gemm chooses for this problem (host-side query;
 * enqueues nothing): the workgroup tile (tile_m x tile_n outputs), the depth
 * of its LDS ring (stages), the number of k ranges (splits > 1: FP32 partial
 * sums in ws plus a fixed-order reduction kernel) and the kernel launches
 * that makes. a_mode / b_mode are the operands' scale modes (the plan differs
 * with block scales). Outputs may be NULL. PURO_ERR_SHAPE for negative sizes,
 * PURO_ERR_UNSUPPORTED for a mode the GEMM does not take. For tests and
 * benchmarks that need to know which kernel configuration runs. */
puro_status puro_fp8_gemm_plan(int64_t M, int64_t N, int64_t K, puro_scale_mode a_mode,
                               puro_scale_mode b_mode, int* tile_m, int* tile_n, int* stages,
                               int* splits, int* launches);
puro_status puro_fp8_gemm(int64_t M, int64_t N, int64_t K,
                          const puro_fp8_operand* A, const puro_fp8_operand* B,
                          void* D, puro_out_dtype d_type, int64_t ldd, int accumulate,
                          void* ws, size_t ws_bytes, hipStream_t stream);

/* GEMM with the BF16 bias / residual epilogue of the linear layers around
 * the FP8 GEMMs: D = BF16(alpha * acc + bias[n] + residual[m, n]), the sum
 * in binary32 and one rounding (BF16 output only; either term may be NULL).
 * Qwen2's QKV projection carries a bias, and the attention output and MLP
 * down projections add into the residual stream, which stays BF16 (Appendix
 * C precision flow): fusing the add removes a BF16 read and write of Y.
 * bias: BF16 [N], 16-byte aligned. residual: BF16 [M, N] with row pitch
 * N <= ldr <= 2^22, ldr % 4 == 0, 16-byte aligned; it may be D itself (ldr == ldd,
 * an in-place residual add) but must not otherwise overlap D. Operands,
 * scales, workspace and errors as puro_fp8_gemm; accumulate is not offered. */
puro_status puro_fp8_gemm_epilogue(int64_t M, int64_t N, int64_t K, const puro_fp8_operand* A,
                                   const puro_fp8_operand* B, uint16_t* D, int64_t ldd, const uint16_t* bias,
                                   const uint16_t* residual, int64_t ldr, void* ws, size_t ws_bytes,
                                   hipStream_t stream);

/* -------------------------------------------------------- linear layer ---
 * Y = X W^T with X [M, K] and W [N, K] in BF16 (dense rows), and its backward
 * pass, as a sequence of the calls above (Section 3.2; Appendix C).
 *
 * Recipe: blockwise = 0 -> one scale per tensor (rule `rnd`); blockwise = 1
 * -> X and dY in 1x128 groups along each GEMM's reduction dimension (row
 * groups for Fprop and Dgrad, column groups for Wgrad), W in 128x128 blocks,
 * power-of-two scales (rule POW2_FLOOR if rnd says so, else POW2). */
typedef struct {
    puro_fp8_format x_fmt, w_fmt, dy_fmt;
    int blockwise;
    puro_scale_rounding rnd;
} puro_linear_recipe;

/* What the forward pass keeps for the backward pass (caller-allocated):
 * the quantised input, transposed for Wgrad (Section 3.2 keeps the quantised
 * input for Wgrad), and the quantised weight, transposed for Dgrad.
 *   xq_t    [K, M] FP8;  x_scale: per-tensor [1], blockwise [M/128, K]
 *   wq_t    [K, N] FP8;  w_scale: per-tensor [1], blockwise [N/128, K/128]
 * Blockwise scales are stored k-block-major (the group index along the
 * reduction dimension of the GEMM that reads them outermost): x_scale[b][k]
 * is the scale of xq_t row k, m in [128 b, 128 b + 128); w_scale[b][c] that
 * of the block of wq_t rows [128 c, 128 c + 128) and columns [128 b, ...).
 * The Wgrad and Dgrad GEMMs then read a k block's scales as one contiguous
 * run. (puro_quantize_fp8 and puro_fp8_gemm use the row-major layouts.)  */
typedef struct {
    uint8_t* xq_t;
    float* x_scale;
    uint8_t* wq_t;
    float* w_scale;
} puro_linear_saved;

/* Byte sizes of the four saved buffers (sizes[0..3] in the struct's order);
 * returns their sum. */
size_t puro_linear_saved_bytes(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* recipe,
                               size_t sizes[4]);
size_t puro_linear_fwd_workspace_size(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* recipe);
size_t puro_linear_bwd_workspace_size(int64_t M, int64_t N, int64_t K, const puro_linear_recipe* recipe);

/* Forward: quantise X and W, Y [M, N] (BF16) = Fprop, fill `saved`.
 * Requirements: M, N, K multiples of 16 (of 128 when blockwise) and at most
 * 2^22 (each is the row pitch of an FP8 operand of one of the three GEMMs);
 * larger sizes return PURO_ERR_SHAPE before anything is enqueued (this also
 * holds for the backward). */
puro_status puro_linear_fwd(const uint16_t* X, const uint16_t* W, int64_t M, int64_t N, int64_t K,
                            const puro_linear_recipe* recipe, uint16_t* Y,
                            const puro_linear_saved* saved, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/* Backward: quantise dY [M, N]; dX [M, K] (BF16) = Dgrad and dW [N, K] (FP32)
 * = Wgrad (dW += when accumulate_dW != 0). dX or dW may be NULL to skip that
 * GEMM. */
puro_status puro_linear_bwd(const uint16_t* dY, const puro_linear_saved* saved,
                            int64_t M, int64_t N, int64_t K, const puro_linear_recipe* recipe,
                            uint16_t* dX, float* dW, int accumulate_dW,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------- LM head with cross-entropy loss ---
 * Section 3.1.3 of the paper names the language-model head as the layer whose
 * cost sets the pipeline's last stage apart; Appendix C keeps it in BF16. For
 * hidden states X [M, K] and the output embedding W [V, K] (BF16, dense rows)
 * and one target vocabulary id per row, targets [M] (int32):
 *   forward:  z = X W^T; lse[m] = log sum_v exp(z[m, v]); loss[m] = lse[m] - z[m, t_m]
 *   backward: dz = g (exp(z - lse) - onehot(t)); dX = dz W (BF16 [M, K]);
 *             dW = dz^T X (FP32 [V, K], overwritten)
 * The logits are never stored: the forward reduces each 128-column block of
 * the GEMM's output tile to (max, sum exp) in its epilogue; the backward
 * recomputes the logits in chunks of 8192 vocabulary columns and writes only
 * the chunk's dz to the workspace (BF16; under PURO_LM_HEAD_FP8 its E4M3
 * copies, in 1x128 row and 128x1 column groups, made in the same epilogue).
 * g is the loss's upstream gradient (1 for the sum over tokens, 1/M for
 * their mean).
 * Recipes: PURO_LM_HEAD_BF16 (BF16 GEMMs with binary32 accumulation, dz
 * rounded to BF16), PURO_LM_HEAD_FP8 (Section 3.2's blockwise recipe: X in
 * 1x128 groups, W in 128x128 blocks, each dz chunk rounded to BF16 and then
 * in 1x128 + 128x1 groups; E4M3, power-of-two scales).
 * Requirements: M, V, K positive multiples of 128, at most 2^21; X, W, lse,
 * loss, dX, dW 16-byte aligned; targets in [0, V) (a row whose target lies
 * outside gets loss NaN and no onehot term). lse and loss are FP32 [M]. ws:
 * puro_lm_head_ce_workspace_size(M, V, K, recipe, backward) bytes (the
 * backward's includes the quantised or transposed operands and one chunk). All
 * pointers are device memory owned by the caller; nothing is allocated or
 * synchronised; invalid arguments return before anything is enqueued. */
typedef enum { PURO_LM_HEAD_BF16 = 0, PURO_LM_HEAD_FP8 = 1 } puro_lm_head_recipe;
size_t puro_lm_head_ce_workspace_size(int64_t M, int64_t V, int64_t K, puro_lm_head_recipe recipe, int backward);
puro_status puro_lm_head_ce_fwd(const uint16_t* X, const uint16_t* W, const int32_t* targets, int64_t M,
                                int64_t V, int64_t K, puro_lm_head_recipe recipe, float* lse, float* loss,
                                void* ws, size_t ws_bytes, hipStream_t stream);
puro_status puro_lm_head_ce_bwd(const uint16_t* X, const uint16_t* W, const int32_t* targets, const float* lse,
                                int64_t M, int64_t V, int64_t K, puro_lm_head_recipe recipe, float grad_scale,
                                uint16_t* dX, float* dW, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------- MuonH ---
 * Section 3.3 (Hyperball Optimization), equation hyperball-update: a wrapped
 * matrix keeps its initial Frobenius radius R; with the Muon update u and the
 * weight learning rate eta,
 *     W~ = W - eta R u / ||u||_F,    W' = R W~ / ||W~||_F.
 * The paper takes Muon from its training framework; the Muon update here is
 * the published method's:
 *     buf' = mu buf + (1 - mu) G;  V = (1 - mu) G + mu buf' (nesterov) or buf'
 *     X_0 = V / (||V||_F + 1e-7), transposed when rows > cols;
 *     ns_steps times: A = X X^T, B = b A + c A A^T, X = a X + B X,
 *     (a, b, c) = (3.4445, -4.7750, 2.0315); u = X (turned back).
 * FP32 state (W, G, buf), each momentum product and sum rounded to binary32
 * in that order with (1 - mu) rounded first; Newton-Schulz in BF16 with
 * binary32 accumulation, each of A, B and X rounded once to BF16; the
 * hyperball step from the BF16 u in binary32 with double-precision norms.
 *
 * puro_muonh_step updates `count` matrices of one shape stored back to back:
 * W [count][rows][cols] (FP32, in place), buf (FP32, in place), G (FP32),
 * radius [count] (FP32 device array: each matrix's R). Optional outputs:
 * w_bf16 (BF16 copy of W'), u_out (BF16 u, W's layout). ns_steps: 5 in the
 * method; 0 applies the hyperball step to X_0 (a test hook). u = 0 (all of V
 * zero) leaves W's direction and only projects it. rows, cols: positive
 * multiples of 128, at most 2^21; count in [1, 65535]; pointers 16-byte
 * aligned device memory owned by the caller. ws:
 * puro_muonh_workspace_size(count, rows, cols) bytes. Matrices may not
 * overlap W, G, buf or the outputs.
 *
 * puro_newton_schulz_bf16 runs `steps` Newton-Schulz steps on X [count][r][c]
 * (BF16, r <= c, already normalised) into out (same layout); the steps of
 * puro_muonh_step, exposed for per-step checks. */
size_t puro_muonh_workspace_size(int64_t count, int64_t rows, int64_t cols);
puro_status puro_muonh_step(int64_t count, int64_t rows, int64_t cols, float* W, uint16_t* w_bf16, const float* G,
                            float* buf, const float* radius, float mu, int nesterov, float eta, int ns_steps,
                            uint16_t* u_out, void* ws, size_t ws_bytes, hipStream_t stream);
size_t puro_newton_schulz_workspace_size(int64_t count, int64_t r, int64_t c);
puro_status puro_newton_schulz_bf16(int64_t count, int64_t r, int64_t c, const uint16_t* X, int steps,
                                    uint16_t* out, void* ws, size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PURO_H */
