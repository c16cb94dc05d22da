// Declarations shared by the GEMM's host planner (gemm.hip) and its kernel
// variants (gemm_kernel.hip, compiled once per operand-format pair and scale
// kind so that the instantiations build in parallel).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"

namespace puro {
namespace gemm_detail {

constexpr int kBK = 128;                   // k block of the grouped scales (and of split-K ranges)

struct Params {
    const uint8_t* A;
    const uint8_t* B;
    const float* sa;
    const float* sb;
    void* D;
    float* partial;
    int64_t lda, ldb, ldd;
    int M, N, K;
    int a_mode, b_mode;
    int a_kmajor, b_kmajor;    // grouped scales k-block-major rather than row-major
    int ld_sa, ld_sb;          // scale pitch: K/128 (row-major) or the row (block) count (k-major)
    uint32_t sa_bytes, sb_bytes;  // sizes of the scale arrays (grouped modes)
    int ksteps, ksteps_per_split, splits;
    int gm;                    // tile rows per group within an XCD's range of tiles
    int tiles_m, tiles_n;
    int accumulate;
    float alpha;               // host-known factor of the sums (with the per-tensor scales)
    const uint16_t* bias;      // OUT kOutBF16Epi: optional bias [N] and residual [M, N] (pitch ldr)
    const uint16_t* residual;
    int64_t ldr;
    float res_scale;           // factor of the residual
    int upper;                 // only the tiles on or above the diagonal (square tiles, M == N)
    int nt_out;                // interior tiles store D with non-temporal (streaming) stores
    int batch;                 // problems of one launch: A, B, D advance by bsa, bsb, bsd bytes,
    int64_t bsa, bsb, bsd;     // the residual by bsr elements, the split-K partials by
    int64_t bsr;               // splits * M * N floats

    // LM-head output kinds (kOutLseStats, kOutSoftmaxGrad; 128-column wave tiles)
    const int32_t* targets;    // target vocabulary id per row
    int col0;                  // vocabulary column of this GEMM's column 0
    float2* stats;             // [M][stats_ld]: (max, sum exp(z - max)) per 128-column block
    int64_t stats_ld;
    float* zt;                 // [M]: the target's logit
    const float* lse;          // [M]
    float grad_scale;
    uint8_t* q8;               // kOutSoftmaxGradQ: dz's FP8 copies (the GemmProblem fields)
    float* q8_scale;
    uint8_t* q8t;
    float* q8t_scale;
};

struct TileCfg {
    int bm, bn;          // workgroup tile
    int wm, wn;          // wave grid (wave tile bm/wm x bn/wn)
    int sl, nst;         // k bytes per pipeline slice, ring stages
    int prod;            // producer waves issue the global->LDS loads
    float fixed_us;      // time model: per wave of work units ...
    float slice_us;      // ... plus per k slice of a unit (MI355X, all CUs busy)
};
// Four MFMA waves (one per SIMD) in a 2x2 grid. The large wave tiles need
// the least LDS traffic per MFMA (128x128: 16 MFMAs per 16 KB of fragment
// reads); the 128x128 tiles give more work units on narrow problems, with a
// deep ring (one workgroup per CU) or a short one (two per CU). A 128x128
// tile moves as many bytes global->LDS per k slice as the texture unit
// passes (about 64 B per clock per CU) while its MFMAs run, so its loads
// often wait for queue space: the deep-ring variant adds four producer waves
// that issue them (the tile's registers leave room for two waves per SIMD),
// 15-20% faster on long-K Wgrad than issuing them from the MFMA waves. The
// time constants are least-squares fits to measured kernel times on the
// Qwen2-1.5B layer shapes.
#define PURO_TILE_LIST(X)                                 \
    X(0, 256, 256, 2, 2, 128, 2, 0, 7.86f, 1.322f)        \
    X(1, 256, 192, 2, 2, 128, 2, 0, 6.37f, 1.120f)        \
    X(2, 128, 128, 2, 2, 128, 4, 1, 6.65f, 0.379f)        \
    X(3, 128, 128, 2, 2, 128, 2, 0, 4.37f, 0.803f)
#define PURO_TILE_ROW(i, bm, bn, wm, wn, sl, nst, prod, f, s) {bm, bn, wm, wn, sl, nst, prod, f, s},

// The bias / residual epilogue: the BF16 bias of columns n..n+3 and the BF16
// residual of row m at those columns added to four binary32 results (the
// sum stays binary32 until the output's one rounding).
// The residual is multiplied by rs in the same fused step as its addition
// (rs = 1 adds it exactly as a plain sum).
__device__ __forceinline__ void add_epilogue4(float4& v, const uint16_t* bias, const uint16_t* residual,
                                              int64_t ldr, int64_t m, int64_t n, float rs) {
    if (bias) {
        const uint2 b = *reinterpret_cast<const uint2*>(bias + n);
        v.x += bf16lo(b.x); v.y += bf16hi(b.x); v.z += bf16lo(b.y); v.w += bf16hi(b.y);
    }
    if (residual) {
        const uint2 r = *reinterpret_cast<const uint2*>(residual + m * ldr + n);
        v.x = fmaf(rs, bf16lo(r.x), v.x); v.y = fmaf(rs, bf16hi(r.x), v.y);
        v.z = fmaf(rs, bf16lo(r.y), v.z); v.w = fmaf(rs, bf16hi(r.y), v.w);
    }
}
__device__ __forceinline__ float add_epilogue1(float v, const uint16_t* bias, const uint16_t* residual, int64_t ldr,
                                               int64_t m, int64_t n, float rs) {
    if (bias) v += __uint_as_float((uint32_t)bias[n] << 16);
    if (residual) v = fmaf(rs, __uint_as_float((uint32_t)residual[m * ldr + n] << 16), v);
    return v;
}

// Enqueue the kernel of tile configuration `cfg` (index into the list above)
// for output kind `out` (kOutBF16, kOutF32, kOutBF16Epi, or 2: split-K
// partial sums) over `grid` workgroups; defined in gemm_kernel.hip for each
// (FA, FB, GROUPED).
template <int FA, int FB, bool GROUPED>
void launch_variant(const Params& prm, int cfg, int out, int grid, hipStream_t stream);

}  // namespace gemm_detail
}  // namespace puro
