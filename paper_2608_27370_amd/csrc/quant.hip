// amax and FP8 quantisation kernels for gfx950.
//
// Section 3.2 of the paper: each linear layer quantises its BF16 operands to
// FP8 right before the GEMM, with scales computed online from the data: one
// per tensor, one per 128 consecutive values along the GEMM's reduction
// dimension (activations, gradients), or one per 128x128 block (weights),
// block scales being powers of two.
//
// These passes are bound by HBM bandwidth: every element is read once as BF16
// (16-byte vector loads, coalesced along rows) and written as one FP8 byte
// per requested copy. Each thread owns an 8x8 sub-block of a 128x128 tile.
// A transposed copy starts as an in-register 8x8 byte transpose; the
// transposed blocks meet in LDS, from where the block stores whole 128-byte
// runs of the transposed rows (16 bytes per lane).
// Per-tensor scaling needs the whole tensor's amax before any encoding: a
// first pass writes per-block partial maxima (no atomics, no zero-initialised
// state); the quantise pass reduces them in every block (few partials) or
// reads the amax a one-block reduction kernel wrote (many partials).
// Loads go through buffer descriptors whose range check supplies the zeros
// outside a tensor, so they carry no branches and never wait on each other.

#include <algorithm>
#include <atomic>
#include <mutex>

#include "device_common.h"
#include "kernels.h"

namespace puro {

namespace {

constexpr int kThreads = 256;
constexpr int kTile = 128;
typedef int v4i __attribute__((ext_vector_type(4)));
// Above this many partial maxima a one-block kernel reduces them once,
// rather than every block of the quantise pass reading them all.
constexpr int kMaxInlinePartials = 2048;

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, 64));
    return v;
}

// Block-wide max of a per-thread value (256 threads); result in every thread.
__device__ __forceinline__ uint32_t block_max(uint32_t v, uint32_t* red) {
    v = wave_max(v);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    return max(max(red[0], red[1]), max(red[2], red[3]));
}

// ---------------------------------------------------------------- amax ---
// Sources of the values a pass reads: the BF16 tensor itself; the SwiGLU of a
// fused gate/up output [rows, 2 cols] (gate = columns [0, cols), up =
// columns [cols, 2 cols)), rounded to BF16 as the tensor H = silu(gate) * up
// would hold it; the RMSNorm y = x * rstd * gamma of x [rows, cols],
// rounded to BF16 (rstd per row from the row pass, gamma per column); or the
// SwiGLU's backward [dg | du] [rows, cols] from dH [rows, cols / 2] and the
// saved gate/up output, rounded to BF16.
enum : int { kSrcBf16 = 0, kSrcSwiglu = 1, kSrcRmsnorm = 2, kSrcSwigluBwd = 3 };

// Partial maxima of one or two tensors in one launch: blocks [0, j0.P) cover
// the rows of the first tensor in P contiguous ranges, the rest the second.
template <bool DENSE, int SRC>
__global__ __launch_bounds__(kThreads) void amax_partial_kernel(AmaxJob j0, AmaxJob j1) {
    __shared__ uint32_t red[4];
    const bool second = (int)blockIdx.x >= j0.P;
    const uint16_t* x = second ? j1.x : j0.x;
    const int64_t rows = second ? j1.rows : j0.rows;
    const int64_t ld = second ? j1.ld : j0.ld;
    const uint32_t cpr = second ? j1.cpr : j0.cpr;
    uint32_t* partial = second ? j1.partial : j0.partial;
    const int P = second ? j1.P : j0.P;
    const int bid = second ? (int)blockIdx.x - j0.P : (int)blockIdx.x;
    const int64_t r0 = rows * bid / P, r1 = rows * (bid + 1) / P;
    const uint32_t n = (uint32_t)((r1 - r0) * cpr);
    uint32_t m = 0;
    constexpr int U = 8;
    for (uint32_t j0i = threadIdx.x; j0i < n; j0i += kThreads * U) {
        uint4 v[U], vu[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t j = j0i + u * kThreads;
            v[u] = vu[u] = make_uint4(0, 0, 0, 0);
            if (j < n) {
                const uint16_t* p;
                if constexpr (DENSE) {
                    p = x + (r0 * cpr + j) * 8;
                } else {
                    const uint32_t rr = j / cpr, cc = j - rr * cpr;
                    p = x + (r0 + rr) * ld + (int64_t)cc * 8;
                }
                v[u] = *reinterpret_cast<const uint4*>(p);
                // the up value of the same position, cols (= 8 cpr) further on
                if constexpr (SRC == kSrcSwiglu) vu[u] = *reinterpret_cast<const uint4*>(p + 8 * cpr);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
            if constexpr (SRC == kSrcSwiglu) {
                const uint32_t wu[4] = {vu[u].x, vu[u].y, vu[u].z, vu[u].w};
                const uint32_t wg[4] = {w[0], w[1], w[2], w[3]};
                swiglu8(wg, wu, w);
            }
            m = max(m, absmax_bits8(w));
        }
    }
    m = block_max(m, red);
    if (threadIdx.x == 0) partial[bid] = m;
}

__global__ __launch_bounds__(kThreads) void amax_finalize_kernel(const uint32_t* __restrict__ partial,
                                                                 int P, float* __restrict__ amax) {
    __shared__ uint32_t red[4];
    uint32_t m = 0;
    for (int i = threadIdx.x; i < P; i += kThreads) m = max(m, partial[i]);
    m = block_max(m, red);
    if (threadIdx.x == 0) *amax = __uint_as_float(m << 16);
}

// ------------------------------------------------------------ RMSNorm ---
// One wave per row, four rows per block: the row's sum of squares in binary32
// (each lane over its 8-column chunks in order, then a butterfly across the
// wave), rstd = 1 / sqrt(sum / cols + eps) stored per row; with AMAX, a second
// sweep over the row (now in cache) forms y = BF16(x * rstd * gamma) and the
// block writes the largest |y| pattern of its rows as a partial maximum.
template <bool AMAX>
__global__ __launch_bounds__(kThreads) void rmsnorm_rows_kernel(const uint16_t* __restrict__ x, int64_t rows,
                                                                int64_t cols, int64_t ld,
                                                                const uint16_t* __restrict__ gamma, float eps,
                                                                float* __restrict__ rstd,
                                                                uint32_t* __restrict__ partial) {
    __shared__ uint32_t red[4];
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t cpr = cols / 8;
    const bool live = row < rows;
    const uint16_t* xr = x + (live ? row : 0) * ld;
    float ss = 0.0f;
    if (live) {
        for (int64_t c = lane; c < cpr; c += 64) {
            const uint4 v = *reinterpret_cast<const uint4*>(xr + c * 8);
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float lo = bf16lo(w[i]), hi = bf16hi(w[i]);
                ss = fmaf(lo, lo, ss);
                ss = fmaf(hi, hi, ss);
            }
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
    const float r = 1.0f / sqrtf(ss / (float)cols + eps);
    if (live && lane == 0) rstd[row] = r;
    if constexpr (AMAX) {
        uint32_t m = 0;
        if (live) {
            for (int64_t c = lane; c < cpr; c += 64) {
                const uint4 v = *reinterpret_cast<const uint4*>(xr + c * 8);
                const uint4 gv = *reinterpret_cast<const uint4*>(gamma + c * 8);
                const uint32_t w[4] = {v.x, v.y, v.z, v.w}, gw[4] = {gv.x, gv.y, gv.z, gv.w};
                uint32_t y[4];
                rmsnorm8(w, r, gw, y);
                m = max(m, absmax_bits8(y));
            }
        }
        m = block_max(m, red);
        if (threadIdx.x == 0) partial[blockIdx.x] = m;
    }
}

// ------------------------------------------------------------ quantise ---
struct Tile {
    int cc, rg;       // column chunk (8 columns) and row group (8 rows) of this thread
    int64_t row0;     // first of the thread's 8 rows
    int64_t col;      // first of the thread's 8 columns
    bool col_ok;
};

// The thread's 8x8 block in tile (bx, by) (tile column, tile row).
__device__ __forceinline__ Tile tile_coords(int64_t cols, int64_t bx, int64_t by) {
    Tile t;
    t.cc = threadIdx.x & 15;
    t.rg = threadIdx.x >> 4;
    t.row0 = by * kTile + t.rg * 8;
    t.col = bx * kTile + t.cc * 8;
    t.col_ok = t.col < cols;
    return t;
}
__device__ __forceinline__ Tile tile_coords(int64_t cols) { return tile_coords(cols, blockIdx.x, blockIdx.y); }

// Buffer descriptor over `bytes` bytes from `base` (32-bit raw data): loads
// at offsets at or beyond `bytes` return zeros and touch no memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
constexpr uint32_t kOOB = 0x80000000u;   // an offset beyond every descriptor's range (ld < 2^23)

// The thread's 8x8 block, zeros outside the tensor, by buffer loads over the
// tile's rows: positions outside the tensor read as zeros through the
// descriptor's range check, so the loads carry no branches and issue back to
// back (and independent loads issued before them are not waited for). With
// the SwiGLU source each value is computed from the gate and up values at the
// same position of the two halves of a row (zeros outside give silu(0) * 0 = 0).
template <int SRC>
__device__ __forceinline__ void load_8x8(const QuantArgs& a, const Tile& t, uint32_t w[8][4]);

// The SwiGLU backward source: the thread's 8 columns of [dg | du] come from
// the same 8 columns c of dH and of the gate half (g), and for dg of the up
// half (u, columns F + c); a chunk never straddles F = cols / 2 (F % 8 == 0).
__device__ __forceinline__ void load_swiglu_bwd_8x8(const QuantArgs& a, const Tile& t, uint32_t w[8][4]) {
    const int64_t F = a.cols / 2;
    const int64_t tr0 = t.row0 - t.rg * 8;
    const int64_t vr = a.cols == 0 ? 0 : max((int64_t)0, min((int64_t)kTile, a.rows - tr0));
    const uint32_t bh = vr == 0 ? 0u : (uint32_t)(((vr - 1) * a.ld + F) * 2);
    const uint32_t bg = vr == 0 ? 0u : (uint32_t)(((vr - 1) * a.ld2 + 2 * F) * 2);
    const __amdgpu_buffer_rsrc_t rh = buffer_rsrc(vr == 0 ? a.x : a.x + tr0 * a.ld, bh);
    const __amdgpu_buffer_rsrc_t rg = buffer_rsrc(vr == 0 ? a.x2 : a.x2 + tr0 * a.ld2, bg);
    const bool dg = t.col < F;
    const int64_t c = dg ? t.col : t.col - F;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t r = t.rg * 8 + i;
        const v4i h = __builtin_amdgcn_raw_buffer_load_b128(rh, t.col_ok ? (uint32_t)((r * a.ld + c) * 2) : kOOB, 0, 0);
        const v4i g = __builtin_amdgcn_raw_buffer_load_b128(rg, t.col_ok ? (uint32_t)((r * a.ld2 + c) * 2) : kOOB, 0, 0);
        const v4i u = __builtin_amdgcn_raw_buffer_load_b128(
            rg, (t.col_ok && dg) ? (uint32_t)((r * a.ld2 + F + c) * 2) : kOOB, 0, 0);
        const uint32_t hw[4] = {(uint32_t)h.x, (uint32_t)h.y, (uint32_t)h.z, (uint32_t)h.w};
        const uint32_t gw[4] = {(uint32_t)g.x, (uint32_t)g.y, (uint32_t)g.z, (uint32_t)g.w};
        const uint32_t uw[4] = {(uint32_t)u.x, (uint32_t)u.y, (uint32_t)u.z, (uint32_t)u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j)
            w[i][j] = pack_bf16x2(swiglu_bwd1(bf16lo(hw[j]), bf16lo(gw[j]), bf16lo(uw[j]), dg),
                                  swiglu_bwd1(bf16hi(hw[j]), bf16hi(gw[j]), bf16hi(uw[j]), dg));
    }
}

template <int SRC>
__device__ __forceinline__ void load_8x8(const QuantArgs& a, const Tile& t, uint32_t w[8][4]) {
    if constexpr (SRC == kSrcSwigluBwd) {
        load_swiglu_bwd_8x8(a, t, w);
        return;
    }
    const int64_t tr0 = t.row0 - t.rg * 8;                        // the tile's first row
    const int64_t vr = a.cols == 0 ? 0 : max((int64_t)0, min((int64_t)kTile, a.rows - tr0));
    // rows tr0 .. tr0 + vr - 1: the last one ends at column cols (2 cols with the SwiGLU source)
    const int64_t width = SRC == kSrcSwiglu ? 2 * a.cols : a.cols;
    const uint32_t bytes = vr == 0 ? 0u : (uint32_t)(((vr - 1) * a.ld + width) * 2);
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(vr == 0 ? a.x : a.x + tr0 * a.ld, bytes);
    uint32_t wu[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const uint32_t off = t.col_ok ? (uint32_t)(((t.rg * 8 + i) * a.ld + t.col) * 2) : kOOB;
        const v4i v = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
        w[i][0] = v.x; w[i][1] = v.y; w[i][2] = v.z; w[i][3] = v.w;
        if constexpr (SRC == kSrcSwiglu) {
            const uint32_t offu = t.col_ok ? off + (uint32_t)(a.cols * 2) : kOOB;
            const v4i vu = __builtin_amdgcn_raw_buffer_load_b128(rs, offu, 0, 0);
            wu[i][0] = vu.x; wu[i][1] = vu.y; wu[i][2] = vu.z; wu[i][3] = vu.w;
        }
    }
    if constexpr (SRC == kSrcSwiglu) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t g[4] = {w[i][0], w[i][1], w[i][2], w[i][3]};
            swiglu8(g, wu[i], w[i]);
        }
    }
    if constexpr (SRC == kSrcRmsnorm) {
        // the rows' rstd (zeros past the last row) and the columns' gamma
        const __amdgpu_buffer_rsrc_t rr = buffer_rsrc(a.rstd, (uint32_t)(a.rows * 4));
        const __amdgpu_buffer_rsrc_t rg = buffer_rsrc(a.gamma, (uint32_t)(a.cols * 2));
        const uint32_t roff = (uint32_t)(t.row0 * 4);
        const v4i r0 = __builtin_amdgcn_raw_buffer_load_b128(rr, roff, 0, 0);
        const v4i r1 = __builtin_amdgcn_raw_buffer_load_b128(rr, roff + 16, 0, 0);
        const v4i gv = __builtin_amdgcn_raw_buffer_load_b128(rg, t.col_ok ? (uint32_t)(t.col * 2) : kOOB, 0, 0);
        const uint32_t gw[4] = {(uint32_t)gv.x, (uint32_t)gv.y, (uint32_t)gv.z, (uint32_t)gv.w};
        const int rs[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) rmsnorm8(w[i], __int_as_float(rs[i]), gw, w[i]);
    }
}

__device__ __forceinline__ void store_rows(const QuantArgs& a, const Tile& t, const uint2 c[8]) {
    if (!t.col_ok) return;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t r = t.row0 + i;
        if (r < a.rows) *reinterpret_cast<uint2*>(a.q + r * a.cols + t.col) = c[i];
    }
}

// qT [cols, rows] of the tile whose first element is (row0, col0), from the
// codes c of every thread's 8x8 block. Column j of a thread's block becomes
// 8 bytes of LDS row col + j (LDS row r = qT row col0 + r, 128 bytes = the
// tile's rows); then each lane stores 16 bytes, eight lanes one whole
// 128-byte run of a qT row. The 16-byte chunk h of LDS row r sits at
// position h ^ ((r >> 3) & 7): the 8-byte writes of a wave (rows 8 apart
// across lanes) then spread over the banks, and a wave's 16-byte reads of 8
// consecutive rows cover all 64 banks four times (the minimum). rows % 16 ==
// 0, so a 16-byte run never crosses the end of a qT row. Ends with a barrier,
// after which the LDS buffer may be reused. qT not 16-byte aligned: 8-byte
// stores straight from registers.
__device__ __forceinline__ void store_transposed_ct(const QuantArgs& a, const Tile& t, int64_t row0, int64_t col0,
                                                    const uint2 ct[8], uint8_t* lds) {
    if ((reinterpret_cast<uintptr_t>(a.qT) & 15) != 0) {
        if (!t.col_ok || t.row0 >= a.rows) return;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            *reinterpret_cast<uint2*>(a.qT + (t.col + j) * a.rows + t.row0) = ct[j];
        return;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int r = t.cc * 8 + j;
        const int pos = (((t.rg >> 1) ^ (r >> 3 & 7)) << 4) + ((t.rg & 1) << 3);
        *reinterpret_cast<uint2*>(lds + r * kTile + pos) = ct[j];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kTile * kTile / 16 / kThreads; ++i) {
        const int q = i * kThreads + threadIdx.x;
        const int r = q >> 3, h = q & 7;
        const uint4 v = *reinterpret_cast<const uint4*>(lds + r * kTile + ((h ^ (r >> 3 & 7)) << 4));
        const int64_t col = col0 + r, row = row0 + h * 16;
        if (col < a.cols && row < a.rows) *reinterpret_cast<uint4*>(a.qT + col * a.rows + row) = v;
    }
    __syncthreads();
}

// The same from the codes of the thread's 8x8 block in row order.
__device__ __forceinline__ void store_transposed(const QuantArgs& a, const Tile& t, int64_t row0, int64_t col0,
                                                 const uint2 c[8], uint8_t* lds) {
    uint2 ct[8];
    transpose8x8(c, ct);
    store_transposed_ct(a, t, row0, col0, ct, lds);
}


// Scale of a per-tensor quantisation: s (stored) and the multiplier r, and
// whether encoding must take the saturating path (the amax was supplied and
// values beyond it saturate, the floor rule clips the top values, or the
// amax or r is not finite).
struct TensorScale {
    float s, r;
    bool safe;
};

template <int FMT>
__device__ __forceinline__ TensorScale tensor_scale(const QuantArgs& a, float amax) {
    float s, r;
    bool saturate = a.supplied != 0;
    constexpr float fm = Fp8Traits<FMT>::kMax;
    if (a.pow2) {
        if (amax != amax) {
            s = r = __uint_as_float(0x7FC00000u);
        } else {
            // |amax| as a BF16-or-wider magnitude: reuse the exponent rule on its top bits
            const uint32_t bits = __float_as_uint(fabsf(amax));
            int e;
            if (bits == 0) e = 0;
            else if (bits >= 0x7F800000u) e = 127;
            else if ((bits >> 23) == 0) e = -127;
            else {
                const bool above = (bits & 0x7FFFFFu) > 0x600000u;   // significand > 1.75
                e = (int)(bits >> 23) - 127 - Fp8Traits<FMT>::kEmax + (a.pow2 != 2 && above ? 1 : 0);
                e = e < -127 ? -127 : (e > 127 ? 127 : e);
                // the floor rule (pow2 == 2) saturates the top values of such a tensor
                saturate = saturate || (a.pow2 == 2 && above);
            }
            s = exp2i(e);
            r = exp2i(-e);
        }
    } else if (amax == 0.0f) {
        s = r = 1.0f;
    } else {
        s = amax / fm;
        r = fm / amax;
    }
    return {s, r, saturate || !(fabsf(amax) <= 3.4028235e38f) || !(fabsf(r) <= 3.4028235e38f)};
}

// Partial maxima of a tensor's amax pass as this thread reads them (its
// share of at most kMaxInlinePartials), issued before the tile loads so
// that they return first and the reduction overlaps the tile's arrival.
struct PartialShare {
    uint32_t v[kMaxInlinePartials / kThreads];
};

// Buffer loads: entries past the partials (all of them when the amax is a
// device scalar) read as zeros, which leave the maximum unchanged.
__device__ __forceinline__ PartialShare load_partials(const QuantArgs& a, bool active = true) {
    PartialShare p;
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(a.partial, (!active || a.amax) ? 0u : (uint32_t)a.npartial * 4u);
#pragma unroll
    for (int u = 0; u < kMaxInlinePartials / kThreads; ++u)
        p.v[u] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, (u * kThreads + threadIdx.x) * 4u, 0, 0);
    return p;
}

// The tensor's amax: the supplied or finalised device scalar, or the block's
// reduction of the partial maxima (every thread gets it).
__device__ __forceinline__ float tensor_amax(const QuantArgs& a, const PartialShare& p, uint32_t* red) {
    if (a.amax) return *a.amax;
    uint32_t m = 0;
#pragma unroll
    for (int u = 0; u < kMaxInlinePartials / kThreads; ++u) m = max(m, p.v[u]);
    m = block_max(m, red);
    return __uint_as_float(m << 16);
}

// Partial maxima of a source's values, one per 128x128 tile (1-D grid over
// the tiles, row-major): the amax pass of a per-tensor quantisation whose
// values are formed from several inputs.
template <int SRC>
__global__ __launch_bounds__(kThreads) void tile_amax_kernel(QuantArgs a, int gx, uint32_t* partial) {
    __shared__ uint32_t red[4];
    const Tile t = tile_coords(a.cols, (int)blockIdx.x % gx, (int)blockIdx.x / gx);
    uint32_t w[8][4];
    load_8x8<SRC>(a, t, w);
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) m = max(m, absmax_bits8(w[i]));
    m = block_max(m, red);
    if (threadIdx.x == 0) partial[blockIdx.x] = m;
}

// Per-tensor quantisation of one or two tensors in one launch (1-D grid:
// the first tensor's tiles, then the second's). Each block loads the partial
// maxima of both tensors and its tile's BF16 values before reducing any of
// them, so that the amax reduction overlaps the arrival of the tile.
template <int FMT, int SRC>
__global__ __launch_bounds__(kThreads) void quant_tensor_kernel(QuantArgs a0, QuantArgs a1, int tiles0,
                                                                int gx0, int gx1) {
    __shared__ uint32_t red[4];
    __shared__ __attribute__((aligned(16))) uint8_t tq[kTile * kTile];
    const bool two = (int)gridDim.x > tiles0;   // a second tensor follows the first one's tiles
    const bool second = (int)blockIdx.x >= tiles0;
    const QuantArgs& a = second ? a1 : a0;
    const int tile = second ? (int)blockIdx.x - tiles0 : (int)blockIdx.x;
    const int gx = second ? gx1 : gx0;
    const Tile t = tile_coords(a.cols, tile % gx, tile / gx);
    const PartialShare p0 = load_partials(a0);
    const PartialShare p1 = load_partials(a1, two);
    uint32_t w[8][4];
    load_8x8<SRC>(a, t, w);
    // the scales (every block derives the same values; block 0 stores them)
    const TensorScale sc0 = tensor_scale<FMT>(a0, tensor_amax(a0, p0, red));
    const TensorScale sc1 = two ? tensor_scale<FMT>(a1, tensor_amax(a1, p1, red)) : sc0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        if (a0.scale) a0.scale[0] = sc0.s;
        if (two && a1.scale) a1.scale[0] = sc1.s;
    }
    const TensorScale sc = second ? sc1 : sc0;
    uint2 c[8];
    if (sc.safe) {
#pragma unroll
        for (int i = 0; i < 8; ++i) c[i] = encode8<FMT, true>(w[i], sc.r);
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) c[i] = encode8<FMT, false>(w[i], sc.r);
    }
    if (a.q) store_rows(a, t, c);
    if (a.qT) store_transposed(a, t, (int64_t)(tile / gx) * kTile, (int64_t)(tile % gx) * kTile, c, tq);
}

// 1x128 row groups (q, scale) and/or 128x1 column groups (qT, scaleT).
template <int FMT, bool ROWS, bool COLS, int SRC>
__global__ __launch_bounds__(kThreads) void quant_groups_kernel(QuantArgs a) {
    __shared__ uint32_t colmax[4][kTile / 2];     // packed pairs of column maxima per wave
    __shared__ __attribute__((aligned(16))) uint8_t tq[COLS ? kTile * kTile : 16];
    const Tile t = tile_coords(a.cols);
    uint32_t w[8][4];
    load_8x8<SRC>(a, t, w);
    const bool floor_rule = a.pow2 == 2;

    if constexpr (ROWS) {
        uint2 c[8];
        float srow[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint32_t m = absmax_bits8(w[i]);
#pragma unroll
            for (int o = 8; o >= 1; o >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, o, 16));
            if (m <= 0x7F7Fu) {                      // finite group
                const int e = pow2_exponent_bf16<FMT>(m, floor_rule);
                srow[i] = exp2i(e);
                if (floor_rule && floor_rule_saturates(m)) c[i] = encode8<FMT, true>(w[i], exp2i(-e));
                else if (e > -127) c[i] = encode8_pow2<FMT>(w[i], srow[i]);
                else c[i] = encode8<FMT, false>(w[i], exp2i(-e));
            } else if (m == 0x7F80u) {               // an infinity: largest scale, saturate
                srow[i] = exp2i(127);
                c[i] = encode8<FMT, true>(w[i], exp2i(-127));
            } else {                                 // a NaN: NaN scale, NaN codes
                srow[i] = __uint_as_float(0x7FC00000u);
                c[i] = encode8<FMT, true>(w[i], srow[i]);
            }
        }
        store_rows(a, t, c);
        if (t.cc == 0) {
            const int64_t ng = a.cols / kTile;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int64_t r = t.row0 + i;
                if (r < a.rows) a.scale[a.kmajor ? (int64_t)blockIdx.x * a.rows + r : r * ng + blockIdx.x] = srow[i];
            }
        }
    }
    if constexpr (COLS) {
        // column maxima over the tile's 128 rows, two columns per word (the
        // two magnitude patterns of a word in its halves): 8 rows in-thread,
        // 4 row groups per wave (lanes 16 apart), 4 waves through LDS
        uint32_t cm[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t m = mag2(w[0][j]);
#pragma unroll
            for (int i = 1; i < 8; ++i) m = pk_max_u16(m, mag2(w[i][j]));
            m = pk_max_u16(m, (uint32_t)__shfl_xor((int)m, 16, 64));
            m = pk_max_u16(m, (uint32_t)__shfl_xor((int)m, 32, 64));
            cm[j] = m;
        }
        const int wv = threadIdx.x >> 6;
        if ((threadIdx.x & 63) < 16) {
#pragma unroll
            for (int j = 0; j < 4; ++j) colmax[wv][t.cc * 4 + j] = cm[j];
        }
        __syncthreads();
        uint32_t cw[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = t.cc * 4 + j;
            cw[j] = pk_max_u16(pk_max_u16(colmax[0][k], colmax[1][k]), pk_max_u16(colmax[2][k], colmax[3][k]));
        }
        float rcol[8], scol[8];
        bool finite = true, normal = true;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t m = (j & 1) ? (cw[j >> 1] >> 16) : (cw[j >> 1] & 0xFFFFu);
            if (m <= 0x7F7Fu) {
                const int e = pow2_exponent_bf16<FMT>(m, floor_rule);
                scol[j] = exp2i(e);
                rcol[j] = exp2i(-e);
                normal = normal && e > -127;
                if (floor_rule && floor_rule_saturates(m)) finite = false;   // take the saturating path
            } else if (m == 0x7F80u) {
                scol[j] = exp2i(127);
                rcol[j] = exp2i(-127);
                finite = false;
            } else {
                scol[j] = rcol[j] = __uint_as_float(0x7FC00000u);
                finite = false;
            }
        }
        uint2 ct[8];
        if (finite && normal) {
            // transpose the BF16 block first: each column then shares one
            // scale, and its codes come out in the transposed copy's order
            uint32_t wt[8][4];
            transpose8x8_b16(w, wt);
#pragma unroll
            for (int j = 0; j < 8; ++j) ct[j] = encode8_pow2<FMT>(wt[j], scol[j]);
        } else {
            uint2 c[8];
            if (finite) {
#pragma unroll
                for (int i = 0; i < 8; ++i) c[i] = encode8_cols<FMT, false>(w[i], rcol);
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) c[i] = encode8_cols<FMT, true>(w[i], rcol);
            }
            transpose8x8(c, ct);
        }
        store_transposed_ct(a, t, (int64_t)blockIdx.y * kTile, (int64_t)blockIdx.x * kTile, ct, tq);
        if (t.rg == 0 && t.col_ok) {
            const int64_t ng = a.rows / kTile;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                a.scaleT[a.kmajor ? (int64_t)blockIdx.y * a.cols + t.col + j : (t.col + j) * ng + blockIdx.y] = scol[j];
        }
    }
}

// One scale per 128x128 block; optional transposed copy with transposed scales.
template <int FMT>
__global__ __launch_bounds__(kThreads) void quant_block_kernel(QuantArgs a) {
    __shared__ uint32_t red[4];
    __shared__ __attribute__((aligned(16))) uint8_t tq[kTile * kTile];
    const Tile t = tile_coords(a.cols);
    uint32_t w[8][4];
    load_8x8<kSrcBf16>(a, t, w);
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) m = max(m, absmax_bits8(w[i]));
    m = block_max(m, red);
    float s;
    uint2 c[8];
    const bool floor_rule = a.pow2 == 2;
    if (m <= 0x7F7Fu) {
        const int e = pow2_exponent_bf16<FMT>(m, floor_rule);
        s = exp2i(e);
        const float r = exp2i(-e);
        if (floor_rule && floor_rule_saturates(m)) {
#pragma unroll
            for (int i = 0; i < 8; ++i) c[i] = encode8<FMT, true>(w[i], r);
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) c[i] = encode8<FMT, false>(w[i], r);
        }
    } else {
        const bool inf = m == 0x7F80u;
        s = inf ? exp2i(127) : __uint_as_float(0x7FC00000u);
        const float r = inf ? exp2i(-127) : s;
#pragma unroll
        for (int i = 0; i < 8; ++i) c[i] = encode8<FMT, true>(w[i], r);
    }
    store_rows(a, t, c);
    if (a.qT) store_transposed(a, t, (int64_t)blockIdx.y * kTile, (int64_t)blockIdx.x * kTile, c, tq);
    if (threadIdx.x == 0) {
        // block (by, bx) of q; scaleT holds the transposed copy's blocks
        const int64_t by = blockIdx.y, bx = blockIdx.x, nby = a.rows / kTile, nbx = a.cols / kTile;
        a.scale[a.kmajor ? bx * nby + by : by * nbx + bx] = s;
        if (a.scaleT) a.scaleT[a.kmajor ? by * nbx + bx : bx * nby + by] = s;
    }
}

template <int FMT, int SRC>
void launch_quantize_fmt(int mode, const QuantArgs& a, hipStream_t stream) {
    // at least one block, so that an empty tensor still gets its scale written
    const int64_t gx = (a.cols + kTile - 1) / kTile, gy = (a.rows + kTile - 1) / kTile;
    const dim3 grid((unsigned)(gx > 0 ? gx : 1), (unsigned)(gy > 0 ? gy : 1));
    switch (mode) {
    case kQTensor:
        quant_tensor_kernel<FMT, SRC><<<grid.x * grid.y, kThreads, 0, stream>>>(a, a, (int)(grid.x * grid.y),
                                                                              (int)grid.x, 1);
        break;
    case kQRow:
        if (a.qT) quant_groups_kernel<FMT, true, true, SRC><<<grid, kThreads, 0, stream>>>(a);
        else quant_groups_kernel<FMT, true, false, SRC><<<grid, kThreads, 0, stream>>>(a);
        break;
    case kQCol:
        quant_groups_kernel<FMT, false, true, SRC><<<grid, kThreads, 0, stream>>>(a);
        break;
    case kQBlock:
        if constexpr (SRC == kSrcBf16) quant_block_kernel<FMT><<<grid, kThreads, 0, stream>>>(a);
        break;
    }
}

}  // namespace

int amax_num_partials(int64_t rows, int64_t cols) {
    if (rows <= 0 || cols <= 0) return 0;
    const int64_t chunks = rows * (cols / 8);
    int64_t P = chunks / (kThreads * 8);    // ~8 vector loads per thread
    if (P < 1) P = 1;
    if (P > 4096) P = 4096;
    if (P > rows) P = rows;                 // whole rows per block
    return (int)P;
}

void launch_amax_partials(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                          uint32_t* partial, int P, hipStream_t stream, bool swiglu) {
    const AmaxJob j{x, rows, ld, partial, (uint32_t)(cols / 8), P};
    if (swiglu) amax_partial_kernel<false, kSrcSwiglu><<<P, kThreads, 0, stream>>>(j, j);
    else if (ld == cols) amax_partial_kernel<true, kSrcBf16><<<P, kThreads, 0, stream>>>(j, j);
    else amax_partial_kernel<false, kSrcBf16><<<P, kThreads, 0, stream>>>(j, j);
}

void launch_amax_finalize(const uint32_t* partial, int P, float* amax, hipStream_t stream) {
    amax_finalize_kernel<<<1, kThreads, 0, stream>>>(partial, P, amax);
}

void launch_quantize(int fmt, int mode, const QuantArgs& a, hipStream_t stream, bool swiglu) {
    if (swiglu) {
        if (fmt == kE4M3) launch_quantize_fmt<kE4M3, kSrcSwiglu>(mode, a, stream);
        else launch_quantize_fmt<kE5M2, kSrcSwiglu>(mode, a, stream);
    } else {
        if (fmt == kE4M3) launch_quantize_fmt<kE4M3, kSrcBf16>(mode, a, stream);
        else launch_quantize_fmt<kE5M2, kSrcBf16>(mode, a, stream);
    }
}

// Workspace: the partial maxima, then the amax scalar.
size_t quant_tensor_ws_bytes(int64_t rows, int64_t cols) {
    return ((size_t)amax_num_partials(rows, cols) * sizeof(uint32_t) + 255) / 256 * 256 + sizeof(float);
}

namespace {

// Amax source of a per-tensor quantisation whose partial maxima are in ws:
// reduced by every quantise block (few partials) or once by a one-block
// kernel into the amax slot of ws.
void amax_source(QuantArgs& a, int P, void* ws, hipStream_t stream) {
    uint32_t* partial = reinterpret_cast<uint32_t*>(ws);
    a.supplied = 0;
    if (P > kMaxInlinePartials) {
        float* amax = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(ws) + ((size_t)P * 4 + 255) / 256 * 256);
        launch_amax_finalize(partial, P, amax, stream);
        a.amax = amax;
    } else {
        // an empty tensor (P = 0) reduces to amax 0: scale 1
        a.amax = nullptr;
        a.partial = partial;
        a.npartial = P;
    }
}

int64_t tiles_x(int64_t cols) { const int64_t g = (cols + kTile - 1) / kTile; return g > 0 ? g : 1; }
int64_t tiles_y(int64_t rows) { const int64_t g = (rows + kTile - 1) / kTile; return g > 0 ? g : 1; }

}  // namespace

void launch_quantize_tensor(int fmt, QuantArgs a, void* ws, hipStream_t stream, bool swiglu) {
    const int P = amax_num_partials(a.rows, a.cols);
    if (P > 0) launch_amax_partials(a.x, a.rows, a.cols, a.ld, reinterpret_cast<uint32_t*>(ws), P, stream, swiglu);
    amax_source(a, P, ws, stream);
    launch_quantize(fmt, kQTensor, a, stream, swiglu);
}

void launch_quantize_tensor_pair(int fmt, QuantArgs a0, void* ws0, QuantArgs a1, void* ws1,
                                 hipStream_t stream) {
    const int P0 = amax_num_partials(a0.rows, a0.cols), P1 = amax_num_partials(a1.rows, a1.cols);
    const bool dense = a0.ld == a0.cols && a1.ld == a1.cols;
    if (P0 == 0 || P1 == 0 || P0 + P1 > (int64_t)INT32_MAX) {
        launch_quantize_tensor(fmt, a0, ws0, stream);
        launch_quantize_tensor(fmt, a1, ws1, stream);
        return;
    }
    const AmaxJob j0{a0.x, a0.rows, a0.ld, reinterpret_cast<uint32_t*>(ws0), (uint32_t)(a0.cols / 8), P0};
    const AmaxJob j1{a1.x, a1.rows, a1.ld, reinterpret_cast<uint32_t*>(ws1), (uint32_t)(a1.cols / 8), P1};
    if (dense) amax_partial_kernel<true, kSrcBf16><<<P0 + P1, kThreads, 0, stream>>>(j0, j1);
    else amax_partial_kernel<false, kSrcBf16><<<P0 + P1, kThreads, 0, stream>>>(j0, j1);
    amax_source(a0, P0, ws0, stream);
    amax_source(a1, P1, ws1, stream);
    const int64_t gx0 = tiles_x(a0.cols), gx1 = tiles_x(a1.cols);
    const int64_t t0 = gx0 * tiles_y(a0.rows), t1 = gx1 * tiles_y(a1.rows);
    const unsigned grid = (unsigned)(t0 + t1);
    if (fmt == kE4M3)
        quant_tensor_kernel<kE4M3, kSrcBf16><<<grid, kThreads, 0, stream>>>(a0, a1, (int)t0, (int)gx0, (int)gx1);
    else
        quant_tensor_kernel<kE5M2, kSrcBf16><<<grid, kThreads, 0, stream>>>(a0, a1, (int)t0, (int)gx0, (int)gx1);
}

size_t rmsnorm_ws_bytes(int64_t rows) {
    const int64_t P = rows > 0 ? (rows + 3) / 4 : 0;
    return ((size_t)P * sizeof(uint32_t) + 255) / 256 * 256 + sizeof(float);
}

void launch_rmsnorm_quantize(int fmt, int mode, QuantArgs a, float eps, void* ws, hipStream_t stream) {
    const int64_t P = a.rows > 0 ? (a.rows + 3) / 4 : 0;
    uint32_t* partial = reinterpret_cast<uint32_t*>(ws);
    if (P > 0) {
        if (mode == kQTensor)
            rmsnorm_rows_kernel<true><<<(unsigned)P, kThreads, 0, stream>>>(a.x, a.rows, a.cols, a.ld, a.gamma, eps,
                                                                           const_cast<float*>(a.rstd), partial);
        else
            rmsnorm_rows_kernel<false><<<(unsigned)P, kThreads, 0, stream>>>(a.x, a.rows, a.cols, a.ld, a.gamma, eps,
                                                                            const_cast<float*>(a.rstd), partial);
    }
    if (mode == kQTensor) amax_source(a, (int)P, ws, stream);
    if (fmt == kE4M3) launch_quantize_fmt<kE4M3, kSrcRmsnorm>(mode, a, stream);
    else launch_quantize_fmt<kE5M2, kSrcRmsnorm>(mode, a, stream);
}

size_t swiglu_bwd_ws_bytes(int64_t rows, int64_t cols) {
    const int64_t P = tiles_x(cols) * tiles_y(rows);
    return ((size_t)P * sizeof(uint32_t) + 255) / 256 * 256 + sizeof(float);
}

void launch_swiglu_bwd_quantize(int fmt, int mode, QuantArgs a, void* ws, hipStream_t stream) {
    if (mode == kQTensor) {
        const int64_t gx = tiles_x(a.cols), P = gx * tiles_y(a.rows);
        if (a.rows > 0 && a.cols > 0) {
            tile_amax_kernel<kSrcSwigluBwd><<<(unsigned)P, kThreads, 0, stream>>>(a, (int)gx,
                                                                                 reinterpret_cast<uint32_t*>(ws));
            amax_source(a, (int)P, ws, stream);
        } else {
            amax_source(a, 0, ws, stream);
        }
    }
    if (fmt == kE4M3) launch_quantize_fmt<kE4M3, kSrcSwigluBwd>(mode, a, stream);
    else launch_quantize_fmt<kE5M2, kSrcSwigluBwd>(mode, a, stream);
}

// ---- scratch for callers that cannot allocate ------------------------------
// puro_quantize_fp8_static keeps the per-tensor amax pass's partial maxima
// (and the reduced amax) here instead of in a caller workspace: a file-scope
// device array, one copy per GPU the library runs on, held until the process
// ends. Host code never passes the array's name to a kernel (there it is a
// host-side stand-in): it looks up each device's address once, with that
// device current, and passes that.
namespace {
__device__ __attribute__((aligned(256))) uint8_t scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;
}  // namespace

hipError_t static_scratch(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_ptr[dev].load(std::memory_order_acquire);
        if (!p) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (!p) return hipErrorInvalidSymbol;
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *ptr = p;
    return hipSuccess;
}

}  // namespace puro
