// BF16 matrix transpose (gfx950), for the operands whose reduction runs down
// their columns: the LM head's backward GEMMs and the Newton-Schulz update.

#include <hip/hip_runtime.h>

#include "kernels.h"

namespace puro {

namespace {

constexpr int kT = 64;   // tile edge

// dst [C, R] (pitch ldd) = src [R, C] (pitch lds) of problem blockIdx.z, in
// 64 x 64 tiles; R, C and both pitches are multiples of 8 (a 16-byte chunk
// never straddles an edge). Each thread moves two 16-byte chunks in and two
// out. The tile sits in LDS as 64 rows of 33 words (one padding word): a
// wave's column reads (8 source rows x 8 columns, the lanes' chunks) then
// fall on 32 distinct banks, two lanes sharing each word.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ src, int64_t R, int64_t C,
                                                             int64_t lds, uint16_t* __restrict__ dst, int64_t ldd,
                                                             int64_t bs_src, int64_t bs_dst) {
    constexpr int kW = kT / 2 + 1;       // words per LDS row
    __shared__ uint32_t t[kT * kW];
    src += blockIdx.z * bs_src;
    dst += blockIdx.z * bs_dst;
    const int64_t r0 = (int64_t)blockIdx.y * kT, c0 = (int64_t)blockIdx.x * kT;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int q = threadIdx.x + 256 * k;
        const int row = q >> 3, ch = q & 7;
        const int64_t r = r0 + row, c = c0 + ch * 8;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (r < R && c < C) v = *reinterpret_cast<const uint4*>(src + r * lds + c);
        uint32_t* w = t + row * kW + ch * 4;
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int q = threadIdx.x + 256 * k;
        const int cc = q >> 3, ch = q & 7;   // destination row c0 + cc, source rows r0 + 8 ch ..
        const int64_t c = c0 + cc, r = r0 + ch * 8;
        uint32_t e[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t word = t[(ch * 8 + i) * kW + (cc >> 1)];
            e[i] = (cc & 1) ? (word >> 16) : (word & 0xFFFFu);
        }
        if (c < C && r < R)
            *reinterpret_cast<uint4*>(dst + c * ldd + r) =
                make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16));
    }
}

// The lower tiles of a symmetric matrix from the upper ones: destination
// tile (blockIdx.y, blockIdx.x) of 64 x 64 takes the transpose of tile
// (blockIdx.x, blockIdx.y) when its rows lie in a tg-tile below the diagonal
// one of its columns (the tiles a GEMM computing only its upper tiles left
// unwritten); other blocks exit at once. Staged through LDS as above.
__global__ __launch_bounds__(256) void mirror_lower_bf16_kernel(uint16_t* __restrict__ A, int64_t ld, int tg,
                                                                int64_t bs) {
    const int64_t r0 = (int64_t)blockIdx.y * kT, c0 = (int64_t)blockIdx.x * kT;
    if (r0 / tg <= c0 / tg) return;
    constexpr int kW = kT / 2 + 1;
    __shared__ uint32_t t[kT * kW];
    A += blockIdx.z * bs;
    // source: rows c0.., columns r0.. (the transposed position, in the upper tiles)
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int q = threadIdx.x + 256 * k;
        const int row = q >> 3, ch = q & 7;
        const uint4 v = *reinterpret_cast<const uint4*>(A + (c0 + row) * ld + r0 + ch * 8);
        uint32_t* w = t + row * kW + ch * 4;
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int q = threadIdx.x + 256 * k;
        const int cc = q >> 3, ch = q & 7;   // destination row r0 + cc, source rows c0 + 8 ch ..
        uint32_t e[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t word = t[(ch * 8 + i) * kW + (cc >> 1)];
            e[i] = (cc & 1) ? (word >> 16) : (word & 0xFFFFu);
        }
        *reinterpret_cast<uint4*>(A + (r0 + cc) * ld + c0 + ch * 8) =
            make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16));
    }
}

}  // namespace

void transpose_bf16(const uint16_t* src, int64_t R, int64_t C, int64_t lds, uint16_t* dst, int64_t ldd,
                    hipStream_t stream, int batch, int64_t bs_src, int64_t bs_dst) {
    if (R <= 0 || C <= 0 || batch <= 0) return;
    const dim3 grid((unsigned)((C + kT - 1) / kT), (unsigned)((R + kT - 1) / kT), (unsigned)batch);
    transpose_bf16_kernel<<<grid, 256, 0, stream>>>(src, R, C, lds, dst, ldd, bs_src, bs_dst);
}

void mirror_lower_bf16(uint16_t* A, int64_t R, int64_t ld, int tg, hipStream_t stream, int batch, int64_t bs) {
    if (R <= 0 || batch <= 0) return;
    const dim3 grid((unsigned)(R / kT), (unsigned)(R / kT), (unsigned)batch);
    mirror_lower_bf16_kernel<<<grid, 256, 0, stream>>>(A, ld, tg, bs);
}

}  // namespace puro
