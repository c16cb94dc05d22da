// BF16 matrix transpose (gfx950), for the operands whose reduction runs down
// their columns: the LM head's backward GEMMs and the Newton-Schulz update.

#include <hip/hip_runtime.h>

#include "kernels.h"

namespace puro {

namespace {

constexpr int kT = 64;   // tile edge

// dst [C, R] (pitch ldd) = src [R, C] (pitch lds) of problem blockIdx.z; 64 x
// 64 tiles through LDS (one padding column keeps the column reads on distinct
// banks), 256 threads, each moving 16 elements.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ src, int64_t R, int64_t C,
                                                             int64_t lds, uint16_t* __restrict__ dst, int64_t ldd,
                                                             int64_t bs_src, int64_t bs_dst) {
    __shared__ uint16_t t[kT][kT + 2];
    src += blockIdx.z * bs_src;
    dst += blockIdx.z * bs_dst;
    const int64_t r0 = (int64_t)blockIdx.y * kT, c0 = (int64_t)blockIdx.x * kT;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
#pragma unroll
    for (int i = 0; i < kT; i += 4) {
        const int64_t r = r0 + ty + i, c = c0 + tx;
        t[ty + i][tx] = (r < R && c < C) ? src[r * lds + c] : (uint16_t)0;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kT; i += 4) {
        const int64_t c = c0 + ty + i, r = r0 + tx;
        if (c < C && r < R) dst[c * ldd + r] = t[tx][ty + i];
    }
}

}  // namespace

void transpose_bf16(const uint16_t* src, int64_t R, int64_t C, int64_t lds, uint16_t* dst, int64_t ldd,
                    hipStream_t stream, int batch, int64_t bs_src, int64_t bs_dst) {
    if (R <= 0 || C <= 0 || batch <= 0) return;
    const dim3 grid((unsigned)((C + kT - 1) / kT), (unsigned)((R + kT - 1) / kT), (unsigned)batch);
    transpose_bf16_kernel<<<grid, 256, 0, stream>>>(src, R, C, lds, dst, ldd, bs_src, bs_dst);
}

}  // namespace puro
