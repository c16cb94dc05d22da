// Scaled FP8 GEMM for gfx950: D[m, n] = sum_k A[m, k] * B[n, k].
//
// Section 3.2 of the paper runs the Fprop, Dgrad and Wgrad GEMMs of every
// linear layer on FP8 operands with higher-precision accumulation; operands
// carry a per-tensor scale or power-of-two scales per 128 values along k
// (per row, or per 128x128 block).
//
// Design (CDNA4):
//  * Both operands reduction-contiguous ("TN"); Dgrad and Wgrad are posed
//    this way by feeding the transposed FP8 copies the quantiser writes.
//  * Workgroup tile BM x BN, k-step 128 bytes (one 128-wide scale group).
//    Operand tiles are staged global -> LDS with buffer_load ... lds
//    (16 bytes per lane, no VGRP staging), double-buffered: the loads for
//    k-step t+1 are in flight while k-step t is multiplied.
//  * LDS rows are 128 bytes; the 16-byte chunk c of row r is stored at
//    position c ^ (r & 7), so the eight lanes of a ds_read_b128 phase hit
//    eight different 16-byte bank groups (conflict-free); the XOR is applied
//    on the global side because the DMA writes lane l at base + 16 l.
//  * v_mfma_scale_f32_32x32x64_f8f6f4: 32x32 outputs per 64-long k slice.
//    Grouped scales become the instruction's E8M0 operands (exact powers of
//    two, applied inside the MFMA); per-tensor scales multiply the FP32
//    result once in the epilogue. The instruction is issued with the B tile
//    as its first operand, so each lane's accumulators hold four consecutive
//    output columns of one row, stored as one 8-byte (BF16) or 16-byte
//    (FP32) vector.
//  * Out-of-range rows and the k tail are zero-filled by the buffer
//    descriptor's range check (num_records) rather than by branches.
//  * Tiles are remapped so the eight XCDs (workgroups are dealt round-robin
//    to them) each own a contiguous range of tiles, grouped by row panels to
//    share operand panels in that XCD's L2.
//  * Small grids split K into slices whose FP32 partial sums a second kernel
//    adds in a fixed order (deterministic).

#include "device_common.h"
#include "kernels.h"

namespace puro {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kBK = 128;                   // bytes of k per stage
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data format
constexpr uint32_t kOOB = 0x80000000u;     // offset that fails the range check

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
    int ld_sa, ld_sb;          // scale row pitch (K/128) for grouped modes
    int ksteps, ksteps_per_split, splits;
    int tiles_m, tiles_n;
    int accumulate;
    float alpha;               // host-known part of the per-tensor scale (1)
};

__device__ __forceinline__ uint32_t e8m0_of(float s) { return (__float_as_uint(s) >> 23) & 0xFFu; }

__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;  // quiet NaN
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

template <int BM, int BN, int WM, int WN, int FA, int FB, int OUT, bool GROUPED, int GM>
__global__ __launch_bounds__(WM * WN * 64) void gemm_fp8_kernel(Params p) {
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int A_BYTES = BM * kBK, B_BYTES = BN * kBK;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int A_LOADS = BM / 8 / NW, B_LOADS = BN / 8 / NW;   // 1 KB DMA loads per wave
    static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "tile / wave mismatch");

    __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WN, wn = wave % WN;

    // ---- tile index: contiguous ranges per XCD, grouped by GM row panels
    const int T = gridDim.x;
    const int b = blockIdx.x;
    const int lt = (T % 8 == 0) ? (b % 8) * (T / 8) + b / 8 : b;
    const int per_split = p.tiles_m * p.tiles_n;
    const int ks = lt / per_split;
    const int rem = lt - ks * per_split;
    const int group = rem / (GM * p.tiles_n);
    const int first_m = group * GM;
    const int gsz = min(GM, p.tiles_m - first_m);
    const int r2 = rem - group * GM * p.tiles_n;
    const int tm = first_m + r2 % gsz, tn = r2 / gsz;
    const int m0 = tm * BM, n0 = tn * BN;
    const int kb0 = ks * p.ksteps_per_split;
    const int kb1 = min(kb0 + p.ksteps_per_split, p.ksteps);

    const int valid_m = min(BM, p.M - m0), valid_n = min(BN, p.N - n0);
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.A + (int64_t)m0 * p.lda), 0, (int)(valid_m * p.lda), kRsrcWord3);
    const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.B + (int64_t)n0 * p.ldb), 0, (int)(valid_n * p.ldb), kRsrcWord3);

    // per-lane source offsets of the DMA loads. Lane l of DMA load q fills
    // LDS row (wave * LOADS + q) * 8 + l / 8 at chunk position l % 8, so it
    // fetches source chunk (l % 8) ^ (row & 7) = (l % 8) ^ (l / 8).
    const int lrow = lane >> 3;
    const int kch = ((lane & 7) ^ lrow) * 16;
    const uint32_t baseA = (uint32_t)((wave * A_LOADS * 8 + lrow) * p.lda) + kch;
    const uint32_t baseB = (uint32_t)((wave * B_LOADS * 8 + lrow) * p.ldb) + kch;
    const uint32_t stepA = (uint32_t)(8 * p.lda), stepB = (uint32_t)(8 * p.ldb);

    auto load_stage = [&](int stage, int kb) {
        const int k0 = kb * kBK;
        const bool kin = k0 + kch < p.K;
        uint8_t* sA = smem + stage * STAGE;
        uint8_t* sB = sA + A_BYTES;
#pragma unroll
        for (int q = 0; q < A_LOADS; ++q) {
            const uint32_t off = kin ? baseA + q * stepA + k0 : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void_t*)(sA + (wave * A_LOADS + q) * 1024),
                                                     16, off, 0, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < B_LOADS; ++q) {
            const uint32_t off = kin ? baseB + q * stepB + k0 : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void_t*)(sB + (wave * B_LOADS + q) * 1024),
                                                     16, off, 0, 0, 0);
        }
    };

    // grouped scales: E8M0 of the lane's A row (per fragment i) and B row (per j)
    int rowA[FM], rowB[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) rowA[i] = min(m0 + wm * WTM + i * 32 + (lane & 31), p.M - 1);
#pragma unroll
    for (int j = 0; j < FN; ++j) rowB[j] = min(n0 + wn * WTN + j * 32 + (lane & 31), p.N - 1);
    uint32_t scA[FM], scB[FN];
    auto load_scales = [&](int kb) {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            if (p.a_mode == kSTensor) scA[i] = 127u;
            else {
                const int r = p.a_mode == kSRow ? rowA[i] : rowA[i] >> 7;
                scA[i] = e8m0_of(p.sa[(int64_t)r * p.ld_sa + kb]);
            }
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            if (p.b_mode == kSTensor) scB[j] = 127u;
            else {
                const int r = p.b_mode == kSRow ? rowB[j] : rowB[j] >> 7;
                scB[j] = e8m0_of(p.sb[(int64_t)r * p.ld_sb + kb]);
            }
        }
    };

    v16f acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // LDS read addresses of the fragments (row within the stage, swizzle key)
    const int fr = lane & 31;           // fragment row of this lane
    const int khalf = (lane >> 5) * 2;  // first of this lane's two 16-byte chunks in a 64-byte slice

    if (kb0 < kb1) load_stage(0, kb0);
    for (int kb = kb0; kb < kb1; ++kb) {
        const int stage = (kb - kb0) & 1;
        if constexpr (GROUPED) load_scales(kb);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (kb + 1 < kb1) load_stage(stage ^ 1, kb + 1);
        const uint8_t* sA = smem + stage * STAGE;
        const uint8_t* sB = sA + A_BYTES;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            v8i af[FM], bf[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int r = wm * WTM + i * 32 + fr;
                const uint8_t* row = sA + r * kBK;
                const int c0 = kk * 4 + khalf;
                const uint4 lo = *reinterpret_cast<const uint4*>(row + ((c0 ^ (r & 7)) << 4));
                const uint4 hi = *reinterpret_cast<const uint4*>(row + (((c0 + 1) ^ (r & 7)) << 4));
                af[i] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int r = wn * WTN + j * 32 + fr;
                const uint8_t* row = sB + r * kBK;
                const int c0 = kk * 4 + khalf;
                const uint4 lo = *reinterpret_cast<const uint4*>(row + ((c0 ^ (r & 7)) << 4));
                const uint4 hi = *reinterpret_cast<const uint4*>(row + (((c0 + 1) ^ (r & 7)) << 4));
                bf[j] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    if constexpr (GROUPED)
                        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                            bf[j], af[i], acc[i][j], FB, FA, 0, (int)scB[j], 0, (int)scA[i]);
                    else
                        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                            bf[j], af[i], acc[i][j], FB, FA, 0, 127, 0, 127);
                }
        }
    }

    // ---- epilogue: lane holds, for fragment (i, j), output row
    // m = i*32 + (lane & 31) and columns n = j*32 + 8 g + 4 (lane >> 5) + {0..3}
    float alpha = p.alpha;
    if (OUT != 2) {
        if (p.a_mode == kSTensor) alpha *= p.sa[0];
        if (p.b_mode == kSTensor) alpha *= p.sb[0];
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int m = m0 + wm * WTM + i * 32 + (lane & 31);
        if (m >= p.M) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = n0 + wn * WTN + j * 32 + g * 8 + (lane >> 5) * 4;
                if (n >= p.N) continue;
                float v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1];
                float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
                if constexpr (OUT == 2) {
                    // split-K partial sums, dense [splits][M][N] FP32 (N % 4 == 0)
                    float* dst = p.partial + ((int64_t)ks * p.M + m) * p.N + n;
                    *reinterpret_cast<float4*>(dst) = make_float4(v0, v1, v2, v3);
                } else {
                    v0 *= alpha; v1 *= alpha; v2 *= alpha; v3 *= alpha;
                    const bool full = n + 3 < p.N;
                    if constexpr (OUT == kOutF32) {
                        float* dst = reinterpret_cast<float*>(p.D) + (int64_t)m * p.ldd + n;
                        if (full) {
                            if (p.accumulate) {
                                const float4 o = *reinterpret_cast<const float4*>(dst);
                                v0 += o.x; v1 += o.y; v2 += o.z; v3 += o.w;
                            }
                            *reinterpret_cast<float4*>(dst) = make_float4(v0, v1, v2, v3);
                        } else {
                            const float vv[4] = {v0, v1, v2, v3};
                            for (int t = 0; t < 4 && n + t < p.N; ++t)
                                dst[t] = p.accumulate ? dst[t] + vv[t] : vv[t];
                        }
                    } else {
                        uint16_t* dst = reinterpret_cast<uint16_t*>(p.D) + (int64_t)m * p.ldd + n;
                        if (full) {
                            if (p.accumulate) {
                                const uint2 o = *reinterpret_cast<const uint2*>(dst);
                                v0 += bf16lo(o.x); v1 += bf16hi(o.x); v2 += bf16lo(o.y); v3 += bf16hi(o.y);
                            }
                            const uint2 w = make_uint2(f32_to_bf16(v0) | (f32_to_bf16(v1) << 16),
                                                       f32_to_bf16(v2) | (f32_to_bf16(v3) << 16));
                            *reinterpret_cast<uint2*>(dst) = w;
                        } else {
                            const float vv[4] = {v0, v1, v2, v3};
                            for (int t = 0; t < 4 && n + t < p.N; ++t) {
                                float v = vv[t];
                                if (p.accumulate) v += __uint_as_float((uint32_t)dst[t] << 16);
                                dst[t] = (uint16_t)f32_to_bf16(v);
                            }
                        }
                    }
                }
            }
        }
    }
}

// Fixed-order sum of the split-K partials, scaling and output conversion.
template <int OUT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ partial, int splits,
                                                            int M, int N, const float* sa, const float* sb,
                                                            int a_tensor, int b_tensor, void* D,
                                                            int64_t ldd, int accumulate) {
    const int64_t nq = N / 4;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)M * nq) return;
    const int64_t m = idx / nq;
    const int n = (int)(idx - m * nq) * 4;
    float alpha = 1.0f;
    if (a_tensor) alpha *= sa[0];
    if (b_tensor) alpha *= sb[0];
    float4 s = *reinterpret_cast<const float4*>(partial + m * N + n);
    for (int k = 1; k < splits; ++k) {
        const float4 t = *reinterpret_cast<const float4*>(partial + ((int64_t)k * M + m) * N + n);
        s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
    }
    s.x *= alpha; s.y *= alpha; s.z *= alpha; s.w *= alpha;
    if constexpr (OUT == kOutF32) {
        float* dst = reinterpret_cast<float*>(D) + m * ldd + n;
        if (accumulate) {
            const float4 o = *reinterpret_cast<const float4*>(dst);
            s.x += o.x; s.y += o.y; s.z += o.z; s.w += o.w;
        }
        *reinterpret_cast<float4*>(dst) = s;
    } else {
        uint16_t* dst = reinterpret_cast<uint16_t*>(D) + m * ldd + n;
        if (accumulate) {
            const uint2 o = *reinterpret_cast<const uint2*>(dst);
            s.x += bf16lo(o.x); s.y += bf16hi(o.x); s.z += bf16lo(o.y); s.w += bf16hi(o.y);
        }
        *reinterpret_cast<uint2*>(dst) = make_uint2(f32_to_bf16(s.x) | (f32_to_bf16(s.y) << 16),
                                                    f32_to_bf16(s.z) | (f32_to_bf16(s.w) << 16));
    }
}

// ---- tile configurations and the plan for a problem ---------------------------

struct Plan {
    int bm, bn;          // tile
    int splits;          // k slices
    int ksteps_per_split;
};

constexpr int kCUs = 256;

Plan make_plan(int64_t M, int64_t N, int64_t K, int out) {
    const int ksteps = (int)((K + kBK - 1) / kBK);
    Plan best{256, 256, 1, ksteps};
    const int64_t big_tiles = ((M + 255) / 256) * ((N + 255) / 256);
    if (big_tiles < kCUs / 2) {
        const int64_t small_tiles = ((M + 127) / 128) * ((N + 127) / 128);
        if (small_tiles > big_tiles) best = Plan{128, 128, 1, ksteps};
    }
    const int64_t tiles = ((M + best.bm - 1) / best.bm) * ((N + best.bn - 1) / best.bn);
    if (tiles == 0) return best;
    // split K when the grid covers well under the CUs and the k range is long
    // enough; split-K needs N % 4 == 0 for the vector partials
    if (tiles < kCUs / 2 && ksteps >= 8 && (N % 4) == 0) {
        int s = (int)((kCUs + tiles - 1) / tiles);
        if (s > ksteps / 4) s = ksteps / 4;
        if (s > 16) s = 16;
        if (s > 1) {
            best.ksteps_per_split = (ksteps + s - 1) / s;
            best.splits = (ksteps + best.ksteps_per_split - 1) / best.ksteps_per_split;
        }
    }
    (void)out;
    return best;
}

template <int BM, int BN, int WM, int WN, int FA, int FB, int OUT>
void launch_cfg(const Params& prm, bool grouped, int grid, hipStream_t stream) {
    constexpr int GM = 8;
    if (grouped)
        gemm_fp8_kernel<BM, BN, WM, WN, FA, FB, OUT, true, GM><<<grid, WM * WN * 64, 0, stream>>>(prm);
    else
        gemm_fp8_kernel<BM, BN, WM, WN, FA, FB, OUT, false, GM><<<grid, WM * WN * 64, 0, stream>>>(prm);
}

template <int BM, int BN, int FA, int FB>
void launch_tile(const Params& prm, int out, bool grouped, int grid, hipStream_t stream) {
    if (out == 2) launch_cfg<BM, BN, 2, 2, FA, FB, 2>(prm, grouped, grid, stream);
    else if (out == kOutF32) launch_cfg<BM, BN, 2, 2, FA, FB, kOutF32>(prm, grouped, grid, stream);
    else launch_cfg<BM, BN, 2, 2, FA, FB, kOutBF16>(prm, grouped, grid, stream);
}

template <int FA, int FB>
void launch_fmt(const Params& prm, const Plan& pl, int out, bool grouped, int grid, hipStream_t stream) {
    if (pl.bm == 256) launch_tile<256, 256, FA, FB>(prm, out, grouped, grid, stream);
    else launch_tile<128, 128, FA, FB>(prm, out, grouped, grid, stream);
}

}  // namespace

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int out) {
    const Plan pl = make_plan(M, N, K, out);
    if (pl.splits <= 1) return 0;
    return (size_t)pl.splits * (size_t)M * (size_t)N * sizeof(float);
}

void launch_gemm(const GemmProblem& g, void* ws, hipStream_t stream) {
    const Plan pl = make_plan(g.M, g.N, g.K, g.out);
    Params prm{};
    prm.A = g.A; prm.B = g.B; prm.sa = g.sa; prm.sb = g.sb;
    prm.D = g.D; prm.partial = reinterpret_cast<float*>(ws);
    prm.lda = g.lda; prm.ldb = g.ldb; prm.ldd = g.ldd;
    prm.M = (int)g.M; prm.N = (int)g.N; prm.K = (int)g.K;
    prm.a_mode = g.sa_mode; prm.b_mode = g.sb_mode;
    prm.ld_sa = (int)(g.K / kBK); prm.ld_sb = (int)(g.K / kBK);
    prm.ksteps = (int)((g.K + kBK - 1) / kBK);
    prm.ksteps_per_split = pl.ksteps_per_split;
    prm.splits = pl.splits;
    prm.tiles_m = (int)((g.M + pl.bm - 1) / pl.bm);
    prm.tiles_n = (int)((g.N + pl.bn - 1) / pl.bn);
    prm.accumulate = g.accumulate;
    prm.alpha = 1.0f;
    const bool grouped = g.sa_mode != kSTensor || g.sb_mode != kSTensor;
    const int out = pl.splits > 1 ? 2 : g.out;
    const int grid = prm.tiles_m * prm.tiles_n * pl.splits;
    if (g.fa == kE4M3 && g.fb == kE4M3) launch_fmt<kE4M3, kE4M3>(prm, pl, out, grouped, grid, stream);
    else if (g.fa == kE5M2 && g.fb == kE4M3) launch_fmt<kE5M2, kE4M3>(prm, pl, out, grouped, grid, stream);
    else if (g.fa == kE4M3 && g.fb == kE5M2) launch_fmt<kE4M3, kE5M2>(prm, pl, out, grouped, grid, stream);
    else launch_fmt<kE5M2, kE5M2>(prm, pl, out, grouped, grid, stream);
    if (pl.splits > 1) {
        const int64_t n = g.M * (g.N / 4);
        const int blocks = (int)((n + 255) / 256);
        if (g.out == kOutF32)
            splitk_reduce_kernel<kOutF32><<<blocks, 256, 0, stream>>>(
                prm.partial, pl.splits, prm.M, prm.N, g.sa, g.sb, g.sa_mode == kSTensor,
                g.sb_mode == kSTensor, g.D, g.ldd, g.accumulate);
        else
            splitk_reduce_kernel<kOutBF16><<<blocks, 256, 0, stream>>>(
                prm.partial, pl.splits, prm.M, prm.N, g.sa, g.sb, g.sa_mode == kSTensor,
                g.sb_mode == kSTensor, g.D, g.ldd, g.accumulate);
    }
}

}  // namespace puro
