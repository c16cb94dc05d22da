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

constexpr int kBK = 128;                   // k block of the grouped scales (and of split-K ranges)
constexpr int kSL = 64;                    // bytes of k per pipeline slice
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
    uint32_t sa_bytes, sb_bytes;  // sizes of the scale arrays (grouped modes)
    int ksteps, ksteps_per_split, splits;
    int tiles_m, tiles_n;
    int accumulate;
    float alpha;               // host-known part of the per-tensor scale (1)
};

__device__ __forceinline__ uint32_t e8m0_of(float s) { return (__float_as_uint(s) >> 23) & 0xFFu; }

typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// Two FP32 values -> two BF16 (round to nearest even) in one word, low half
// first: the conversion instruction (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((v2f){a, b}, v2bf));
}
__device__ __forceinline__ uint16_t to_bf16(float a) { return (uint16_t)pack_bf16x2(a, 0.0f); }

typedef int v4i __attribute__((ext_vector_type(4)));

// Raw buffer descriptor (base, num_records bytes; 32-bit data format); every
// field is made wave-uniform so that it lives in SGPRs.
__device__ __forceinline__ v4i make_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = (uint64_t)base;
    v4i r;
    r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r.y = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xFFFFu));
    r.z = __builtin_amdgcn_readfirstlane((int)bytes);
    r.w = (int)kRsrcWord3;
    return r;
}

// LDS byte address of a __shared__ object (the value M0 takes for a DMA).
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
}

// Global -> LDS DMA of BYTES (16 or 4) per lane: lane l's data lands at
// LDS address lds + BYTES * l; offsets at or beyond the descriptor's
// num_records read as zero. Issued from inline assembly so that the
// compiler, which cannot tell which LDS bytes a DMA writes, does not make
// every later LDS read wait for it: the kernel waits explicitly
// (s_waitcnt vmcnt(0) + barrier) before reading a stage. M0 is saved and
// restored around the DMA (the compiler may keep a value there), and one wait
// state separates the M0 write from the DMA that reads it.
template <int BYTES>
__device__ __forceinline__ void dma_to_lds(v4i rsrc, uint32_t lds, uint32_t voff) {
    lds = (uint32_t)__builtin_amdgcn_readfirstlane((int)lds);   // wave-uniform by construction
    uint32_t saved;
    if constexpr (BYTES == 16)
        asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                     "buffer_load_dwordx4 %2, %3, 0 offen lds\n\ts_mov_b32 m0, %0"
                     : "=&s"(saved) : "s"(lds), "v"(voff), "s"(rsrc) : "memory");
    else
        asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                     "buffer_load_dword %2, %3, 0 offen lds\n\ts_mov_b32 m0, %0"
                     : "=&s"(saved) : "s"(lds), "v"(voff), "s"(rsrc) : "memory");
}

template <int BM, int BN, int WM, int WN, int FA, int FB, int OUT, bool GROUPED, int GM, int NST>
__global__ __launch_bounds__(WM * WN * 64) void gemm_fp8_kernel(Params p) {
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int A_BYTES = BM * kSL, B_BYTES = BN * kSL;
    constexpr int STAGE = A_BYTES + B_BYTES;        // one 64-byte k slice of both tiles
    // 1 KB DMA loads (16 rows of 64 bytes) per wave and slice; when the row
    // blocks do not divide evenly, the surplus loads repeat earlier blocks
    // (the same bytes to the same place), so every wave issues the same
    // number of loads and can wait on an exact count
    constexpr int A_BLK = BM / 16, B_BLK = BN / 16;
    constexpr int A_PER = (A_BLK + NW - 1) / NW, B_PER = (B_BLK + NW - 1) / NW;
    constexpr int SC_BLK = (BM + BN) / 64;          // 64 scales per 4-byte DMA load
    constexpr int LOADS = A_PER + B_PER + (GROUPED ? 1 : 0);
    static_assert(BM % 16 == 0 && BN % 16 == 0 && (BM + BN) % 64 == 0, "tile shape");
    static_assert(NST >= 3 && NST <= 4, "pipeline depth");

    __shared__ __attribute__((aligned(1024))) uint8_t smem[NST * STAGE];
    // grouped scales of a slice's rows (A then B), float, DMA'd like the operands
    __shared__ __attribute__((aligned(16))) float ssc[GROUPED ? NST * (BM + BN) : 1];

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
    // k slices [s0, s1) of 64 bytes: this split's 128-wide k blocks, twice
    const int s0 = 2 * ks * p.ksteps_per_split;
    const int s1 = 2 * min((ks + 1) * p.ksteps_per_split, p.ksteps);

    const int valid_m = min(BM, p.M - m0), valid_n = min(BN, p.N - n0);
    const v4i ra = make_rsrc(p.A + (int64_t)m0 * p.lda, (uint32_t)(valid_m * p.lda));
    const v4i rb = make_rsrc(p.B + (int64_t)n0 * p.ldb, (uint32_t)(valid_n * p.ldb));

    // LDS layout of a slice: row r of a tile is 64 bytes (four 16-byte chunks)
    // and its chunk c sits at position c ^ key(r), key(r) = ((r >> 1) & 3) ^
    // ((r >> 3) & 1). Among 16 consecutive rows the rows sharing a 64-byte
    // position in a 256-byte bank line get distinct keys, and so do the rows
    // of 8 consecutive rows sharing a position in a 128-byte line: the 16 (or
    // 8) lanes of a ds_read_b128 phase, reading consecutive rows at the same
    // logical chunk, hit distinct banks with 64 (or 32) four-byte banks.
    // Lane l of a DMA load fills row 16 * blk + l / 4 at position l % 4; since
    // blocks are 16 rows, key(row) = ((l >> 3) & 3) ^ ((l >> 5) & 1) for every
    // block, so each lane fetches one fixed chunk of its row.
    const int dkey = ((lane >> 3) & 3) ^ ((lane >> 5) & 1);
    const int kch = ((lane & 3) ^ dkey) * 16;
    const uint32_t rowA = (uint32_t)((lane >> 2) * p.lda), rowB = (uint32_t)((lane >> 2) * p.ldb);
    const uint32_t blkA = (uint32_t)(16 * p.lda), blkB = (uint32_t)(16 * p.ldb);
    const uint32_t smem_lds = lds_addr(smem);
    const uint32_t ssc_lds = lds_addr(ssc);

    v4i rsa{}, rsb{};
    if constexpr (GROUPED) {
        rsa = make_rsrc(p.sa, p.a_mode == kSTensor ? 0u : p.sa_bytes);
        rsb = make_rsrc(p.sb, p.b_mode == kSTensor ? 0u : p.sb_bytes);
    }

    // all LOADS DMA loads of slice `sl` into ring stage `st`
    auto load_slice = [&](int st, int sl) {
        const int k0 = sl * kSL;
        // the k tail (K % 64 != 0) reads out of range on purpose: zeros
        const uint32_t off = (k0 + kch < p.K) ? (uint32_t)(k0 + kch) : kOOB;
        const uint32_t sbase = smem_lds + st * STAGE;
#pragma unroll
        for (int q = 0; q < A_PER; ++q) {
            const int blk = (wave * A_PER + q) % A_BLK;
            dma_to_lds<16>(ra, sbase + blk * 1024, rowA + blk * blkA + off);
        }
#pragma unroll
        for (int q = 0; q < B_PER; ++q) {
            const int blk = (wave * B_PER + q) % B_BLK;
            dma_to_lds<16>(rb, sbase + A_BYTES + blk * 1024, rowB + blk * blkB + off);
        }
        if constexpr (GROUPED) {
            // lane l of scale load t brings the scale of tile row 64 t + l
            // (A rows, then B rows) for the 128-wide k block of the slice
            const int t = wave % SC_BLK;
            const int r = t * 64 + lane;
            const bool is_a = t * 64 < BM;
            const int row = is_a ? m0 + r : n0 + (r - BM);
            const int mode = is_a ? p.a_mode : p.b_mode;
            const int ld = is_a ? p.ld_sa : p.ld_sb;
            const int srow = mode == kSBlock ? row >> 7 : row;
            const uint32_t soff = (uint32_t)(srow * ld + (sl >> 1)) * 4u;
            const uint32_t dst = ssc_lds + (st * (BM + BN) + t * 64) * 4;
            dma_to_lds<4>(is_a ? rsa : rsb, dst, soff);
        }
    };

    v16f acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int fr = lane & 31;                 // fragment row of this lane
    const int c0 = (lane >> 5) * 2;           // this lane's two 16-byte chunks of a slice row
    // key of the lane's fragment rows (fragments start at multiples of 32)
    const int key = ((fr >> 1) & 3) ^ ((fr >> 3) & 1);
    const int pos0 = (c0 ^ key) << 4, pos1 = ((c0 + 1) ^ key) << 4;

    // prologue: slices s0 .. s0 + NST - 2 in flight
#pragma unroll
    for (int t = 0; t < NST - 1; ++t)
        if (s0 + t < s1) load_slice(t, s0 + t);

    for (int sl = s0; sl < s1; ++sl) {
        const int st = (sl - s0) % NST;
        // this wave's loads of slice sl are done once at most `later` slices
        // issued after it remain outstanding
        const int later = min(s1 - 1 - sl, NST - 2);
        if (later >= 2) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(2 * LOADS) : "memory");
        else if (later == 1) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(LOADS) : "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        // every wave's loads of slice sl have landed, and every wave is done
        // with slice sl - 1, whose stage the next load reuses
        __syncthreads();
        const uint8_t* sA = smem + st * STAGE;
        const uint8_t* sB = sA + A_BYTES;
        uint32_t scA[FM], scB[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i)
            scA[i] = (GROUPED && p.a_mode != kSTensor)
                         ? e8m0_of(ssc[st * (BM + BN) + wm * WTM + i * 32 + fr]) : 127u;
#pragma unroll
        for (int j = 0; j < FN; ++j)
            scB[j] = (GROUPED && p.b_mode != kSTensor)
                         ? e8m0_of(ssc[st * (BM + BN) + BM + wn * WTN + j * 32 + fr]) : 127u;
        v8i af[FM], bf[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const uint8_t* row = sA + (wm * WTM + i * 32 + fr) * kSL;
            const uint4 lo = *reinterpret_cast<const uint4*>(row + pos0);
            const uint4 hi = *reinterpret_cast<const uint4*>(row + pos1);
            af[i] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const uint8_t* row = sB + (wn * WTN + j * 32 + fr) * kSL;
            const uint4 lo = *reinterpret_cast<const uint4*>(row + pos0);
            const uint4 hi = *reinterpret_cast<const uint4*>(row + pos1);
            bf[j] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
        }
        if (sl + NST - 1 < s1) load_slice((st + NST - 1) % NST, sl + NST - 1);
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

    // ---- epilogue. Lane l holds, for fragment (i, j), wave-tile row
    // i*32 + (l & 31) and columns j*32 + 8g + 4(l >> 5) + {0..3}, g = 0..3.
    // Written straight to memory that would scatter 16-byte pieces over 32
    // rows per store; instead each wave stages its FP32 tile in its own part
    // of the (now idle) stage buffers, 16-byte chunks XOR-swizzled by row so
    // that both the writes and the row reads are free of bank conflicts, and
    // then stores whole rows: consecutive lanes on consecutive 16-byte chunks
    // (4 FP32 values), converted and scaled on the way out.
    float alpha = p.alpha;
    if (OUT != 2) {
        if (p.a_mode == kSTensor) alpha *= p.sa[0];
        if (p.b_mode == kSTensor) alpha *= p.sb[0];
    }
    constexpr int ROWB = WTN * 4;                 // bytes of one staged wave-tile row (FP32)
    constexpr int CPR = ROWB / 16;                // 16-byte chunks per row
    constexpr int REGION = NST * STAGE / NW;      // LDS bytes per wave
    constexpr int RFIT = (REGION / ROWB) / 32 * 32;
    constexpr int RPP = RFIT < WTM ? RFIT : WTM;  // rows per pass
    // XOR key of the chunk swizzle: 16 distinct keys when rows have 16*k chunks, else 8
    constexpr int SWZ = (CPR % 16 == 0) ? 15 : 7;
    static_assert(RPP >= 32 && WTM % RPP == 0 && (RPP * CPR) % 64 == 0, "epilogue tiling");
    static_assert(CPR % 8 == 0, "row swizzle needs 8k chunks per row");
    uint8_t* ep = smem + wave * REGION;
    const int mrow0 = m0 + wm * WTM;
    const int ncol0 = n0 + wn * WTN;
    float* const part = p.partial + (int64_t)ks * p.M * p.N;
    __syncthreads();   // every wave is done with the last stage
#pragma unroll
    for (int pass = 0; pass < WTM / RPP; ++pass) {
#pragma unroll
        for (int ii = 0; ii < RPP / 32; ++ii) {
            const int i = pass * (RPP / 32) + ii;
            const int r = ii * 32 + (lane & 31);
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int chunk = j * 8 + g * 2 + (lane >> 5);
                    float4 v = make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                           acc[i][j][4 * g + 3]);
                    *reinterpret_cast<float4*>(ep + r * ROWB + ((chunk ^ (r & SWZ)) << 4)) = v;
                }
        }
        __syncthreads();
#pragma unroll
        for (int it = 0; it < RPP * CPR / 64; ++it) {
            const int q = it * 64 + lane;
            const int r = q / CPR, c = q % CPR;
            float4 v = *reinterpret_cast<const float4*>(ep + r * ROWB + ((c ^ (r & SWZ)) << 4));
            const int m = mrow0 + pass * RPP + r;
            const int n = ncol0 + c * 4;
            if (m >= p.M || n >= p.N) continue;
            if constexpr (OUT == 2) {
                // split-K partial sums, dense [splits][M][N] FP32 (N % 4 == 0)
                *reinterpret_cast<float4*>(part + (int64_t)m * p.N + n) = v;
                continue;
            }
            v.x *= alpha; v.y *= alpha; v.z *= alpha; v.w *= alpha;
            if (n + 3 < p.N) {
                if constexpr (OUT == kOutF32) {
                    float4* dst = reinterpret_cast<float4*>(reinterpret_cast<float*>(p.D) + (int64_t)m * p.ldd + n);
                    if (p.accumulate) {
                        const float4 o = *dst;
                        v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
                    }
                    *dst = v;
                } else {
                    uint2* dst = reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(p.D) + (int64_t)m * p.ldd + n);
                    if (p.accumulate) {
                        const uint2 o = *dst;
                        v.x += bf16lo(o.x); v.y += bf16hi(o.x); v.z += bf16lo(o.y); v.w += bf16hi(o.y);
                    }
                    *dst = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
                }
            } else {
                // ragged right edge: element by element
                const float vv[4] = {v.x, v.y, v.z, v.w};
                for (int t = 0; t < 4 && n + t < p.N; ++t) {
                    if constexpr (OUT == kOutF32) {
                        float* dst = reinterpret_cast<float*>(p.D) + (int64_t)m * p.ldd + n + t;
                        *dst = p.accumulate ? *dst + vv[t] : vv[t];
                    } else {
                        uint16_t* dst = reinterpret_cast<uint16_t*>(p.D) + (int64_t)m * p.ldd + n + t;
                        *dst = to_bf16(p.accumulate ? vv[t] + __uint_as_float((uint32_t)*dst << 16) : vv[t]);
                    }
                }
            }
        }
        if (pass + 1 < WTM / RPP) __syncthreads();   // the next pass reuses the region
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
        *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(s.x, s.y), pack_bf16x2(s.z, s.w));
    }
}

// ---- tile configurations and the plan for a problem ---------------------------

struct Plan {
    int cfg;             // index into kTiles
    int bm, bn;          // tile
    int splits;          // k slices
    int ksteps_per_split;
};

struct TileCfg {
    int bm, bn;
    float eff;           // relative MFMA efficiency of the configuration
};
// 256x256 and 256x192: 8 waves (2 per SIMD) in a 4x2 grid (wave tiles 64x128,
// 64x96); 128x128: 4 waves in 2x2 (wave tiles 64x64) for small problems.
constexpr TileCfg kTiles[] = {{256, 256, 1.0f}, {256, 192, 0.95f}, {128, 128, 0.35f}};
constexpr int kCUs = 256;

// Pick the tile shape and the k split with the smallest estimated time: MFMA
// time of the waves of work units over the CUs, plus the traffic of split-K
// partial sums (written, then read by the reduction) when splitting.
Plan make_plan(int64_t M, int64_t N, int64_t K, int out) {
    const int ksteps = (int)((K + kBK - 1) / kBK);
    Plan best{0, 256, 256, 1, ksteps};
    double best_cost = -1.0;
    for (int c = 0; c < 3; ++c) {
        const TileCfg t = kTiles[c];
        const int64_t tiles = ((M + t.bm - 1) / t.bm) * ((N + t.bn - 1) / t.bn);
        if (tiles == 0) return best;
        const int max_s = (N % 4 == 0) ? (ksteps / 4 < 16 ? ksteps / 4 : 16) : 1;
        for (int s = 1; s <= (max_s > 1 ? max_s : 1); ++s) {
            const int kps = (ksteps + s - 1) / s;
            const int splits = kps > 0 ? (ksteps + kps - 1) / kps : 1;
            if (splits != s) continue;
            const int64_t units = tiles * splits;
            const int64_t waves = (units + kCUs - 1) / kCUs;
            // cycles: one k-step of a tile is bm*bn*128*2 FLOP at 8192 FLOP/clk
            double cost = (double)waves * t.bm * t.bn * (kps > 0 ? kps : 1) * 256.0 / 8192.0 / t.eff;
            if (splits > 1)   // partials written and read back, mostly in the 256 MB MALL (~8 KB/clk)
                cost += 2.0 * splits * (double)M * N * 4.0 / 8192.0;
            if (best_cost < 0 || cost < best_cost) {
                best_cost = cost;
                best = Plan{c, t.bm, t.bn, splits, kps};
            }
        }
    }
    (void)out;
    return best;
}

template <int BM, int BN, int WM, int WN, int FA, int FB, int OUT>
void launch_cfg(const Params& prm, bool grouped, int grid, hipStream_t stream) {
    constexpr int GM = 8;
    constexpr int NST = 4;
    if (grouped)
        gemm_fp8_kernel<BM, BN, WM, WN, FA, FB, OUT, true, GM, NST><<<grid, WM * WN * 64, 0, stream>>>(prm);
    else
        gemm_fp8_kernel<BM, BN, WM, WN, FA, FB, OUT, false, GM, NST><<<grid, WM * WN * 64, 0, stream>>>(prm);
}

template <int BM, int BN, int WM, int WN, int FA, int FB>
void launch_tile(const Params& prm, int out, bool grouped, int grid, hipStream_t stream) {
    if (out == 2) launch_cfg<BM, BN, WM, WN, FA, FB, 2>(prm, grouped, grid, stream);
    else if (out == kOutF32) launch_cfg<BM, BN, WM, WN, FA, FB, kOutF32>(prm, grouped, grid, stream);
    else launch_cfg<BM, BN, WM, WN, FA, FB, kOutBF16>(prm, grouped, grid, stream);
}

template <int FA, int FB>
void launch_fmt(const Params& prm, const Plan& pl, int out, bool grouped, int grid, hipStream_t stream) {
    if (pl.cfg == 0) launch_tile<256, 256, 4, 2, FA, FB>(prm, out, grouped, grid, stream);
    else if (pl.cfg == 1) launch_tile<256, 192, 4, 2, FA, FB>(prm, out, grouped, grid, stream);
    else launch_tile<128, 128, 2, 2, FA, FB>(prm, out, grouped, grid, stream);
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
    auto scale_bytes = [&](int mode, int64_t rows) -> uint32_t {
        if (mode == kSTensor) return 4u;
        const int64_t srows = mode == kSRow ? rows : (rows + 127) / 128;
        return (uint32_t)(srows * (g.K / kBK) * 4);
    };
    prm.sa_bytes = scale_bytes(g.sa_mode, g.M);
    prm.sb_bytes = scale_bytes(g.sb_mode, g.N);
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
