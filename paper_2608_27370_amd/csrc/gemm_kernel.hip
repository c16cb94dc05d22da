// Scaled FP8 GEMM kernel for gfx950: D[m, n] = sum_k A[m, k] * B[n, k].
//
// Section 3.2 of the paper runs the Fprop, Dgrad and Wgrad GEMMs of every
// linear layer on FP8 operands with higher-precision accumulation; operands
// carry a per-tensor scale or power-of-two scales per 128 values along k
// (per row, or per 128x128 block).
//
// Design (CDNA4):
//  * Both operands reduction-contiguous ("TN"); Dgrad and Wgrad are posed
//    this way by feeding the transposed FP8 copies the quantiser writes.
//  * Four waves per workgroup, one per SIMD, in a 2x2 grid; workgroup tiles
//    up to 256x256 (wave tiles up to 128x128, accumulators in AGPRs).
//  * Operand tiles move global -> LDS by buffer_load ... lds (16 bytes per
//    lane, no VGPR staging) in k slices of SL = 128 bytes: one 1 KB DMA load
//    covers 8 rows x 128 bytes, whole cache lines. A ring of NST slices
//    keeps the next ones in flight while one is multiplied.
//  * Within a slice the wave works in 64-byte k steps; the fragments of
//    the next step are read from LDS into a second register set while the
//    MFMAs of the current one run, and the DMA loads are spread between
//    the MFMAs too. The loop body has no branches and waits on constant
//    counts; one barrier per slice.
//  * LDS rows are XOR-swizzled in 16-byte chunks (conflict-free reads; the
//    swizzle is applied on the global side because the DMA writes lane l at
//    base + 16 l).
//  * v_mfma_scale_f32_32x32x64_f8f6f4: 32x32 outputs per 64-long k step.
//    Grouped scales become the instruction's E8M0 operands (exact powers of
//    two, applied inside the MFMA); per-tensor scales multiply the FP32
//    result once in the epilogue. The instruction is issued with the B tile
//    as its first operand, so each lane's accumulators hold four consecutive
//    output columns of one row.
//  * Out-of-range rows and the k tail are zero-filled by the buffer
//    descriptor's range check (num_records) rather than by branches.
//  * Tiles are remapped so the eight XCDs (workgroups are dealt round-robin
//    to them) each own a contiguous range of tiles, grouped by row panels to
//    share operand panels in that XCD's L2.
//  * The epilogue stages each wave's FP32 tile in the idle ring and stores
//    whole rows; interior tiles take a branch-free path that issues all LDS
//    reads of a pass before its stores.
//  * Small grids split K into ranges whose FP32 partial sums a second kernel
//    adds in a fixed order (deterministic).

// This file is compiled once per operand-format pair and scale kind
// (PURO_FA, PURO_FB, PURO_GROUPED), each object holding that variant's tile
// configurations and output kinds.

#include <climits>
#include <type_traits>

#include "device_common.h"
#include "gemm_common.h"
#include "kernels.h"

#if !defined(PURO_FA) || !defined(PURO_FB) || !defined(PURO_GROUPED)
#error "gemm_kernel.hip is compiled with -DPURO_FA=<0|1> -DPURO_FB=<0|1> -DPURO_GROUPED=<0|1>"
#endif

namespace puro {
namespace gemm_detail {

namespace {


typedef int v8i __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data format
constexpr uint32_t kOOB = 0x80000000u;     // offset that fails the range check


// f(std::integral_constant<int, i>) for i = 0 .. N-1, each call with its own
// compile-time index (no loop left for the unroller to decide on).
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<N, I + 1>(f);
    }
}

constexpr int cgcd(int a, int b) { return b == 0 ? a : cgcd(b, a % b); }



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

// dz's E4M3 copies from a wave's staged 128 x 128 BF16 tile (row r at
// ep + 256 r, its 16-byte chunk c at position c ^ (r & 15)), for the LM
// head's backward: the same codes and power-of-two scales as the 1x128 +
// 128x1 quantiser gives for that BF16 dz (its groups are 128-aligned, so
// each lies in one wave tile), written where the dX and dW GEMMs read them.
//  * rows: lane l quantises staged rows l and l + 64, each one 1x128 group;
//  * columns: lane l takes 8 columns (chunk c = l & 15) over the row blocks
//    of 8 rows b = (l >> 4) + 4 k; the 4 lanes of a chunk share the column
//    maxima through two shuffles, each 8 x 8 block is transposed in
//    registers and its 8 columns' codes go to the transposed copy.
__device__ __forceinline__ void quantize_staged_dz(const Params& p, const uint8_t* ep, int64_t mrow0, int64_t ncol0,
                                                   int lane) {
    typedef unsigned int v4u __attribute__((ext_vector_type(4)));
    constexpr int F = kE4M3;
    const int64_t M = p.M, N = p.N;
    auto chunk = [&](int r, int c) __attribute__((always_inline)) {
        return *reinterpret_cast<const v4u*>(ep + r * 256 + ((c ^ (r & 15)) << 4));
    };
    // ---- rows
    const __amdgpu_buffer_rsrc_t rq =
        __builtin_amdgcn_make_buffer_rsrc(p.q8 + mrow0 * N + ncol0, 0, (int)(127 * N + 128), 0x00020000);
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
        const int r = lane + 64 * rr;
        uint32_t w[16][4];
        uint32_t m = 0;
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            const v4u v = chunk(r, c);
            w[c][0] = v.x; w[c][1] = v.y; w[c][2] = v.z; w[c][3] = v.w;
            m = max(m, absmax_bits8(w[c]));
        }
        float s;
        uint2 q[16];
        if (m <= 0x7F7Fu) {
            const int e = pow2_exponent_bf16<F>(m);
            s = exp2i(e);
            if (e > -127) {
#pragma unroll
                for (int c = 0; c < 16; ++c) q[c] = encode8_pow2<F>(w[c], s);
            } else {
#pragma unroll
                for (int c = 0; c < 16; ++c) q[c] = encode8<F, false>(w[c], exp2i(-e));
            }
        } else {
            // an infinity: the largest scale, saturated codes; a NaN: NaN scale and codes
            const bool inf = m == 0x7F80u;
            s = inf ? exp2i(127) : __uint_as_float(0x7FC00000u);
            const float rinv = inf ? exp2i(-127) : s;
#pragma unroll
            for (int c = 0; c < 16; ++c) q[c] = encode8<F, true>(w[c], rinv);
        }
#pragma unroll
        for (int c = 0; c < 16; c += 2)
            __builtin_amdgcn_raw_buffer_store_b128(v4u{q[c].x, q[c].y, q[c + 1].x, q[c + 1].y}, rq,
                                                   (int)(r * N + c * 8), 0, 0);
        p.q8_scale[(ncol0 / 128) * M + mrow0 + r] = s;
    }
    // ---- columns
    const int cb = lane & 15, b0 = lane >> 4;
    uint32_t cm[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const v4u v = chunk((b0 + 4 * k) * 8 + i, cb);
            cm[0] = pk_max_u16(cm[0], mag2(v.x)); cm[1] = pk_max_u16(cm[1], mag2(v.y));
            cm[2] = pk_max_u16(cm[2], mag2(v.z)); cm[3] = pk_max_u16(cm[3], mag2(v.w));
        }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        cm[j] = pk_max_u16(cm[j], (uint32_t)__shfl_xor((int)cm[j], 16, 64));
        cm[j] = pk_max_u16(cm[j], (uint32_t)__shfl_xor((int)cm[j], 32, 64));
    }
    float scol[8], rcol[8];
    bool finite = true, normal = true;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t m = (j & 1) ? (cm[j >> 1] >> 16) : (cm[j >> 1] & 0xFFFFu);
        if (m <= 0x7F7Fu) {
            const int e = pow2_exponent_bf16<F>(m);
            scol[j] = exp2i(e);
            rcol[j] = exp2i(-e);
            normal = normal && e > -127;
        } else if (m == 0x7F80u) {
            scol[j] = exp2i(127);
            rcol[j] = exp2i(-127);
            finite = false;
        } else {
            scol[j] = rcol[j] = __uint_as_float(0x7FC00000u);
            finite = false;
        }
    }
    // the transposed copy's rows ncol0 + 8 cb + j hold columns mrow0 + 8 b + (0..7)
    const __amdgpu_buffer_rsrc_t rt =
        __builtin_amdgcn_make_buffer_rsrc(p.q8t + ncol0 * M + mrow0, 0, (int)(127 * M + 128), 0x00020000);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int b = b0 + 4 * k;
        uint32_t w[8][4];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const v4u v = chunk(b * 8 + i, cb);
            w[i][0] = v.x; w[i][1] = v.y; w[i][2] = v.z; w[i][3] = v.w;
        }
        uint2 ct[8];
        if (finite && normal) {
            uint32_t wt[8][4];
            transpose8x8_b16(w, wt);
#pragma unroll
            for (int j = 0; j < 8; ++j) ct[j] = encode8_pow2<F>(wt[j], scol[j]);
        } else {
            uint2 c[8];
            if (finite) {
#pragma unroll
                for (int i = 0; i < 8; ++i) c[i] = encode8_cols<F, false>(w[i], rcol);
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) c[i] = encode8_cols<F, true>(w[i], rcol);
            }
            transpose8x8(c, ct);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j)
            __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(unsigned int __attribute__((ext_vector_type(2))), ct[j]),
                                                  rt, (int)((cb * 8 + j) * M + b * 8), 0, 0);
    }
    if (b0 == 0) {
#pragma unroll
        for (int j = 0; j < 8; ++j) p.q8t_scale[(mrow0 / 128) * N + ncol0 + cb * 8 + j] = scol[j];
    }
}

// PROD: the workgroup has NW more waves that only issue the global->LDS
// loads (producers); the NW MFMA waves (consumers) then only read LDS and
// multiply, so a load that cannot issue (the texture unit's queue full)
// does not hold up their matrix instructions. Both kinds meet at the one
// barrier per slice.
template <int BM, int BN, int WM, int WN, int FA, int FB, int OUT, bool GROUPED, int SL, int NST, bool PROD>
__global__ __launch_bounds__(WM * WN * 64 * (PROD ? 2 : 1)) void gemm_fp8_kernel(Params p) {
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int KH = SL / 64;                     // 64-byte MFMA k steps per slice
    constexpr int A_BYTES = BM * SL, B_BYTES = BN * SL;
    constexpr int STAGE = A_BYTES + B_BYTES;        // one SL-byte k slice of both tiles
    // 1 KB DMA loads (RPL rows of SL bytes) per wave and slice; when the row
    // blocks do not divide evenly, the surplus loads repeat earlier blocks
    // (the same bytes to the same place), so every wave issues the same
    // number of loads and can wait on an exact count
    constexpr int RPL = 1024 / SL;                  // rows per DMA load
    constexpr int CPR = SL / 16;                    // 16-byte chunks per LDS row
    constexpr int A_BLK = BM / RPL, B_BLK = BN / RPL;
    constexpr int A_PER = (A_BLK + NW - 1) / NW, B_PER = (B_BLK + NW - 1) / NW;
    constexpr int SC_BLK = (BM + BN) / 64;          // 64 scales per 4-byte DMA load
    constexpr int SC_PER = GROUPED ? (SC_BLK + NW - 1) / NW : 0;
    constexpr int LOADS = A_PER + B_PER + SC_PER;
    static_assert(SL == 64 || SL == 128, "slice width");
    static_assert(BM % 32 == 0 && BN % 32 == 0 && (BM + BN) % 64 == 0, "tile shape");
    static_assert(NST >= 2 && (NST - 1) * LOADS <= 63, "pipeline depth");

    __shared__ __attribute__((aligned(1024))) uint8_t smem[NST * STAGE];
    // grouped scales of a slice's rows (A then B), float, DMA'd like the operands
    __shared__ __attribute__((aligned(16))) float ssc[GROUPED ? NST * (BM + BN) : 1];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave_id = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool producer = PROD && wave_id >= NW;
    // consumer waves 0..NW-1; a producer takes the DMA share of consumer wave_id - NW
    const int wave = producer ? wave_id - NW : wave_id;
    const int wm = wave / WN, wn = wave % WN;

    // ---- tile index: contiguous ranges per XCD, grouped by p.gm row panels
    const int T = gridDim.x;
    const int b = blockIdx.x;
    int lt = (T % 8 == 0) ? (b % 8) * (T / 8) + b / 8 : b;
    // a symmetric product computes only the tiles on or above the diagonal
    const int per_split = p.upper ? p.tiles_m * (p.tiles_m + 1) / 2 : p.tiles_m * p.tiles_n;
    if (p.batch > 1) {
        // problem bi of a batched launch: its operands, output and partials
        const int bi = lt / (per_split * p.splits);
        lt -= bi * per_split * p.splits;
        p.A += bi * p.bsa;
        p.B += bi * p.bsb;
        p.D = reinterpret_cast<uint8_t*>(p.D) + bi * p.bsd;
        if (p.residual) p.residual += bi * p.bsr;
        p.partial += (int64_t)bi * p.splits * p.M * p.N;
    }
    const int ks = lt / per_split;
    const int rem = lt - ks * per_split;
    int tm, tn;
    if (p.upper) {
        // row tm of the upper triangle holds tiles_n - tm tiles (a uniform scalar walk)
        int r = rem;
        tm = 0;
        while (r >= p.tiles_n - tm) {
            r -= p.tiles_n - tm;
            ++tm;
        }
        tn = tm + r;
    } else {
        const int group = rem / (p.gm * p.tiles_n);
        const int first_m = group * p.gm;
        const int gsz = min(p.gm, p.tiles_m - first_m);
        const int r2 = rem - group * p.gm * p.tiles_n;
        tm = first_m + r2 % gsz;
        tn = r2 / gsz;
    }
    const int m0 = tm * BM, n0 = tn * BN;
    // per-tensor scales, applied to the FP32 sums in the epilogue (loaded
    // here so that their latency hides behind the main loop)
    float alpha = p.alpha;
    if (OUT != 2) {
        if (p.a_mode == kSTensor) alpha *= p.sa[0];
        if (p.b_mode == kSTensor) alpha *= p.sb[0];
    }
    // k slices [s0, s1) of SL bytes: this split's 128-wide k blocks
    constexpr int SPB = kBK / SL;                   // slices per 128-wide k block
    const int s0 = SPB * ks * p.ksteps_per_split;
    const int s1 = SPB * min((ks + 1) * p.ksteps_per_split, p.ksteps);

    const int valid_m = min(BM, p.M - m0), valid_n = min(BN, p.N - n0);
    const v4i ra = make_rsrc(p.A + (int64_t)m0 * p.lda, (uint32_t)(valid_m * p.lda));
    const v4i rb = make_rsrc(p.B + (int64_t)n0 * p.ldb, (uint32_t)(valid_n * p.ldb));

    // LDS layout of a slice: row r of a tile is SL bytes (CPR 16-byte chunks)
    // and its logical chunk c sits at position c ^ key(r). The 16 (or 8)
    // lanes of a ds_read_b128 phase read 16 (8) consecutive rows at the same
    // logical chunk; the keys make them hit distinct banks with 64 (32)
    // four-byte banks:
    //  * SL = 64, key(r) = ((r >> 1) & 3) ^ ((r >> 3) & 1): of 16 consecutive
    //    rows, those sharing a 64-byte position in a 256-byte bank line get
    //    distinct keys, and so do those of 8 rows in a 128-byte line;
    //  * SL = 128, key(r) = (r & 7) ^ ((r >> 3) & 1): of 16 consecutive rows
    //    the 8 even (odd) ones, which share the lower (upper) half of a
    //    256-byte bank line, get distinct keys, and 8 consecutive rows in a
    //    128-byte line get the keys 0..7.
    // Lane l of a DMA load fills row RPL * blk + l / CPR at position l % CPR,
    // so it fetches the logical chunk (l % CPR) ^ key(row) of that row.
    auto row_key = [](int r) { return SL == 64 ? ((r >> 1) & 3) ^ ((r >> 3) & 1) : (r & 7) ^ ((r >> 3) & 1); };
    // logical k byte a lane fetches in a load of an even / odd row block
    const int kch0 = ((lane % CPR) ^ row_key(lane / CPR)) * 16;
    const int kch1 = ((lane % CPR) ^ row_key(RPL + lane / CPR)) * 16;
    const uint32_t rowA = (uint32_t)((lane / CPR) * p.lda), rowB = (uint32_t)((lane / CPR) * p.ldb);
    const uint32_t blkA = (uint32_t)(RPL * p.lda), blkB = (uint32_t)(RPL * p.ldb);
    const uint32_t smem_lds = lds_addr(smem);
    const uint32_t ssc_lds = lds_addr(ssc);

    v4i rsa{}, rsb{};
    // Scale load j of this wave brings entries 64 t .. 64 t + 63 (t = its
    // chunk) of a slice's scale vector: BM entries for A, then BN for B. A
    // row-scaled operand has one entry per tile row, a block-scaled one one
    // per 128-row block (entries past that are unused). The element lane l
    // loads for k block kb is sc_base[j] + kb * sc_kstride[j] (row-major
    // scales: stride 1; k-major: the array's row pitch), or nothing when
    // sc_base[j] < 0; all of it is fixed before the main loop.
    int sc_base[SC_PER > 0 ? SC_PER : 1], sc_kstride[SC_PER > 0 ? SC_PER : 1];
    bool sc_is_a[SC_PER > 0 ? SC_PER : 1];
    if constexpr (GROUPED) {
        rsa = make_rsrc(p.sa, p.a_mode == kSTensor ? 0u : p.sa_bytes);
        rsb = make_rsrc(p.sb, p.b_mode == kSTensor ? 0u : p.sb_bytes);
#pragma unroll
        for (int j = 0; j < SC_PER; ++j) {
            const int t = (wave * SC_PER + j) % SC_BLK;
            const bool is_a = t * 64 < BM;
            const int r = t * 64 + lane - (is_a ? 0 : BM);
            const int mode = is_a ? p.a_mode : p.b_mode;
            const bool km = is_a ? p.a_kmajor : p.b_kmajor;
            const int ld = is_a ? p.ld_sa : p.ld_sb;
            const int row0 = is_a ? m0 : n0;
            const int rows = is_a ? p.M : p.N;
            int unit = -1;   // row (row scales) or 128-row block (block scales) of this lane's entry
            if (mode == kSBlock) {
                // the 128-row blocks the tile's rows touch: from row0's to (row0 + BM - 1)'s
                const int b = (row0 >> 7) + r;
                const int last = (row0 + (is_a ? BM : BN) - 1) >> 7;
                if (b <= last && b < (rows + 127) >> 7) unit = b;
            } else if (mode == kSRow) {
                if (row0 + r < rows) unit = row0 + r;
            }
            sc_is_a[j] = is_a;
            sc_base[j] = unit < 0 ? -1 : (km ? unit : unit * ld);
            sc_kstride[j] = km ? ld : 1;
        }
    }
    (void)sc_base; (void)sc_kstride; (void)sc_is_a;

    // DMA load q (0 <= q < LOADS) of this wave for slice `sl` into ring
    // stage `st`. With `valid` false the load still issues (so that every
    // wave always has the same number in flight and waits on constant
    // counts) but reads out of range: no memory traffic, zeros into a stage
    // no later slice uses.
    auto dma_one = [&](int st, int sl, int q, bool valid) __attribute__((always_inline)) {
        const int k0 = sl * SL;
        const uint32_t sbase = smem_lds + st * STAGE;
        if (q < A_PER + B_PER) {
            const bool is_a = q < A_PER;
            const int blk = is_a ? (wave * A_PER + q) % A_BLK : (wave * B_PER + (q - A_PER)) % B_BLK;
            const int kch = (blk & 1) ? kch1 : kch0;
            // the k tail (K % SL != 0) also reads out of range on purpose: zeros
            const uint32_t off = (valid && k0 + kch < p.K) ? (uint32_t)(k0 + kch) : kOOB;
            if (is_a) dma_to_lds<16>(ra, sbase + blk * 1024, rowA + blk * blkA + off);
            else dma_to_lds<16>(rb, sbase + A_BYTES + blk * 1024, rowB + blk * blkB + off);
        } else if constexpr (GROUPED) {
            const int j = q - A_PER - B_PER;
            const int t = (wave * SC_PER + j) % SC_BLK;
            const int kb = sl / SPB;
            const uint32_t soff = (valid && sc_base[j] >= 0) ? (uint32_t)(sc_base[j] + kb * sc_kstride[j]) * 4u : kOOB;
            const uint32_t dst = ssc_lds + (st * (BM + BN) + t * 64) * 4;
            dma_to_lds<4>(sc_is_a[j] ? rsa : rsb, dst, soff);
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
    const int c0 = (lane >> 5) * 2;           // first of this lane's two chunks in a 64-byte k step
    // key of the lane's fragment rows (fragments start at multiples of 32)
    const int key = row_key(fr);

    // The operand fragments of one 64-byte k step as this wave holds them:
    // for each 32-row fragment (A fragments first) 32 bytes of k per lane,
    // bytes 32 (l >> 5) .. + 31 of the step in row l & 31, from two 16-byte
    // LDS reads; and the E8M0 scale of each fragment row.
    struct Frags {
        v8i f[FM + FN];
        uint32_t sc[FM + FN];
    };
    // the LDS entry of each fragment row's scale within a stage's scale
    // vector (block scales: the row's 128-row block counted from the block
    // of the tile's first row, which need not start a block when the tile
    // is 192 rows), and whether the operand has grouped scales at all
    int sc_off[FM + FN];
    bool sc_on[FM + FN];
#pragma unroll
    for (int fi = 0; fi < FM + FN; ++fi) {
        const bool is_a = fi < FM;
        const int r = is_a ? wm * WTM + fi * 32 + fr : wn * WTN + (fi - FM) * 32 + fr;   // tile row
        const int row0 = is_a ? m0 : n0;
        const int mode = is_a ? p.a_mode : p.b_mode;
        sc_off[fi] = (is_a ? 0 : BM) + (mode == kSBlock ? ((row0 + r) >> 7) - (row0 >> 7) : r);
        sc_on[fi] = mode != kSTensor;
    }
    // read piece t of k step h of the slice in stage st: t < FM + FN are
    // the operand fragments, the rest the scales (their raw binary32 bits:
    // scales_e8m0 turns them into the instruction's operands once they have
    // landed, so that no read waits on its own result)
    constexpr int NPIECE = (FM + FN) * (GROUPED ? 2 : 1);
    auto read_piece = [&](Frags& f, int st, int h, int t) __attribute__((always_inline)) {
        if (t < FM + FN) {
            const uint8_t* row = t < FM ? smem + st * STAGE + (wm * WTM + t * 32 + fr) * SL
                                        : smem + st * STAGE + A_BYTES + (wn * WTN + (t - FM) * 32 + fr) * SL;
            const int cc = 4 * h + c0;
            const v4i lo = *reinterpret_cast<const v4i*>(row + ((cc ^ key) << 4));
            const v4i hi = *reinterpret_cast<const v4i*>(row + (((cc + 1) ^ key) << 4));
            f.f[t] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        } else {
            const int fi = t - (FM + FN);
            f.sc[fi] = __float_as_uint(ssc[st * (BM + BN) + sc_off[fi]]);
        }
    };
    // the E8M0 exponent of each scale (127, a factor of 1, for a per-tensor
    // scaled operand, whose factor the epilogue applies)
    auto scales_e8m0 = [&](Frags& f) __attribute__((always_inline)) {
        if constexpr (GROUPED) {
#pragma unroll
            for (int fi = 0; fi < FM + FN; ++fi) f.sc[fi] = sc_on[fi] ? (f.sc[fi] >> 23) & 0xFFu : 127u;
        }
    };
    auto mfma_one = [&](const Frags& f, int t) __attribute__((always_inline)) {
        const int i = t / FN, j = t % FN;
        if constexpr (FA == kBF16) {
            // BF16: the lane's 32 bytes are 16 k values; each half feeds one
            // 32x32x16 instruction. A and B split k the same way, so the two
            // instructions together add every product of the 64-byte step.
            const v4i blo = __builtin_shufflevector(f.f[FM + j], f.f[FM + j], 0, 1, 2, 3);
            const v4i bhi = __builtin_shufflevector(f.f[FM + j], f.f[FM + j], 4, 5, 6, 7);
            const v4i alo = __builtin_shufflevector(f.f[i], f.f[i], 0, 1, 2, 3);
            const v4i ahi = __builtin_shufflevector(f.f[i], f.f[i], 4, 5, 6, 7);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, blo),
                                                                __builtin_bit_cast(v8bf, alo), acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, bhi),
                                                                __builtin_bit_cast(v8bf, ahi), acc[i][j], 0, 0, 0);
        } else if constexpr (GROUPED)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                f.f[FM + j], f.f[i], acc[i][j], FB, FA, 0, (int)f.sc[FM + j], 0, (int)f.sc[i]);
        else
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                f.f[FM + j], f.f[i], acc[i][j], FB, FA, 0, 127, 0, 127);
    };

    // One pipeline step: the MFMAs of k step h of slice sl (fragments in
    // `cur`, read during the previous step) with the LDS reads of the next
    // k step (into `nxt`) and, in a slice's last k step, the DMA loads of
    // slice sl + NST interleaved between them, so that LDS and memory
    // latency hide behind the MFMAs.
    // Before the reads of the next slice (in its last k step) a wave waits
    // until at most NST - 2 slices of its DMA loads remain in flight (every
    // wave always has NST - 1 in flight then, so its loads of slice sl + 1
    // have landed) and until its reads of slice sl are complete
    // (lgkmcnt(0)). After the barrier every wave is at that point: slice
    // sl + 1 is in LDS and the stage of slice sl is free for the DMA of slice
    // sl + NST. The loop body has no branches: reads past the last slice
    // fetch stale LDS data that is never used, and DMA loads past it read
    // nothing.
    constexpr int NMFMA = FM * FN;
    auto step = [&](int sl, int h, Frags& cur, Frags& nxt) __attribute__((always_inline)) {
        const bool last = h == KH - 1;
        if (last) {
            if constexpr (PROD)
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            else
                asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" :: "n"((NST - 2) * LOADS) : "memory");
            __syncthreads();
        }
        const int st = (sl - s0) % NST;
        const int rst = last ? (sl + 1 - s0) % NST : st;   // stage and k step read into nxt
        const int rh = last ? 0 : h + 1;
        const bool refill = sl + NST < s1;
        // fragment read u goes after MFMA u * NMFMA / NPIECE (the first half
        // of the step), DMA load q after MFMA q * NMFMA / LOADS (constant loop
        // bounds, so that everything unrolls and the fragments stay in
        // registers). A slice's k steps share its scales (one 128-wide k
        // block): the last step reads the next slice's, two after each of
        // MFMAs NMFMA / 2 .. NMFMA / 2 + 3, and makes them operands after its
        // last MFMA; the other steps pass theirs on.
        if constexpr (GROUPED) {
            if (!last) {
#pragma unroll
                for (int fi = 0; fi < FM + FN; ++fi) nxt.sc[fi] = cur.sc[fi];
            }
        }
#pragma unroll
        for (int t = 0; t < NMFMA; ++t) {
            mfma_one(cur, t);
#pragma unroll
            for (int u = 0; u < FM + FN; ++u)
                if (u * NMFMA / NPIECE == t) read_piece(nxt, rst, rh, u);
            if (last) {
#pragma unroll
                for (int u = FM + FN; u < NPIECE; ++u)
                    if (NMFMA / 2 + (u - FM - FN) / 2 == t) read_piece(nxt, rst, rh, u);
            }
            if (last && !PROD) {
#pragma unroll
                for (int q = 0; q < LOADS; ++q)
                    if (q * NMFMA / LOADS == t) dma_one(st, sl + NST, q, refill);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if (last) scales_e8m0(nxt);
    };

    // prologue: slices s0 .. s0 + NST - 1 in flight, then k step 0 of slice s0 read
    if (!PROD || producer) {
#pragma unroll
        for (int t = 0; t < NST; ++t)
#pragma unroll
            for (int q = 0; q < LOADS; ++q) dma_one(t, s0 + t, q, s0 + t < s1);
        asm volatile("s_waitcnt vmcnt(%0)" :: "n"((NST - 1) * LOADS) : "memory");
    }
    __syncthreads();
    if constexpr (PROD) {
        if (producer) {
            // per slice: slice sl + 1 landed, then (after the barrier at which
            // the consumers have read all of slice sl) its stage refilled with
            // slice sl + NST; the same barriers as the consumers' loop and
            // epilogue
            for (int sl = s0; sl < s1; ++sl) {
                asm volatile("s_waitcnt vmcnt(%0)" :: "n"((NST - 2) * LOADS) : "memory");
                __syncthreads();
                const int st = (sl - s0) % NST;
#pragma unroll
                for (int q = 0; q < LOADS; ++q) dma_one(st, sl + NST, q, sl + NST < s1);
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();   // the epilogue's barrier: the ring is idle
            return;
        }
    }
    Frags F0, F1;
#pragma unroll
    for (int t = 0; t < NPIECE; ++t) read_piece(F0, 0, 0, t);
    scales_e8m0(F0);
    if constexpr (KH == 2) {
        for (int sl = s0; sl < s1; ++sl) {
            step(sl, 0, F0, F1);
            step(sl, 1, F1, F0);
        }
    } else {
        int sl = s0;
        for (; sl + 1 < s1; sl += 2) {
            step(sl, 0, F0, F1);
            step(sl + 1, 0, F1, F0);
        }
        if (sl < s1) step(sl, 0, F0, F1);
    }
    // the loads issued for slices past the end write zeros into the ring,
    // which the epilogue reuses: let them land first
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    // ---- The LM head's forward statistics, straight from the accumulators.
    // Of each of its rows i*32 + (l & 31), lane l holds the 64 columns
    // j*32 + 8g + 4(l >> 5) + {0..3} of the wave tile; lane l ^ 32 holds the
    // other 64. A row's maximum and its sum of e^(z - max) over the 128
    // columns are the lane's over its 64 sums, combined with the partner's by
    // one exchange each: no staging, every logit read once. The exponent is
    // one FMA, z log2(e) - max log2(e), fed to the exp2 instruction. Its
    // rounding errs by a relative 2^-24 of |z| on each term and of |max| on
    // all of them alike, far inside the error of a binary32 log-sum-exp.
    if constexpr (OUT == kOutLseStats) {
        static_assert(!PROD && FN == 4 && WTN == 128, "LM-head statistics: 128-column wave tiles");
        const int mrow0 = m0 + wm * WTM, ncol0 = n0 + wn * WTN;
        if (ncol0 >= p.N) return;      // a wave tile wholly past N (the ragged last tile) has no block
        const int hl = lane >> 5;
        // each row's target column, relative to the lane's first column of
        // the wave tile (4 hl), or out of range
        int tcol[FM];
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int64_t m = (int64_t)mrow0 + i * 32 + (lane & 31);
            tcol[i] = m < p.M ? p.targets[m] - p.col0 - ncol0 - 4 * hl : INT_MIN;
        }
        constexpr float kLog2e = 1.44269504088896340736f;
        static_for<FM>([&](auto i_c) __attribute__((always_inline)) {
            constexpr int i = decltype(i_c)::value;
            float v[FN * 16];
#pragma unroll
            for (int e = 0; e < FN * 16; ++e)
                asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v[e]) : "a"(acc[i][e / 16][e % 16]));
            if (alpha != 1.0f) {
#pragma unroll
                for (int e = 0; e < FN * 16; ++e) v[e] *= alpha;
            }
            float mq[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
            for (int e = 4; e < FN * 16; ++e) mq[e % 4] = fmaxf(mq[e % 4], v[e]);
            float mx = fmaxf(fmaxf(mq[0], mq[1]), fmaxf(mq[2], mq[3]));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const float m2 = mx * kLog2e;
            float sq[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int e = 0; e < FN * 16; ++e) sq[e % 4] += __builtin_amdgcn_exp2f(fmaf(v[e], kLog2e, -m2));
            float sum = (sq[0] + sq[1]) + (sq[2] + sq[3]);
            sum += __shfl_xor(sum, 32, 64);
            const int64_t m = (int64_t)mrow0 + i * 32 + (lane & 31);
            if (hl == 0 && m < p.M) p.stats[m * p.stats_ld + ncol0 / 128] = make_float2(mx, sum);
            // the target's logit, where this wave tile holds it: entry
            // (j, g, t) of fragment row i is column j*32 + 8g + t past the
            // lane's first (rare: a branch taken by the whole wave or not)
            const int tc = tcol[i];
            const bool mine = tc >= 0 && tc < WTN && ((tc >> 2) & 1) == 0;
            if (__builtin_amdgcn_ballot_w64(mine)) {
                float zt = 0.0f;
#pragma unroll
                for (int e = 0; e < FN * 16; ++e) {
                    const int j = e / 16, g = (e % 16) / 4, t = e % 4;
                    zt = tc == j * 32 + 8 * g + t ? v[e] : zt;
                }
                if (mine) p.zt[m] = zt;
            }
        });
        return;
    }

    // ---- epilogue. Lane l holds, for fragment (i, j), wave-tile row
    // i*32 + (l & 31) and columns j*32 + 8g + 4(l >> 5) + {0..3}, g = 0..3.
    // Written straight to memory that would scatter 16-byte pieces over 32
    // rows per store; instead each wave stages its FP32 tile in its own part
    // of the (now idle) stage buffers, 16-byte chunks XOR-swizzled by row so
    // that both the writes and the row reads are free of bank conflicts, and
    // then stores whole rows: consecutive lanes on consecutive 16-byte chunks
    // (4 FP32 values), converted and scaled on the way out.
    constexpr int ROWB = WTN * 4;                 // bytes of one staged wave-tile row (FP32)
    constexpr int ECPR = ROWB / 16;               // 16-byte chunks per staged row
    constexpr int REGION = NST * STAGE / NW;      // LDS bytes per wave
    constexpr int RFIT = REGION / ROWB;          // rows that fit in the region
    // rows per pass: WTM halved until it fits
    constexpr int RPP = WTM <= RFIT ? WTM : (WTM / 2 <= RFIT ? WTM / 2 : WTM / 4);
    // XOR key of the chunk swizzle: 16 distinct keys when rows have 16*k chunks, else 8
    constexpr int SWZ = (ECPR % 16 == 0) ? 15 : 7;
    static_assert(RPP >= 32 && WTM % RPP == 0 && (RPP * ECPR) % 64 == 0, "epilogue tiling");
    static_assert(ECPR % 8 == 0, "row swizzle needs 8k chunks per row");
    uint8_t* ep = smem + wave * REGION;
    const int mrow0 = m0 + wm * WTM;
    const int ncol0 = n0 + wn * WTN;
    float* const part = p.partial + (int64_t)ks * p.M * p.N;
    // a tile inside the matrix whose sums overwrite the output (or, binary32,
    // add to it) stores whole 4-column vectors everywhere: a branch-free path
    // that issues all of a pass's LDS reads before its stores
    constexpr int ES = (OUT == kOutF32 || OUT == 2) ? 4 : 2;    // bytes per output element
    const int64_t ldo = OUT == 2 ? (int64_t)p.N : p.ldd;          // output pitch (elements)
    // (and whose rows, and residual rows, lie within 2^31 bytes of its first:
    // the fast path addresses them with 32-bit buffer offsets)
    const bool fast = m0 + BM <= p.M && n0 + BN <= p.N && (OUT == 2 || OUT == kOutF32 || !p.accumulate) &&
                      (int64_t)WTM * ldo * ES <= INT32_MAX &&
                      (OUT != kOutBF16Epi || (int64_t)WTM * p.ldr * 2 <= INT32_MAX);
    // the bias of the lane's columns in the fast path below: lane chunk
    // (it * 64 + lane) % ECPR repeats with period ECPR / gcd(64, ECPR) in it
    constexpr int EP = ECPR / ((ECPR & -ECPR) < 64 ? (ECPR & -ECPR) : 64);
    uint2 eb[OUT == kOutBF16Epi ? EP : 1];
    if constexpr (OUT == kOutBF16Epi) {
        const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t*>(p.bias), 0, p.bias ? p.N * 2 : 0, 0x00020000);
#pragma unroll
        for (int it = 0; it < EP; ++it)
            eb[it] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(
                rb, (uint32_t)((ncol0 + ((it * 64 + lane) % ECPR) * 4) * 2), 0, 0));
    }
    __syncthreads();   // every wave is done with the last stage
    // A plain BF16 output of a tile inside the matrix, 128-column wave tiles:
    // the lane rounds its sums to BF16 first and stages those, half the LDS
    // bytes of the binary32 staging below, and the whole wave tile fits its
    // region in one pass. Staged row r is 256 bytes, 32 units of 8 bytes
    // (four columns), and unit u sits at position u ^ 2 (r & 15): the two
    // units of each 16-byte chunk stay side by side and in order, so a chunk
    // reads back with one 16-byte load and leaves with one 16-byte store (a
    // store covers four whole rows); a chunk's position in its row depends
    // on r & 15, so the 16 lanes of a read phase, one row's 16 chunks, hit
    // distinct banks.
    // The LM head's backward output (dz of the logits) takes the same path:
    // each lane forms dz = g (exp(z - lse) - [column == target]) from its
    // sums directly, with the lse and target column of its FM rows loaded
    // first, and rounds it to BF16. The exponential is 2^t (1 + c): with
    // lse log2(e) split per row into its binary32 rounding P and the rest,
    // t = z log2(e)_hi - P is one FMA, which rounds once as z - lse would,
    // and 1 + c, the rest of the exponent times ln 2, is another.
    // Its dz kinds take every wave tile this way (M and N are multiples of
    // 128, so a wave tile lies wholly inside the output or wholly outside):
    // kOutSoftmaxGradQ quantises the staged tile (below).
    constexpr bool kDz = OUT == kOutSoftmaxGrad || OUT == kOutSoftmaxGradQ;
    static_assert(!kDz || (ECPR == 32 && WTM == 128 && WTM * 256 <= REGION), "dz kinds: 128 x 128 wave tiles");
    if constexpr ((OUT == kOutBF16 || OUT == kOutBF16Epi || kDz) && ECPR == 32 && WTM * 256 <= REGION) {
        if constexpr (kDz) {
            if (mrow0 + WTM > p.M || ncol0 + WTN > p.N) return;
        }
        if (kDz || fast) {
            // per row: P = lse log2(e)_hi rounded, K = 1 - (the rest of
            // lse log2(e)) ln 2 (rounded once), and the target's column
            // relative to the lane's first column of the wave tile
            constexpr float kL2eHi = 1.44269502162933349609375f;     // log2(e) rounded to binary32
            constexpr float kL2eLo = 1.925962989e-8f;                // log2(e) - kL2eHi
            constexpr float kLn2 = 0.693147180559945309f;
            constexpr float kL2eLoLn2 = kL2eLo * kLn2;
            float row_p[kDz ? FM : 1], row_k[kDz ? FM : 1];
            int row_tgt[kDz ? FM : 1];
            if constexpr (kDz) {
#pragma unroll
                for (int i = 0; i < FM; ++i) {
                    const int64_t m = (int64_t)mrow0 + i * 32 + (lane & 31);
                    row_tgt[i] = p.targets[m] - p.col0 - ncol0 - 4 * (lane >> 5);
                    const float l = p.lse[m];
                    row_p[i] = l * kL2eHi;
                    row_k[i] = 1.0f - (fmaf(l, kL2eHi, -row_p[i]) + l * kL2eLo) * kLn2;
                }
            }
            (void)row_p; (void)row_k; (void)row_tgt;
            // The bias / residual epilogue in the same one pass: the wave's
            // residual block arrives in its LDS region by DMA, each 16-byte
            // chunk already where the staged output chunk will sit (the lane
            // that lands chunk position q of row r loads the residual's chunk
            // q ^ (r & 15)); the lane then reads the four residual values of
            // each of its output units there, forms alpha acc + bias + rs
            // residual in binary32 with one rounding to BF16, and writes the
            // result over them. The bias of the lane's 64 columns is loaded
            // into registers once.
            uint2 bq[OUT == kOutBF16Epi ? FN * 4 : 1];
            if constexpr (OUT == kOutBF16Epi) {
                if (p.bias) {
                    const __amdgpu_buffer_rsrc_t rbq = __builtin_amdgcn_make_buffer_rsrc(
                        const_cast<uint16_t*>(p.bias), 0, p.N * 2, 0x00020000);
#pragma unroll
                    for (int e = 0; e < FN * 4; ++e)
                        bq[e] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(
                            rbq, (uint32_t)((ncol0 + (e / 4) * 32 + 8 * (e % 4) + 4 * (lane >> 5)) * 2), 0, 0));
                }
                if (p.residual) {
                    const v4i rr = make_rsrc(p.residual + (int64_t)mrow0 * p.ldr + ncol0,
                                             (uint32_t)((WTM - 1) * p.ldr * 2 + WTN * 2));
                    const uint32_t ep_lds = smem_lds + wave * REGION;
#pragma unroll
                    for (int q = 0; q < WTM / 4; ++q) {          // 1 KB: four rows of 256 bytes
                        const int r = q * 4 + (lane >> 4), c = (lane & 15) ^ (r & 15);
                        dma_to_lds<16>(rr, ep_lds + q * 1024, (uint32_t)((r * p.ldr + c * 8) * 2));
                    }
                }
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            }
            (void)bq;
            // one fragment row i of the wave tile; `onehot` when some lane's
            // row has its target among the lane's columns of this wave tile
            // (a few rows in a hundred), else dz is g e throughout
            auto stage_row = [&](auto scaled, auto onehot, auto epi, int i) __attribute__((always_inline)) {
                {
                    const int r = i * 32 + (lane & 31);
#pragma unroll
                    for (int j = 0; j < FN; ++j) {
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            // read at the point of use (a copy the compiler
                            // may not hoist): otherwise it moves accumulators
                            // to VGPRs ahead of the branch, and spills
                            float v0, v1, v2, v3;
                            asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v0) : "a"(acc[i][j][4 * g]));
                            asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v1) : "a"(acc[i][j][4 * g + 1]));
                            asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v2) : "a"(acc[i][j][4 * g + 2]));
                            asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v3) : "a"(acc[i][j][4 * g + 3]));
                            if constexpr (decltype(scaled)::value) {
                                v0 *= alpha; v1 *= alpha; v2 *= alpha; v3 *= alpha;
                            }
                            if constexpr (kDz) {
                                // the four sums are columns j*32 + 8g + {0..3} past the
                                // lane's first: tr is the target's position among them
                                const int tr = row_tgt[i] - (j * 32 + 8 * g);
                                const float P = row_p[i], K = row_k[i], gs = p.grad_scale;
                                auto dz = [&](float z, int c) __attribute__((always_inline)) {
                                    // 2^(z log2 e - lse log2 e) = 2^t (1 + c)
                                    const float e = __builtin_amdgcn_exp2f(fmaf(z, kL2eHi, -P)) * fmaf(z, kL2eLoLn2, K);
                                    if constexpr (decltype(onehot)::value) return fmaf(gs, e, c == tr ? -gs : 0.0f);
                                    else return gs * e;
                                };
                                v0 = dz(v0, 0); v1 = dz(v1, 1); v2 = dz(v2, 2); v3 = dz(v3, 3);
                            }
                            const int u = j * 8 + 2 * g + (lane >> 5);
                            uint2* const pos = reinterpret_cast<uint2*>(ep + r * 256 + ((u ^ (2 * (r & 15))) << 3));
                            if constexpr (OUT == kOutBF16Epi) {
                                // each term only when given: adding +0 would turn a -0 sum into +0
                                if constexpr ((decltype(epi)::value & 1) != 0) {
                                    const uint2 b = bq[j * 4 + g];
                                    v0 += bf16lo(b.x); v1 += bf16hi(b.x); v2 += bf16lo(b.y); v3 += bf16hi(b.y);
                                }
                                if constexpr ((decltype(epi)::value & 2) != 0) {
                                    const uint2 rv = *pos;
                                    const float rs = p.res_scale;
                                    v0 = fmaf(rs, bf16lo(rv.x), v0); v1 = fmaf(rs, bf16hi(rv.x), v1);
                                    v2 = fmaf(rs, bf16lo(rv.y), v2); v3 = fmaf(rs, bf16hi(rv.y), v3);
                                }
                            }
                            *pos = make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
                        }
                        // one fragment at a time: otherwise every accumulator
                        // is read into VGPRs before the first write
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
            };
            auto stage = [&](auto scaled, auto epi) __attribute__((always_inline)) {
#pragma unroll
                for (int i = 0; i < FM; ++i) {
                    if constexpr (kDz) {
                        // set for the lane that holds its row's target (and
                        // maybe for its partner lane): a wave-uniform branch
                        if (__builtin_amdgcn_ballot_w64((unsigned)row_tgt[i] < (unsigned)WTN))
                            stage_row(scaled, std::true_type{}, epi, i);
                        else
                            stage_row(scaled, std::false_type{}, epi, i);
                    } else {
                        stage_row(scaled, std::false_type{}, epi, i);
                    }
                }
            };
            // epi: bit 0 a bias, bit 1 a residual (bias / residual epilogue only)
            auto stage_epi = [&](auto epi) __attribute__((always_inline)) {
                if (alpha == 1.0f) stage(std::false_type{}, epi);
                else stage(std::true_type{}, epi);
            };
            if constexpr (OUT == kOutBF16Epi) {
                const int which = (p.bias ? 1 : 0) | (p.residual ? 2 : 0);
                if (which == 3) stage_epi(std::integral_constant<int, 3>{});
                else if (which == 2) stage_epi(std::integral_constant<int, 2>{});
                else if (which == 1) stage_epi(std::integral_constant<int, 1>{});
                else stage_epi(std::integral_constant<int, 0>{});
            } else {
                stage_epi(std::integral_constant<int, 0>{});
            }
            // the region belongs to this wave alone
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            if constexpr (OUT == kOutSoftmaxGradQ) {
                quantize_staged_dz(p, ep, mrow0, ncol0, lane);
                return;
            }
            // iteration it: lane l takes chunk l & 15 of staged row 4 it + (l >> 4);
            // (r & 15) repeats every 4 iterations, so four lane addresses serve
            // all of them with compile-time offsets
            typedef unsigned int v4u __attribute__((ext_vector_type(4)));
            const int rl = lane >> 4, cl = lane & 15;
            uint32_t la[4];
#pragma unroll
            for (int ph = 0; ph < 4; ++ph) {
                const int r = 4 * ph + rl;
                la[ph] = r * 256 + ((cl ^ (r & 15)) << 4);
            }
            const uint32_t row_bytes = (uint32_t)(p.ldd * 2);
            const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
                reinterpret_cast<uint8_t*>(p.D) + ((int64_t)mrow0 * p.ldd + ncol0) * 2, 0,
                (int)((WTM - 1) * row_bytes + WTN * 2), 0x00020000);
            const int voff = (int)(rl * row_bytes + cl * 16);
            constexpr int IT16 = WTM / 4, EG16 = 4;
            auto store_all = [&](auto nt_c) __attribute__((always_inline)) {
                constexpr int AUX = decltype(nt_c)::value ? 2 : 0;   // 2: the non-temporal bit
#pragma unroll
                for (int g0 = 0; g0 < IT16; g0 += EG16) {
                    v4u d[EG16];
#pragma unroll
                    for (int e = 0; e < EG16; ++e) {
                        const int it = g0 + e, ph = it % 4;
                        d[e] = *reinterpret_cast<const v4u*>(ep + la[ph] + (it - ph) * 4 * 256);
                    }
#pragma unroll
                    for (int e = 0; e < EG16; ++e)
                        __builtin_amdgcn_raw_buffer_store_b128(d[e], rd, voff, (int)((g0 + e) * 4 * row_bytes), AUX);
                }
            };
            if (p.nt_out) store_all(std::true_type{});
            else store_all(std::false_type{});
            return;
        }
    }
    // Fast-path addressing. Iteration it of a pass covers staged row r and
    // chunk c with it * 64 + lane = r * ECPR + c. That map repeats every FP
    // iterations, FR rows further on, and the rows' chunk swizzle every NPH
    // such periods. So the lane parts of the LDS addresses (NPH x FP) and of
    // the output and residual offsets (FP) are computed here, once per tile;
    // an iteration adds a compile-time LDS offset and a wave-uniform row
    // offset (the buffer access's scalar operand). No store then computes a
    // 64-bit address.
    constexpr int FP = EP;
    constexpr int FR = 64 * FP / ECPR;
    constexpr int NPH = (SWZ + 1) / cgcd(FR, SWZ + 1);
    const uint32_t row_bytes = (uint32_t)(ldo * ES);
    const uint32_t rrow_bytes = OUT == kOutBF16Epi ? (uint32_t)(p.ldr * 2) : 0u;
    uint32_t laddr[NPH][FP], goff[FP], roff[FP];
#pragma unroll
    for (int vv = 0; vv < FP; ++vv) {
        const int q = vv * 64 + lane;
        const int rv = q / ECPR, cv = q % ECPR;
        goff[vv] = rv * row_bytes + cv * 4 * ES;
        roff[vv] = rv * rrow_bytes + cv * 8;
#pragma unroll
        for (int ph = 0; ph < NPH; ++ph) {
            const int r = ph * FR + rv;
            laddr[ph][vv] = r * ROWB + ((cv ^ (r & SWZ)) << 4);
        }
    }
    // the wave tile's output (and residual) rows as buffers: base at its
    // first element, range over its last row's WTN elements
    const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
        OUT == 2 ? (void*)(part + (int64_t)mrow0 * p.N + ncol0)
                 : (void*)(reinterpret_cast<uint8_t*>(p.D) + ((int64_t)mrow0 * p.ldd + ncol0) * ES),
        0, fast ? (int)((WTM - 1) * row_bytes + WTN * ES) : 0, 0x00020000);
    const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
        OUT == kOutBF16Epi && p.residual ? const_cast<uint16_t*>(p.residual + (int64_t)mrow0 * p.ldr + ncol0) : nullptr,
        0, OUT == kOutBF16Epi && p.residual && fast ? (int)((WTM - 1) * rrow_bytes + WTN * 2) : 0, 0x00020000);
    (void)laddr; (void)goff; (void)roff; (void)rd; (void)rres;
    // one pass per constant: the accumulators are indexed by the pass, and a
    // loop the unroller leaves rolled would move them to scratch memory
    static_for<WTM / RPP>([&](auto pass_c) __attribute__((always_inline)) {
        constexpr int pass = decltype(pass_c)::value;
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
        // the region belongs to this wave alone: once its own writes are
        // done other lanes of the wave may read them (and the next pass
        // writes only after this pass's reads have returned their data)
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        constexpr int IT = RPP * ECPR / 64;
        if (fast) {
            // the residual is loaded before the LDS reads of its group of
            // iterations, so that its latency overlaps those reads and the
            // group's stores wait once (a load issued after stores waits for
            // them); an absent residual is a zero-range buffer (no branch, no
            // traffic). Groups of at most 16 iterations keep the residual and
            // the staged values in registers beside the accumulators of the
            // passes still to come.
            // With ACC (binary32 output added to what D holds) each group
            // first loads the outputs it replaces, with the stores' own
            // addressing, in the same place as the residual.
            auto run_groups = [&](auto acc_c) __attribute__((always_inline)) {
                constexpr bool ACC = decltype(acc_c)::value;
                constexpr int EG = ((OUT == kOutBF16Epi || ACC) && IT > 16) ? IT / 2 : IT;
                static_assert(IT % EG == 0 && EG % FP == 0, "epilogue groups");
                typedef unsigned int v4a __attribute__((ext_vector_type(4)));
#pragma unroll
                for (int g0 = 0; g0 < IT; g0 += EG) {
                    v4a ea[ACC ? EG : 1];
                    if constexpr (ACC) {
#pragma unroll
                        for (int e = 0; e < EG; ++e) {
                            const int u = (g0 + e) / FP, vv = (g0 + e) % FP;
                            ea[e] = __builtin_bit_cast(v4a, __builtin_amdgcn_raw_buffer_load_b128(
                                rd, (int)goff[vv], (int)((pass * RPP + u * FR) * row_bytes), 0));
                        }
                    }
                    (void)ea;
                    uint2 er[OUT == kOutBF16Epi ? EG : 1];
                    if constexpr (OUT == kOutBF16Epi) {
#pragma unroll
                        for (int e = 0; e < EG; ++e) {
                            const int u = (g0 + e) / FP, vv = (g0 + e) % FP;
                            er[e] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(
                                rres, (int)roff[vv], (int)((pass * RPP + u * FR) * rrow_bytes), 0));
                        }
                    }
                    float4 v[EG];
#pragma unroll
                    for (int e = 0; e < EG; ++e) {
                        const int u = (g0 + e) / FP, vv = (g0 + e) % FP, ph = u % NPH;
                        v[e] = *reinterpret_cast<const float4*>(ep + laddr[ph][vv] + (u - ph) * FR * ROWB);
                    }
                    if constexpr (OUT != 2) {
                        if (alpha != 1.0f) {
#pragma unroll
                            for (int e = 0; e < EG; ++e) {
                                v[e].x *= alpha; v[e].y *= alpha; v[e].z *= alpha; v[e].w *= alpha;
                            }
                        }
                    }
                    // AUX 2 is the buffer store's non-temporal bit
                    auto store_group = [&](auto nt_c) __attribute__((always_inline)) {
                        constexpr int AUX = decltype(nt_c)::value ? 2 : 0;
#pragma unroll
                        for (int e = 0; e < EG; ++e) {
                            const int u = (g0 + e) / FP, vv = (g0 + e) % FP;
                            const int soff = (int)((pass * RPP + u * FR) * row_bytes);
                            float4 w = v[e];
                            if constexpr (OUT == kOutBF16Epi) {
                                // each term only when given: adding +0 would turn a -0 sum into +0
                                if (p.bias) {
                                    const uint2 b = eb[vv];
                                    w.x += bf16lo(b.x); w.y += bf16hi(b.x); w.z += bf16lo(b.y); w.w += bf16hi(b.y);
                                }
                                if (p.residual) {
                                    const uint2 rv = er[e];
                                    const float rs = p.res_scale;
                                    w.x = fmaf(rs, bf16lo(rv.x), w.x); w.y = fmaf(rs, bf16hi(rv.x), w.y);
                                    w.z = fmaf(rs, bf16lo(rv.y), w.z); w.w = fmaf(rs, bf16hi(rv.y), w.w);
                                }
                            }
                            if constexpr (ES == 4) {
                                if constexpr (ACC) {
                                    const float4 o = __builtin_bit_cast(float4, ea[e]);
                                    w.x += o.x; w.y += o.y; w.z += o.z; w.w += o.w;
                                }
                                typedef unsigned int v4u __attribute__((ext_vector_type(4)));
                                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, w), rd, (int)goff[vv], soff, AUX);
                            } else {
                                typedef unsigned int v2u __attribute__((ext_vector_type(2)));
                                __builtin_amdgcn_raw_buffer_store_b64(v2u{pack_bf16x2(w.x, w.y), pack_bf16x2(w.z, w.w)}, rd,
                                                                      (int)goff[vv], soff, AUX);
                            }
                        }
                    };
                    if (OUT != 2 && p.nt_out) store_group(std::true_type{});
                    else store_group(std::false_type{});
                }
            };
            if constexpr (OUT == kOutF32) {
                if (p.accumulate) run_groups(std::true_type{});
                else run_groups(std::false_type{});
            } else {
                run_groups(std::false_type{});
            }
            return;
        }
#pragma unroll
        for (int it = 0; it < IT; ++it) {
            const int q = it * 64 + lane;
            const int r = q / ECPR, c = q % ECPR;
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
                if constexpr (OUT == kOutBF16Epi) add_epilogue4(v, p.bias, p.residual, p.ldr, m, n, p.res_scale);
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
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    if (n + t >= p.N) continue;
                    if constexpr (OUT == kOutF32) {
                        float* dst = reinterpret_cast<float*>(p.D) + (int64_t)m * p.ldd + n + t;
                        *dst = p.accumulate ? *dst + vv[t] : vv[t];
                    } else {
                        uint16_t* dst = reinterpret_cast<uint16_t*>(p.D) + (int64_t)m * p.ldd + n + t;
                        float o = p.accumulate ? vv[t] + __uint_as_float((uint32_t)*dst << 16) : vv[t];
                        if constexpr (OUT == kOutBF16Epi) o = add_epilogue1(o, p.bias, p.residual, p.ldr, m, n + t, p.res_scale);
                        *dst = to_bf16(o);
                    }
                }
            }
        }
    });
}

template <int BM, int BN, int WM, int WN, int SL, int NST, int PROD, int FA, int FB, bool GROUPED, int OUT>
void launch_cfg(const Params& prm, int grid, hipStream_t stream) {
    constexpr int threads = WM * WN * 64 * (PROD ? 2 : 1);
    gemm_fp8_kernel<BM, BN, WM, WN, FA, FB, OUT, GROUPED, SL, NST, PROD != 0><<<grid, threads, 0, stream>>>(prm);
}

template <int BM, int BN, int WM, int WN, int SL, int NST, int PROD, int FA, int FB, bool GROUPED>
void launch_tile(const Params& prm, int out, int grid, hipStream_t stream) {
    // the LM-head kinds exist for BF16 operands and blockwise E4M3 operands,
    // on 128-column wave tiles
    constexpr bool lm = (FA == kBF16 && FB == kBF16 && !GROUPED) || (FA == kE4M3 && FB == kE4M3 && GROUPED);
    if (out == 2) launch_cfg<BM, BN, WM, WN, SL, NST, PROD, FA, FB, GROUPED, 2>(prm, grid, stream);
    else if (out == kOutF32) launch_cfg<BM, BN, WM, WN, SL, NST, PROD, FA, FB, GROUPED, kOutF32>(prm, grid, stream);
    else if (out == kOutBF16Epi)
        launch_cfg<BM, BN, WM, WN, SL, NST, PROD, FA, FB, GROUPED, kOutBF16Epi>(prm, grid, stream);
    else if (out == kOutLseStats || out == kOutSoftmaxGrad) {
        if constexpr (lm && BN / WN == 128) {
            if (out == kOutLseStats) launch_cfg<BM, BN, WM, WN, SL, NST, PROD, FA, FB, GROUPED, kOutLseStats>(prm, grid, stream);
            else launch_cfg<BM, BN, WM, WN, SL, NST, PROD, FA, FB, GROUPED, kOutSoftmaxGrad>(prm, grid, stream);
        }
    } else if (out == kOutSoftmaxGradQ) {
        // the blockwise E4M3 recipe's backward, 128 x 128 wave tiles
        if constexpr (FA == kE4M3 && FB == kE4M3 && GROUPED && BM / WM == 128 && BN / WN == 128)
            launch_cfg<BM, BN, WM, WN, SL, NST, PROD, FA, FB, GROUPED, kOutSoftmaxGradQ>(prm, grid, stream);
    } else launch_cfg<BM, BN, WM, WN, SL, NST, PROD, FA, FB, GROUPED, kOutBF16>(prm, grid, stream);
}

}  // namespace

template <int FA, int FB, bool GROUPED>
void launch_variant(const Params& prm, int cfg, int out, int grid, hipStream_t stream) {
#define PURO_TILE_CASE(i, bm, bn, wm, wn, sl, nst, prod, f, s) \
    case i: launch_tile<bm, bn, wm, wn, sl, nst, prod, FA, FB, GROUPED>(prm, out, grid, stream); break;
    switch (cfg) { PURO_TILE_LIST(PURO_TILE_CASE) }
#undef PURO_TILE_CASE
}

template void launch_variant<PURO_FA, PURO_FB, (PURO_GROUPED != 0)>(const Params&, int, int, int, hipStream_t);

}  // namespace gemm_detail
}  // namespace puro
