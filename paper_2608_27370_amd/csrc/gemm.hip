// Host side of the scaled FP8 GEMM: the plan for a problem (tile
// configuration and k split), its launch, and the fixed-order split-K
// reduction kernel. The GEMM kernel itself is in gemm_kernel.hip.

#include <type_traits>

#include "device_common.h"
#include "gemm_common.h"
#include "kernels.h"

namespace puro {

using namespace gemm_detail;

namespace {

// Fixed-order sum of the split-K partials, scaling and output conversion.
// Batched launches: problem bi's partials follow problem bi-1's, its output
// starts bsd bytes and its residual bsr elements after the previous one's.
template <int OUT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ partial, int splits,
                                                            int M, int N, const float* sa, const float* sb,
                                                            int a_tensor, int b_tensor, void* D,
                                                            int64_t ldd, int accumulate, const uint16_t* bias,
                                                            const uint16_t* residual, int64_t ldr, float alpha0,
                                                            float res_scale, int batch, int64_t bsd,
                                                            int64_t bsr) {
    const int64_t nq = N / 4;
    int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)M * nq * batch) return;
    const int64_t bi = idx / ((int64_t)M * nq);
    idx -= bi * M * nq;
    partial += bi * splits * (int64_t)M * N;
    D = reinterpret_cast<uint8_t*>(D) + bi * bsd;
    if (residual) residual += bi * bsr;
    const int64_t m = idx / nq;
    const int n = (int)(idx - m * nq) * 4;
    float alpha = alpha0;
    if (a_tensor) alpha *= sa[0];
    if (b_tensor) alpha *= sb[0];
    float4 s = *reinterpret_cast<const float4*>(partial + m * N + n);
    for (int k = 1; k < splits; ++k) {
        const float4 t = *reinterpret_cast<const float4*>(partial + ((int64_t)k * M + m) * N + n);
        s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
    }
    s.x *= alpha; s.y *= alpha; s.z *= alpha; s.w *= alpha;
    if constexpr (OUT == kOutBF16Epi) add_epilogue4(s, bias, residual, ldr, m, n, res_scale);
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

constexpr TileCfg kTiles[] = {PURO_TILE_LIST(PURO_TILE_ROW)};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);
constexpr int kCUs = 256;
constexpr int kLdsBytes = 160 * 1024;

struct Plan {
    int cfg;             // index into kTiles
    int splits;          // k ranges (split-K)
    int ksteps_per_split;
};

// Workgroups of a configuration that fit on one CU (by LDS).
int per_cu(const TileCfg& t, bool grouped) {
    const int lds = (t.bm + t.bn) * t.sl * t.nst + (grouped ? (t.bm + t.bn) * 4 * t.nst : 0);
    const int n = kLdsBytes / lds;
    return n < 1 ? 1 : n;
}

// Pick the tile configuration and k split with the smallest modelled time:
// waves of work units over the CUs, each a fixed cost plus a cost per k
// slice (lower when part of the GPU idles and the clock rises; higher with
// block scales), plus the split-K partial sums written and read back.
Plan make_plan(int64_t M, int64_t N, int64_t K, bool grouped, int batch = 1, bool upper = false) {
    const int ksteps = (int)((K + kBK - 1) / kBK);
    Plan best{0, 1, ksteps};
    double best_cost = -1.0;
    for (int c = 0; c < kNumTiles; ++c) {
        const TileCfg t = kTiles[c];
        if (upper && t.bm != t.bn) continue;   // the upper-triangle walk takes square tiles
        const int64_t tm_ = (M + t.bm - 1) / t.bm, tn_ = (N + t.bn - 1) / t.bn;
        const int64_t tiles = (upper ? tm_ * (tm_ + 1) / 2 : tm_ * tn_) * batch;
        if (tiles == 0) return best;
        const int64_t slots = (int64_t)kCUs * per_cu(t, grouped);
        const int max_s = (N % 4 == 0) ? (ksteps / 4 < 16 ? ksteps / 4 : 16) : 1;
        for (int s = 1; s <= (max_s > 1 ? max_s : 1); ++s) {
            const int kps = (ksteps + s - 1) / s;
            const int splits = kps > 0 ? (ksteps + kps - 1) / kps : 1;
            if (splits != s) continue;
            const int64_t units = tiles * splits;
            const int64_t waves = (units + slots - 1) / slots;
            const double busy = units < slots ? (double)units / slots : 1.0;
            double cost = (double)waves * (t.fixed_us + t.slice_us * (kps > 0 ? kps : 1) * (1.0 - 0.332 * (1.0 - busy)));
            if (grouped) cost *= 1.14;
            if (splits > 1) cost += 0.289e-6 * splits * (double)M * N * 4.0 * batch;
            if (best_cost < 0 || cost < best_cost) {
                best_cost = cost;
                best = Plan{c, splits, kps};
            }
        }
    }
    return best;
}

// Tile rows per group of an XCD's contiguous range of tiles (the order in
// which that XCD's CUs take them): 4 (the QKV Wgrad's 24-tile ranges become
// 4 x 6 tiles, 10 operand panels per XCD instead of 11 at 8). On the
// 28-layer step with the workload's operands, groups of 2 and 8 rows for
// the short reductions over many tile columns (the gate/up Fprop, the down
// Dgrad) measured 1% slower than 4 (results bitwise the same).
constexpr int kGroupRows = 4;

size_t plan_workspace_bytes(int64_t M, int64_t N, const Plan& pl, int batch = 1) {
    if (pl.splits <= 1) return 0;
    return (size_t)batch * (size_t)pl.splits * (size_t)M * (size_t)N * sizeof(float);
}

// Enqueue the GEMM of `g` with plan `pl`; `ws` holds plan_workspace_bytes.
// Bytes per operand element, and whether the operands carry grouped scales.
int elem_bytes(const GemmProblem& g) { return g.fa == kBF16 ? 2 : 1; }
bool grouped_scales(const GemmProblem& g) {
    return g.sa_mode == kSRow || g.sa_mode == kSBlock || g.sb_mode == kSRow || g.sb_mode == kSBlock;
}

void run_plan(const GemmProblem& g, const Plan& pl, void* ws, hipStream_t stream) {
    const TileCfg t = kTiles[pl.cfg];
    // the kernel walks k in bytes of an operand row
    const int eb = elem_bytes(g);
    Params prm{};
    prm.A = g.A; prm.B = g.B; prm.sa = g.sa; prm.sb = g.sb;
    prm.D = g.D; prm.partial = reinterpret_cast<float*>(ws);
    prm.lda = g.lda * eb; prm.ldb = g.ldb * eb; prm.ldd = g.ldd;
    prm.M = (int)g.M; prm.N = (int)g.N; prm.K = (int)(g.K * eb);
    prm.a_mode = g.sa_mode; prm.b_mode = g.sb_mode;
    prm.a_kmajor = g.sa_kmajor; prm.b_kmajor = g.sb_kmajor;
    auto scale_ld = [&](int mode, bool km, int64_t rows) -> int {
        if (!km) return (int)(g.K / kBK);
        return (int)(mode == kSBlock ? (rows + 127) / 128 : rows);
    };
    prm.ld_sa = scale_ld(g.sa_mode, g.sa_kmajor, g.M);
    prm.ld_sb = scale_ld(g.sb_mode, g.sb_kmajor, g.N);
    auto scale_bytes = [&](int mode, int64_t rows) -> uint32_t {
        if (mode == kSTensor) return 4u;
        const int64_t srows = mode == kSRow ? rows : (rows + 127) / 128;
        return (uint32_t)(srows * (g.K / kBK) * 4);
    };
    prm.sa_bytes = scale_bytes(g.sa_mode, g.M);
    prm.sb_bytes = scale_bytes(g.sb_mode, g.N);
    prm.ksteps = (int)((g.K * eb + kBK - 1) / kBK);
    prm.ksteps_per_split = pl.ksteps_per_split;
    prm.splits = pl.splits;
    prm.tiles_m = (int)((g.M + t.bm - 1) / t.bm);
    prm.tiles_n = (int)((g.N + t.bn - 1) / t.bn);
    prm.accumulate = g.accumulate;
    prm.gm = kGroupRows;
    prm.alpha = g.alpha;
    prm.bias = g.bias;
    prm.residual = g.residual;
    prm.ldr = g.ldr;
    prm.res_scale = g.res_scale;
    prm.upper = g.upper;
    prm.nt_out = g.nt_out;
    const int ob = g.out == kOutF32 ? 4 : 2;
    prm.batch = g.batch;
    prm.bsa = g.bsa * eb; prm.bsb = g.bsb * eb; prm.bsd = g.bsd * ob; prm.bsr = g.bsr;
    prm.targets = g.targets; prm.col0 = g.col0;
    prm.stats = g.stats; prm.stats_ld = g.stats_ld; prm.zt = g.zt;
    prm.lse = g.lse; prm.grad_scale = g.grad_scale;
    prm.q8 = g.q8; prm.q8_scale = g.q8_scale; prm.q8t = g.q8t; prm.q8t_scale = g.q8t_scale;
    const bool grouped = grouped_scales(g);
    const int out = pl.splits > 1 ? 2 : g.out;
    const int grid = (g.upper ? prm.tiles_m * (prm.tiles_m + 1) / 2 : prm.tiles_m * prm.tiles_n) * pl.splits * g.batch;
    auto launch = [&](auto fa, auto fb) {
        constexpr int FA = decltype(fa)::value, FB = decltype(fb)::value;
        if (grouped) launch_variant<FA, FB, true>(prm, pl.cfg, out, grid, stream);
        else launch_variant<FA, FB, false>(prm, pl.cfg, out, grid, stream);
    };
    using E4 = std::integral_constant<int, kE4M3>;
    using E5 = std::integral_constant<int, kE5M2>;
    if (g.fa == kBF16) launch_variant<kBF16, kBF16, false>(prm, pl.cfg, out, grid, stream);
    else if (g.fa == kE4M3 && g.fb == kE4M3) launch(E4{}, E4{});
    else if (g.fa == kE5M2 && g.fb == kE4M3) launch(E5{}, E4{});
    else if (g.fa == kE4M3 && g.fb == kE5M2) launch(E4{}, E5{});
    else launch(E5{}, E5{});
    if (pl.splits > 1) {
        const int64_t n = g.M * (g.N / 4) * g.batch;
        const int blocks = (int)((n + 255) / 256);
        if (g.out == kOutF32)
            splitk_reduce_kernel<kOutF32><<<blocks, 256, 0, stream>>>(
                prm.partial, pl.splits, prm.M, prm.N, g.sa, g.sb, g.sa_mode == kSTensor,
                g.sb_mode == kSTensor, g.D, g.ldd, g.accumulate, nullptr, nullptr, 0, g.alpha, 1.0f, g.batch,
                prm.bsd, 0);
        else if (g.out == kOutBF16Epi)
            splitk_reduce_kernel<kOutBF16Epi><<<blocks, 256, 0, stream>>>(
                prm.partial, pl.splits, prm.M, prm.N, g.sa, g.sb, g.sa_mode == kSTensor,
                g.sb_mode == kSTensor, g.D, g.ldd, 0, g.bias, g.residual, g.ldr, g.alpha, g.res_scale, g.batch,
                prm.bsd, g.bsr);
        else
            splitk_reduce_kernel<kOutBF16><<<blocks, 256, 0, stream>>>(
                prm.partial, pl.splits, prm.M, prm.N, g.sa, g.sb, g.sa_mode == kSTensor,
                g.sb_mode == kSTensor, g.D, g.ldd, g.accumulate, nullptr, nullptr, 0, g.alpha, 1.0f, g.batch,
                prm.bsd, 0);
    }
}

}  // namespace

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int out, int batch) {
    // enough for the plan with or without block scales
    (void)out;
    // enough for the plans with or without block scales, and (square
    // problems) for the upper-triangle plans
    size_t w = 0;
    for (int u = 0; u < (M == N ? 2 : 1); ++u)
        for (int gr = 0; gr < 2; ++gr) {
            const size_t v = plan_workspace_bytes(M, N, make_plan(M, N, K, gr != 0, batch, u != 0), batch);
            w = v > w ? v : w;
        }
    return w;
}

void gemm_plan(int64_t M, int64_t N, int64_t K, bool grouped, int* tile_m, int* tile_n, int* stages,
               int* splits) {
    const Plan p = make_plan(M, N, K, grouped);
    *tile_m = kTiles[p.cfg].bm;
    *tile_n = kTiles[p.cfg].bn;
    *stages = kTiles[p.cfg].nst;
    *splits = p.splits;
}

void launch_gemm(const GemmProblem& g, void* ws, hipStream_t stream) {
    const int64_t kb = g.K * elem_bytes(g);
    if (g.out == kOutLseStats || g.out == kOutSoftmaxGrad || g.out == kOutSoftmaxGradQ) {
        // the LM-head epilogues reduce over 128-column wave tiles: the
        // 256 x 256 configuration, unsplit
        run_plan(g, Plan{0, 1, (int)((kb + kBK - 1) / kBK)}, ws, stream);
        return;
    }
    run_plan(g, make_plan(g.M, g.N, kb, grouped_scales(g), g.batch, g.upper != 0), ws, stream);
}

int gemm_tile(const GemmProblem& g) {
    if (g.out == kOutLseStats || g.out == kOutSoftmaxGrad || g.out == kOutSoftmaxGradQ) return kTiles[0].bm;
    return kTiles[make_plan(g.M, g.N, g.K * elem_bytes(g), grouped_scales(g), g.batch, g.upper != 0).cfg].bm;
}

}  // namespace puro
