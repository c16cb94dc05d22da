// The language-model head with its cross-entropy loss (gfx950).
//
// Section 3.1.3 of the paper names the LM head as the layer whose cost sets
// the pipeline's last stage apart; Appendix C keeps it in BF16 while the
// transformer's linear layers run in FP8. For hidden states X [M, K], the
// output embedding W [V, K] and one target id per row:
//
//   forward:  z = X W^T, lse_m = log sum_v exp(z_mv), loss_m = lse_m - z_{m,t_m}
//   backward: dz = g (exp(z - lse) - onehot(t)), dX = dz W, dW = dz^T X
//
// The logits are never stored. The forward's GEMM reduces each 128-column
// block of every row to (max, sum of exp(z - max)) in its epilogue (and keeps
// the target's logit); one block per row then combines the blocks into lse
// and the loss. The backward walks the vocabulary in chunks: the chunk's
// logits are recomputed by the same GEMM, whose epilogue writes dz (BF16)
// instead; the chunk's dz then feeds the dX GEMM (accumulated over chunks in
// binary32) and the dW GEMM of the chunk's rows of W.
//
// Recipes: BF16 operands throughout (the transposed copies that the backward
// GEMMs read, X^T and W^T, are made once per call, and each dz chunk's),
// or the blockwise FP8
// recipe of Section 3.2: X in 1x128 groups (rows for the logits, columns for
// dW), W in 128x128 blocks (the transposed copy for dX shares the block
// scales), and each dz chunk quantised in 1x128 + 128x1 groups (by the
// chunk GEMM's epilogue, from the BF16 dz it forms, as the quantiser would);
// E4M3 with power-of-two scales.

#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace puro {

namespace {

__global__ __launch_bounds__(256) void f32_to_bf16_kernel(const float* __restrict__ src, uint16_t* __restrict__ dst,
                                                          int64_t n4) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n4) return;
    const float4 v = reinterpret_cast<const float4*>(src)[i];
    reinterpret_cast<uint2*>(dst)[i] = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
}

__global__ __launch_bounds__(256) void fill_f32_kernel(float* __restrict__ dst, float v, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) dst[i] = v;
}

// lse and loss of one row from its blocks' (max, sum exp(z - max)): the
// largest block maximum M, then lse = M + log sum_b s_b exp(m_b - M); blocks
// past the vocabulary (max -inf, sum 0) drop out. loss = lse - z_target (NaN
// when no block held the target).
__global__ __launch_bounds__(256) void lse_rows_kernel(const float2* __restrict__ stats, int64_t ld, int nblk,
                                                       const float* __restrict__ zt, float* __restrict__ lse,
                                                       float* __restrict__ loss) {
    __shared__ float red[4];
    const int64_t m = blockIdx.x;
    const float2* st = stats + m * ld;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    float mx = -__builtin_inff();
    for (int b = threadIdx.x; b < nblk; b += 256) mx = fmaxf(mx, st[b].x);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    if (lane == 0) red[w] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    float s = 0.0f;
    for (int b = threadIdx.x; b < nblk; b += 256) {
        const float2 v = st[b];
        if (v.y != 0.0f) s += v.y * exp_f32(v.x - mx);   // NaN sums propagate
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
    if (lane == 0) red[w] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        const float l = mx + logf((red[0] + red[1]) + (red[2] + red[3]));
        lse[m] = l;
        loss[m] = l - zt[m];
    }
}

constexpr size_t kAl = 256;
size_t al(size_t v) { return (v + kAl - 1) / kAl * kAl; }

// Workspace regions, in bytes from the start.
struct LmLayout {
    size_t stats, zt;                               // forward
    size_t xq, xs, xqt, xst, wq, wsc, wqt, wsct;    // FP8 operands
    size_t xt, wt;                                  // BF16 transposed operands
    size_t dz, dzt, dzq, dzs, dzqt, dzst, dxacc;    // backward chunk and dX
    size_t gemm, total;
};

struct Carve {
    size_t used = 0;
    size_t take(size_t b) { const size_t at = used; used = al(used + b); return at; }
};

}  // namespace

int64_t lm_head_chunk(int64_t V) { return V < kLmChunk ? V : kLmChunk; }

static LmLayout lm_layout(int64_t M, int64_t V, int64_t K, int fp8, bool bwd) {
    Carve c;
    LmLayout l{};
    const int64_t Vc = lm_head_chunk(V);
    if (!bwd) {
        l.stats = c.take((size_t)M * (V / 128) * sizeof(float2));
        l.zt = c.take((size_t)M * sizeof(float));
    }
    if (fp8) {
        l.xq = c.take((size_t)M * K);
        l.xs = c.take((size_t)M * (K / 128) * 4);
        l.wq = c.take((size_t)V * K);
        l.wsc = c.take((size_t)(V / 128) * (K / 128) * 4);
        if (bwd) {
            l.xqt = c.take((size_t)M * K);
            l.xst = c.take((size_t)M * (K / 128) * 4);
            l.wqt = c.take((size_t)V * K);
            l.wsct = c.take((size_t)(V / 128) * (K / 128) * 4);
        }
    } else if (bwd) {
        l.xt = c.take((size_t)M * K * 2);
        l.wt = c.take((size_t)V * K * 2);
    }
    size_t g = 0;
    if (bwd) {
        // the FP8 recipe's chunk GEMM writes dz's E4M3 copies directly
        if (!fp8) l.dz = c.take((size_t)M * Vc * 2);
        if (fp8) {
            l.dzq = c.take((size_t)M * Vc);
            l.dzs = c.take((size_t)M * (Vc / 128) * 4);
            l.dzqt = c.take((size_t)M * Vc);
            l.dzst = c.take((size_t)M * (Vc / 128) * 4);
        } else {
            l.dzt = c.take((size_t)M * Vc * 2);
        }
        l.dxacc = c.take((size_t)M * K * 4);
        // the split-K partials of the dX and dW GEMMs, for a full chunk and
        // for the last (possibly narrower) one
        const int64_t eb = fp8 ? 1 : 2;
        const int64_t last = V - (V - 1) / Vc * Vc;
        for (const int64_t n : {Vc, last}) {
            const size_t g1 = gemm_workspace_bytes(M, K, n * eb, kOutF32);
            const size_t g2 = gemm_workspace_bytes(n, K, M * eb, kOutF32);
            g = g1 > g ? g1 : g;
            g = g2 > g ? g2 : g;
        }
    }
    l.gemm = c.take(g);
    l.total = c.used;
    return l;
}

size_t lm_head_ws_bytes(int64_t M, int64_t V, int64_t K, int fp8, bool bwd) {
    return lm_layout(M, V, K, fp8, bwd).total;
}

namespace {

// Quantise X (1x128 rows, k-major scales; with qt also the 128x1 column copy)
// and W (128x128 blocks, row-major scales: the same array serves the
// transposed copy as k-major block scales), E4M3, power-of-two scales.
void quantize_lm_operands(const uint16_t* X, const uint16_t* W, int64_t M, int64_t V, int64_t K, uint8_t* w8,
                          const LmLayout& l, bool bwd, hipStream_t stream) {
    QuantArgs ax{};
    ax.x = X; ax.rows = M; ax.cols = K; ax.ld = K;
    ax.q = w8 + l.xq; ax.scale = reinterpret_cast<float*>(w8 + l.xs);
    ax.qT = bwd ? w8 + l.xqt : nullptr; ax.scaleT = bwd ? reinterpret_cast<float*>(w8 + l.xst) : nullptr;
    ax.pow2 = 1; ax.kmajor = 1;
    launch_quantize(kE4M3, kQRow, ax, stream);
    QuantArgs aw{};
    aw.x = W; aw.rows = V; aw.cols = K; aw.ld = K;
    aw.q = w8 + l.wq; aw.scale = reinterpret_cast<float*>(w8 + l.wsc);
    aw.qT = bwd ? w8 + l.wqt : nullptr; aw.scaleT = bwd ? reinterpret_cast<float*>(w8 + l.wsct) : nullptr;
    aw.pow2 = 1; aw.kmajor = 0;
    launch_quantize(kE4M3, kQBlock, aw, stream);
}

// The logits GEMM of vocabulary columns [c0, c0 + n) with an LM-head output kind.
GemmProblem logits_problem(const uint16_t* X, const uint16_t* W, int64_t M, int64_t K, int64_t c0, int64_t n,
                           int fp8, uint8_t* w8, const LmLayout& l, int out) {
    GemmProblem g{};
    g.M = M; g.N = n; g.K = K;
    g.out = out;
    g.col0 = (int)c0;
    if (fp8) {
        g.A = w8 + l.xq; g.lda = K; g.fa = kE4M3; g.sa_mode = kSRow; g.sa_kmajor = 1;
        g.sa = reinterpret_cast<const float*>(w8 + l.xs);
        g.B = w8 + l.wq + c0 * K; g.ldb = K; g.fb = kE4M3; g.sb_mode = kSBlock; g.sb_kmajor = 0;
        g.sb = reinterpret_cast<const float*>(w8 + l.wsc) + (c0 / 128) * (K / 128);
    } else {
        g.A = reinterpret_cast<const uint8_t*>(X); g.lda = K; g.fa = kBF16; g.sa_mode = kSNone;
        g.B = reinterpret_cast<const uint8_t*>(W + c0 * K); g.ldb = K; g.fb = kBF16; g.sb_mode = kSNone;
    }
    return g;
}

}  // namespace

void launch_lm_head_fwd(const uint16_t* X, const uint16_t* W, const int32_t* targets, int64_t M, int64_t V,
                        int64_t K, int fp8, float* lse, float* loss, void* ws, hipStream_t stream) {
    uint8_t* w8 = reinterpret_cast<uint8_t*>(ws);
    const LmLayout l = lm_layout(M, V, K, fp8, false);
    float* zt = reinterpret_cast<float*>(w8 + l.zt);
    fill_f32_kernel<<<(unsigned)((M + 255) / 256), 256, 0, stream>>>(zt, __builtin_nanf(""), M);
    if (fp8) quantize_lm_operands(X, W, M, V, K, w8, l, false, stream);
    GemmProblem g = logits_problem(X, W, M, K, 0, V, fp8, w8, l, kOutLseStats);
    g.targets = targets;
    g.stats = reinterpret_cast<float2*>(w8 + l.stats);
    g.stats_ld = V / 128;
    g.zt = zt;
    g.D = nullptr; g.ldd = V;
    launch_gemm(g, nullptr, stream);
    lse_rows_kernel<<<(unsigned)M, 256, 0, stream>>>(g.stats, g.stats_ld, (int)(V / 128), zt, lse, loss);
}

void launch_lm_head_bwd(const uint16_t* X, const uint16_t* W, const int32_t* targets, const float* lse, int64_t M,
                        int64_t V, int64_t K, int fp8, float grad_scale, uint16_t* dX, float* dW, void* ws,
                        hipStream_t stream) {
    uint8_t* w8 = reinterpret_cast<uint8_t*>(ws);
    const LmLayout l = lm_layout(M, V, K, fp8, true);
    const int64_t Vc = lm_head_chunk(V);
    if (fp8) {
        quantize_lm_operands(X, W, M, V, K, w8, l, true, stream);
    } else {
        transpose_bf16(X, M, K, K, reinterpret_cast<uint16_t*>(w8 + l.xt), M, stream);
        transpose_bf16(W, V, K, K, reinterpret_cast<uint16_t*>(w8 + l.wt), V, stream);
    }
    float* dxacc = reinterpret_cast<float*>(w8 + l.dxacc);
    uint16_t* dz = reinterpret_cast<uint16_t*>(w8 + l.dz);
    void* gws = w8 + l.gemm;
    for (int64_t c0 = 0; c0 < V; c0 += Vc) {
        const int64_t n = (V - c0) < Vc ? (V - c0) : Vc;
        // dz of the chunk's columns: the logits recomputed, the gradient
        // written as BF16 [M, n] or (FP8) as its E4M3 copies in 1x128 rows
        // (for dX) and 128x1 columns (for dW), k-major scales
        GemmProblem g = logits_problem(X, W, M, K, c0, n, fp8, w8, l, fp8 ? kOutSoftmaxGradQ : kOutSoftmaxGrad);
        g.targets = targets;
        g.lse = lse;
        g.grad_scale = grad_scale;
        g.D = fp8 ? nullptr : dz; g.ldd = n;
        if (fp8) {
            g.q8 = w8 + l.dzq; g.q8_scale = reinterpret_cast<float*>(w8 + l.dzs);
            g.q8t = w8 + l.dzqt; g.q8t_scale = reinterpret_cast<float*>(w8 + l.dzst);
        }
        launch_gemm(g, nullptr, stream);
        GemmProblem gx{}, gw{};
        gx.M = M; gx.N = K; gx.K = n; gx.out = kOutF32; gx.D = dxacc; gx.ldd = K; gx.accumulate = c0 > 0;
        gw.M = n; gw.N = K; gw.K = M; gw.out = kOutF32; gw.D = dW + c0 * K; gw.ldd = K;
        if (fp8) {
            // dX += dzq [M, n] (WqT columns [c0, c0 + n)), block scales k-major
            gx.A = w8 + l.dzq; gx.lda = n; gx.fa = kE4M3; gx.sa_mode = kSRow; gx.sa_kmajor = 1;
            gx.sa = reinterpret_cast<const float*>(w8 + l.dzs);
            gx.B = w8 + l.wqt + c0; gx.ldb = V; gx.fb = kE4M3; gx.sb_mode = kSBlock; gx.sb_kmajor = 1;
            gx.sb = reinterpret_cast<const float*>(w8 + l.wsc) + (c0 / 128) * (K / 128);
            // dW rows [c0, c0 + n) = dzqT [n, M] (XqT)^T
            gw.A = w8 + l.dzqt; gw.lda = M; gw.fa = kE4M3; gw.sa_mode = kSRow; gw.sa_kmajor = 1;
            gw.sa = reinterpret_cast<const float*>(w8 + l.dzst);
            gw.B = w8 + l.xqt; gw.ldb = M; gw.fb = kE4M3; gw.sb_mode = kSRow; gw.sb_kmajor = 1;
            gw.sb = reinterpret_cast<const float*>(w8 + l.xst);
        } else {
            uint16_t* dzt = reinterpret_cast<uint16_t*>(w8 + l.dzt);
            transpose_bf16(dz, M, n, n, dzt, M, stream);
            gx.A = reinterpret_cast<const uint8_t*>(dz); gx.lda = n; gx.fa = kBF16; gx.sa_mode = kSNone;
            gx.B = reinterpret_cast<const uint8_t*>(reinterpret_cast<uint16_t*>(w8 + l.wt) + c0); gx.ldb = V;
            gx.fb = kBF16; gx.sb_mode = kSNone;
            gw.A = reinterpret_cast<const uint8_t*>(dzt); gw.lda = M; gw.fa = kBF16; gw.sa_mode = kSNone;
            gw.B = w8 + l.xt; gw.ldb = M; gw.fb = kBF16; gw.sb_mode = kSNone;
        }
        launch_gemm(gx, gws, stream);
        launch_gemm(gw, gws, stream);
    }
    const int64_t n4 = M * K / 4;
    f32_to_bf16_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, stream>>>(dxacc, dX, n4);
}

}  // namespace puro
