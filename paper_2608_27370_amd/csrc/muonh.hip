// MuonH: the Muon update under the hyperball wrapper (gfx950), for `count`
// matrices of one shape stored back to back.
//
// Section 3.3 (Hyperball Optimization), equation hyperball-update: each
// wrapped matrix keeps its initial Frobenius radius R; with the Muon update u
// and the weight learning rate eta,
//
//   W~ = W - eta R u / ||u||_F,     W' = R W~ / ||W~||_F.
//
// The Muon update (momentum with a Nesterov look-ahead, then the quintic
// Newton-Schulz orthogonalisation; the paper states neither, so these follow
// the published method):
//
//   buf' = mu buf + (1 - mu) G,   V = (1 - mu) G + mu buf'   (FP32 state)
//   X_0  = V / (||V|| + 1e-7), transposed when rows > cols (r <= c below)
//   A = X X^T,  B = b A + c A A^T,  X' = a X + B X        (BF16, 5 steps)
//
// Passes (n elements per matrix):
//   momentum     G, buf -> buf'; sums of V^2 in double per block      HBM, 12 n B
//   scale        one block per matrix: 1 / (||V|| + eps)
//   start        G, buf' -> X_0 in both orientations (BF16)            HBM, 12 n B
//   per step     three batched BF16 GEMMs (A, B, X') and the transpose of X'
//   reduce       sums of W^2, W.u, u^2 in double per block             HBM, 6 n B
//   coeffs       k1 = eta R / ||u||, ||W~||^2 = ||W||^2 - 2 k1 W.u + k1^2 ||u||^2,
//                k2 = R / ||W~||
//   apply        W' = k2 (W - k1 u), its BF16 copy, u                  HBM, 12-16 n B
// The GEMMs keep X and X^T: the Gram product reduces along X's rows and the
// update along X^T's rows, and both operands of the kernel are
// reduction-contiguous.

#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace puro {

namespace {

constexpr int kRed = 512;            // reduction blocks per matrix
constexpr double kNsEps = 1e-7;
constexpr float kNsA = 3.4445f, kNsB = -4.7750f, kNsC = 2.0315f;

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Sum of the 256 threads' v (three values at once); result valid in thread 0.
__device__ __forceinline__ void block_sum3(double& a, double& b, double& c) {
    __shared__ double red[3][4];
    a = wave_sum(a); b = wave_sum(b); c = wave_sum(c);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (lane == 0) { red[0][w] = a; red[1][w] = b; red[2][w] = c; }
    __syncthreads();
    if (threadIdx.x == 0) {
        a = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
        b = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
        c = (red[2][0] + red[2][1]) + (red[2][2] + red[2][3]);
    }
}

// The momentum update in binary32, each product and sum rounded on its own:
// the pragma keeps the compiler from fusing a product into the sum.
__device__ __forceinline__ float momentum_buf(float g, float b, float mu, float om) {
#pragma clang fp contract(off)
    return mu * b + om * g;
}
__device__ __forceinline__ float nesterov_v(float g, float nb, float mu, float om) {
#pragma clang fp contract(off)
    return om * g + mu * nb;
}
__device__ __forceinline__ float momentum1(float g, float& b, float mu, float om, int nesterov) {
    b = momentum_buf(g, b, mu, om);
    return nesterov ? nesterov_v(g, b, mu, om) : b;
}

// buf <- buf' and the partial sums of V^2 of block blockIdx.x of matrix
// blockIdx.y; n4 float4 per matrix.
__global__ __launch_bounds__(256) void momentum_kernel(const float* __restrict__ G, float* __restrict__ buf,
                                                       int64_t n4, float mu, float om, int nesterov,
                                                       double* __restrict__ partial) {
    const int64_t off = (int64_t)blockIdx.y * n4;
    const float4* g4 = reinterpret_cast<const float4*>(G) + off;
    float4* b4 = reinterpret_cast<float4*>(buf) + off;
    double s = 0.0, z1 = 0.0, z2 = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)kRed * 256) {
        const float4 g = g4[i];
        float4 b = b4[i];
        const float v0 = momentum1(g.x, b.x, mu, om, nesterov), v1 = momentum1(g.y, b.y, mu, om, nesterov);
        const float v2 = momentum1(g.z, b.z, mu, om, nesterov), v3 = momentum1(g.w, b.w, mu, om, nesterov);
        b4[i] = b;
        s += (double)v0 * v0 + (double)v1 * v1 + (double)v2 * v2 + (double)v3 * v3;
    }
    block_sum3(s, z1, z2);
    if (threadIdx.x == 0) partial[(int64_t)blockIdx.y * kRed + blockIdx.x] = s;
}

// scale[b] = 1 / (||V_b|| + eps) from the kRed partial sums, summed in a fixed order.
__global__ __launch_bounds__(256) void ns_scale_kernel(const double* __restrict__ partial, float* __restrict__ scale) {
    double s = 0.0, z1 = 0.0, z2 = 0.0;
    for (int i = threadIdx.x; i < kRed; i += 256) s += partial[(int64_t)blockIdx.x * kRed + i];
    block_sum3(s, z1, z2);
    if (threadIdx.x == 0) scale[blockIdx.x] = (float)(1.0 / (sqrt(s) + kNsEps));
}

// X_0 = BF16(V * scale) of a 64 x 64 tile of V [rows, cols] (matrix
// blockIdx.z), written in V's layout (xv, pitch cols) and transposed (xt,
// pitch rows). V is recomputed from G and buf' with the same binary32 steps.
__global__ __launch_bounds__(256) void ns_start_kernel(const float* __restrict__ G, const float* __restrict__ buf,
                                                       int64_t rows, int64_t cols, float mu, float om, int nesterov,
                                                       const float* __restrict__ scale, uint16_t* __restrict__ xv,
                                                       uint16_t* __restrict__ xt) {
    __shared__ uint16_t t[64][66];
    const int64_t n = rows * cols;
    const int64_t bz = blockIdx.z;
    G += bz * n; buf += bz * n; xv += bz * n; xt += bz * n;
    const float s = scale[bz];
    const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    // rows and columns are multiples of 128: every tile is whole
#pragma unroll 4
    for (int i = 0; i < 64; i += 4) {
        const int64_t idx = (r0 + ty + i) * cols + c0 + tx;
        const float b = buf[idx];
        const float g = G[idx];
        // buf already holds buf': recompute V from it without updating it again
        const float v = nesterov ? nesterov_v(g, b, mu, om) : b;
        const uint16_t x = to_bf16(__fmul_rn(v, s));
        xv[idx] = x;
        t[ty + i][tx] = x;
    }
    __syncthreads();
#pragma unroll 4
    for (int i = 0; i < 64; i += 4) xt[(c0 + ty + i) * rows + r0 + tx] = t[tx][ty + i];
}

// Partial sums of W^2, W.u and u^2 (u BF16) of block blockIdx.x of matrix blockIdx.y.
__global__ __launch_bounds__(256) void hyperball_reduce_kernel(const float* __restrict__ W,
                                                               const uint16_t* __restrict__ u, int64_t n4,
                                                               double* __restrict__ partial) {
    const int64_t off = (int64_t)blockIdx.y * n4;
    const float4* w4 = reinterpret_cast<const float4*>(W) + off;
    const uint2* u4 = reinterpret_cast<const uint2*>(u) + off;
    double ww = 0.0, wu = 0.0, uu = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)kRed * 256) {
        const float4 w = w4[i];
        const uint2 q = u4[i];
        const float a[4] = {w.x, w.y, w.z, w.w};
        const float b[4] = {bf16lo(q.x), bf16hi(q.x), bf16lo(q.y), bf16hi(q.y)};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            ww += (double)a[j] * a[j];
            wu += (double)a[j] * b[j];
            uu += (double)b[j] * b[j];
        }
    }
    block_sum3(ww, wu, uu);
    if (threadIdx.x == 0) {
        double* p = partial + ((int64_t)blockIdx.y * kRed + blockIdx.x) * 3;
        p[0] = ww; p[1] = wu; p[2] = uu;
    }
}

// k[2b] = k1 = eta R / ||u|| (0 for u = 0: no displacement) and k[2b + 1] =
// k2 = R / ||W - k1 u||, with ||W - k1 u||^2 expanded in the sums.
__global__ __launch_bounds__(256) void hyperball_coeffs_kernel(const double* __restrict__ partial,
                                                               const float* __restrict__ radius, float eta,
                                                               float* __restrict__ k) {
    double ww = 0.0, wu = 0.0, uu = 0.0;
    for (int i = threadIdx.x; i < kRed; i += 256) {
        const double* p = partial + ((int64_t)blockIdx.x * kRed + i) * 3;
        ww += p[0]; wu += p[1]; uu += p[2];
    }
    block_sum3(ww, wu, uu);
    if (threadIdx.x == 0) {
        const double R = radius[blockIdx.x];
        const float k1 = uu > 0.0 ? (float)((double)eta * R / sqrt(uu)) : 0.0f;
        const double t2 = ww - 2.0 * (double)k1 * wu + (double)k1 * (double)k1 * uu;
        k[2 * blockIdx.x] = k1;
        k[2 * blockIdx.x + 1] = (float)(R / sqrt(t2 > 0.0 ? t2 : 0.0));
    }
}

// W' = k2 * (W - k1 u) in place, with the optional BF16 copy of W' and of u.
__global__ __launch_bounds__(256) void hyperball_apply_kernel(float* __restrict__ W, const uint16_t* __restrict__ u,
                                                              int64_t n4, const float* __restrict__ k,
                                                              uint16_t* __restrict__ w_bf16,
                                                              uint16_t* __restrict__ u_out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n4) return;
    const int64_t off = (int64_t)blockIdx.y * n4;
    const float k1 = k[2 * blockIdx.y], k2 = k[2 * blockIdx.y + 1];
    float4* w4 = reinterpret_cast<float4*>(W) + off;
    const uint2 q = reinterpret_cast<const uint2*>(u)[off + i];
    float4 w = w4[i];
    w.x = __fmul_rn(k2, fmaf(-k1, bf16lo(q.x), w.x));
    w.y = __fmul_rn(k2, fmaf(-k1, bf16hi(q.x), w.y));
    w.z = __fmul_rn(k2, fmaf(-k1, bf16lo(q.y), w.z));
    w.w = __fmul_rn(k2, fmaf(-k1, bf16hi(q.y), w.w));
    w4[i] = w;
    if (w_bf16) reinterpret_cast<uint2*>(w_bf16)[off + i] = make_uint2(pack_bf16x2(w.x, w.y), pack_bf16x2(w.z, w.w));
    if (u_out) reinterpret_cast<uint2*>(u_out)[off + i] = q;
}

constexpr size_t kAl = 256;
size_t al(size_t v) { return (v + kAl - 1) / kAl * kAl; }

struct NsLayout {
    size_t x, xt, xn, xnt, a, b, partial, scal, gemm, total;
};

// r <= c: the oriented shape.
NsLayout ns_layout(int64_t count, int64_t r, int64_t c) {
    NsLayout l{};
    size_t at = 0;
    auto take = [&](size_t bytes) { const size_t o = at; at = al(at + bytes); return o; };
    const size_t xb = (size_t)count * r * c * 2, ab = (size_t)count * r * r * 2;
    l.x = take(xb); l.xt = take(xb); l.xn = take(xb); l.xnt = take(xb);
    l.a = take(ab); l.b = take(ab);
    l.partial = take((size_t)count * kRed * 3 * sizeof(double));
    l.scal = take((size_t)count * 2 * sizeof(float));
    // split-K partials of the three products (K in bytes of BF16 rows)
    size_t g = gemm_workspace_bytes(r, r, 2 * c, kOutBF16, (int)count);
    const size_t g2 = gemm_workspace_bytes(r, r, 2 * r, kOutBF16Epi, (int)count);
    const size_t g3 = gemm_workspace_bytes(r, c, 2 * r, kOutBF16Epi, (int)count);
    g = g2 > g ? g2 : g;
    g = g3 > g ? g3 : g;
    l.gemm = take(g);
    l.total = at;
    return l;
}

// `steps` Newton-Schulz steps on x [count][r][c] (with xt its transpose),
// ping-ponging with xn/xnt; returns which buffers hold the result (0: x/xt, 1:
// xn/xnt). The transposed copy of the result is made only when `need_t`.
int ns_steps(uint8_t* w8, const NsLayout& l, int64_t count, int64_t r, int64_t c, int steps, bool need_t,
             hipStream_t stream) {
    uint16_t* X[2] = {reinterpret_cast<uint16_t*>(w8 + l.x), reinterpret_cast<uint16_t*>(w8 + l.xn)};
    uint16_t* Xt[2] = {reinterpret_cast<uint16_t*>(w8 + l.xt), reinterpret_cast<uint16_t*>(w8 + l.xnt)};
    uint16_t* A = reinterpret_cast<uint16_t*>(w8 + l.a);
    uint16_t* B = reinterpret_cast<uint16_t*>(w8 + l.b);
    void* gws = w8 + l.gemm;
    const int bt = (int)count;
    int cur = 0;
    for (int s = 0; s < steps; ++s) {
        GemmProblem gram{};
        gram.M = r; gram.N = r; gram.K = c;
        gram.A = reinterpret_cast<const uint8_t*>(X[cur]); gram.lda = c; gram.fa = kBF16; gram.sa_mode = kSNone;
        gram.B = reinterpret_cast<const uint8_t*>(X[cur]); gram.ldb = c; gram.fb = kBF16; gram.sb_mode = kSNone;
        gram.D = A; gram.ldd = r; gram.out = kOutBF16;
        gram.batch = bt; gram.bsa = r * c; gram.bsb = r * c; gram.bsd = r * r;
        gram.upper = 1;   // X X^T is symmetric: the upper tiles, then their mirror
        launch_gemm(gram, gws, stream);
        mirror_lower_bf16(A, r, r, gemm_tile(gram), stream, bt, r * r);
        GemmProblem poly{};
        poly.M = r; poly.N = r; poly.K = r;
        poly.A = reinterpret_cast<const uint8_t*>(A); poly.lda = r; poly.fa = kBF16; poly.sa_mode = kSNone;
        poly.B = reinterpret_cast<const uint8_t*>(A); poly.ldb = r; poly.fb = kBF16; poly.sb_mode = kSNone;
        poly.D = B; poly.ldd = r; poly.out = kOutBF16Epi;
        poly.residual = A; poly.ldr = r; poly.alpha = kNsC; poly.res_scale = kNsB;
        poly.batch = bt; poly.bsa = r * r; poly.bsb = r * r; poly.bsd = r * r; poly.bsr = r * r;
        poly.upper = 1;   // b A + c A A^T is symmetric too
        launch_gemm(poly, gws, stream);
        mirror_lower_bf16(B, r, r, gemm_tile(poly), stream, bt, r * r);
        GemmProblem upd{};
        upd.M = r; upd.N = c; upd.K = r;
        upd.A = reinterpret_cast<const uint8_t*>(B); upd.lda = r; upd.fa = kBF16; upd.sa_mode = kSNone;
        upd.B = reinterpret_cast<const uint8_t*>(Xt[cur]); upd.ldb = r; upd.fb = kBF16; upd.sb_mode = kSNone;
        upd.D = X[1 - cur]; upd.ldd = c; upd.out = kOutBF16Epi;
        upd.residual = X[cur]; upd.ldr = c; upd.res_scale = kNsA;
        upd.batch = bt; upd.bsa = r * r; upd.bsb = r * c; upd.bsd = r * c; upd.bsr = r * c;
        launch_gemm(upd, gws, stream);
        cur = 1 - cur;
        if (s + 1 < steps || need_t) transpose_bf16(X[cur], r, c, c, Xt[cur], r, stream, bt, r * c, r * c);
    }
    return cur;
}

}  // namespace

size_t muonh_ws_bytes(int64_t count, int64_t rows, int64_t cols) {
    const int64_t r = rows < cols ? rows : cols, c = rows < cols ? cols : rows;
    return ns_layout(count, r, c).total;
}

size_t newton_schulz_ws_bytes(int64_t count, int64_t r, int64_t c) { return ns_layout(count, r, c).total; }

void launch_newton_schulz(const uint16_t* X, int64_t count, int64_t r, int64_t c, int steps, uint16_t* out,
                          void* ws, hipStream_t stream) {
    uint8_t* w8 = reinterpret_cast<uint8_t*>(ws);
    const NsLayout l = ns_layout(count, r, c);
    const size_t xb = (size_t)count * r * c * 2;
    hipMemcpyAsync(w8 + l.x, X, xb, hipMemcpyDeviceToDevice, stream);
    transpose_bf16(X, r, c, c, reinterpret_cast<uint16_t*>(w8 + l.xt), r, stream, (int)count, r * c, r * c);
    const int cur = ns_steps(w8, l, count, r, c, steps, false, stream);
    hipMemcpyAsync(out, w8 + (cur ? l.xn : l.x), xb, hipMemcpyDeviceToDevice, stream);
}

void launch_muonh_step(int64_t count, int64_t rows, int64_t cols, float* W, uint16_t* w_bf16, const float* G,
                       float* buf, const float* radius, float mu, int nesterov, float eta, int steps,
                       uint16_t* u_out, void* ws, hipStream_t stream) {
    uint8_t* w8 = reinterpret_cast<uint8_t*>(ws);
    const bool tr = rows > cols;
    const int64_t r = tr ? cols : rows, c = tr ? rows : cols;
    const NsLayout l = ns_layout(count, r, c);
    const int64_t n4 = rows * cols / 4;
    const float om = 1.0f - mu;
    double* partial = reinterpret_cast<double*>(w8 + l.partial);
    float* scal = reinterpret_cast<float*>(w8 + l.scal);
    const dim3 red((unsigned)kRed, (unsigned)count);
    momentum_kernel<<<red, 256, 0, stream>>>(G, buf, n4, mu, om, nesterov, partial);
    ns_scale_kernel<<<(unsigned)count, 256, 0, stream>>>(partial, scal);
    // X_0 in V's layout and transposed; with rows > cols, X = V^T
    uint16_t* xv = reinterpret_cast<uint16_t*>(w8 + (tr ? l.xt : l.x));
    uint16_t* xtv = reinterpret_cast<uint16_t*>(w8 + (tr ? l.x : l.xt));
    const dim3 sg((unsigned)(cols / 64), (unsigned)(rows / 64), (unsigned)count);
    ns_start_kernel<<<sg, 256, 0, stream>>>(G, buf, rows, cols, mu, om, nesterov, scal, xv, xtv);
    const int cur = ns_steps(w8, l, count, r, c, steps, tr, stream);
    // u in W's layout: X itself, or its transpose when the matrix was turned
    const uint16_t* u = reinterpret_cast<const uint16_t*>(w8 + (cur ? (tr ? l.xnt : l.xn) : (tr ? l.xt : l.x)));
    hyperball_reduce_kernel<<<red, 256, 0, stream>>>(W, u, n4, partial);
    hyperball_coeffs_kernel<<<(unsigned)count, 256, 0, stream>>>(partial, radius, eta, scal);
    const dim3 ag((unsigned)((n4 + 255) / 256), (unsigned)count);
    hyperball_apply_kernel<<<ag, 256, 0, stream>>>(W, u, n4, scal, w_bf16, u_out);
}

}  // namespace puro
