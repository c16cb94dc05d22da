// Device helpers shared by the quantiser and GEMM kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace puro {

// FP8 format ids; the values double as the MFMA operand-format selectors of
// the gfx950 f8f6f4 instructions (0 = E4M3, 1 = E5M2). kBF16 marks BF16
// GEMM operands (the 32x32x16 BF16 matrix instruction).
enum : int { kE4M3 = 0, kE5M2 = 1, kBF16 = 2 };

template <int FMT> struct Fp8Traits;
template <> struct Fp8Traits<kE4M3> {
    static constexpr float kMax = 448.0f;
    static constexpr uint32_t kMaxBits = 0x43E00000u;  // 448.0f
    static constexpr int kEmax = 8;                    // 448 = 1.75 * 2^8
};
template <> struct Fp8Traits<kE5M2> {
    static constexpr float kMax = 57344.0f;
    static constexpr uint32_t kMaxBits = 0x47600000u;  // 57344.0f
    static constexpr int kEmax = 15;                   // 57344 = 1.75 * 2^15
};

__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// Two binary32 values -> two BF16 (round to nearest even) in one word, low
// half first: the conversion instruction (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((v2f){a, b}, v2bf));
}
__device__ __forceinline__ uint16_t to_bf16(float a) { return (uint16_t)pack_bf16x2(a, 0.0f); }

// e^x in binary32 within about 2 ulp: 2^(x log2 e) by the exp2 instruction,
// with the rounding error of the product x log2 e (exact from an FMA, plus
// the low part of log2 e) applied as a first-order factor, so that the error
// does not grow with |x|. Overflows to infinity above x = 88.72 and gives 0
// below -103; e^(+inf) = inf, e^(-inf) = 0, NaN stays NaN.
__device__ __forceinline__ float exp_f32(float x) {
    constexpr float kL2eHi = 1.44269502162933349609375f;      // log2 e rounded to binary32
    constexpr float kL2eLo = 1.925962989e-8f;                 // log2 e - kL2eHi
    constexpr float kLn2 = 0.693147180559945309f;
    const float t = x * kL2eHi;
    // the correction only where it matters and stays finite (the result is
    // exactly 0 or infinity beyond)
    const float err = fabsf(x) < 100.0f ? fmaf(x, kL2eHi, -t) + x * kL2eLo : 0.0f;   // x log2 e - t
    return __builtin_amdgcn_exp2f(t) * (1.0f + err * kLn2);
}

// e^x as m * 2^n, m in [1, 2) within about 2 ulp, n an integer: the exp2
// instruction only ever sees the fraction of x log2 e, so results that lie
// below binary32's normal range (where that instruction flushes to zero) keep
// their significand. For finite x with |x| < 2^24.
__device__ __forceinline__ float exp_split(float x, int& n) {
    constexpr float kL2eHi = 1.44269502162933349609375f;
    constexpr float kL2eLo = 1.925962989e-8f;
    constexpr float kLn2 = 0.693147180559945309f;
    const float t = x * kL2eHi;
    const float err = fmaf(x, kL2eHi, -t) + x * kL2eLo;
    const float fl = floorf(t);
    n = (int)fl;
    return __builtin_amdgcn_exp2f(t - fl) * (1.0f + err * kLn2);
}

// Gate values below kDeepGate take the scaled evaluation: there 1 + e^-g equals
// e^-g in binary32, so silu(g) = g e^g, and e^g and the reciprocal of 1 + e^-g
// approach or leave binary32's normal range. Below kFarGate the result is
// zero in binary32 (|silu(g)| < 2^-270), and e^-g overflows in the direct
// evaluation, which then gives -0 as binary32 arithmetic does.
constexpr float kDeepGate = -64.0f;
constexpr float kFarGate = -192.0f;

// x * y * z * e^g for g in [kFarGate, kDeepGate): the factors' significands
// multiplied (magnitude in [1/8, 2)) and the exponents added, then one ldexp,
// which rounds once (correctly into the subnormal range) instead of flushing;
// no intermediate product overflows or underflows.
__device__ __forceinline__ float mul_exp_deep(float x, float y, float z, float g) {
    int n, ex, ey, ez;
    const float m = exp_split(g, n);
    const float mx = __builtin_frexpf(x, &ex);
    const float my = __builtin_frexpf(y, &ey);
    const float mz = __builtin_frexpf(z, &ez);
    return __builtin_ldexpf(mx * my * mz * m, n + ex + ey + ez);
}

// SwiGLU of one gate/up pair in binary32: silu(g) * u with silu(g) = g / (1 + e^-g),
// the quotient as g times the reciprocal instruction's 1 / (1 + e^-g) (about
// 1 ulp); altogether within about 5 ulp of the exact value. Deep in the
// negative tail (g < -64) silu(g) u = g u e^g in the scaled form above, so
// that no step flushes a value below binary32's normal range to zero.
__device__ __forceinline__ float swiglu1(float g, float u) {
    if (g < kDeepGate && g >= kFarGate) return mul_exp_deep(g, u, 1.0f, g);
    return g * __builtin_amdgcn_rcpf(1.0f + exp_f32(-g)) * u;
}

// Eight SwiGLU values, BF16 (round to nearest even), from four words of gate
// values and four words of up values (two BF16 values per word, low first).
__device__ __forceinline__ void swiglu8(const uint32_t g[4], const uint32_t u[4], uint32_t h[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
        h[i] = pack_bf16x2(swiglu1(bf16lo(g[i]), bf16lo(u[i])), swiglu1(bf16hi(g[i]), bf16hi(u[i])));
}

// The SwiGLU's backward for one element in binary32: from dH and the saved
// gate g and up u, dg = dH * u * silu'(g) with silu'(g) = s (1 + g (1 - s)),
// s = 1 / (1 + e^-g) (the reciprocal instruction), or du = dH * silu(g) =
// dH * g * s. Deep in the negative tail (g < -64, where s = e^g and 1 - s = 1
// in binary32) dg = dH u e^g (1 + g) and du = dH g e^g in the scaled form.
__device__ __forceinline__ float swiglu_bwd1(float dh, float g, float u, bool dg) {
    if (g < kDeepGate && g >= kFarGate) return dg ? mul_exp_deep(dh, u, 1.0f + g, g) : mul_exp_deep(dh, g, 1.0f, g);
    const float sg = __builtin_amdgcn_rcpf(1.0f + exp_f32(-g));
    return dg ? dh * u * (sg * fmaf(g, 1.0f - sg, 1.0f)) : dh * (g * sg);
}

// Eight RMSNorm outputs, BF16 (round to nearest even): x * r * gamma in
// binary32 from four words of x, the row's r = rstd and four words of gamma.
__device__ __forceinline__ void rmsnorm8(const uint32_t x[4], float r, const uint32_t g[4], uint32_t y[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
        y[i] = pack_bf16x2(bf16lo(x[i]) * r * bf16lo(g[i]), bf16hi(x[i]) * r * bf16hi(g[i]));
}

// Hardware conversion of two binary32 values to two FP8 codes (RNE), written
// into byte pair HI (false: bytes 0-1, true: bytes 2-3) of `old`. In range it
// rounds exactly like the encoding this library defines; it does not
// saturate (too-large values become NaN/Inf) and gives NaN a sign, which the
// callers below handle.
template <int FMT, bool HI>
__device__ __forceinline__ uint32_t cvt_pk(float a, float b, uint32_t old) {
    if constexpr (FMT == kE4M3)
        return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, HI);
    else
        return (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(a, b, (int)old, HI);
}

// Four values already known to lie within [-FMAX, FMAX] in magnitude up to
// one binary32 rounding of the scale (never NaN): hardware path.
template <int FMT>
__device__ __forceinline__ uint32_t encode4_fast(float a, float b, float c, float d) {
    uint32_t w = cvt_pk<FMT, false>(a, b, 0u);
    return cvt_pk<FMT, true>(c, d, w);
}

// One value of any kind: saturate finite and infinite magnitudes above FMAX
// to +-FMAX, map every NaN to 0x7F.
template <int FMT>
__device__ __forceinline__ uint32_t encode1_safe(float v) {
    uint32_t u = __float_as_uint(v);
    uint32_t m = u & 0x7FFFFFFFu;
    bool nan = m > 0x7F800000u;
    m = m < Fp8Traits<FMT>::kMaxBits ? m : Fp8Traits<FMT>::kMaxBits;
    float c = __uint_as_float((u & 0x80000000u) | m);
    uint32_t code = cvt_pk<FMT, false>(c, 0.0f, 0u) & 0xFFu;
    return nan ? 0x7Fu : code;
}

template <int FMT>
__device__ __forceinline__ uint32_t encode4_safe(float a, float b, float c, float d) {
    return encode1_safe<FMT>(a) | (encode1_safe<FMT>(b) << 8) | (encode1_safe<FMT>(c) << 16) |
           (encode1_safe<FMT>(d) << 24);
}

// Encode 8 BF16 values (4 packed words) times r into 8 codes (2 words).
template <int FMT, bool SAFE>
__device__ __forceinline__ uint2 encode8(const uint32_t w[4], float r) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf16lo(w[i]) * r;
        v[2 * i + 1] = bf16hi(w[i]) * r;
    }
    uint2 out;
    if constexpr (SAFE) {
        out.x = encode4_safe<FMT>(v[0], v[1], v[2], v[3]);
        out.y = encode4_safe<FMT>(v[4], v[5], v[6], v[7]);
    } else {
        out.x = encode4_fast<FMT>(v[0], v[1], v[2], v[3]);
        out.y = encode4_fast<FMT>(v[4], v[5], v[6], v[7]);
    }
    return out;
}

// Encode with one multiplier per column of the 8x8 block (column-grouped scales).
template <int FMT, bool SAFE>
__device__ __forceinline__ uint2 encode8_cols(const uint32_t w[4], const float r[8]) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf16lo(w[i]) * r[2 * i];
        v[2 * i + 1] = bf16hi(w[i]) * r[2 * i + 1];
    }
    uint2 out;
    if constexpr (SAFE) {
        out.x = encode4_safe<FMT>(v[0], v[1], v[2], v[3]);
        out.y = encode4_safe<FMT>(v[4], v[5], v[6], v[7]);
    } else {
        out.x = encode4_fast<FMT>(v[0], v[1], v[2], v[3]);
        out.y = encode4_fast<FMT>(v[4], v[5], v[6], v[7]);
    }
    return out;
}

// Codes of the 8 BF16 values of w divided by the power of two s, one
// v_cvt_scalef32_pk_{fp8,bf8}_bf16 per pair: the instruction rounds x / s
// exactly as v_cvt_pk_{fp8,bf8}_f32 rounds it (the same codes as encode8
// with r = 1 / s, verified bit for bit over every BF16 pattern on the
// hardware), and like it does not saturate: for groups whose values stay
// within the format after scaling. s must be a normal binary32 number.
typedef short short2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
template <int FMT, bool HI>
__device__ __forceinline__ short2_t cvt_scaled_pk(short2_t old, uint32_t x, float s) {
    const bf16x2_t v = __builtin_bit_cast(bf16x2_t, x);
    if constexpr (FMT == kE4M3) return __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(old, v, s, HI);
    else return __builtin_amdgcn_cvt_scalef32_pk_bf8_bf16(old, v, s, HI);
}
template <int FMT>
__device__ __forceinline__ uint2 encode8_pow2(const uint32_t w[4], float s) {
    short2_t a = cvt_scaled_pk<FMT, false>(short2_t{0, 0}, w[0], s);
    a = cvt_scaled_pk<FMT, true>(a, w[1], s);
    short2_t b = cvt_scaled_pk<FMT, false>(short2_t{0, 0}, w[2], s);
    b = cvt_scaled_pk<FMT, true>(b, w[3], s);
    return make_uint2(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b));
}

// 8x8 transpose of 16-bit values: w[i] holds row i (word j = columns 2j and
// 2j + 1, the low half first), wt[c] column c in the same form. One byte
// permute per output word: a pair of rows' halves meet in one word.
__device__ __forceinline__ void transpose8x8_b16(const uint32_t w[8][4], uint32_t wt[8][4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            wt[2 * j][k] = __builtin_amdgcn_perm(w[2 * k + 1][j], w[2 * k][j], 0x05040100u);      // low halves
            wt[2 * j + 1][k] = __builtin_amdgcn_perm(w[2 * k + 1][j], w[2 * k][j], 0x07060302u);  // high halves
        }
}

// Both halves' unsigned 16-bit maxima in one instruction (v_pk_max_u16).
typedef unsigned short ushort2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pk_max_u16(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(ushort2_t, a),
                                                                  __builtin_bit_cast(ushort2_t, b)));
}
// The two BF16 magnitude patterns of a word, in place.
__device__ __forceinline__ uint32_t mag2(uint32_t w) { return w & 0x7FFF7FFFu; }

// Largest BF16 magnitude pattern among 8 values (4 words); as integers the
// magnitude patterns order like the magnitudes, and NaN patterns exceed Inf.
__device__ __forceinline__ uint32_t absmax_bits8(const uint32_t w[4]) {
    const uint32_t m = pk_max_u16(pk_max_u16(mag2(w[0]), mag2(w[1])), pk_max_u16(mag2(w[2]), mag2(w[3])));
    return max(m & 0xFFFFu, m >> 16);
}

// Power-of-two scale exponent; amax given as its BF16 magnitude pattern
// (finite, non-NaN), amax = 0 -> 0, clamped to [-127, 127]. Writing
// amax = f * 2^E with f in [1, 2) and FMAX = 1.75 * 2^Emax:
//  * default rule, the smallest e with amax <= FMAX * 2^e: e = E - Emax,
//    plus one when f > 1.75;
//  * OCP-MX rule (floor): e = E - Emax, floor(log2 amax) - Emax; values of
//    a group whose amax has f > 1.75 may then saturate.
template <int FMT>
__device__ __forceinline__ int pow2_exponent_bf16(uint32_t mag, bool floor_rule = false) {
    if (mag == 0) return 0;
    if (mag >= 0x7F80u) return 127;                 // infinity
    uint32_t bits = mag << 16;
    int ef = (int)(bits >> 23);
    if (ef == 0) return -127;                        // subnormal: far below the clamp
    int e = ef - 127 - Fp8Traits<FMT>::kEmax + (!floor_rule && (bits & 0x7FFFFFu) > 0x600000u ? 1 : 0);
    return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// Under the floor rule, whether a group with this amax (BF16 magnitude
// pattern) can hold values beyond FMAX after scaling (significand > 1.75).
__device__ __forceinline__ bool floor_rule_saturates(uint32_t mag) { return (mag & 0x7Fu) > 0x60u; }

// 2^e as binary32 for e in [-127, 127] (2^-127 is subnormal).
__device__ __forceinline__ float exp2i(int e) {
    return e >= -126 ? __uint_as_float((uint32_t)(e + 127) << 23) : __uint_as_float(0x00400000u);
}

// 8x8 byte transpose: in[i] holds row i (bytes 0..7 = columns 0..7, as a
// uint2), out[j] holds column j (bytes 0..7 = rows 0..7).
__device__ __forceinline__ void transpose8x8(const uint2 in[8], uint2 out[8]) {
    // 4x4 byte transpose of four words (rows) -> four words (columns)
    auto t4 = [](uint32_t a, uint32_t b, uint32_t c, uint32_t d, uint32_t o[4]) {
        // interleave bytes of (a, b) and (c, d)
        uint32_t ab_lo = __builtin_amdgcn_perm(b, a, 0x05010400u);  // a0 b0 a1 b1
        uint32_t ab_hi = __builtin_amdgcn_perm(b, a, 0x07030602u);  // a2 b2 a3 b3
        uint32_t cd_lo = __builtin_amdgcn_perm(d, c, 0x05010400u);  // c0 d0 c1 d1
        uint32_t cd_hi = __builtin_amdgcn_perm(d, c, 0x07030602u);  // c2 d2 c3 d3
        o[0] = __builtin_amdgcn_perm(cd_lo, ab_lo, 0x05040100u);    // a0 b0 c0 d0
        o[1] = __builtin_amdgcn_perm(cd_lo, ab_lo, 0x07060302u);    // a1 b1 c1 d1
        o[2] = __builtin_amdgcn_perm(cd_hi, ab_hi, 0x05040100u);    // a2 b2 c2 d2
        o[3] = __builtin_amdgcn_perm(cd_hi, ab_hi, 0x07060302u);    // a3 b3 c3 d3
    };
    uint32_t tl[4], tr[4], bl[4], br[4];
    t4(in[0].x, in[1].x, in[2].x, in[3].x, tl);  // rows 0-3, cols 0-3
    t4(in[0].y, in[1].y, in[2].y, in[3].y, tr);  // rows 0-3, cols 4-7
    t4(in[4].x, in[5].x, in[6].x, in[7].x, bl);  // rows 4-7, cols 0-3
    t4(in[4].y, in[5].y, in[6].y, in[7].y, br);  // rows 4-7, cols 4-7
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        out[j] = make_uint2(tl[j], bl[j]);
        out[4 + j] = make_uint2(tr[j], br[j]);
    }
}

}  // namespace puro
