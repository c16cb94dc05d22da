/*
 * Scaled FP8 GEMM of the oracle, in FP64, one output element at a time.
 *
 * Section 3.2 of the paper: the Fprop, Dgrad and Wgrad GEMMs of a linear layer
 * take FP8 operands and accumulate in higher precision; the operands carry
 * either one scale per tensor or one scale per 128-long group along the
 * reduction dimension (activations, gradients) or per 128x128 block (weights).
 *
 * For D[m][n] = sum_k A[m][k] * B[n][k] (both operands stored with the
 * reduction index k contiguous):
 *
 *   ref[m][n] = sum over k-blocks kb of sa(m, kb) * sb(n, kb)
 *                 * sum_{k in kb} val_a(A[m][k]) * val_b(B[n][k])
 *   den[m][n] = sum_k | sa(m, kb(k)) * val_a(A[m][k]) * sb(n, kb(k)) * val_b(B[n][k]) |
 *
 * where val_x is the 256-entry decode table of the operand's format, and the
 * scale mode of an operand with rows indexed by i is
 *   0: one scale s[0]; 1: s[i * ld_s + kb] (a scale per row and k-block);
 *   2: s[(i / 128) * ld_s + kb] (a scale per 128x128 block).
 * kblock is the k-block length (128 for grouped scales, K for one block).
 *
 * Test infrastructure only; plain loops, k ascending, no blocking.
 */
#include <math.h>
#include <stdint.h>

static double scale_at(const float* s, int mode, int64_t ld_s, int64_t i, int64_t kb)
{
    if (mode == 0) return (double)s[0];
    if (mode == 1) return (double)s[i * ld_s + kb];
    return (double)s[(i / 128) * ld_s + kb];
}

static void one_entry(int64_t m, int64_t n, int64_t K, int64_t kblock,
                      const uint8_t* a, int64_t lda, const double* lut_a,
                      const float* sa, int sa_mode, int64_t ld_sa,
                      const uint8_t* b, int64_t ldb, const double* lut_b,
                      const float* sb, int sb_mode, int64_t ld_sb,
                      double* ref, double* den)
{
    double acc = 0.0, mag = 0.0;
    for (int64_t k0 = 0; k0 < K; k0 += kblock) {
        int64_t kb = k0 / kblock;
        double s = scale_at(sa, sa_mode, ld_sa, m, kb) * scale_at(sb, sb_mode, ld_sb, n, kb);
        double part = 0.0, part_mag = 0.0;
        int64_t k1 = k0 + kblock < K ? k0 + kblock : K;
        for (int64_t k = k0; k < k1; ++k) {
            double p = lut_a[a[m * lda + k]] * lut_b[b[n * ldb + k]];
            part += p;
            part_mag += fabs(p);
        }
        acc += s * part;
        mag += fabs(s) * part_mag;
    }
    *ref = acc;
    *den = mag;
}

void oracle_gemm_fp64(int64_t M, int64_t N, int64_t K, int64_t kblock,
                      const uint8_t* a, int64_t lda, const double* lut_a,
                      const float* sa, int sa_mode, int64_t ld_sa,
                      const uint8_t* b, int64_t ldb, const double* lut_b,
                      const float* sb, int sb_mode, int64_t ld_sb,
                      double* ref, double* den)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n)
            one_entry(m, n, K, kblock, a, lda, lut_a, sa, sa_mode, ld_sa,
                      b, ldb, lut_b, sb, sb_mode, ld_sb, &ref[m * N + n], &den[m * N + n]);
}

void oracle_gemm_fp64_entries(int64_t count, const int64_t* ms, const int64_t* ns,
                              int64_t K, int64_t kblock,
                              const uint8_t* a, int64_t lda, const double* lut_a,
                              const float* sa, int sa_mode, int64_t ld_sa,
                              const uint8_t* b, int64_t ldb, const double* lut_b,
                              const float* sb, int sb_mode, int64_t ld_sb,
                              double* ref, double* den)
{
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t i = 0; i < count; ++i)
        one_entry(ms[i], ns[i], K, kblock, a, lda, lut_a, sa, sa_mode, ld_sa,
                  b, ldb, lut_b, sb, sb_mode, ld_sb, &ref[i], &den[i]);
}
