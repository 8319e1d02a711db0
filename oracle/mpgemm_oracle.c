/*
 * CPU ORACLE for LUT-based mixed-precision GEMM -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load this library.  It shares no code with the HIP path: it never sees the
 * packed weight layout, the reinterpreted scale/zero, or the GPU table layout.
 *
 * What it computes is the plain definition of the operation the paper's LUT
 * method reformulates (LUT Tensor Core, Section 3.1.2, Eq. 1 and Eq. 3; LMMA
 * semantics O = A x W^T + Acc, Section 3.3.1):
 *
 *     y[m, n] = sum_k  a[m, k] * r[n, k],     r[n, k] = s * (q[n, k] - z)   (Eq. 1)
 *
 * evaluated element by element in float64 (every product is exact in float64
 * for FP16 inputs, so the result is the real-valued product up to the rounding
 * of the final sum), or in int64 for INT8 activations.  It also holds the plain
 * definition of the precompute step's outputs (Section 3.1.1-3.1.2: per 4
 * activations, the half table of signed partial sums selected by Eq. 5) and the
 * FP32 per-token absmax INT8 activation quantizer used by the INT8 workload.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -shared -fPIC (see build.py).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define WFMT_UINT 0
#define WFMT_BINARY 1
#define WFMT_TERNARY 2

/* Real-valued weight r = s * (q - z) of one element (Eq. 1).
 * BINARY codes {0,1} stand for {-1,+1}: r = s * (2q - 1).
 * TERNARY codes are the integers {-1,0,+1}: r = s * w. */
static double weight_value(int wfmt, const void *codes, int64_t idx, double s, double z)
{
    if (wfmt == WFMT_UINT) {
        double q = (double)((const uint8_t *)codes)[idx];
        return s * (q - z);
    }
    if (wfmt == WFMT_BINARY) {
        double q = (double)((const uint8_t *)codes)[idx];
        return s * (2.0 * q - 1.0);
    }
    return s * (double)((const int8_t *)codes)[idx];
}

/* Integer weight of the INT8-activation path (BINARY or TERNARY only). */
static int64_t weight_int(int wfmt, const void *codes, int64_t idx)
{
    if (wfmt == WFMT_BINARY)
        return 2 * (int64_t)((const uint8_t *)codes)[idx] - 1;
    return (int64_t)((const int8_t *)codes)[idx];
}

/*
 * Dense FP mpGEMM, float64.  Computes y[i][c] for the row subset rows[0..n_rows)
 * and column subset cols[0..n_cols) (NULL subset = all rows / all columns).
 *   a      [M][K]   activations (float64 copies of the FP16 inputs)
 *   codes  [N][K]   uint8 (UINT, BINARY) or int8 (TERNARY)
 *   group  quantization group along K; 0 = one scale for the whole tensor
 *   scales [N][K/group] or [1];  zeros same shape as scales, UINT only
 *   acc    optional [n_rows][n_cols] added to the result (the "+Acc" term), may be NULL
 * Returns 0, or -1 on an invalid argument.
 */
int oracle_mpgemm_f64(int64_t M, int64_t N, int64_t K, const double *a,
                      const void *codes, int wfmt, int64_t group,
                      const double *scales, const double *zeros,
                      const int64_t *rows, int64_t n_rows,
                      const int64_t *cols, int64_t n_cols,
                      const double *acc, double *y)
{
    if (M < 0 || N < 0 || K < 0 || !codes || !scales || !y)
        return -1;
    if (group < 0 || (group > 0 && K % group != 0))
        return -1;
    if (wfmt == WFMT_UINT && !zeros)
        return -1;
    int64_t nr = rows ? n_rows : M;
    int64_t nc = cols ? n_cols : N;
    int64_t n_groups = group ? K / group : 1;
    int rc = 0;
#pragma omp parallel
    {
        double *r = (double *)malloc(sizeof(double) * (size_t)(K > 0 ? K : 1));
        if (!r) {
#pragma omp atomic write
            rc = -1;
        } else {
#pragma omp for schedule(dynamic, 4)
            for (int64_t c = 0; c < nc; ++c) {
                int64_t n = cols ? cols[c] : c;
                /* dequantize one weight row, element by element (Eq. 1) */
                for (int64_t k = 0; k < K; ++k) {
                    int64_t sidx = group ? n * n_groups + k / group : 0;
                    double s = scales[sidx];
                    double z = (wfmt == WFMT_UINT) ? zeros[sidx] : 0.0;
                    r[k] = weight_value(wfmt, codes, n * K + k, s, z);
                }
                for (int64_t i = 0; i < nr; ++i) {
                    int64_t m = rows ? rows[i] : i;
                    const double *am = a + m * K;
                    double sum = 0.0;
                    for (int64_t k = 0; k < K; ++k)
                        sum += am[k] * r[k];
                    if (acc)
                        sum += acc[i * nc + c];
                    y[i * nc + c] = sum;
                }
            }
            free(r);
        }
    }
    return rc;
}

/*
 * Per-token absmax INT8 quantizer, in FP32 with no fused multiply-add
 * (the activation-quantized workload; the paper names INT8 activations,
 * Sections 2.1 and 3.3.1, without fixing the quantizer):
 *   amax = max_k |a_k|;  amax == 0  ->  q = 0, s_a = 0;
 *   inv = 127 / amax (correctly rounded);  q_k = clamp(rint(a_k * inv), -127, 127)
 *   (round half to even);  s_a = amax / 127.
 */
void oracle_quantize_int8(int64_t M, int64_t K, const float *a, int8_t *q, float *s_a)
{
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        const float *am = a + m * K;
        float amax = 0.0f;
        for (int64_t k = 0; k < K; ++k) {
            float v = fabsf(am[k]);
            if (v > amax)
                amax = v;
        }
        if (amax == 0.0f) {
            for (int64_t k = 0; k < K; ++k)
                q[m * K + k] = 0;
            s_a[m] = 0.0f;
            continue;
        }
        volatile float inv = 127.0f / amax;
        for (int64_t k = 0; k < K; ++k) {
            volatile float prod = am[k] * inv;
            float r = rintf(prod);
            if (r > 127.0f)
                r = 127.0f;
            if (r < -127.0f)
                r = -127.0f;
            q[m * K + k] = (int8_t)r;
        }
        volatile float sa = amax / 127.0f;
        s_a[m] = sa;
    }
}

/*
 * Dense integer mpGEMM of INT8 activations with BINARY or TERNARY weights:
 *   acc[i][c] = sum_k int64(qa[m][k]) * w[n][k]
 * (subsets as in oracle_mpgemm_f64; acc_in optional, added).  Returns -1 for UINT.
 */
int oracle_mpgemm_i64(int64_t M, int64_t N, int64_t K, const int8_t *qa,
                      const void *codes, int wfmt,
                      const int64_t *rows, int64_t n_rows,
                      const int64_t *cols, int64_t n_cols,
                      const int64_t *acc_in, int64_t *acc)
{
    if (wfmt != WFMT_BINARY && wfmt != WFMT_TERNARY)
        return -1;
    int64_t nr = rows ? n_rows : M;
    int64_t nc = cols ? n_cols : N;
    (void)N;
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t c = 0; c < nc; ++c) {
        int64_t n = cols ? cols[c] : c;
        for (int64_t i = 0; i < nr; ++i) {
            int64_t m = rows ? rows[i] : i;
            int64_t sum = 0;
            for (int64_t k = 0; k < K; ++k)
                sum += (int64_t)qa[m * K + k] * weight_int(wfmt, codes, n * K + k);
            if (acc_in)
                sum += acc_in[i * nc + c];
            acc[i * nc + c] = sum;
        }
    }
    (void)M;
    return 0;
}

/*
 * FP32 output of the integer path: y = (float(acc) * s_a[row]) * s_w[col],
 * two round-to-nearest-even FP32 multiplies in that order.
 */
void oracle_int_output_f32(int64_t n_rows, int64_t n_cols, const int64_t *acc,
                           const float *s_a, const float *s_w, float *y)
{
    for (int64_t i = 0; i < n_rows; ++i)
        for (int64_t c = 0; c < n_cols; ++c) {
            volatile float t = (float)acc[i * n_cols + c] * s_a[i];
            volatile float u = t * s_w[c];
            y[i * n_cols + c] = u;
        }
}

/*
 * Half tables of the precompute step (Section 3.1.2, Eq. 4-5), float64.
 * For token m and group j of 4 consecutive activations a_0..a_3 (a_i = a[m][4j+i]),
 * the full table over a 4-bit pattern p = W_3 W_2 W_1 W_0 (MSB first) is
 *     LUT[p] = sum_i a_i * (2 * bit_{3-i}(p) - 1)        (bits {0,1} read as {-1,+1})
 * i.e. the pattern's most significant bit belongs to the first activation.
 * The half table keeps the patterns whose MSB is 0:  T[idx] = LUT[0 idx], idx in [0, 8).
 * K must be a multiple of 4.  Output T[m][j][idx].
 */
void oracle_half_tables_f64(int64_t M, int64_t K, const double *a, double *T)
{
    int64_t J = K / 4;
    for (int64_t m = 0; m < M; ++m)
        for (int64_t j = 0; j < J; ++j) {
            const double *g = a + m * K + 4 * j;
            for (int idx = 0; idx < 8; ++idx) {
                double t = 0.0;
                for (int i = 0; i < 4; ++i) {
                    int bit = (idx >> (3 - i)) & 1; /* i = 0 is the MSB, always 0 here */
                    t += g[i] * (bit ? 1.0 : -1.0);
                }
                T[(m * J + j) * 8 + idx] = t;
            }
        }
}

/* Same definition on INT8 activations, exact in int64. */
void oracle_half_tables_i64(int64_t M, int64_t K, const int8_t *qa, int64_t *T)
{
    int64_t J = K / 4;
    for (int64_t m = 0; m < M; ++m)
        for (int64_t j = 0; j < J; ++j) {
            const int8_t *g = qa + m * K + 4 * j;
            for (int idx = 0; idx < 8; ++idx) {
                int64_t t = 0;
                for (int i = 0; i < 4; ++i) {
                    int bit = (idx >> (3 - i)) & 1;
                    t += (int64_t)g[i] * (bit ? 1 : -1);
                }
                T[(m * J + j) * 8 + idx] = t;
            }
        }
}

/* Activation sums over each quantization group q: S[m][q] = sum_{k in q} a[m][k]. */
void oracle_group_sums_f64(int64_t M, int64_t K, int64_t group, const double *a, double *S)
{
    int64_t G = group ? group : K;
    int64_t Q = K / G;
    for (int64_t m = 0; m < M; ++m)
        for (int64_t q = 0; q < Q; ++q) {
            double s = 0.0;
            for (int64_t k = q * G; k < (q + 1) * G; ++k)
                s += a[m * K + k];
            S[m * Q + q] = s;
        }
}

void oracle_group_sums_i64(int64_t M, int64_t K, int64_t group, const int8_t *qa, int64_t *S)
{
    int64_t G = group ? group : K;
    int64_t Q = K / G;
    for (int64_t m = 0; m < M; ++m)
        for (int64_t q = 0; q < Q; ++q) {
            int64_t s = 0;
            for (int64_t k = q * G; k < (q + 1) * G; ++k)
                s += qa[m * K + k];
            S[m * Q + q] = s;
        }
}

/*
 * Per-token power-of-two normalizer of the FP16 table path:
 *   amax = max_k |a[m][k]|,  amax = f * 2^e with f in [0.5, 1)  ->  mult[m] = 2^e
 *   (mult = 1 when amax == 0).  Tables are built from a * 2^-e and the
 *   result is multiplied back by 2^e, which is exact in binary floating point.
 */
void oracle_token_pow2(int64_t M, int64_t K, const double *a, double *mult)
{
    for (int64_t m = 0; m < M; ++m) {
        double amax = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double v = fabs(a[m * K + k]);
            if (v > amax)
                amax = v;
        }
        if (amax == 0.0) {
            mult[m] = 1.0;
            continue;
        }
        int e = 0;
        (void)frexp(amax, &e);
        mult[m] = ldexp(1.0, e);
    }
}

/*
 * INT8 table quantization (Section 3.1.3): an approximation of the FP16-activation
 * path, so this follows the method's steps in order instead of a closed form.
 *   1. per token, the power-of-two normalization of the FP16 table path:
 *      x = a * 2^-e with max |a| = f 2^e, f in [0.5, 1)  (exact; it changes no code,
 *      only the unit of the scale);
 *   2. per group j of 4 activations, the 8-entry half table of Eq. 5 as exact real
 *      numbers, T[idx] = -x0 + (+-x1) + (+-x2) + (+-x3) (bit 2 of idx selects the
 *      sign of x1, bit 1 of x2, bit 0 of x3: the first activation is the MSB of a
 *      pattern, and the half table keeps the patterns whose MSB is 0);
 *   3. each table quantized on its own to INT8 with a symmetric scale: with
 *      amax = max_idx |T[idx]|, q = round(127 T / amax), ties to even (|q| <= 127
 *      by construction), and scale = amax / 127 rounded to the nearest FP32 value;
 *      q = 0 and scale = 0 for an all-zero table.  The paper asks for one INT8
 *      precision per table and fixes neither rounding nor scale format; this is the
 *      reading.
 * Exactness of this float64 evaluation: every x is an integer multiple of
 * u = 2^(-24-e) (FP16 values are multiples of 2^-24) below 1 in magnitude, so every
 * T is n u with |n| < 2^42 and its sums are exact in float64, in any order, and so
 * is 127 T (|127 n| < 2^49).  When 127 T / amax = 127 n / n_max is not a half-integer
 * it lies at least 1 / (2 n_max) > 2^-43 away from every half-integer, more than the
 * float64 division's rounding error (at most 2^-47 below 128), so rint of the
 * rounded quotient is the exact round-half-to-even.  The FP32 scale is the float64
 * quotient rounded to FP32; amax / 127 has a binary expansion of period 7 (or
 * terminates), so that second rounding never meets a tie the first one created.
 * Outputs q[m][j][8] (int8), scale[m][j] (float32), mult[m] = 2^e (float64).
 */
void oracle_lut8_tables(int64_t M, int64_t K, const float *a, int8_t *q, float *scale, double *mult)
{
    int64_t J = K / 4;
    for (int64_t m = 0; m < M; ++m) {
        float amax = 0.0f;
        for (int64_t k = 0; k < K; ++k) {
            float v = fabsf(a[m * K + k]);
            if (v > amax)
                amax = v;
        }
        int e = 0;
        if (amax != 0.0f)
            (void)frexpf(amax, &e);
        const double down = ldexp(1.0, -e);
        mult[m] = ldexp(1.0, e);
        for (int64_t j = 0; j < J; ++j) {
            double x[4], t[8], tmax = 0.0;
            for (int i = 0; i < 4; ++i)
                x[i] = (double)a[m * K + 4 * j + i] * down;
            for (int idx = 0; idx < 8; ++idx) {
                double s = -x[0];
                s += (idx & 4) ? x[1] : -x[1];
                s += (idx & 2) ? x[2] : -x[2];
                s += (idx & 1) ? x[3] : -x[3];
                t[idx] = s;
                if (fabs(s) > tmax)
                    tmax = fabs(s);
            }
            for (int idx = 0; idx < 8; ++idx)
                q[(m * J + j) * 8 + idx] = tmax == 0.0 ? 0 : (int8_t)rint((127.0 * t[idx]) / tmax);
            scale[m * J + j] = tmax == 0.0 ? 0.0f : (float)(tmax / 127.0);
        }
    }
}

/*
 * FP mpGEMM with INT8-quantized tables (Section 3.1.3 on top of Section 3.1):
 * continues from oracle_lut8_tables with
 *   4. the lookup of Eq. 4-6: the full table entry of a 4-bit pattern p is
 *      L(p) = scale * q[p & 7] when its MSB is 0 and -scale * q[~p & 7] when it is 1
 *      (the negated row of the inverted low bits);
 *   5. bit-serial weights (Section 3.2.1) with the reinterpretation of Eq. 2: plane b
 *      of 4 consecutive codes forms the pattern (first code = MSB), every plane uses
 *      the same table, and y = 2^e sum_q s'_q (sum_{j in q} sum_b 2^b L(p_b) - z'_q S_q)
 *      (Eq. 3) with s' = s/2, z' = 2z + 1 - 2^b (UINT), s' = s/2, z' = -1 with codes
 *      q = w + 1 (TERNARY), s' = s, z' = 0 (BINARY), and S_q the sum of x over
 *      quantization group q; float64 from step 4 on.
 * Arguments as oracle_mpgemm_f64 plus the bit width `bits`; a is float32 here.
 */
int oracle_mpgemm_lut8(int64_t M, int64_t N, int64_t K, const float *a, const void *codes, int wfmt,
                       int bits, int64_t group, const double *scales, const double *zeros,
                       const int64_t *rows, int64_t n_rows, const int64_t *cols, int64_t n_cols,
                       double *y)
{
    if (K % 4 != 0 || bits < 1 || bits > 4)
        return -1;
    const int64_t G = group ? group : K;
    if (K % G != 0 || G % 4 != 0)
        return -1;
    const int64_t J = K / 4, Q = K / G;
    const int64_t R = rows ? n_rows : M, C = cols ? n_cols : N;
    int8_t *q = (int8_t *)malloc((size_t)(M * J * 8));
    float *sc = (float *)malloc((size_t)(M * J) * sizeof(float));
    double *mult = (double *)malloc((size_t)M * sizeof(double));
    double *S = (double *)malloc((size_t)(M * Q) * sizeof(double));
    if (!q || !sc || !mult || !S) {
        free(q); free(sc); free(mult); free(S);
        return -1;
    }
    oracle_lut8_tables(M, K, a, q, sc, mult);
    for (int64_t m = 0; m < M; ++m)
        for (int64_t g = 0; g < Q; ++g) {
            double s = 0.0;
            for (int64_t k = g * G; k < (g + 1) * G; ++k)
                s += (double)a[m * K + k] / mult[m];
            S[m * Q + g] = s;
        }
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t ci = 0; ci < C; ++ci) {
        const int64_t n = cols ? cols[ci] : ci;
        for (int64_t ri = 0; ri < R; ++ri) {
            const int64_t m = rows ? rows[ri] : ri;
            double total = 0.0;
            for (int64_t g = 0; g < Q; ++g) {
                const double s = scales[group ? n * Q + g : 0];
                double sp, zp;
                if (wfmt == WFMT_BINARY) {
                    sp = s;
                    zp = 0.0;
                } else if (wfmt == WFMT_TERNARY) {
                    sp = 0.5 * s;
                    zp = -1.0;
                } else {
                    sp = 0.5 * s;
                    zp = 2.0 * zeros[group ? n * Q + g : 0] + 1.0 - (double)(1 << bits);
                }
                double acc = 0.0;
                for (int64_t j = g * G / 4; j < (g + 1) * G / 4; ++j) {
                    int code[4];
                    for (int i = 0; i < 4; ++i) {
                        const int64_t idx = n * K + 4 * j + i;
                        if (wfmt == WFMT_TERNARY)
                            code[i] = (int)((const int8_t *)codes)[idx] + 1;
                        else
                            code[i] = (int)((const uint8_t *)codes)[idx] & ((1 << bits) - 1);
                    }
                    const int8_t *qt = q + (m * J + j) * 8;
                    const double scale = (double)sc[m * J + j];
                    for (int b = 0; b < bits; ++b) {
                        int p = 0;
                        for (int i = 0; i < 4; ++i)
                            p = (p << 1) | ((code[i] >> b) & 1);
                        const double L = (p & 8) ? -scale * (double)qt[~p & 7] : scale * (double)qt[p & 7];
                        acc += (double)(1 << b) * L;
                    }
                }
                total += sp * (acc - zp * S[m * Q + g]);
            }
            y[ri * C + ci] = mult[m] * total;
        }
    }
    free(q); free(sc); free(mult); free(S);
    return 0;
}
