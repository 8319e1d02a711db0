/*
 * Host sanitizer driver for the CPU oracle (test infrastructure): calls every
 * entry point of oracle/mpgemm_oracle.c on small inputs whose buffers are sized
 * exactly as each function's contract states, with row and column subsets, the
 * optional accumulator, all weight formats, per-tensor and per-group scales, and
 * the zero token.  Built with -fsanitize=address,undefined by
 * tests/test_oracle_sanitized.py; any out-of-bounds access, leak or undefined
 * behaviour aborts the run.  Prints "ok" at the end.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_mpgemm_f64(int64_t M, int64_t N, int64_t K, const double *a, const void *codes, int wfmt,
                      int64_t group, const double *scales, const double *zeros, const int64_t *rows,
                      int64_t n_rows, const int64_t *cols, int64_t n_cols, const double *acc, double *y);
void oracle_quantize_int8(int64_t M, int64_t K, const float *a, int8_t *q, float *s_a);
int oracle_mpgemm_i64(int64_t M, int64_t N, int64_t K, const int8_t *qa, const void *codes, int wfmt,
                      const int64_t *rows, int64_t n_rows, const int64_t *cols, int64_t n_cols,
                      const int64_t *acc_in, int64_t *acc);
void oracle_int_output_f32(int64_t n_rows, int64_t n_cols, const int64_t *acc, const float *s_a,
                           const float *s_w, float *y);
void oracle_half_tables_f64(int64_t M, int64_t K, const double *a, double *T);
void oracle_half_tables_i64(int64_t M, int64_t K, const int8_t *qa, int64_t *T);
void oracle_group_sums_f64(int64_t M, int64_t K, int64_t group, const double *a, double *S);
void oracle_group_sums_i64(int64_t M, int64_t K, int64_t group, const int8_t *qa, int64_t *S);
void oracle_token_pow2(int64_t M, int64_t K, const double *a, double *mult);
void oracle_lut8_tables(int64_t M, int64_t K, const float *a, int8_t *q, float *scale, double *mult);
int oracle_mpgemm_lut8(int64_t M, int64_t N, int64_t K, const float *a, const void *codes, int wfmt, int bits,
                       int64_t group, const double *scales, const double *zeros, const int64_t *rows,
                       int64_t n_rows, const int64_t *cols, int64_t n_cols, double *y);

static uint64_t st = 0x2408600312345ull;
static double rnd(void) { /* uniform in [-1, 1) */
    st = st * 6364136223846793005ull + 1442695040888963407ull;
    return (double)(st >> 11) / (double)(1ull << 52) - 1.0;
}
static void *xmalloc(size_t n) {
    void *p = malloc(n ? n : 1);
    if (!p) { fprintf(stderr, "out of memory\n"); exit(2); }
    return p;
}

static int run(int64_t M, int64_t N, int64_t K, int wfmt, int bits, int64_t group) {
    const int64_t Q = group ? K / group : 1;
    double *a = xmalloc(sizeof(double) * M * K);
    float *af = xmalloc(sizeof(float) * M * K);
    for (int64_t i = 0; i < M * K; ++i) af[i] = (float)(a[i] = (i / K == 1) ? 0.0 : 3.0 * rnd());
    uint8_t *cu = xmalloc(N * K);
    int8_t *ct = xmalloc(N * K);
    for (int64_t i = 0; i < N * K; ++i) {
        const uint64_t r = (uint64_t)((rnd() + 1.0) * 1000.0);
        cu[i] = (uint8_t)(r % (wfmt == 1 ? 2u : (1u << bits)));
        ct[i] = (int8_t)((int)(r % 3u) - 1);
    }
    const void *codes = wfmt == 2 ? (const void *)ct : (const void *)cu;
    double *s = xmalloc(sizeof(double) * N * Q), *z = xmalloc(sizeof(double) * N * Q);
    for (int64_t i = 0; i < N * Q; ++i) { s[i] = 0.05 + 0.01 * rnd(); z[i] = 1.5 + rnd(); }
    const int64_t rows[2] = {M - 1, 0}, cols[3] = {N - 1, 0, N / 2};
    double *y = xmalloc(sizeof(double) * M * N), *acc = xmalloc(sizeof(double) * 2 * 3);
    for (int i = 0; i < 6; ++i) acc[i] = rnd();
    int rc = 0;
    rc |= oracle_mpgemm_f64(M, N, K, a, codes, wfmt, group, s, z, NULL, 0, NULL, 0, NULL, y);
    rc |= oracle_mpgemm_f64(M, N, K, a, codes, wfmt, group, s, z, rows, 2, cols, 3, acc, y);
    rc |= oracle_mpgemm_lut8(M, N, K, af, codes, wfmt, bits, group, s, z, NULL, 0, NULL, 0, y);
    rc |= oracle_mpgemm_lut8(M, N, K, af, codes, wfmt, bits, group, s, z, rows, 2, cols, 3, y);
    const int64_t J = K / 4;
    double *T = xmalloc(sizeof(double) * M * J * 8), *S = xmalloc(sizeof(double) * M * Q), *mult = xmalloc(sizeof(double) * M);
    oracle_half_tables_f64(M, K, a, T);
    oracle_group_sums_f64(M, K, group, a, S);
    oracle_token_pow2(M, K, a, mult);
    int8_t *q8 = xmalloc(M * J * 8);
    float *sc = xmalloc(sizeof(float) * M * J);
    oracle_lut8_tables(M, K, af, q8, sc, mult);
    if (wfmt != 0) {
        int8_t *qa = xmalloc(M * K);
        float *sa = xmalloc(sizeof(float) * M), *sw = xmalloc(sizeof(float) * N), *yf = xmalloc(sizeof(float) * M * N);
        int64_t *ti = xmalloc(sizeof(int64_t) * M * J * 8), *si = xmalloc(sizeof(int64_t) * M * Q);
        int64_t *ai = xmalloc(sizeof(int64_t) * M * N), *ain = xmalloc(sizeof(int64_t) * 6);
        for (int i = 0; i < 6; ++i) ain[i] = i - 3;
        for (int64_t i = 0; i < N; ++i) sw[i] = 0.03f;
        oracle_quantize_int8(M, K, af, qa, sa);
        rc |= oracle_mpgemm_i64(M, N, K, qa, codes, wfmt, NULL, 0, NULL, 0, NULL, ai);
        oracle_int_output_f32(M, N, ai, sa, sw, yf);
        rc |= oracle_mpgemm_i64(M, N, K, qa, codes, wfmt, rows, 2, cols, 3, ain, ai);
        oracle_half_tables_i64(M, K, qa, ti);
        oracle_group_sums_i64(M, K, group, qa, si);
        free(qa); free(sa); free(sw); free(yf); free(ti); free(si); free(ai); free(ain);
    }
    free(a); free(af); free(cu); free(ct); free(s); free(z); free(y); free(acc);
    free(T); free(S); free(mult); free(q8); free(sc);
    return rc;
}

int main(void) {
    int rc = 0;
    rc |= run(3, 5, 256, 0, 2, 128);  /* UINT2, per group, a zero token */
    rc |= run(2, 7, 384, 0, 4, 384);  /* UINT4, per channel */
    rc |= run(3, 4, 128, 0, 1, 0);    /* UINT1, per tensor */
    rc |= run(2, 5, 256, 1, 1, 0);    /* BINARY, per tensor */
    rc |= run(3, 6, 512, 1, 1, 512);  /* BINARY, per channel */
    rc |= run(2, 3, 256, 2, 2, 0);    /* TERNARY, per tensor */
    rc |= run(3, 9, 128, 2, 2, 128);  /* TERNARY, per channel */
    if (rc) {
        fprintf(stderr, "an oracle entry point rejected valid arguments\n");
        return 1;
    }
    printf("ok\n");
    return 0;
}
