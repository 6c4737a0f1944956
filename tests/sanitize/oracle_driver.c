/*
 * A driver for the CPU oracle under AddressSanitizer and UndefinedBehaviour-
 * Sanitizer (test infrastructure; built and run by tests/test_sanitize.py).
 * It runs every entry point of oracle/lamp_oracle.c on small seeded inputs:
 * every mode and flag of the forward pass (with statistics and query-block
 * subsets), ragged lengths, empty inputs, windows, GQA, the decode form, the
 * logit entry points, the codecs and the exponentials.  Any sanitizer report
 * aborts (-fno-sanitize-recover=all); the exit status is 0 otherwise.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int lamp_oracle_fwd_ex(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int N, int d,
                       int causal, int window, int bq, int bk, int nk, double delta, double tau, unsigned flags,
                       uint64_t seed, double *o, double *lse, uint8_t *mask, const int64_t *qblocks,
                       int64_t nqblocks, int nthreads, uint64_t *stats);
int lamp_oracle_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int M, int N,
                       int d, int causal, int window, int tk, double delta, double tau, unsigned flags, double *o,
                       double *lse, uint8_t *mask, const int64_t *rows, int64_t nrows, int nthreads);
int oracle_logits8(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                   int window, int row0, int nrows, uint8_t *out, int nthreads);
int oracle_logits16(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                    int window, int row0, int nrows, uint16_t *out, int nthreads);
int oracle_logits16_step(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                         int window, int row0, int nrows, uint16_t *out, int nthreads);
int oracle_logits_sim(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                      int window, int row0, int nrows, int high, double *out, int nthreads);
int oracle_logits8_sr(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                      int window, int row0, int nrows, uint64_t seed, uint8_t *out, int nthreads);
int oracle_round_fmt(int fmt_id, const double *x, double *y, int64_t n);
int oracle_encode_fmt(int fmt_id, const double *x, uint32_t *c, int64_t n);
int oracle_decode_fmt(int fmt_id, const uint32_t *c, double *y, int64_t n);
int oracle_exp_doc(const double *x, double *y, int64_t n);
int oracle_tables(uint8_t *lut8, uint16_t *exp16);
int oracle_round_sim(int p, const double *x, double *y, int64_t n);
int oracle_shift_sim(int p, const double *mu, const double *y, double *s, int64_t n);
int oracle_sim_exp(int p, const double *s, double *e, int64_t n);
int oracle_e4m3_of_f32_bits(uint64_t start, int64_t count, uint8_t *out, int nthreads);

static uint64_t g_state = 0x9E3779B97F4A7C15ull;

static uint64_t next64(void)
{
    /* splitmix64 (Steele, Lea, Flood 2014): only to draw test inputs */
    uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* bf16 bit patterns of roughly N(0, gain^2)-sized values */
static void fill_bf16(uint16_t *x, size_t n, double gain)
{
    for (size_t i = 0; i < n; ++i) {
        double u = 0.0;
        for (int r = 0; r < 4; ++r) u += (double)(next64() >> 11) * 0x1p-53;
        float f = (float)((u - 2.0) * 1.7 * gain);
        uint32_t b;
        memcpy(&b, &f, 4);
        x[i] = (uint16_t)(b >> 16);
    }
}

static int failures = 0;

static void check(int rc, const char *what)
{
    if (rc != 0) {
        fprintf(stderr, "%s returned %d\n", what, rc);
        ++failures;
    }
}

static void run_fwd(int B, int Hq, int Hkv, int N, int d, int causal, int window, int bq, int bk, int nk, double tau,
                    unsigned flags, double gain, int subset, int nthreads)
{
    size_t nq = (size_t)B * Hq * N * d, nk_ = (size_t)B * Hkv * N * d;
    uint16_t *q = malloc(nq * 2 + 2), *k = malloc(nk_ * 2 + 2), *v = malloc(nk_ * 2 + 2);
    fill_bf16(q, nq, gain);
    fill_bf16(k, nk_, gain);
    fill_bf16(v, nk_, 1.0);
    int nqb = (N + bq - 1) / bq, ntiles = (N + bk * nk - 1) / (bk * nk);
    double *o = malloc(nq * sizeof(double) + 8), *lse = malloc((size_t)B * Hq * N * sizeof(double) + 8);
    uint8_t *mask = malloc((size_t)B * Hq * nqb * ntiles * nk + 1);
    uint64_t *stats = calloc((size_t)8 + nk + 1, sizeof(uint64_t));
    int64_t blocks[2] = {0, (int64_t)B * Hq * nqb - 1};
    check(lamp_oracle_fwd_ex(q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, 0x1p-8, tau, flags, 7, o, lse,
                             mask, subset ? blocks : NULL, subset ? 2 : 0, nthreads, stats),
          "lamp_oracle_fwd_ex");
    free(q); free(k); free(v); free(o); free(lse); free(mask); free(stats);
}

int main(void)
{
    const double taus[5] = {INFINITY, 1.0, 0.5, 0x1p-5, 0.0};
    /* every mode x flag combination the oracle accepts, on a ragged causal shape */
    const unsigned flag_sets[8] = {0, 1, 2, 3, 4, 5, 8, 16};
    for (int f = 0; f < 8; ++f)
        for (int t = 0; t < 5; ++t) run_fwd(1, 2, 1, 77, 16, 1, 0, 32, 8, 4, taus[t], flag_sets[f], 1.0, 0, 1);
    /* saturating inputs, windows, GQA, non-causal, query-block subsets */
    run_fwd(1, 1, 1, 96, 32, 1, 0, 32, 8, 4, 0.5, 0, 8.0, 0, 1);
    run_fwd(1, 1, 1, 96, 32, 1, 0, 32, 8, 4, 0.5, 1, 8.0, 0, 1);
    run_fwd(2, 4, 2, 100, 16, 1, 17, 16, 4, 4, 0.5, 0, 1.0, 1, 1);
    run_fwd(1, 2, 2, 64, 8, 0, 0, 64, 16, 4, 0x1p-5, 0, 1.0, 1, 1);
    run_fwd(1, 1, 1, 5, 8, 1, 0, 32, 8, 4, 0.5, 0, 1.0, 0, 1);          /* N < bq */
    run_fwd(1, 1, 1, 33, 8, 1, 0, 16, 8, 3, 0.25, 0, 1.0, 0, 1);        /* nk = 3 */
    run_fwd(0, 1, 1, 64, 8, 1, 0, 16, 8, 4, 0.5, 0, 1.0, 0, 1);         /* B = 0 */
    run_fwd(1, 1, 1, 0, 8, 1, 0, 16, 8, 4, 0.5, 0, 1.0, 0, 1);          /* N = 0 */
    run_fwd(2, 2, 1, 70, 16, 1, 0, 16, 8, 4, 0.5, 0, 1.0, 0, 4);         /* several threads */
    /* the decode form */
    {
        int B = 2, Hq = 4, Hkv = 2, M = 3, N = 130, d = 16;
        uint16_t *q = malloc((size_t)B * Hq * M * d * 2), *k = malloc((size_t)B * Hkv * N * d * 2),
                 *v = malloc((size_t)B * Hkv * N * d * 2);
        fill_bf16(q, (size_t)B * Hq * M * d, 2.0);
        fill_bf16(k, (size_t)B * Hkv * N * d, 2.0);
        fill_bf16(v, (size_t)B * Hkv * N * d, 1.0);
        int np = (N + 63) / 64 * 64;
        double *o = malloc((size_t)B * Hq * M * d * 8), *lse = malloc((size_t)B * Hq * M * 8);
        uint8_t *mask = malloc((size_t)B * Hq * M * np);
        for (int t = 0; t < 5; ++t) {
            check(lamp_oracle_decode(q, k, v, B, Hq, Hkv, M, N, d, 1, 0, 64, 0x1p-8, taus[t], 0, o, lse, mask, NULL, 0,
                                     1), "lamp_oracle_decode");
            check(lamp_oracle_decode(q, k, v, B, Hq, Hkv, M, N, d, 1, 40, 64, 0x1p-8, taus[t], 0, o, lse, mask, NULL,
                                     0, 1), "lamp_oracle_decode window");
        }
        free(q); free(k); free(v); free(o); free(lse); free(mask);
    }
    /* the logit entry points */
    {
        int N = 48, d = 32;
        uint16_t *q = malloc((size_t)2 * N * d * 2), *k = malloc((size_t)N * d * 2);
        fill_bf16(q, (size_t)2 * N * d, 4.0);
        fill_bf16(k, (size_t)N * d, 4.0);
        uint8_t *y8 = malloc((size_t)2 * 20 * N);
        uint16_t *y16 = malloc((size_t)2 * 20 * N * 2);
        double *ys = malloc((size_t)2 * 20 * N * 8);
        check(oracle_logits8(q, k, 1, 2, 1, N, d, 1, 7, 5, 20, y8, 1), "oracle_logits8");
        check(oracle_logits8_sr(q, k, 1, 2, 1, N, d, 1, 0, 5, 20, 3, y8, 1), "oracle_logits8_sr");
        check(oracle_logits16(q, k, 1, 2, 1, N, d, 0, 0, 5, 20, y16, 1), "oracle_logits16");
        check(oracle_logits16_step(q, k, 1, 2, 1, N, d, 0, 0, 5, 20, y16, 1), "oracle_logits16_step");
        check(oracle_logits_sim(q, k, 1, 2, 1, N, d, 1, 0, 5, 20, 0, ys, 1), "oracle_logits_sim 8");
        check(oracle_logits_sim(q, k, 1, 2, 1, N, d, 1, 0, 5, 20, 1, ys, 1), "oracle_logits_sim 16");
        free(q); free(k); free(y8); free(y16); free(ys);
    }
    /* codecs, exponentials, tables */
    {
        enum { n = 4096 };
        static double x[n], y[n], s[n];
        static uint32_t c[n];
        for (int i = 0; i < n; ++i) x[i] = ldexp((double)(next64() >> 11) * 0x1p-53 - 0.5, (int)(i % 64) - 40);
        for (int f = 0; f < 6; ++f) {
            check(oracle_round_fmt(f, x, y, n), "oracle_round_fmt");
            for (int i = 0; i < n; ++i) y[i] = fabs(y[i]);
            check(oracle_round_fmt(f, y, y, n), "oracle_round_fmt abs");
            check(oracle_encode_fmt(f, y, c, n), "oracle_encode_fmt");
            check(oracle_decode_fmt(f, c, s, n), "oracle_decode_fmt");
        }
        for (int i = 0; i < n; ++i) x[i] = -fabs(x[i]) * 1e3;
        check(oracle_exp_doc(x, y, n), "oracle_exp_doc");
        static uint8_t lut8[256];
        static uint16_t exp16[65536];
        check(oracle_tables(lut8, exp16), "oracle_tables");
        for (int p = 3; p <= 11; p += 8) {
            check(oracle_round_sim(p, x, y, n), "oracle_round_sim");
            for (int i = 0; i < n; ++i) s[i] = fabs(x[i]) * 1e-3;
            check(oracle_shift_sim(p, s, x, y, n), "oracle_shift_sim");
            check(oracle_sim_exp(p, y, s, n), "oracle_sim_exp");
        }
        static uint8_t e8[1 << 16];
        check(oracle_e4m3_of_f32_bits(0x43E00000u - 100, 1 << 16, e8, 1), "oracle_e4m3_of_f32_bits");
    }
    if (failures) {
        fprintf(stderr, "%d calls failed\n", failures);
        return 1;
    }
    printf("oracle driver: all calls clean\n");
    return 0;
}
