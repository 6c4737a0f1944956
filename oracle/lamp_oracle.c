/*
 * lamp_oracle.c -- plain, slow CPU oracle for the LampAttention forward pass.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the independent reference that the
 * GPU library is checked against.  It shares no code, header, table or
 * constant generator with the GPU library, and nothing in the product path may
 * call it: only the test suite, the smoke check and the benchmark's
 * cpu_baseline leg load it.
 *
 * What it computes follows the paper (LampAttention: look-ahead mixed-precision
 * FlashAttention) section by section:
 *   - online softmax state (mu, omega) and its update: Sec. 2 (opening);
 *   - block threat T_theta, descending sort, safety-margin test: Sec. 3.1,
 *     Eq. (7) ("stage 1");
 *   - block-LAMP multidimensional knapsack: Sec. 3.1, Eq. (8) ("stage 2");
 *   - the kernel as a whole: Sec. 3.2, Algorithm 1;
 *   - number formats e4m3 / ue5m3 / e4m11 / ue5m11 and the 8-bit exp LUT:
 *     Sec. 3.3, "Floating-point formats";
 *   - recursive FMA accumulation in FP32 with rounding after every step:
 *     Sec. 4.1.
 * Where the paper is silent or ambiguous, the reading taken is stated at the
 * place it is used (marked "reading:").
 *
 * Everything is fp64 except where the method fixes another precision (the
 * fp32 FMA of the 8-bit accumulation, the formats above).  Build with
 * -ffp-contract=off: every fused multiply-add below is an explicit fma().
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <float.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Number formats (Sec. 3.3).                                                */
/* ------------------------------------------------------------------------ */

/* A binary floating-point format with `mbits` stored mantissa bits, exponent
 * bias `bias`, gradual underflow (subnormals) and a largest finite value
 * `maxval`.  Rounding is round-to-nearest-even; values beyond maxval saturate
 * to +-maxval (reading: no QK-Norm is assumed, so overflow saturates). */
typedef struct {
    int ebits, mbits, bias, is_signed;
    double maxval;
} ofmt_t;

/* e4m3 accumulator: OCP E4M3FN, bias 7, largest finite 448 (Sec. 3.3). */
static const ofmt_t F_E4M3 = {4, 3, 7, 1, 448.0};
/* e4m11 high-precision accumulator: bias 7, all codes finite,
 * largest (2 - 2^-11) * 2^8 = 511.875 (Sec. 3.3). */
static const ofmt_t F_E4M11 = {4, 11, 7, 1, 511.875};
/* ue5m3 / ue5m11 shifted logits mu_hat - y >= 0 (Sec. 3.3); the paper does
 * not state a bias, reading: 15. */
static const ofmt_t F_UE5M3_SHIFT = {5, 3, 15, 0, 122880.0};
static const ofmt_t F_UE5M11_SHIFT = {5, 11, 15, 0, 131040.0};
/* ue5m3 / ue5m11 exponentials: bias 31 so that code 11111000 is 1.0, smallest
 * normal 2^-30, smallest subnormal 2^-33 resp. 2^-41 (Sec. 3.3). */
static const ofmt_t F_UE5M3_EXP = {5, 3, 31, 0, 1.875};
static const ofmt_t F_UE5M11_EXP = {5, 11, 31, 0, 2.0 - 0x1p-11};

/* Round an exact double to the format grid (RNE, subnormals, saturation);
 * *sat (may be NULL) is set to 1 when the rounded magnitude exceeded the
 * largest value and was clamped to it. */
static double round_to_fmt_s(double x, const ofmt_t *f, int *sat)
{
    if (isnan(x)) return x;
    if (x == 0.0) return x;                       /* keeps the sign of zero */
    double ax = fabs(x);
    if (isinf(ax)) {
        if (sat) *sat = 1;
        return copysign(f->maxval, x);
    }
    int E;
    (void)frexp(ax, &E);                          /* ax = fr * 2^E, fr in [0.5,1) */
    int e = E - 1;                                /* ax in [2^e, 2^(e+1)) */
    int emin = 1 - f->bias;                       /* smallest normal exponent */
    if (e < emin) e = emin;
    double quantum = ldexp(1.0, e - f->mbits);
    double r = nearbyint(ax / quantum) * quantum; /* default mode: ties to even */
    if (r > f->maxval) {
        r = f->maxval;
        if (sat) *sat = 1;
    }
    return copysign(r, x);
}

static double round_to_fmt(double x, const ofmt_t *f) { return round_to_fmt_s(x, f, NULL); }

/* Code of a value that already lies on the grid. */
static uint32_t encode_fmt(double v, const ofmt_t *f)
{
    uint32_t sign = (f->is_signed && signbit(v)) ? 1u : 0u;
    double a = fabs(v);
    int emin = 1 - f->bias;
    uint32_t e, m;
    if (a < ldexp(1.0, emin)) {
        e = 0;
        m = (uint32_t)(a / ldexp(1.0, emin - f->mbits));
    } else {
        int E;
        (void)frexp(a, &E);
        int eu = E - 1;
        e = (uint32_t)(eu + f->bias);
        m = (uint32_t)(a / ldexp(1.0, eu - f->mbits)) - (1u << f->mbits);
    }
    return (sign << (f->ebits + f->mbits)) | (e << f->mbits) | m;
}

static double decode_fmt(uint32_t code, const ofmt_t *f)
{
    uint32_t m = code & ((1u << f->mbits) - 1u);
    uint32_t e = (code >> f->mbits) & ((1u << f->ebits) - 1u);
    int sign = f->is_signed ? (int)((code >> (f->ebits + f->mbits)) & 1u) : 0;
    double v;
    if (e == 0) v = ldexp((double)m, 1 - f->bias - f->mbits);
    else v = ldexp((double)((1u << f->mbits) | m), (int)e - f->bias - f->mbits);
    return sign ? -v : v;
}

static const ofmt_t *fmt_by_id(int id)
{
    switch (id) {
    case 0: return &F_E4M3;
    case 1: return &F_E4M11;
    case 2: return &F_UE5M3_SHIFT;
    case 3: return &F_UE5M11_SHIFT;
    case 4: return &F_UE5M3_EXP;
    case 5: return &F_UE5M11_EXP;
    default: return NULL;
    }
}

/* Exported codec entry points (used by the tests to pin the codecs). */
int oracle_round_fmt(int fmt_id, const double *x, double *y, int64_t n)
{
    const ofmt_t *f = fmt_by_id(fmt_id);
    if (!f) return -1;
    for (int64_t i = 0; i < n; ++i) y[i] = round_to_fmt(x[i], f);
    return 0;
}

int oracle_encode_fmt(int fmt_id, const double *x, uint32_t *c, int64_t n)
{
    const ofmt_t *f = fmt_by_id(fmt_id);
    if (!f) return -1;
    for (int64_t i = 0; i < n; ++i) c[i] = encode_fmt(round_to_fmt(x[i], f), f);
    return 0;
}

int oracle_decode_fmt(int fmt_id, const uint32_t *c, double *y, int64_t n)
{
    const ofmt_t *f = fmt_by_id(fmt_id);
    if (!f) return -1;
    for (int64_t i = 0; i < n; ++i) y[i] = decode_fmt(c[i], f);
    return 0;
}

/* e4m3 code of every fp32 bit pattern in [start, start+count): used to check
 * the GPU's rounding exhaustively.  NaN patterns give 0xFF. */
int oracle_e4m3_of_f32_bits(uint64_t start, int64_t count, uint8_t *out, int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t i = 0; i < count; ++i) {
        uint32_t b = (uint32_t)(start + (uint64_t)i);
        float x;
        memcpy(&x, &b, 4);
        if (isnan(x)) { out[i] = 0xFF; continue; }
        out[i] = (uint8_t)encode_fmt(round_to_fmt((double)x, &F_E4M3), &F_E4M3);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* exp_doc: the one documented fp64 exponential used for the rescale factor  */
/* lambda_hat = exp(mu - mu_hat).  The paper takes alpha_hat in high          */
/* precision (Sec. 2.2, last paragraph); both the oracle and the GPU library  */
/* evaluate it with the same operations in the same order so that the        */
/* stage-2 decisions, which depend on omega_hat, agree bit for bit:           */
/*   x < -700 -> 0;                                                          */
/*   n = rint(RN(x * LOG2E));  r = fma(-n, LN2_HI, x);  r = fma(-n, LN2_LO, r) */
/*   p = Horner in fma of sum_{k=0}^{13} r^k / k!  (coefficients RN64(1/k!)) */
/*   result = ldexp(p, n).                                                   */
/* LN2_HI is ln 2 truncated to 32 significant bits (so n*LN2_HI is exact),   */
/* LN2_LO = RN64(ln 2 - LN2_HI), LOG2E = RN64(1/ln 2).                        */
/* ------------------------------------------------------------------------ */
static const double ED_LOG2E = 0x1.71547652b82fep+0;
static const double ED_LN2_HI = 0x1.62e42fee00000p-1;
static const double ED_LN2_LO = 0x1.a39ef35793c76p-33;
static const double ED_C[14] = {
    0x1.0000000000000p+0, 0x1.0000000000000p+0, 0x1.0000000000000p-1,
    0x1.5555555555555p-3, 0x1.5555555555555p-5, 0x1.1111111111111p-7,
    0x1.6c16c16c16c17p-10, 0x1.a01a01a01a01ap-13, 0x1.a01a01a01a01ap-16,
    0x1.71de3a556c734p-19, 0x1.27e4fb7789f5cp-22, 0x1.ae64567f544e4p-26,
    0x1.1eed8eff8d898p-29, 0x1.6124613a86d09p-33};

static double exp_doc(double x)
{
    if (x < -700.0) return 0.0;
    double n = nearbyint(x * ED_LOG2E);
    double r = fma(-n, ED_LN2_HI, x);
    r = fma(-n, ED_LN2_LO, r);
    double p = ED_C[13];
    for (int k = 12; k >= 0; --k) p = fma(p, r, ED_C[k]);
    return ldexp(p, (int)n);
}

int oracle_exp_doc(const double *x, double *y, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) y[i] = exp_doc(x[i]);
    return 0;
}

int oracle_exp_doc_constants(double *out /* 17 */)
{
    out[0] = ED_LOG2E;
    out[1] = ED_LN2_HI;
    out[2] = ED_LN2_LO;
    for (int k = 0; k < 14; ++k) out[3 + k] = ED_C[k];
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Exponential tables (Sec. 3.3): the 8-bit exp is a look-up table from the  */
/* ue5m3 shift code to the ue5m3 exp code, E = RN(exp(-s)), correctly         */
/* rounded (Sec. 4.1 models the exponentials as correctly rounded); the       */
/* 16-bit exp uses the same rule on ue5m11.  exp is evaluated in long double  */
/* and every entry is checked to lie clearly away from a rounding midpoint;  */
/* an entry that does not is reported as an error (never seen for these     */
/* inputs; the test suite re-derives every entry in 60-digit arithmetic).     */
/* ------------------------------------------------------------------------ */
static uint8_t g_lut8[256];
static uint16_t g_exp16[65536];
static int g_tables_ok = 0;

static int cr_exp_neg(double s, const ofmt_t *f, uint32_t *code)
{
    long double e = expl(-(long double)s);
    long double elo = e * (1.0L - 0x1p-60L), ehi = e * (1.0L + 0x1p-60L);
    double r = round_to_fmt((double)e, f);
    uint32_t c = encode_fmt(r, f);
    uint32_t cmax = (1u << (f->ebits + f->mbits)) - 1u;
    /* The enclosure [elo, ehi] of exp(-s) must lie strictly between the
     * midpoints to the neighbouring grid values; then the exact value rounds
     * to r as well. */
    if (c > 0) {
        long double mb = ((long double)decode_fmt(c - 1, f) + (long double)r) / 2;
        if (!(elo > mb)) return -1;
    }
    if (c < cmax) {
        long double ma = ((long double)r + (long double)decode_fmt(c + 1, f)) / 2;
        if (!(ehi < ma)) return -1;
    }
    *code = c;
    return 0;
}

static int build_tables(void)
{
    if (g_tables_ok) return 0;
    for (uint32_t c = 0; c < 256; ++c) {
        uint32_t e;
        if (cr_exp_neg(decode_fmt(c, &F_UE5M3_SHIFT), &F_UE5M3_EXP, &e)) return -1;
        g_lut8[c] = (uint8_t)e;
    }
    for (uint32_t c = 0; c < 65536; ++c) {
        uint32_t e;
        if (cr_exp_neg(decode_fmt(c, &F_UE5M11_SHIFT), &F_UE5M11_EXP, &e)) return -1;
        g_exp16[c] = (uint16_t)e;
    }
    g_tables_ok = 1;
    return 0;
}

int oracle_tables(uint8_t *lut8, uint16_t *exp16)
{
    int rc = build_tables();
    if (rc) return rc;
    if (lut8) memcpy(lut8, g_lut8, sizeof g_lut8);
    if (exp16) memcpy(exp16, g_exp16, sizeof g_exp16);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* The "SIM" precision profile (Sec. 4.1): the numerics of the paper's own   */
/* simulation, which stores the 8-bit and 16-bit numbers in FP32 with the    */
/* mantissa cut to 3 and 11 bits, accumulates by recursive FP32 FMA with a    */
/* rounding after every step, and models the exponentials as correctly        */
/* rounded.  Readings: "cut" is round-to-nearest-even (as for the hardware    */
/* formats); the exponent range is FP32's, with FP32's gradual underflow (the */
/* quantum below 2^-126 is 2^(-126-p)); there is no saturation, overflow      */
/* gives an infinity as in FP32.                                              */
/* ------------------------------------------------------------------------ */

/* Round an exact double to p stored mantissa bits in FP32's exponent range. */
static double round_sim(double x, int p)
{
    if (x == 0.0 || !isfinite(x)) return x;
    double ax = fabs(x);
    int E;
    (void)frexp(ax, &E);
    int e = E - 1;                                /* ax in [2^e, 2^(e+1)) */
    if (e < -126) e = -126;
    double quantum = ldexp(1.0, e - p);
    double r = nearbyint(ax / quantum) * quantum; /* ties to even */
    if (r >= 0x1p128) r = INFINITY;
    return copysign(r, x);
}

/* Round the exact real hi + lo, given as hi = RN64(hi + lo) and its error lo
 * (|lo| <= ulp(hi)/2), to p mantissa bits.  Only when hi is exactly halfway
 * between two grid values can lo change the result: then its sign decides. */
static double round_sim_sum(double hi, double lo, int p)
{
    double r = round_sim(hi, p);
    if (lo == 0.0 || hi == 0.0 || !isfinite(hi)) return r;
    double ah = fabs(hi);
    int E;
    (void)frexp(ah, &E);
    int e = E - 1;
    if (e < -126) e = -126;
    double quantum = ldexp(1.0, e - p);
    double t = ah / quantum;
    if (t - floor(t) != 0.5) return r;
    double mag = ((lo > 0.0) == (hi > 0.0)) ? (floor(t) + 1.0) * quantum : floor(t) * quantum;
    if (mag >= 0x1p128) mag = INFINITY;
    return copysign(mag, hi);
}

/* x rounded toward zero to p mantissa bits in FP32's exponent range. */
static double trunc_sim(double x, int p)
{
    if (x == 0.0 || !isfinite(x)) return x;
    double ax = fabs(x);
    int E;
    (void)frexp(ax, &E);
    int e = E - 1;
    if (e < -126) e = -126;
    double quantum = ldexp(1.0, e - p);
    return copysign(floor(ax / quantum) * quantum, x);
}

static long double round_sim_ld(long double x, int p)
{
    if (x == 0.0L) return x;
    int E;
    (void)frexpl(x, &E);
    int e = E - 1;
    if (e < -126) e = -126;
    long double quantum = ldexpl(1.0L, e - p);
    return nearbyintl(x / quantum) * quantum;
}

static int g_sim_fail = 0;   /* set if an exponential lies too close to a midpoint */

/* E = RN_p(exp(-s)) for a shift s >= 0, correctly rounded: exp is evaluated
 * in long double, and the enclosure exp(-s) (1 -+ 2^-60) must round to one
 * value (otherwise g_sim_fail is raised; the test suite re-derives every
 * value that occurs in 60-digit arithmetic). */
static double sim_exp(double s, int p)
{
    long double e = expl(-(long double)s);
    long double a = round_sim_ld(e * (1.0L - 0x1p-60L), p), b = round_sim_ld(e * (1.0L + 0x1p-60L), p);
    if (a != b) __atomic_store_n(&g_sim_fail, 1, __ATOMIC_RELAXED);
    return (double)round_sim_ld(e, p);
}

/* Shifted exponential in the SIM profile: s = RN_p(max(0, mu_hat - y)) of the
 * exact difference (a TwoSum gives it as hi + lo), E = RN_p(exp(-s)); p = 11
 * for the 16-bit path, 3 for the 8-bit one. */
static double shifted_exp_sim(double mu_hat, double y, int high)
{
    const int p = high ? 11 : 3;
    double a = mu_hat, b = -y;
    double hi = a + b, bb = hi - a;
    double lo = (a - (hi - bb)) + (b - bb);
    double x = (hi > 0.0) ? round_sim_sum(hi, lo, p) : 0.0;
    return sim_exp(x, p);
}

int oracle_round_sim(int p, const double *x, double *y, int64_t n)
{
    if (p != 3 && p != 11) return -1;
    for (int64_t i = 0; i < n; ++i) y[i] = round_sim(x[i], p);
    return 0;
}

/* s[i] = RN_p(max(0, mu[i] - y[i])) from the exact difference. */
int oracle_shift_sim(int p, const double *mu, const double *y, double *s, int64_t n)
{
    if (p != 3 && p != 11) return -1;
    for (int64_t i = 0; i < n; ++i) {
        double a = mu[i], b = -y[i];
        double hi = a + b, bb = hi - a;
        double lo = (a - (hi - bb)) + (b - bb);
        s[i] = (hi > 0.0) ? round_sim_sum(hi, lo, p) : 0.0;
    }
    return 0;
}

int oracle_sim_exp(int p, const double *s, double *e, int64_t n)
{
    if (p != 3 && p != 11) return -1;
    g_sim_fail = 0;
    for (int64_t i = 0; i < n; ++i) e[i] = sim_exp(s[i], p);
    return g_sim_fail ? -2 : 0;
}

double oracle_trunc_sim3(double x) { return trunc_sim(x, 3); }

/* ------------------------------------------------------------------------ */
/* Logits.                                                                   */
/* ------------------------------------------------------------------------ */

static float bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* Scale applied to Q before accumulation (Sec. 3.3: the 1/sqrt(d) scaling
 * is applied before the product is accumulated): s = RN32(1/sqrt(d)). */
static float scale_of(int d)
{
    return (float)(1.0 / sqrt((double)d));
}

float oracle_scale(int d) { return scale_of(d); }

/* q_tilde = RN32(q * s). */
static void prescale(const uint16_t *q, int d, float s, float *qt)
{
    for (int c = 0; c < d; ++c) qt[c] = (float)((double)bf16_to_f32(q[c]) * (double)s);
}

/* Low-precision logit (Sec. 4.1 and Alg. 1): recursive summation with one
 * FP32 FMA per step, the running sum rounded to e4m3 after every step,
 * channels in ascending order, starting from +0.  *sat (may be NULL) is set
 * when some step was clamped to +-448 (Sec. 3.3 assumes QK-Norm keeps the
 * sums in range; these inputs need not). */
static double logit8_s(const float *qt, const uint16_t *k, int d, int *sat)
{
    float acc = 0.0f;
    for (int c = 0; c < d; ++c) {
        float t = fmaf(qt[c], bf16_to_f32(k[c]), acc);
        acc = (float)round_to_fmt_s((double)t, &F_E4M3, sat);
    }
    return (double)acc;
}

static double logit8(const float *qt, const uint16_t *k, int d) { return logit8_s(qt, k, d, NULL); }

/* High-precision logit (Alg. 1, recompute steps; Sec. 3.3 gives e4m11 as the
 * 16-bit accumulator format).  Reading: the dot product is accumulated by a
 * sequential FP32 FMA chain in ascending channel order, starting from +0,
 * and the sum is rounded once to e4m11 (saturating; *sat set when clamped).
 * This is 16-bit accumulation taken at FP32 accumulation precision, the
 * reading named for the recompute (FP32 accumulation); the paper's own
 * simulation keeps its numbers in FP32 and accumulates by FP32 FMA (Sec. 4.1).
 * The literal alternative of Sec. 3.3, e4m11 as the accumulator itself, is
 * logit16_step below. */
static double logit16_s(const float *qt, const uint16_t *k, int d, int *sat)
{
    float acc = 0.0f;
    for (int c = 0; c < d; ++c) acc = fmaf(qt[c], bf16_to_f32(k[c]), acc);
    return round_to_fmt_s((double)acc, &F_E4M11, sat);
}

static double logit16(const float *qt, const uint16_t *k, int d) { return logit16_s(qt, k, d, NULL); }

/* The literal reading of Sec. 3.3 ("16-bit e4m11 format to accumulate"): the
 * 8-bit recursion with e4m11 in place of e4m3, i.e. every FP32 FMA result
 * rounded to e4m11 (saturating) before the next step. */
static double logit16_step(const float *qt, const uint16_t *k, int d, int *sat)
{
    float acc = 0.0f;
    for (int c = 0; c < d; ++c) {
        float t = fmaf(qt[c], bf16_to_f32(k[c]), acc);
        acc = (float)round_to_fmt_s((double)t, &F_E4M11, sat);
    }
    return (double)acc;
}

/* SIM profile logits: the same recursions with the roundings of the profile
 * (3 mantissa bits after every step; one rounding to 11 bits at the end of
 * the FP32 chain, as for the e4m11 logit).  The profile does not saturate. */
static double logit8_sim_s(const float *qt, const uint16_t *k, int d, int *sat)
{
    (void)sat;
    float acc = 0.0f;
    for (int c = 0; c < d; ++c) {
        float t = fmaf(qt[c], bf16_to_f32(k[c]), acc);
        acc = (float)round_sim((double)t, 3);
    }
    return (double)acc;
}

static double logit8_sim(const float *qt, const uint16_t *k, int d) { return logit8_sim_s(qt, k, d, NULL); }

static double logit16_sim_s(const float *qt, const uint16_t *k, int d, int *sat)
{
    (void)sat;
    float acc = 0.0f;
    for (int c = 0; c < d; ++c) acc = fmaf(qt[c], bf16_to_f32(k[c]), acc);
    return round_sim((double)acc, 11);
}

static double logit16_sim(const float *qt, const uint16_t *k, int d) { return logit16_sim_s(qt, k, d, NULL); }

/* The literal Sec. 3.3 reading in the SIM profile: 11 bits after every step. */
static double logit16_sim_step(const float *qt, const uint16_t *k, int d, int *sat)
{
    (void)sat;
    float acc = 0.0f;
    for (int c = 0; c < d; ++c) {
        float t = fmaf(qt[c], bf16_to_f32(k[c]), acc);
        acc = (float)round_sim((double)t, 11);
    }
    return (double)acc;
}

/* ------------------------------------------------------------------------ */
/* Stochastic rounding of the 8-bit accumulation.                            */
/* ------------------------------------------------------------------------ */
/* Sec. 3.3 ("Floating-point formats") names stochastic rounding (Croci et al.
 * 2022) as the alternative to round-to-nearest for the e4m3 accumulation, to
 * counter swamping.  The paper fixes neither the generator nor the number of
 * random bits; the readings taken:
 *   - each step rounds the FP32 FMA result t (as in the round-to-nearest
 *     recursion) to one of its two e4m3 neighbours: a = min(|t|, 448), lo the
 *     e4m3 number next to a toward zero, u = 2^(max(e, -6) - 3) its spacing
 *     (e the binary exponent of a); the result is lo + u when
 *     floor(2^16 (a - lo) / u) + r >= 2^16 and lo otherwise, with the sign of
 *     t (saturating at 448, as the round-to-nearest recursion; a zero keeps
 *     the sign of t).  r is a uniform 16-bit integer, so the probability of
 *     rounding away from zero is the distance to lo in units of u, cut to
 *     16 bits;
 *   - r comes from the counter-based generator Philox4x32-10 (Salmon, Moraes,
 *     Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011),
 *     key (seed mod 2^32, seed / 2^32), counter (j, i, b*Hq + h, c / 8) for
 *     query row j, key i, query head h of batch b and channel c: each of the
 *     four 32-bit words of one call holds two 16-bit fields, and channel c
 *     takes the low half (c even) or the high half (c odd) of word
 *     (c mod 8) / 2.  The numbers depend on the logit and the channel alone,
 *     not on any blocking. */

/* Philox4x32-10 of counter c under key k (SC 2011: the 4x32 round with
 * multipliers M0, M1 and Weyl key increments W0, W1; ten rounds, the first
 * with the key as given). */
void oracle_philox4x32_10(const uint32_t c_in[4], const uint32_t k_in[2], uint32_t out[4])
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t c0 = c_in[0], c1 = c_in[1], c2 = c_in[2], c3 = c_in[3];
    uint32_t k0 = k_in[0], k1 = k_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { k0 += W0; k1 += W1; }
        const uint64_t p0 = (uint64_t)M0 * c0, p1 = (uint64_t)M1 * c2;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        const uint32_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Stochastic rounding of t to e4m3 with the 16-bit random integer r (above). */
static double sr_e4m3(double t, uint32_t r)
{
    double a = fabs(t);
    if (a > F_E4M3.maxval) a = F_E4M3.maxval;
    int E;
    (void)frexp(a, &E);                 /* a = f 2^E, f in [1/2, 1); a = 0: E = 0 */
    int e = E - 1;
    int emin = 1 - F_E4M3.bias;
    if (e < emin) e = emin;
    double u = ldexp(1.0, e - F_E4M3.mbits);
    double lo = floor(a / u) * u;
    double frac16 = floor((a - lo) / u * 65536.0);
    double res = (frac16 + (double)r >= 65536.0) ? lo + u : lo;
    return copysign(res, t);
}

int oracle_sr_e4m3(const double *t, const uint32_t *r, double *y, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) {
        if (r[i] >= (1u << 16)) return -1;
        y[i] = sr_e4m3(t[i], r[i]);
    }
    return 0;
}

/* 16-bit random integer of channel c of the logit (j, i) of head bh. */
static uint32_t sr_bits(uint64_t seed, int64_t bh, int64_t j, int64_t i, int c, uint32_t w[4], int *have)
{
    if (c % 8 == 0 || !*have) {
        const uint32_t ctr[4] = {(uint32_t)j, (uint32_t)i, (uint32_t)bh, (uint32_t)(c / 8)};
        const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
        oracle_philox4x32_10(ctr, key, w);
        *have = 1;
    }
    return (w[(c % 8) / 2] >> (16 * (c & 1))) & 0xFFFFu;
}

/* Low-precision logit with stochastic rounding: the recursion of logit8 with
 * sr_e4m3 in place of round-to-nearest; *sat (may be NULL) is set when some
 * step's |t| exceeded 448 and was clamped. */
static double logit8_sr_s(const float *qt, const uint16_t *k, int d, uint64_t seed, int64_t bh, int64_t j,
                          int64_t i, int *sat)
{
    float acc = 0.0f;
    uint32_t w[4];
    int have = 0;
    for (int c = 0; c < d; ++c) {
        float t = fmaf(qt[c], bf16_to_f32(k[c]), acc);
        if (sat && fabs((double)t) > F_E4M3.maxval) *sat = 1;
        acc = (float)sr_e4m3((double)t, sr_bits(seed, bh, j, i, c, w, &have));
    }
    return (double)acc;
}

static double logit8_sr(const float *qt, const uint16_t *k, int d, uint64_t seed, int64_t bh, int64_t j, int64_t i)
{
    return logit8_sr_s(qt, k, d, seed, bh, j, i, NULL);
}

static int visible(int64_t i, int64_t j, int causal, int window)
{
    if (causal && i > j) return 0;
    if (window > 0 && i <= j - window) return 0;
    return 1;
}

/* Y8 codes of rows [row0, row0+nrows) of every (b, h): out[B][Hq][nrows][N],
 * invisible entries 0xFF. */
int oracle_logits8(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d,
                   int causal, int window, int row0, int nrows, uint8_t *out, int nthreads)
{
    if (Hq % Hkv) return -1;
    int G = Hq / Hkv;
    float s = scale_of(d);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for collapse(3) schedule(dynamic)
#endif
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < Hq; ++h)
            for (int r = 0; r < nrows; ++r) {
                int64_t j = row0 + r;
                float qt[1024];
                prescale(q + (((int64_t)b * Hq + h) * N + j) * d, d, s, qt);
                const uint16_t *kb = k + ((int64_t)b * Hkv + h / G) * N * d;
                uint8_t *o = out + (((int64_t)b * Hq + h) * nrows + r) * N;
                for (int64_t i = 0; i < N; ++i) {
                    if (!visible(i, j, causal, window)) { o[i] = 0xFF; continue; }
                    o[i] = (uint8_t)encode_fmt(logit8(qt, kb + i * d, d), &F_E4M3);
                }
            }
    return 0;
}

/* Y8 codes with stochastic rounding (seed above), same layout. */
int oracle_logits8_sr(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d,
                      int causal, int window, int row0, int nrows, uint64_t seed, uint8_t *out, int nthreads)
{
    if (Hq % Hkv) return -1;
    int G = Hq / Hkv;
    float s = scale_of(d);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for collapse(3) schedule(dynamic)
#endif
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < Hq; ++h)
            for (int r = 0; r < nrows; ++r) {
                int64_t j = row0 + r;
                float qt[1024];
                prescale(q + (((int64_t)b * Hq + h) * N + j) * d, d, s, qt);
                const uint16_t *kb = k + ((int64_t)b * Hkv + h / G) * N * d;
                uint8_t *o = out + (((int64_t)b * Hq + h) * nrows + r) * N;
                for (int64_t i = 0; i < N; ++i) {
                    if (!visible(i, j, causal, window)) { o[i] = 0xFF; continue; }
                    o[i] = (uint8_t)encode_fmt(logit8_sr(qt, kb + i * d, d, seed, (int64_t)b * Hq + h, j, i), &F_E4M3);
                }
            }
    return 0;
}

/* Y16 codes, same layout; invisible entries 0xFFFF (never compared). */
int oracle_logits16(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d,
                    int causal, int window, int row0, int nrows, uint16_t *out, int nthreads)
{
    if (Hq % Hkv) return -1;
    int G = Hq / Hkv;
    float s = scale_of(d);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for collapse(3) schedule(dynamic)
#endif
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < Hq; ++h)
            for (int r = 0; r < nrows; ++r) {
                int64_t j = row0 + r;
                float qt[1024];
                prescale(q + (((int64_t)b * Hq + h) * N + j) * d, d, s, qt);
                const uint16_t *kb = k + ((int64_t)b * Hkv + h / G) * N * d;
                uint16_t *o = out + (((int64_t)b * Hq + h) * nrows + r) * N;
                for (int64_t i = 0; i < N; ++i) {
                    if (!visible(i, j, causal, window)) { o[i] = 0xFFFF; continue; }
                    o[i] = (uint16_t)encode_fmt(logit16(qt, kb + i * d, d), &F_E4M11);
                }
            }
    return 0;
}

/* Y16 codes by the literal reading of Sec. 3.3 (e4m11 as the accumulator,
 * rounded after every FP32 FMA; logit16_step), same layout as
 * oracle_logits16. */
int oracle_logits16_step(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d,
                         int causal, int window, int row0, int nrows, uint16_t *out, int nthreads)
{
    if (Hq % Hkv) return -1;
    int G = Hq / Hkv;
    float s = scale_of(d);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for collapse(3) schedule(dynamic)
#endif
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < Hq; ++h)
            for (int r = 0; r < nrows; ++r) {
                int64_t j = row0 + r;
                float qt[1024];
                prescale(q + (((int64_t)b * Hq + h) * N + j) * d, d, s, qt);
                const uint16_t *kb = k + ((int64_t)b * Hkv + h / G) * N * d;
                uint16_t *o = out + (((int64_t)b * Hq + h) * nrows + r) * N;
                for (int64_t i = 0; i < N; ++i) {
                    if (!visible(i, j, causal, window)) { o[i] = 0xFFFF; continue; }
                    o[i] = (uint16_t)encode_fmt(logit16_step(qt, kb + i * d, d, NULL), &F_E4M11);
                }
            }
    return 0;
}

/* SIM profile logit values (high = 0: 8-bit recursion, 1: 16-bit), same
 * layout as above; invisible entries NaN. */
int oracle_logits_sim(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d,
                      int causal, int window, int row0, int nrows, int high, double *out, int nthreads)
{
    if (Hq % Hkv) return -1;
    int G = Hq / Hkv;
    float s = scale_of(d);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for collapse(3) schedule(dynamic)
#endif
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < Hq; ++h)
            for (int r = 0; r < nrows; ++r) {
                int64_t j = row0 + r;
                float qt[1024];
                prescale(q + (((int64_t)b * Hq + h) * N + j) * d, d, s, qt);
                const uint16_t *kb = k + ((int64_t)b * Hkv + h / G) * N * d;
                double *o = out + (((int64_t)b * Hq + h) * nrows + r) * N;
                for (int64_t i = 0; i < N; ++i) {
                    if (!visible(i, j, causal, window)) { o[i] = NAN; continue; }
                    o[i] = high ? logit16_sim(qt, kb + i * d, d) : logit8_sim(qt, kb + i * d, d);
                }
            }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* The forward pass (Algorithm 1).                                           */
/* ------------------------------------------------------------------------ */

enum { MASK_LOW = 0, MASK_STAGE1 = 1, MASK_STAGE2 = 2, MASK_INACTIVE = 3 };

/* Variants of Algorithm 1 (flags of lamp_oracle_fwd):
 *  ORACLE_STAGE1_OFF: the first stage is disabled (the paper's appendix on
 *    first-stage recomputation): mu_hat is the running maximum of the 8-bit
 *    logits and only the second stage chooses recomputations;
 *  ORACLE_MU_TRUNC: the 8-bit shifts use mu_hat truncated to e4m3 (Sec. 3.3:
 *    the running maxima may be rounded to e4m3 for the low-precision shifts by
 *    dropping the low mantissa bits).
 * Both apply for 0 < tau < inf; the two end modes ignore them.
 *  ORACLE_SIM: the "SIM" precision profile above (Sec. 4.1) in place of the
 *    hardware formats of Sec. 3.3, in every mode;
 *  ORACLE_SR8: the 8-bit logits rounded stochastically (logit8_sr, with the
 *    seed argument), in the modes that compute them; not with ORACLE_SIM;
 *  ORACLE_Y16_STEP: the 16-bit logits by the literal reading of Sec. 3.3,
 *    e4m11 (or, in the SIM profile, 11 bits) as the accumulator, rounded after
 *    every FP32 FMA (logit16_step), instead of the FP32 chain rounded once.
 *    An alternative reading for study; the GPU library does not build it. */
enum { ORACLE_STAGE1_OFF = 1, ORACLE_MU_TRUNC = 2, ORACLE_SIM = 4, ORACLE_SR8 = 8, ORACLE_Y16_STEP = 16 };

/* Statistics words (lamp_oracle_fwd_ex), counted from the definitions: the
 * (query block, key tile) pairs with an active sub-block, the stage-1 and
 * stage-2 sub-blocks (mask codes 1 and 2), the inactive ones (code 3), the
 * visible 8-bit logits whose recursion was clamped at some step, the visible
 * 16-bit logits of recomputed sub-blocks whose rounding was clamped, two
 * words of the GPU kernel's schedule (left 0 here), then the histogram of
 * 16-bit sub-blocks per active tile, 0..nk. */
enum { OST_TILES = 0, OST_S1, OST_S2, OST_INACTIVE, OST_SAT8, OST_SAT16, OST_HIST = 8 };

/* x truncated (rounded toward zero) to e4m3; reading: values beyond the
 * largest e4m3 number saturate to +-448; infinities are kept. */
static double trunc_e4m3(double x)
{
    if (isinf(x) || x == 0.0) return x;
    double ax = fabs(x);
    if (ax >= F_E4M3.maxval) return copysign(F_E4M3.maxval, x);
    int E;
    (void)frexp(ax, &E);
    int e = E - 1;
    int emin = 1 - F_E4M3.bias;
    if (e < emin) e = emin;
    double quantum = ldexp(1.0, e - F_E4M3.mbits);
    return copysign(floor(ax / quantum) * quantum, x);
}

double oracle_trunc_e4m3(double x) { return trunc_e4m3(x); }

/* Shifted exponential of one logit y against the running maximum mu_hat
 * (Alg. 1, exponential steps; Sec. 3.3): s = RN_shift(max(0, mu_hat - y)),
 * E = table[s].  The difference is exact in fp64 (both operands are
 * multiples of 2^-17 of magnitude <= 512).  Reading: the shift is clamped at
 * 0 (a stage-2 16-bit logit may exceed mu_hat, which stage 2 does not
 * update), so every E <= 1. */
static double shifted_exp(double mu_hat, double y, int high)
{
    double x = mu_hat - y;
    if (x < 0.0) x = 0.0;
    if (high) {
        uint32_t sc = encode_fmt(round_to_fmt(x, &F_UE5M11_SHIFT), &F_UE5M11_SHIFT);
        return decode_fmt(g_exp16[sc], &F_UE5M11_EXP);
    } else {
        uint32_t sc = encode_fmt(round_to_fmt(x, &F_UE5M3_SHIFT), &F_UE5M3_SHIFT);
        return decode_fmt(g_lut8[sc], &F_UE5M3_EXP);
    }
}

typedef struct {
    const uint16_t *q, *k, *v;
    int B, Hq, Hkv, N, d, causal, window, bq, bk, nk;
    double delta, tau;
    unsigned flags;
    uint64_t seed;
    double *o, *lse;
    uint8_t *mask;
    uint64_t *stats;
} fwd_args_t;

/* One query block (Alg. 1, body of the outer parallel loop). */
static void fwd_qblock(const fwd_args_t *A, int b, int h, int qb)
{
    const int d = A->d, N = A->N, bq = A->bq, bk = A->bk, nk = A->nk;
    const int T = bk * nk;                       /* keys per tile */
    const int G = A->Hq / A->Hkv;
    /* Reading for lengths that are not multiples of the block sizes: keys at
     * or beyond N are invisible, and the last query block's rows beyond N do
     * not exist (no visible key: they take part in no test and are not
     * written); the mask holds every sub-block of the ceil(N/T) tiles. */
    const int ntiles = (N + T - 1) / T;
    const int nkb = ntiles * nk;                 /* key sub-blocks per row */
    const int nqbh = (N + bq - 1) / bq;          /* query blocks per head */
    const int64_t q0 = (int64_t)qb * bq;
    const float s = scale_of(d);
    const uint16_t *kbase = A->k + ((int64_t)b * A->Hkv + h / G) * (int64_t)N * d;
    const uint16_t *vbase = A->v + ((int64_t)b * A->Hkv + h / G) * (int64_t)N * d;
    const int pure8 = isinf(A->tau) && A->tau > 0;
    const int all16 = (A->tau == 0.0);
    const int stage1_off = !pure8 && !all16 && (A->flags & ORACLE_STAGE1_OFF);
    const int mu_trunc = !pure8 && !all16 && (A->flags & ORACLE_MU_TRUNC);
    const int sim = (A->flags & ORACLE_SIM) != 0;
    const int sr8 = (A->flags & ORACLE_SR8) != 0;
    const int y16step = (A->flags & ORACLE_Y16_STEP) != 0;
    const int64_t bh = (int64_t)b * A->Hq + h;
    double (*const y8f)(const float *, const uint16_t *, int, int *) = sim ? logit8_sim_s : logit8_s;
    double (*const y16f)(const float *, const uint16_t *, int, int *) =
        sim ? (y16step ? logit16_sim_step : logit16_sim_s) : (y16step ? logit16_step : logit16_s);
    /* statistics of this query block (added to A->stats at the end) */
    uint64_t st_tiles = 0, st_s1 = 0, st_s2 = 0, st_sat8 = 0, st_sat16 = 0, st_hist[17] = {0};
    double (*const expf_)(double, double, int) = sim ? shifted_exp_sim : shifted_exp;

    float *qt = (float *)malloc(sizeof(float) * (size_t)bq * d);
    double *mu = (double *)malloc(sizeof(double) * bq);
    double *om = (double *)malloc(sizeof(double) * bq);
    double *O = (double *)calloc((size_t)bq * d, sizeof(double));
    double *muh = (double *)malloc(sizeof(double) * bq);
    double *lam = (double *)malloc(sizeof(double) * bq);
    double *omh = (double *)malloc(sizeof(double) * bq);
    double *Y = (double *)malloc(sizeof(double) * (size_t)T * bq);   /* [i][j] */
    double *E = (double *)malloc(sizeof(double) * (size_t)T * bq);   /* [i][j] */
    unsigned char *vis = (unsigned char *)malloc((size_t)T * bq);
    double *m8 = (double *)malloc(sizeof(double) * (size_t)nk * bq);
    double *cost = (double *)malloc(sizeof(double) * (size_t)nk * bq);
    int *prec = (int *)malloc(sizeof(int) * nk);  /* 0 low, 1 stage1, 2 stage2, 3 inactive */
    int *order = (int *)malloc(sizeof(int) * nk);
    double *thr = (double *)malloc(sizeof(double) * nk);

    for (int j = 0; j < bq; ++j) {
        if (q0 + j < N) prescale(A->q + (((int64_t)b * A->Hq + h) * N + q0 + j) * d, d, s, qt + (size_t)j * d);
        else memset(qt + (size_t)j * d, 0, sizeof(float) * (size_t)d);
        mu[j] = -INFINITY;
        om[j] = 0.0;
    }
    uint8_t *mrow = A->mask + (((int64_t)b * A->Hq + h) * nqbh + qb) * nkb;
    for (int t = 0; t < nkb; ++t) mrow[t] = MASK_INACTIVE;

    for (int tile = 0; tile < ntiles; ++tile) {
        const int64_t k0 = (int64_t)tile * T;
        int any_active = 0;
        for (int th = 0; th < nk; ++th) {
            int act = 0;
            for (int ii = th * bk; ii < (th + 1) * bk && !act; ++ii)
                for (int j = 0; j < bq; ++j)
                    if (k0 + ii < N && q0 + j < N && visible(k0 + ii, q0 + j, A->causal, A->window)) { act = 1; break; }
            prec[th] = act ? MASK_LOW : MASK_INACTIVE;
            any_active |= act;
        }
        if (!any_active) continue;               /* no state change */
        for (int ii = 0; ii < T; ++ii)
            for (int j = 0; j < bq; ++j)
                vis[(size_t)ii * bq + j] = (unsigned char)(k0 + ii < N && q0 + j < N &&
                                                           visible(k0 + ii, q0 + j, A->causal, A->window));

        /* Low-precision logits of the tile (Alg. 1: accumulate Y in low
         * precision).  In the all-16-bit mode they are never used. */
        if (!all16) {
            for (int ii = 0; ii < T; ++ii)
                for (int j = 0; j < bq; ++j) {
                    int sat = 0;
                    Y[(size_t)ii * bq + j] = vis[(size_t)ii * bq + j]
                        ? (sr8 ? logit8_sr_s(qt + (size_t)j * d, kbase + (k0 + ii) * d, d, A->seed, bh, q0 + j,
                                             k0 + ii, &sat)
                               : y8f(qt + (size_t)j * d, kbase + (k0 + ii) * d, d, &sat)) : NAN;
                    st_sat8 += (uint64_t)sat;
                }
        }
        /* Column maxima per sub-block: m8[theta][j] (Sec. 3.1, C and T). */
        for (int th = 0; th < nk; ++th)
            for (int j = 0; j < bq; ++j) {
                double m = -INFINITY;
                if (!all16)
                    for (int ii = th * bk; ii < (th + 1) * bk; ++ii)
                        if (vis[(size_t)ii * bq + j] && Y[(size_t)ii * bq + j] > m) m = Y[(size_t)ii * bq + j];
                m8[(size_t)th * bq + j] = m;
            }
        for (int j = 0; j < bq; ++j) muh[j] = mu[j];

        if (pure8 || stage1_off) {
            /* The paper's 8-bit baseline (Sec. 4.1), and the first stage
             * disabled: no stage-1 recomputation, the running maximum is
             * taken over the 8-bit logits. */
            for (int th = 0; th < nk; ++th)
                if (prec[th] != MASK_INACTIVE)
                    for (int j = 0; j < bq; ++j)
                        if (m8[(size_t)th * bq + j] > muh[j]) muh[j] = m8[(size_t)th * bq + j];
        } else if (all16) {
            /* Threshold 0: every active sub-block is recomputed in 16 bits
             * (16-bit FlashAttention in the paper's formats). */
            for (int th = 0; th < nk; ++th) {
                if (prec[th] == MASK_INACTIVE) continue;
                prec[th] = MASK_STAGE1;
                for (int ii = th * bk; ii < (th + 1) * bk; ++ii)
                    for (int j = 0; j < bq; ++j) {
                        size_t ix = (size_t)ii * bq + j;
                        if (!vis[ix]) continue;
                        int sat = 0;
                        Y[ix] = y16f(qt + (size_t)j * d, kbase + (k0 + ii) * d, d, &sat);
                        st_sat16 += (uint64_t)sat;
                        if (Y[ix] > muh[j]) muh[j] = Y[ix];
                    }
            }
        } else {
            /* Stage 1 (Sec. 3.1, Eq. (7); Alg. 1): threats
             * T_theta = max_j (m8[theta][j] - mu_j) over columns with a
             * visible entry (exact in fp64, +inf when mu_j = -inf). */
            int na = 0;
            for (int th = 0; th < nk; ++th) {
                if (prec[th] == MASK_INACTIVE) continue;
                double tv = -INFINITY;
                for (int j = 0; j < bq; ++j) {
                    double m = m8[(size_t)th * bq + j];
                    if (m == -INFINITY) continue;
                    double dlt = m - mu[j];
                    if (dlt > tv) tv = dlt;
                }
                thr[th] = tv;
                order[na++] = th;
            }
            /* Sort by threat, descending; reading: ties by ascending theta
             * (insertion sort is stable). */
            for (int a = 1; a < na; ++a) {
                int x = order[a], p = a - 1;
                while (p >= 0 && thr[order[p]] < thr[x]) { order[p + 1] = order[p]; --p; }
                order[p + 1] = x;
            }
            /* Sequential safety-margin test against the running mu_hat.
             * Reading: mu_hat_j > fma(|mu_hat_j|, delta, m8) (exact for the
             * paper's power-of-two delta); columns without a visible entry
             * are not tested; mu_hat = -inf fails. */
            for (int a = 0; a < na; ++a) {
                int th = order[a];
                int pass = 1;
                for (int j = 0; j < bq && pass; ++j) {
                    double m = m8[(size_t)th * bq + j];
                    if (m == -INFINITY) continue;
                    if (!(muh[j] > fma(fabs(muh[j]), A->delta, m))) pass = 0;
                }
                if (pass) continue;
                prec[th] = MASK_STAGE1;
                for (int ii = th * bk; ii < (th + 1) * bk; ++ii)
                    for (int j = 0; j < bq; ++j) {
                        size_t ix = (size_t)ii * bq + j;
                        if (!vis[ix]) continue;
                        int sat = 0;
                        Y[ix] = y16f(qt + (size_t)j * d, kbase + (k0 + ii) * d, d, &sat);
                        st_sat16 += (uint64_t)sat;
                        if (Y[ix] > muh[j]) muh[j] = Y[ix];
                    }
            }
        }

        /* Exponentials against the final mu_hat: 16-bit for stage-1
         * sub-blocks, 8-bit LUT for the rest (Alg. 1); the 8-bit ones
         * against mu_hat truncated to e4m3 with ORACLE_MU_TRUNC. */
        for (int th = 0; th < nk; ++th)
            for (int ii = th * bk; ii < (th + 1) * bk; ++ii)
                for (int j = 0; j < bq; ++j) {
                    size_t ix = (size_t)ii * bq + j;
                    const int high = prec[th] == MASK_STAGE1;
                    const double ref = (!high && mu_trunc) ? (sim ? trunc_sim(muh[j], 3) : trunc_e4m3(muh[j]))
                                                           : muh[j];
                    E[ix] = (prec[th] == MASK_INACTIVE || !vis[ix]) ? 0.0 : expf_(ref, Y[ix], high);
                }
        /* lambda_hat = exp(mu - mu_hat) in high precision (Sec. 2.2):
         * 1 when mu_hat = -inf (no mass yet), 0 when mu = -inf < mu_hat. */
        for (int j = 0; j < bq; ++j) {
            if (muh[j] == -INFINITY) lam[j] = 1.0;
            else if (mu[j] == -INFINITY) lam[j] = 0.0;
            else lam[j] = exp_doc(mu[j] - muh[j]);
            /* S_j = sum_i E_ij, keys ascending.  With the hardware formats
             * the sum is exact in fp64 (every E is a multiple of 2^-41 in
             * [0,1] and a tile holds at most 2^9 of them); in the SIM profile
             * (E down to 2^-137) it is the fp64 sum in this order. */
            double S = 0.0;
            for (int ii = 0; ii < T; ++ii) S += E[(size_t)ii * bq + j];
            omh[j] = fma(lam[j], om[j], S);
        }

        if (!pure8 && !all16) {
            /* Stage 2 (Sec. 3.1, Eq. (8)): per sub-block and column
             * c = sum_{i in theta, ascending} E (omega_hat - E), each
             * operation rounded in fp64. */
            int F = 0;
            for (int th = 0; th < nk; ++th) {
                if (prec[th] != MASK_LOW) continue;
                F |= 1 << th;
                for (int j = 0; j < bq; ++j) {
                    double c = 0.0;
                    for (int ii = th * bk; ii < (th + 1) * bk; ++ii) {
                        size_t ix = (size_t)ii * bq + j;
                        if (!vis[ix]) continue;
                        double tt = omh[j] - E[ix];
                        double pp = E[ix] * tt;
                        c = c + pp;
                    }
                    cost[(size_t)th * bq + j] = c;
                }
            }
            /* Maximise the number of 8-bit sub-blocks: enumerate the
             * recompute set R (a subset of F) by size, then (reading) by
             * ascending bitmask, and take the first R whose complement
             * satisfies xi_j <= (tau*omega_hat_j)*omega_hat_j for every j,
             * xi_j = sum over kept sub-blocks, ascending, in fp64. */
            int R = F;
            int nF = __builtin_popcount((unsigned)F);
            int found = 0;
            for (int sz = 0; sz <= nF && !found; ++sz) {
                for (int msk = 0; msk < (1 << nk) && !found; ++msk) {
                    if ((msk & ~F) || __builtin_popcount((unsigned)msk) != sz) continue;
                    int ok = 1;
                    for (int j = 0; j < bq && ok; ++j) {
                        double xi = 0.0;
                        for (int th = 0; th < nk; ++th)
                            if ((F >> th & 1) && !(msk >> th & 1)) xi = xi + cost[(size_t)th * bq + j];
                        double lim = (A->tau * omh[j]) * omh[j];
                        if (!(xi <= lim)) ok = 0;
                    }
                    if (ok) { R = msk; found = 1; }
                }
            }
            /* Stage-2 recompute (Alg. 1): 16-bit logits and exponentials
             * against the same mu_hat, which is not updated. */
            for (int th = 0; th < nk; ++th) {
                if (!(R >> th & 1)) continue;
                prec[th] = MASK_STAGE2;
                for (int ii = th * bk; ii < (th + 1) * bk; ++ii)
                    for (int j = 0; j < bq; ++j) {
                        size_t ix = (size_t)ii * bq + j;
                        if (!vis[ix]) continue;
                        int sat = 0;
                        Y[ix] = y16f(qt + (size_t)j * d, kbase + (k0 + ii) * d, d, &sat);
                        st_sat16 += (uint64_t)sat;
                        E[ix] = expf_(muh[j], Y[ix], 1);
                    }
            }
        }

        /* State update (Alg. 1): omega, O, mu. */
        for (int j = 0; j < bq; ++j) {
            double S = 0.0;
            for (int ii = 0; ii < T; ++ii) S += E[(size_t)ii * bq + j];
            om[j] = fma(lam[j], om[j], S);
            double *oj = O + (size_t)j * d;
            for (int c = 0; c < d; ++c) oj[c] *= lam[j];
            for (int ii = 0; ii < T; ++ii) {
                double e = E[(size_t)ii * bq + j];
                if (e == 0.0) continue;
                const uint16_t *vr = vbase + (k0 + ii) * d;
                for (int c = 0; c < d; ++c) oj[c] += e * (double)bf16_to_f32(vr[c]);
            }
            mu[j] = muh[j];
        }
        for (int th = 0; th < nk; ++th) mrow[tile * nk + th] = (uint8_t)prec[th];
        int nrec = 0;
        for (int th = 0; th < nk; ++th) {
            st_s1 += prec[th] == MASK_STAGE1;
            st_s2 += prec[th] == MASK_STAGE2;
            nrec += prec[th] == MASK_STAGE1 || prec[th] == MASK_STAGE2;
        }
        ++st_tiles;
        ++st_hist[nrec];
    }
    if (A->stats) {
        uint64_t inactive = 0;
        for (int t = 0; t < nkb; ++t) inactive += mrow[t] == MASK_INACTIVE;
        uint64_t *S = A->stats;
#ifdef _OPENMP
#pragma omp critical(oracle_stats)
#endif
        {
            S[OST_TILES] += st_tiles;
            S[OST_S1] += st_s1;
            S[OST_S2] += st_s2;
            S[OST_INACTIVE] += inactive;
            S[OST_SAT8] += st_sat8;
            S[OST_SAT16] += st_sat16;
            for (int c = 0; c <= nk; ++c) S[OST_HIST + c] += st_hist[c];
        }
    }

    /* Epilogue (Alg. 1): O / omega; lse = mu + ln(omega). */
    for (int j = 0; j < bq && q0 + j < N; ++j) {
        double *dst = A->o + (((int64_t)b * A->Hq + h) * N + q0 + j) * d;
        for (int c = 0; c < d; ++c) dst[c] = O[(size_t)j * d + c] / om[j];
        A->lse[((int64_t)b * A->Hq + h) * N + q0 + j] = mu[j] + log(om[j]);
    }
    free(qt); free(mu); free(om); free(O); free(muh); free(lam); free(omh);
    free(Y); free(E); free(vis); free(m8); free(cost); free(prec); free(order); free(thr);
}

/* lamp_oracle_fwd: Q,K,V bf16 bit patterns [B,H,N,d] (host memory),
 * outputs o [B,Hq,N,d] fp64, lse [B,Hq,N] fp64, mask [B,Hq,ceil(N/bq),
 * ceil(N/(bk*nk))*nk] u8 (any N >= 0; B = 0 or N = 0 computes nothing).
 * If qblocks != NULL only the listed query blocks (flat index
 * (b*Hq + h)*ceil(N/bq) + qb) are computed; other outputs are left untouched.
 * stats != NULL: the statistics words (OST_*, 8 + nk + 1 of them) of the
 * computed query blocks are added to it.
 * Returns 0, or -1 on invalid arguments / -2 on a table failure or, in the SIM
 * profile, an exponential too close to a rounding midpoint to be certified. */
int lamp_oracle_fwd_ex(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       int B, int Hq, int Hkv, int N, int d, int causal, int window,
                       int bq, int bk, int nk, double delta, double tau, unsigned flags, uint64_t seed,
                       double *o, double *lse, uint8_t *mask,
                       const int64_t *qblocks, int64_t nqblocks, int nthreads, uint64_t *stats)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || N < 0 || d <= 0 || d > 1024) return -1;
    if (Hq % Hkv || bq <= 0 || bk <= 0 || nk <= 0 || nk > 16) return -1;
    if (window < 0 || (window > 0 && !causal)) return -1;
    if (!(tau >= 0.0) || !(delta >= 0.0)) return -1;
    if (build_tables()) return -2;
    if (flags & ~(unsigned)(ORACLE_STAGE1_OFF | ORACLE_MU_TRUNC | ORACLE_SIM | ORACLE_SR8 | ORACLE_Y16_STEP)) return -1;
    if ((flags & ORACLE_SR8) && (flags & ORACLE_SIM)) return -1;
    if (B == 0 || N == 0) return 0;                /* nothing to compute */
    g_sim_fail = 0;
    fwd_args_t A = {q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, delta, tau, flags, seed, o, lse, mask,
                    stats};
    const int nqbh = (N + bq - 1) / bq;
    int64_t nqb = (int64_t)B * Hq * nqbh;
    int64_t count = qblocks ? nqblocks : nqb;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int64_t t = 0; t < count; ++t) {
        int64_t f = qblocks ? qblocks[t] : t;
        int qb = (int)(f % nqbh);
        int h = (int)((f / nqbh) % Hq);
        int b = (int)(f / ((int64_t)nqbh * Hq));
        fwd_qblock(&A, b, h, qb);
    }
    return g_sim_fail ? -2 : 0;
}

/* The above without statistics. */
int lamp_oracle_fwd_seeded(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                           int B, int Hq, int Hkv, int N, int d, int causal, int window,
                           int bq, int bk, int nk, double delta, double tau, unsigned flags, uint64_t seed,
                           double *o, double *lse, uint8_t *mask,
                           const int64_t *qblocks, int64_t nqblocks, int nthreads)
{
    return lamp_oracle_fwd_ex(q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, delta, tau, flags, seed, o, lse,
                              mask, qblocks, nqblocks, nthreads, NULL);
}

/* lamp_oracle_fwd: the above with seed 0 (ORACLE_SR8 takes the seeded form). */
int lamp_oracle_fwd(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                    int B, int Hq, int Hkv, int N, int d, int causal, int window,
                    int bq, int bk, int nk, double delta, double tau, unsigned flags,
                    double *o, double *lse, uint8_t *mask,
                    const int64_t *qblocks, int64_t nqblocks, int nthreads)
{
    return lamp_oracle_fwd_seeded(q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, delta, tau, flags, 0,
                                  o, lse, mask, qblocks, nqblocks, nthreads);
}

/* ------------------------------------------------------------------------ */
/* The vector form for single query rows (Sec. 2, "Look-ahead distribution   */
/* of precisions", Eq. (6)): decode against a key/value cache.               */
/* ------------------------------------------------------------------------ */

typedef struct {
    const uint16_t *q, *k, *v;
    int B, Hq, Hkv, M, N, d, causal, window, tk;
    double delta, tau;
    double *o, *lse;
    uint8_t *mask;
} dec_args_t;

typedef struct {
    double key;
    int idx;
} kidx_t;

/* ascending cost; reading: ties by ascending key index */
static int cmp_kidx(const void *pa, const void *pb)
{
    const kidx_t *a = (const kidx_t *)pa, *b = (const kidx_t *)pb;
    if (a->key < b->key) return -1;
    if (a->key > b->key) return 1;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

/* One query row: the online-softmax update of Sec. 2 over key tiles of tk
 * logits, each tile with the two-step look-ahead of Sec. 2:
 *   1. the maximizer c of the tile's 8-bit logits (reading: the first index
 *      attaining the maximum) passes if mu > fl(y_c) + |mu| delta, tested as
 *      mu > fma(|mu|, delta, fl(y_c)) (mu = -inf fails); then mu_hat = mu;
 *      otherwise y_c is recomputed in 16 bits, g_c = 0, and
 *      mu_hat = max(mu, y16_c);
 *   2. Eq. (6), a knapsack with uniform values solved greedily: the costs
 *      p_i (1 - p_i) of the remaining 8-bit logits, taken in the scaled form
 *      E_i (omega_hat - E_i) against tau omega_hat^2 (as in Eq. (8)), are
 *      sorted ascending (ties by index) and accumulated in fp64 while the sum
 *      stays within the limit; the first cost that would pass it and every
 *      later one are recomputed in 16 bits against the same mu_hat.
 * tau = +inf keeps every logit in 8 bits (mu_hat = max(mu, max fl(y)));
 * tau = 0 recomputes every visible logit. */
static void dec_row(const dec_args_t *A, int b, int h, int r)
{
    const int d = A->d, N = A->N, tk = A->tk;
    const int64_t P = (int64_t)N - A->M + r;           /* the query's position */
    const int G = A->Hq / A->Hkv;
    const int ntiles = (N + tk - 1) / tk;
    const float s = scale_of(d);
    const uint16_t *kbase = A->k + ((int64_t)b * A->Hkv + h / G) * (int64_t)N * d;
    const uint16_t *vbase = A->v + ((int64_t)b * A->Hkv + h / G) * (int64_t)N * d;
    const int pure8 = isinf(A->tau) && A->tau > 0;
    const int all16 = (A->tau == 0.0);
    const int64_t row = ((int64_t)b * A->Hq + h) * A->M + r;

    float *qt = (float *)malloc(sizeof(float) * (size_t)d);
    double *O = (double *)calloc((size_t)d, sizeof(double));
    double *Y = (double *)malloc(sizeof(double) * (size_t)tk);
    double *E = (double *)malloc(sizeof(double) * (size_t)tk);
    unsigned char *vis = (unsigned char *)malloc((size_t)tk);
    unsigned char *prec = (unsigned char *)malloc((size_t)tk);
    kidx_t *F = (kidx_t *)malloc(sizeof(kidx_t) * (size_t)tk);
    prescale(A->q + row * d, d, s, qt);
    double mu = -INFINITY, om = 0.0;
    uint8_t *mrow = A->mask + row * (int64_t)ntiles * tk;
    for (int64_t i = 0; i < (int64_t)ntiles * tk; ++i) mrow[i] = MASK_INACTIVE;

    for (int t = 0; t < ntiles; ++t) {
        const int64_t k0 = (int64_t)t * tk;
        int nvis = 0;
        for (int i = 0; i < tk; ++i) {
            vis[i] = (unsigned char)(k0 + i < N && visible(k0 + i, P, A->causal, A->window));
            nvis += vis[i];
            prec[i] = vis[i] ? MASK_LOW : MASK_INACTIVE;
        }
        if (!nvis) continue;                     /* no state change */
        double muh;
        if (all16) {
            muh = mu;
            for (int i = 0; i < tk; ++i) {
                if (!vis[i]) continue;
                Y[i] = logit16(qt, kbase + (k0 + i) * d, d);
                prec[i] = MASK_STAGE1;
                if (Y[i] > muh) muh = Y[i];
            }
        } else {
            int c = -1;
            for (int i = 0; i < tk; ++i) {
                if (!vis[i]) continue;
                Y[i] = logit8(qt, kbase + (k0 + i) * d, d);
                if (c < 0 || Y[i] > Y[c]) c = i;
            }
            if (pure8) {
                muh = Y[c] > mu ? Y[c] : mu;
            } else if (mu > fma(fabs(mu), A->delta, Y[c])) {
                muh = mu;
            } else {
                Y[c] = logit16(qt, kbase + (k0 + c) * d, d);
                prec[c] = MASK_STAGE1;
                muh = Y[c] > mu ? Y[c] : mu;
            }
        }
        for (int i = 0; i < tk; ++i)
            E[i] = vis[i] ? shifted_exp(muh, Y[i], prec[i] == MASK_STAGE1) : 0.0;
        const double lam = (mu == -INFINITY) ? 0.0 : exp_doc(mu - muh);
        double S = 0.0;
        for (int i = 0; i < tk; ++i) S += E[i];  /* exact (multiples of 2^-41) */
        const double omh = fma(lam, om, S);
        if (!pure8 && !all16) {
            int nf = 0;
            for (int i = 0; i < tk; ++i) {
                if (prec[i] != MASK_LOW) continue;
                double tt = omh - E[i];
                F[nf].key = E[i] * tt;
                F[nf].idx = i;
                ++nf;
            }
            qsort(F, (size_t)nf, sizeof(kidx_t), cmp_kidx);
            const double lim = (A->tau * omh) * omh;
            double xi = 0.0;
            int a = 0;
            for (; a < nf; ++a) {
                double nx = xi + F[a].key;
                if (!(nx <= lim)) break;
                xi = nx;
            }
            for (; a < nf; ++a) {                 /* recomputed in 16 bits */
                int i = F[a].idx;
                Y[i] = logit16(qt, kbase + (k0 + i) * d, d);
                E[i] = shifted_exp(muh, Y[i], 1);
                prec[i] = MASK_STAGE2;
            }
        }
        double S2 = 0.0;
        for (int i = 0; i < tk; ++i) S2 += E[i];
        om = fma(lam, om, S2);
        for (int c = 0; c < d; ++c) O[c] *= lam;
        for (int i = 0; i < tk; ++i) {
            if (E[i] == 0.0) continue;
            const uint16_t *vr = vbase + (k0 + i) * d;
            for (int c = 0; c < d; ++c) O[c] += E[i] * (double)bf16_to_f32(vr[c]);
        }
        mu = muh;
        for (int i = 0; i < tk; ++i) mrow[k0 + i] = prec[i];
    }
    double *dst = A->o + row * d;
    for (int c = 0; c < d; ++c) dst[c] = O[c] / om;
    A->lse[row] = mu + log(om);
    free(qt); free(O); free(Y); free(E); free(vis); free(prec); free(F);
}

/* lamp_oracle_decode: q [B,Hq,M,d] (M query rows at positions N-M .. N-1),
 * k, v [B,Hkv,N,d] bf16 bit patterns (host); o [B,Hq,M,d] fp64, lse [B,Hq,M]
 * fp64, mask [B,Hq,M,ceil(N/tk)*tk] u8 per key (0 8-bit, 1 the maximizer
 * recomputed by the look-ahead test (every logit at tau = 0), 2 recomputed by
 * the knapsack, 3 invisible).  rows != NULL computes only the listed rows
 * (flat (b*Hq + h)*M + r).  flags must be 0.  Returns 0, -1 on invalid
 * arguments, -2 on a table failure. */
int lamp_oracle_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       int B, int Hq, int Hkv, int M, int N, int d, int causal, int window, int tk,
                       double delta, double tau, unsigned flags, double *o, double *lse, uint8_t *mask,
                       const int64_t *rows, int64_t nrows, int nthreads)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || M < 0 || N < 0 || M > N || d <= 0 || d > 1024) return -1;
    if (Hq % Hkv || tk <= 0 || window < 0 || (window > 0 && !causal)) return -1;
    if (!(tau >= 0.0) || !(delta >= 0.0) || flags) return -1;
    if (build_tables()) return -2;
    if (B == 0 || M == 0) return 0;
    dec_args_t A = {q, k, v, B, Hq, Hkv, M, N, d, causal, window, tk, delta, tau, o, lse, mask};
    const int64_t total = (int64_t)B * Hq * M;
    const int64_t count = rows ? nrows : total;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int64_t t = 0; t < count; ++t) {
        int64_t f = rows ? rows[t] : t;
        int r = (int)(f % M);
        int h = (int)((f / M) % Hq);
        int b = (int)(f / ((int64_t)M * Hq));
        dec_row(&A, b, h, r);
    }
    return 0;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
