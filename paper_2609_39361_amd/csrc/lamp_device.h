// lamp_device.h -- device numerics of the LampAttention forward pass (gfx950).
//
// Number formats of the method (paper Sec. 3.3), all round-to-nearest-even
// with subnormals:
//   e4m3   8-bit logit accumulator, bias 7, saturating at +-448
//   e4m11  16-bit logit accumulator, bias 7, saturating at +-511.875
//   ue5m3  / ue5m11 shifted logits mu_hat - y >= 0, bias 15
//   ue5m3  / ue5m11 exponentials, bias 31 (code 11111000 = 1.0)
// The 8-bit accumulation (Sec. 4.1: recursive FMA summation in FP32, the sum
// rounded after every step) uses the hardware fp8 conversions: one fp32 FMA
// per multiply-add, and one packed round-to-e4m3 plus one packed decode per
// two accumulators.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lamp {

// Round two fp32 values to e4m3 with the hardware conversion (RNE).  Codes in
// bits [7:0] and [15:8]; bits [31:16] are taken from `old` (passing the
// register being overwritten avoids a register copy).  The conversion does not
// saturate: a value whose rounding exceeds 448 gives a NaN code (0x7F/0xFF),
// and NaN stays NaN through every later FMA and conversion, so an overflow
// anywhere in a chain shows up as a NaN code at its end.
__device__ __forceinline__ uint32_t pk_e4m3(float a, float b, uint32_t old = 0u)
{
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, false);
}

// Saturating variant (the method's definition: RN, then +-448 on overflow):
// clamping first gives the same code, since RN is monotone and 448 is on the
// grid.
__device__ __forceinline__ uint32_t pk_e4m3_sat(float a, float b, uint32_t old = 0u)
{
    a = __builtin_amdgcn_fmed3f(a, -448.0f, 448.0f);
    b = __builtin_amdgcn_fmed3f(b, -448.0f, 448.0f);
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, false);
}

// Pointers into read-only memory that every lane of a wave reads at the same
// address: the constant address space makes the compiler use scalar loads.
typedef const float __attribute__((address_space(4))) *kptr32_t;
typedef const double __attribute__((address_space(4))) *kptr64_t;

// Nonzero iff one of the two codes in bits [15:0] is a NaN code.
__device__ __forceinline__ uint32_t e4m3_nan_bits(uint32_t r)
{
    return ((r & 0x7F7Fu) + 0x0101u) & 0x8080u;
}

// Decode the two e4m3 codes in bits [15:0] (exact).
__device__ __forceinline__ float2 unpk_e4m3(uint32_t r)
{
    auto v = __builtin_amdgcn_cvt_pk_f32_fp8((int)r, false);
    return make_float2(v[0], v[1]);
}

__device__ __forceinline__ float e4m3_value(uint32_t code)
{
    return __builtin_amdgcn_cvt_f32_fp8((int)code, 0);
}

// --- e4m11 -----------------------------------------------------------------
// Round an fp64 value to e4m11 (RNE, subnormal quantum 2^-17, saturating at
// 511.875).  Returns the value (exact in fp32) and its code in *code.
__device__ __forceinline__ float rn_e4m11(double y, uint32_t *code)
{
    double ay = __builtin_fabs(y);
    int e = __builtin_amdgcn_frexp_exp(ay) - 1;          // ay in [2^e, 2^(e+1))
    int qe = (e > -6 ? e : -6) - 11;                     // exponent of the quantum
    double c = __builtin_amdgcn_ldexp(1.5, 52 + qe);     // ulp(c) = 2^qe
    double r = (ay + c) - c;                             // RNE to a multiple of 2^qe
    r = r < 511.875 ? r : 511.875;
    uint32_t sign = __builtin_signbit(y) ? 0x8000u : 0u;
    uint32_t mag;
    if (r < 0x1p-6) {
        mag = (uint32_t)(r * 0x1p17);
    } else {
        uint32_t hi = (uint32_t)(__builtin_bit_cast(uint64_t, r) >> 32);
        uint32_t ex = (hi >> 20) - 1023u + 7u;
        mag = (ex << 11) | ((hi >> 9) & 0x7FFu);
    }
    *code = sign | mag;
    float v = (float)r;
    return sign ? -v : v;
}

// Value of an e4m11 code, exact in fp32, without branches: the significand
// (with its implicit bit for a normal code) scaled by 2^(max(ex, 1) - 18).
// The same rounding of a finite fp32 value, on its bit pattern (identical to
// rn_e4m11((double)x)): from 2^-6 on, round to nearest even at bit 12 of the
// fp32 pattern (a carry moves into the exponent); below, add and subtract
// 1.5 * 2^6, whose ulp is the subnormal quantum 2^-17; then saturate.
__device__ __forceinline__ float rn_e4m11_f32(float x, uint32_t *code)
{
    const uint32_t b = __builtin_bit_cast(uint32_t, x), sign = b & 0x80000000u, ab = b & 0x7FFFFFFFu;
    const float ax = __builtin_bit_cast(float, ab);
    const uint32_t rn = (ab + 0x7FFu + ((ab >> 12) & 1u)) & 0xFFFFF000u;
    const float as = (ax + 96.0f) - 96.0f;
    uint32_t r = ab < 0x3C800000u ? __builtin_bit_cast(uint32_t, as) : rn;   // 0x3C800000 = 2^-6
    r = r < 0x43FFF000u ? r : 0x43FFF000u;                                     // 0x43FFF000 = 511.875
    *code = (sign >> 16) | (r >= 0x3C800000u ? (r >> 12) - 0x3C000u : (uint32_t)(as * 131072.0f));
    return __builtin_bit_cast(float, r | sign);
}

__device__ __forceinline__ float e4m11_value(uint32_t code)
{
    const uint32_t ex = (code >> 11) & 0xFu, m = code & 0x7FFu;
    const float v = __builtin_amdgcn_ldexpf((float)(ex ? m | 0x800u : m), (int)(ex ? ex : 1u) - 18);
    return (code & 0x8000u) ? -v : v;
}

// An e4m11 (or e4m3) value truncated toward zero to e4m3, saturating at 448;
// infinities are kept.  Normal e4m3 magnitudes keep the top 3 fp32 mantissa
// bits; below 2^-6 the e4m3 quantum is 2^-9.
__device__ __forceinline__ float trunc_e4m3(float x)
{
    const float ax = __builtin_fabsf(x);
    if (!(ax < 0x1p-6f)) {
        if (ax >= 448.0f) return ax == __builtin_inff() ? x : __builtin_copysignf(448.0f, x);
        return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, x) & 0xFFF00000u);
    }
    return __builtin_copysignf(__builtin_truncf(ax * 512.0f) * (1.0f / 512.0f), x);
}

// --- shifts ----------------------------------------------------------------
// Shift s = max(mu_hat - y, 2^-14) in fp32.  mu_hat (e4m11 or e4m3) and y are
// multiples of 2^-17 of magnitude <= 511.875, so the fp32 difference is exact
// below 128; from 128 on every exponential below is 0 whatever the rounding.
// Shifts below 2^-14 give the exponential 1.0 in both formats, so they are
// lifted to 2^-14, the smallest normal shift, which keeps the code arithmetic
// free of the subnormal case.
__device__ __forceinline__ float shift_of(float mu_hat, float y)
{
    float x = mu_hat - y;
    return x > 0x1p-14f ? x : 0x1p-14f;
}

// ue5m3 (bias 15) code of a normal shift: RNE on the fp32 bits.  Shifts are
// at most 1024 (code 200); the clamp keeps the table index in range whatever
// the input.
__device__ __forceinline__ uint32_t ue5m3_code(float x)
{
    uint32_t b = __builtin_bit_cast(uint32_t, x);
    uint32_t c = ((b + 0x7FFFFu + ((b >> 20) & 1u)) >> 20) - ((127u - 15u) << 3);
    return c < 255u ? c : 255u;
}

// ue5m11 (bias 15) code of a normal shift, clamped to the table.
__device__ __forceinline__ uint32_t ue5m11_code(float x)
{
    uint32_t b = __builtin_bit_cast(uint32_t, x);
    uint32_t c = ((b + 0x7FFu + ((b >> 12) & 1u)) >> 12) - ((127u - 15u) << 11);
    return c < 65535u ? c : 65535u;
}

// --- exponential codes -------------------------------------------------------
// Value of a ue5m11 (bias 31) exponential code, exact in fp32.
__device__ __forceinline__ float ue5m11e_value(uint32_t c)
{
    uint32_t ex = c >> 11, m = c & 0x7FFu;
    return ex ? __builtin_bit_cast(float, ((ex + 96u) << 23) | (m << 12)) : (float)m * 0x1p-41f;
}

// bf16 bit pattern of a bf16-exact fp32 value.
__device__ __forceinline__ uint32_t bf16_bits(float v)
{
    return __builtin_bit_cast(uint32_t, v) >> 16;
}

__device__ __forceinline__ float bf16_value(uint32_t b)
{
    return __builtin_bit_cast(float, b << 16);
}

// A ue5m11 exponential (12 significant bits, at least 2^-41) as the exact sum
// of two bf16 values: hi keeps the top 8 significant bits (the fp32 pattern
// with its low half cleared), lo = ev - hi holds the remaining 4 and is exact.
__device__ __forceinline__ void split_bf16(float ev, uint32_t &hi, uint32_t &lo)
{
    const uint32_t bits = __builtin_bit_cast(uint32_t, ev);
    hi = bits >> 16;
    lo = __builtin_bit_cast(uint32_t, ev - __builtin_bit_cast(float, bits & 0xFFFF0000u)) >> 16;
}

// --- the SIM profile (Sec. 4.1) -----------------------------------------------
// The numerics of the paper's simulation: numbers kept in FP32 with P = 3 or
// 11 stored mantissa bits, FP32's exponent range and gradual underflow, no
// saturation.  The rounding acts on the FP32 encoding: the fraction field is
// rounded at bit 23-P to nearest, ties to even, a carry moving into the
// exponent (overflow gives an infinity).
template <int P>
__device__ __forceinline__ float rn_sim(float x)
{
    constexpr uint32_t DROP = 23 - P;
    const uint32_t b = __builtin_bit_cast(uint32_t, x);
    return __builtin_bit_cast(float, (b + ((1u << (DROP - 1)) - 1u) + ((b >> DROP) & 1u)) & ~((1u << DROP) - 1u));
}

// mu_hat rounded toward zero to 3 mantissa bits (the optional truncation of
// Sec. 3.3 in the SIM profile); infinities are kept.
__device__ __forceinline__ float trunc_sim3(float x)
{
    return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, x) & 0xFFF00000u);
}

// Exponential tables of the SIM profile: entry ((e - EMIN) << P) | m holds
// RN_P(exp(-s)) for the shift s = (2^P + m) 2^(e-P).  Shifts below 2^EMIN give
// 1 and shifts from 2^EMAX on give 0, so the first and last rows are constant
// and shifts outside the range are clamped to them.
constexpr int SIM8_EMIN = -6, SIM8_EMAX = 7, SIM16_EMIN = -14, SIM16_EMAX = 7;
constexpr int SIM8_N = (SIM8_EMAX - SIM8_EMIN + 1) << 3;
constexpr int SIM16_N = (SIM16_EMAX - SIM16_EMIN + 1) << 11;

// Table index of s = RN_P(max(0, mu - y)), the exact difference rounded once.
// The fp32 difference and its TwoSum error give the exact value; only a
// difference lying exactly halfway between two grid values can round
// differently from its fp32 rounding, and then the sign of the error decides.
// mu and y are finite.
template <int P, int EMIN, int EMAX>
__device__ __forceinline__ uint32_t sim_shift_index(float mu, float y)
{
    const float s = mu - y;
    if (!(s > 0.0f)) return 0u;   // shift 0 (a difference of 0 is exact)
    const float bb = s - mu;
    const float err = (mu - (s - bb)) + (-y - bb);
    constexpr uint32_t DROP = 23 - P, HALF = 1u << (DROP - 1), LOW = (1u << DROP) - 1u;
    const uint32_t b = __builtin_bit_cast(uint32_t, s);
    uint32_t r = (b + (HALF - 1u) + ((b >> DROP) & 1u)) & ~LOW;
    if ((b & LOW) == HALF && err != 0.0f) r = err > 0.0f ? b + HALF : b & ~LOW;
    int e = (int)(r >> 23) - 127;
    e = e < EMIN ? EMIN : (e > EMAX ? EMAX : e);
    return ((uint32_t)(e - EMIN) << P) | ((r >> DROP) & ((1u << P) - 1u));
}

// Column maxima of SIM logits merge through an integer atomic max: the FP32
// pattern mapped to an int that orders like the value (negative patterns
// have their magnitude bits flipped); the map is its own inverse.
__device__ __forceinline__ int ord_of(float y)
{
    const int b = __builtin_bit_cast(int, y);
    return b ^ ((b >> 31) & 0x7FFFFFFF);
}

__device__ __forceinline__ float ord_value(int k)
{
    return __builtin_bit_cast(float, k ^ ((k >> 31) & 0x7FFFFFFF));
}

// --- exp_doc ----------------------------------------------------------------
// The fp64 exponential of the rescale factor lambda_hat = exp(mu - mu_hat)
// (Sec. 2.2: alpha_hat in high precision), fixed operation by operation so
// that it is reproducible: Cody-Waite reduction with ln 2 split into a
// 32-significant-bit head and an fp64 tail, then the degree-13 Taylor
// polynomial in Horner form with fma and coefficients RN64(1/k!), then an
// exact scaling by 2^n.  Arguments below -700 give 0.
//
// EXPDOC_K: log2(e), ln2 head, ln2 tail, then 1/13!, 1/12!, ..., 1/0!.
constexpr int EXPDOC_NK = 17;
__device__ constexpr double EXPDOC_K[EXPDOC_NK] = {
    0x1.71547652b82fep+0, 0x1.62e42fee00000p-1, 0x1.a39ef35793c76p-33,
    0x1.6124613a86d09p-33, 0x1.1eed8eff8d898p-29, 0x1.ae64567f544e4p-26, 0x1.27e4fb7789f5cp-22,
    0x1.71de3a556c734p-19, 0x1.a01a01a01a01ap-16, 0x1.a01a01a01a01ap-13, 0x1.6c16c16c16c17p-10,
    0x1.1111111111111p-7,  0x1.5555555555555p-5,  0x1.5555555555555p-3,  0x1.0000000000000p-1,
    1.0, 1.0};

// k(i) returns EXPDOC_K[i]; the forward kernel reads them from LDS so that the
// compiler does not keep 17 fp64 constants in registers across its main loop.
template <class K>
__device__ __forceinline__ double exp_doc_k(double x, K k)
{
    if (x < -700.0) return 0.0;
    double n = __builtin_rint(x * k(0));
    double r = __builtin_fma(-n, k(1), x);
    r = __builtin_fma(-n, k(2), r);
    double p = k(3);
#pragma unroll
    for (int i = 4; i < EXPDOC_NK; ++i) p = __builtin_fma(p, r, k(i));
    return __builtin_amdgcn_ldexp(p, (int)n);
}

__device__ __forceinline__ double exp_doc(double x)
{
    return exp_doc_k(x, [](int i) { return EXPDOC_K[i]; });
}

// --- wave helpers ------------------------------------------------------------
__device__ __forceinline__ double wave_max_f64(double v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        double o = __shfl_xor(v, m, 64);
        v = o > v ? o : v;
    }
    return v;
}

__device__ __forceinline__ bool wave_any(bool p)
{
    return __ballot(p) != 0ull;
}

} // namespace lamp
