// lamp_sr.h -- stochastic rounding of the 8-bit logit accumulation.
//
// Sec. 3.3 ("Floating-point formats") names stochastic rounding (Croci et al.
// 2022) as the alternative to round-to-nearest for the e4m3 accumulation, to
// counter swamping.  The paper fixes neither the generator nor the number of
// random bits; the library's reading:
//   - each step rounds the FP32 FMA result t to one of its two e4m3
//     neighbours: a = min(|t|, 448), lo the e4m3 number next to a toward zero,
//     u its spacing; the step goes to lo + u when floor(2^20 (a - lo) / u) +
//     r >= 2^20 and to lo otherwise, with the sign of t; r is a uniform
//     20-bit integer;
//   - r comes from the counter-based generator Philox4x64-10 (Salmon, Moraes,
//     Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011)
//     under key (seed, 0) at counter (j, i, b*Hq + h, c / 8) for query row j,
//     key i, query head h of batch b and channel c; the four 64-bit outputs
//     are read as eight 32-bit halves, low half first, and channel c takes
//     the top 20 bits of half c mod 8.
// The random numbers depend on the logit and the channel only, so the 8-bit
// logits are the same under every blocking and in the logits entry point.
#pragma once
#include <stdint.h>

#include "lamp_device.h"

namespace lamp {

// Philox4x64-10: ten rounds of the 4x64 round function; the key is bumped by
// the Weyl constants before every round after the first.
__device__ __forceinline__ void philox4x64_10(uint64_t (&c)[4], uint64_t k0, uint64_t k1)
{
    constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        const uint64_t hi0 = __umul64hi(M0, c[0]), lo0 = M0 * c[0];
        const uint64_t hi1 = __umul64hi(M1, c[2]), lo1 = M1 * c[2];
        const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
}

// The 20-bit random integer of channel u (0..7) of a group from its words.
__device__ __forceinline__ uint32_t sr_r20(const uint64_t (&w)[4], int u)
{
    const uint64_t word = w[u >> 1];
    const uint32_t half = (u & 1) ? (uint32_t)(word >> 32) : (uint32_t)word;
    return half >> 12;
}

// Stochastic rounding of a finite fp32 value to e4m3 (saturating at 448),
// returned as the fp32 value.  In the normal e4m3 range the FP32 pattern has
// exactly 20 bits below e4m3's last mantissa bit: adding r to them carries
// into that bit when the rounding goes up.  Below 2^-6 the spacing is 2^-9
// and the distance to the lower neighbour is taken in units of 2^-29 (all
// steps exact).
__device__ __forceinline__ float sr_e4m3(float t, uint32_t r)
{
    const uint32_t bits = __builtin_bit_cast(uint32_t, t);
    const uint32_t sign = bits & 0x80000000u;
    uint32_t a = bits & 0x7FFFFFFFu;
    a = a < 0x43E00000u ? a : 0x43E00000u;                 // 448
    uint32_t res;
    if (a >= 0x3C800000u) {                                  // 2^-6
        res = (a & 0xFFF00000u) + (((a & 0xFFFFFu) + r) & 0x100000u);
    } else {
        const float af = __builtin_bit_cast(float, a);
        const float lo = __builtin_floorf(af * 512.0f) * (1.0f / 512.0f);
        const uint32_t f20 = (uint32_t)((af - lo) * 536870912.0f);   // 2^29
        res = __builtin_bit_cast(uint32_t, lo + (f20 + r >= 0x100000u ? 1.0f / 512.0f : 0.0f));
    }
    return __builtin_bit_cast(float, res | sign);
}

// 8-bit logits with stochastic rounding for 16 keys and QPL query rows per
// lane: the key rows k32 + kk*D (fp32, kk = 0..15, the same for every lane),
// the query rows qrow[s] (fp32, pre-scaled) of query index j[s]; key index
// i0 + kk; bh = b*Hq + h.  Codes out as in emu8_chunk: acc[s][p] holds the
// e4m3 codes of keys 2p (bits 7:0) and 2p+1 (bits 15:8).
template <int D, int QPL>
__device__ __forceinline__ void sr8_chunk(const float *const (&qrow)[QPL], const float *k32, uint64_t seed,
                                          uint64_t bh, const int (&j)[QPL], int i0, uint32_t (&acc)[QPL][8])
{
    static_assert(D % 8 == 0, "channel groups of 8");
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int p = 0; p < 8; ++p) acc[s][p] = 0u;
    for (int kk = 0; kk < 16; ++kk) {
        const float *krow = k32 + (size_t)kk * D;
        float y[QPL];
#pragma unroll
        for (int s = 0; s < QPL; ++s) y[s] = 0.0f;
        for (int g = 0; g < D / 8; ++g) {
            const float4 ka = *reinterpret_cast<const float4 *>(krow + 8 * g);
            const float4 kb = *reinterpret_cast<const float4 *>(krow + 8 * g + 4);
            const float kv[8] = {ka.x, ka.y, ka.z, ka.w, kb.x, kb.y, kb.z, kb.w};
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
                const float4 qa = *reinterpret_cast<const float4 *>(qrow[s] + 8 * g);
                const float4 qb = *reinterpret_cast<const float4 *>(qrow[s] + 8 * g + 4);
                const float qv[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
                uint64_t w[4] = {(uint64_t)(uint32_t)j[s], (uint64_t)(uint32_t)(i0 + kk), bh, (uint64_t)g};
                philox4x64_10(w, seed, 0);
                float v = y[s];
#pragma unroll
                for (int u = 0; u < 8; ++u) v = sr_e4m3(__builtin_fmaf(qv[u], kv[u], v), sr_r20(w, u));
                y[s] = v;
            }
        }
        // the code of key kk into its byte (exact: y is an e4m3 value)
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            const uint32_t code = pk_e4m3_sat(y[s], 0.0f) & 0xFFu;
#pragma unroll
            for (int p = 0; p < 8; ++p) acc[s][p] |= (p == (kk >> 1)) ? code << (8 * (kk & 1)) : 0u;
        }
    }
}

} // namespace lamp
