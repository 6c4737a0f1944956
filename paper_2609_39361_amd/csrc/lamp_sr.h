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
//     under key (seed, 0) at counter (j, i, b*Hq + h, c / 12) for query row
//     j, key i, query head h of batch b and channel c; each of the four
//     64-bit outputs holds three 20-bit fields (bits 0-19, 20-39, 40-59), and
//     channel c takes field (c mod 12) mod 3 of output (c mod 12) / 3, so
//     one call serves twelve channels.
// The random numbers depend on the logit and the channel only, so the 8-bit
// logits are the same under every blocking and in the logits entry point.
#pragma once
#include <stdint.h>
#include <utility>

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

// The 20-bit random integer of channel u (0..11) of a group from its words.
template <int U>
__device__ __forceinline__ uint32_t sr_r20(const uint64_t (&w)[4])
{
    return (uint32_t)((w[U / 3] >> (20 * (U % 3))) & 0xFFFFFull);
}

// Stochastic rounding of a finite fp32 value to e4m3 (saturating at 448),
// returned as the fp32 value, without branches.  In the normal e4m3 range the
// FP32 pattern has exactly 20 bits below e4m3's last mantissa bit: adding r
// to them carries into that bit when the rounding goes up.  Below 2^-6 the
// spacing is 2^-9: the magnitude in units of 2^-29, truncated to an integer
// (the floor the rounding asks for), takes the same carry step, and the
// result is converted back (all steps exact).
// amax keeps the largest |t| pattern seen, so that a chain whose steps were
// clamped (|t| > 448) can be counted.
__device__ __forceinline__ float sr_e4m3(float t, uint32_t r, uint32_t &amax)
{
    const uint32_t bits = __builtin_bit_cast(uint32_t, t);
    const uint32_t sign = bits & 0x80000000u;
    uint32_t a = bits & 0x7FFFFFFFu;
    amax = amax > a ? amax : a;
    a = a < 0x43E00000u ? a : 0x43E00000u;                                 // 448
    const bool sub = a < 0x3C800000u;                                       // below 2^-6
    const uint32_t n = (uint32_t)(__builtin_bit_cast(float, a) * 536870912.0f);   // 2^29 units, floor
    const uint32_t x = sub ? n : a;
    const uint32_t y = (x & 0xFFF00000u) + (((x & 0xFFFFFu) + r) & 0x100000u);
    const uint32_t ys = __builtin_bit_cast(uint32_t, (float)y * (1.0f / 536870912.0f));
    return __builtin_bit_cast(float, (sub ? ys : y) | sign);
}

// The steps of one row over the channels U... of a group, in order.
template <int NC, int... U>
__device__ __forceinline__ float sr8_steps(const float (&qv)[NC], const float (&kv)[NC], const uint64_t (&w)[4],
                                           float v, uint32_t &amax, std::integer_sequence<int, U...>)
{
    ((v = sr_e4m3(__builtin_fmaf(qv[U], kv[U], v), sr_r20<U>(w), amax)), ...);
    return v;
}

// NC channels from c0 of one key and QPL rows: the group's Philox call, then
// the NC steps of each row's recursion.
template <int NC, int QPL>
__device__ __forceinline__ void sr8_group(const float *const (&qrow)[QPL], const float *krow, int c0, uint64_t seed,
                                          uint64_t bh, const int (&j)[QPL], uint32_t key, float (&y)[QPL],
                                          uint32_t (&amax)[QPL])
{
    static_assert(NC % 4 == 0 && NC <= 12, "whole 4-channel loads, at most one call");
    float kv[NC];
#pragma unroll
    for (int u = 0; u < NC; u += 4) {
        const float4 a = *reinterpret_cast<const float4 *>(krow + c0 + u);
        kv[u] = a.x; kv[u + 1] = a.y; kv[u + 2] = a.z; kv[u + 3] = a.w;
    }
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        float qv[NC];
#pragma unroll
        for (int u = 0; u < NC; u += 4) {
            const float4 a = *reinterpret_cast<const float4 *>(qrow[s] + c0 + u);
            qv[u] = a.x; qv[u + 1] = a.y; qv[u + 2] = a.z; qv[u + 3] = a.w;
        }
        uint64_t w[4] = {(uint64_t)(uint32_t)j[s], (uint64_t)key, bh, (uint64_t)(c0 / 12)};
        philox4x64_10(w, seed, 0);
        y[s] = sr8_steps(qv, kv, w, y[s], amax[s], std::make_integer_sequence<int, NC>{});
    }
}

// 8-bit logits with stochastic rounding for 16 keys and QPL query rows per
// lane: the key rows k32 + kk*D (fp32, kk = 0..15, the same for every lane),
// the query rows qrow[s] (fp32, pre-scaled) of query index j[s]; key index
// i0 + kk; bh = b*Hq + h.  Codes out as in emu8_chunk: acc[s][p] holds the
// e4m3 codes of keys 2p (bits 7:0) and 2p+1 (bits 15:8); sat[s] bit kk is
// set when a step of key kk's chain was clamped (|t| > 448).
template <int D, int QPL>
__device__ __forceinline__ void sr8_chunk(const float *const (&qrow)[QPL], const float *k32, uint64_t seed,
                                          uint64_t bh, const int (&j)[QPL], int i0, uint32_t (&acc)[QPL][8],
                                          uint32_t (&sat)[QPL])
{
    static_assert(D % 4 == 0, "channel groups of 4");
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        sat[s] = 0u;
#pragma unroll
        for (int p = 0; p < 8; ++p) acc[s][p] = 0u;
    }
    for (int kk = 0; kk < 16; ++kk) {
        const float *krow = k32 + (size_t)kk * D;
        const uint32_t key = (uint32_t)(i0 + kk);
        float y[QPL];
        uint32_t amax[QPL];
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            y[s] = 0.0f;
            amax[s] = 0u;
        }
        for (int g = 0; g < D / 12; ++g) sr8_group<12, QPL>(qrow, krow, 12 * g, seed, bh, j, key, y, amax);
        if constexpr (D % 12 != 0) sr8_group<D % 12, QPL>(qrow, krow, D / 12 * 12, seed, bh, j, key, y, amax);
        // the code of key kk into its byte (exact: y is an e4m3 value)
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            const uint32_t code = pk_e4m3_sat(y[s], 0.0f) & 0xFFu;
#pragma unroll
            for (int p = 0; p < 8; ++p) acc[s][p] |= (p == (kk >> 1)) ? code << (8 * (kk & 1)) : 0u;
            sat[s] |= (amax[s] > 0x43E00000u ? 1u : 0u) << kk;
        }
    }
}

} // namespace lamp
