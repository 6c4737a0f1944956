// lamp_sr.h -- stochastic rounding of the 8-bit logit accumulation.
//
// Sec. 3.3 ("Floating-point formats") names stochastic rounding (Croci et al.
// 2022) as the alternative to round-to-nearest for the e4m3 accumulation, to
// counter swamping.  The paper fixes neither the generator nor the number of
// random bits; the library's reading:
//   - each step rounds the FP32 FMA result t to one of its two e4m3
//     neighbours: a = min(|t|, 448), lo the e4m3 number next to a toward zero,
//     u its spacing; the step goes to lo + u when floor(2^16 (a - lo) / u) +
//     r >= 2^16 and to lo otherwise, with the sign of t; r is a uniform
//     16-bit integer;
//   - r comes from the counter-based generator Philox4x32-10 (Salmon, Moraes,
//     Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011)
//     under key (seed mod 2^32, seed / 2^32) at counter (j, i, b*Hq + h,
//     c / 8) for query row j, key i, query head h of batch b and channel c;
//     each of the four 32-bit outputs holds two 16-bit fields, channel c
//     taking the low half (c even) or the high half (c odd) of output
//     (c mod 8) / 2, so one call serves eight channels.
// The random numbers depend on the logit and the channel only, so the 8-bit
// logits are the same under every blocking and in the logits entry point.
//
// The rounding itself is gfx950's stochastic fp32 -> fp8 conversion
// (v_cvt_sr_fp8_f32) on the value clamped to +-448: it adds the top 20 bits
// of its 32-bit random operand to the 20 bits of the FP32 significand below
// e4m3's last bit (below 2^-6: to the bits below the 2^-9 quantum) and
// truncates, which with the operand r << 16 is the rounding above (the low 4
// of those 20 random bits are zero, so they never carry); the library's tests
// check it against the oracle's rounding.
#pragma once
#include <stdint.h>
#include <utility>

#include "lamp_device.h"
#include "lamp_loops.h"

namespace lamp {

// Philox4x32-10: ten rounds of the 4x32 round function; the key is bumped by
// the Weyl constants before every round after the first.
__device__ __forceinline__ void philox4x32_10(uint32_t (&c)[4], uint32_t k0, uint32_t k1)
{
    constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        const uint64_t p0 = (uint64_t)M0 * c[0], p1 = (uint64_t)M1 * c[2];
        // three-input exclusive or in one VALU instruction (bitop3 truth table 0x96)
        const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c[1], k0, 0x96);
        const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c[3], k1, 0x96);
        c[1] = (uint32_t)p1;
        c[3] = (uint32_t)p0;
        c[0] = n0;
        c[2] = n2;
    }
}

// The random operand of channel u (0..7) of a group: its 16-bit field in the
// top half of a word.
template <int U>
__device__ __forceinline__ uint32_t sr_operand(const uint32_t (&w)[4])
{
    return (U & 1) ? (w[U / 2] & 0xFFFF0000u) : (w[U / 2] << 16);
}

// One stochastically rounded step value (fp32, an e4m3 number); amax keeps
// the largest |t| pattern seen, so that a chain whose steps were clamped
// (|t| > 448) can be counted.
__device__ __forceinline__ float sr_e4m3(float t, uint32_t rop, uint32_t &amax)
{
    const uint32_t a = __builtin_bit_cast(uint32_t, t) & 0x7FFFFFFFu;
    amax = amax > a ? amax : a;
    const float tc = __builtin_amdgcn_fmed3f(t, -448.0f, 448.0f);
    return __builtin_amdgcn_cvt_f32_fp8(__builtin_amdgcn_cvt_sr_fp8_f32(tc, (int)rop, 0, 0), 0);
}

// The steps of one row over the channels U... of a group, in order.
template <int NC, int... U>
__device__ __forceinline__ float sr8_steps(const float (&qv)[NC], const float (&kv)[NC], const uint32_t (&w)[4],
                                           float v, uint32_t &amax, std::integer_sequence<int, U...>)
{
    ((v = sr_e4m3(__builtin_fmaf(qv[U], kv[U], v), sr_operand<U>(w), amax)), ...);
    return v;
}

// 8 channels from c0 of one key and QPL rows: the group's Philox call, then
// the 8 steps of each row's recursion.
template <int QPL>
__device__ __forceinline__ void sr8_group(const float *const (&qrow)[QPL], const float *krow, int c0, uint64_t seed,
                                          uint32_t bh, const int (&j)[QPL], uint32_t key, float (&y)[QPL],
                                          uint32_t (&amax)[QPL])
{
    float kv[8];
#pragma unroll
    for (int u = 0; u < 8; u += 4) {
        const float4 a = *reinterpret_cast<const float4 *>(krow + c0 + u);
        kv[u] = a.x; kv[u + 1] = a.y; kv[u + 2] = a.z; kv[u + 3] = a.w;
    }
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        float qv[8];
#pragma unroll
        for (int u = 0; u < 8; u += 4) {
            const float4 a = *reinterpret_cast<const float4 *>(qrow[s] + c0 + u);
            qv[u] = a.x; qv[u + 1] = a.y; qv[u + 2] = a.z; qv[u + 3] = a.w;
        }
        uint32_t w[4] = {(uint32_t)j[s], key, bh, (uint32_t)(c0 / 8)};
        philox4x32_10(w, (uint32_t)seed, (uint32_t)(seed >> 32));
        y[s] = sr8_steps(qv, kv, w, y[s], amax[s], std::make_integer_sequence<int, 8>{});
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
    static_assert(D % 8 == 0, "channel groups of 8");
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
        for (int g = 0; g < D / 8; ++g) sr8_group<QPL>(qrow, krow, 8 * g, seed, (uint32_t)bh, j, key, y, amax);
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

// ---- the pipelined kernel's form: keys by DPP row broadcast --------------
// Channels cb .. cb+7 of the two chains of keys 2P, 2P+1 of each of QPL query
// rows, whose codes share word acc[s][P] (bits 7:0, 15:8): one Philox call per
// chain, then 8 steps of both, each decoding the pair, running both FP32 FMAs
// (the keys by row broadcast) and rounding each value stochastically into its
// byte.  Without CLAMP a |t| above 448 gives a NaN code, which the NaN carries
// to the end of the chain (the caller then re-runs with CLAMP, which is the
// saturating recursion: the two agree up to that step).
template <int P, int QPL, bool CLAMP>
__device__ __forceinline__ void sr8_pair8(const float4 &k0, const float4 &k1, const float4 (&q0)[QPL],
                                          const float4 (&q1)[QPL], const int (&j)[QPL], uint32_t key0,
                                          uint32_t bh, uint32_t g, uint32_t s0, uint32_t s1, uint32_t (&acc)[QPL][8])
{
    const float kv[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        // the query index through an empty statement the compiler cannot move:
        // the generator's rounds stay here, next to their use, instead of being
        // hoisted for every pair and block at once (which exhausts the registers)
        uint32_t js = (uint32_t)j[s];
        asm volatile("" : "+v"(js));
        uint32_t wa[4] = {js, key0 + 2 * P, bh, g};
        uint32_t wb[4] = {js, key0 + 2 * P + 1, bh, g};
        philox4x32_10(wa, s0, s1);
        philox4x32_10(wb, s0, s1);
        const float qv[8] = {q0[s].x, q0[s].y, q0[s].z, q0[s].w, q1[s].x, q1[s].y, q1[s].z, q1[s].w};
        uint32_t word = acc[s][P];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const uint32_t ra = (c & 1) ? (wa[c / 2] & 0xFFFF0000u) : (wa[c / 2] << 16);
            const uint32_t rb = (c & 1) ? (wb[c / 2] & 0xFFFF0000u) : (wb[c / 2] << 16);
            const float2 f = unpk_e4m3(word);
            float ta = fmac_bc<2 * P>(f.x, kv[c], qv[c]);
            float tb = fmac_bc<2 * P + 1>(f.y, kv[c], qv[c]);
            if (CLAMP) {
                ta = __builtin_amdgcn_fmed3f(ta, -448.0f, 448.0f);
                tb = __builtin_amdgcn_fmed3f(tb, -448.0f, 448.0f);
            }
            word = (uint32_t)__builtin_amdgcn_cvt_sr_fp8_f32(ta, (int)ra, (int)word, 0);
            word = (uint32_t)__builtin_amdgcn_cvt_sr_fp8_f32(tb, (int)rb, (int)word, 1);
        }
        acc[s][P] = word;
    }
}

// Y8 with stochastic rounding of one 16-key chunk for QPL query rows of this
// lane, keys read by row broadcast as in emu8_pass (k32 at the chunk's first
// key, layout LY; qrow[s] at the pre-scaled query row of query index j[s];
// key index key0 + i; bh = b*Hq + h).  The loop runs 8 channels of every
// chain at a time, so that each Philox call feeds its 8 steps at once, one key
// pair after the other (a loop, not unrolled, over a switch on the pair: the
// broadcast lane is an immediate, and one pair's chains at a time keep the
// registers of the surrounding kernel free); the loads run 8 channels ahead in
// two buffers written only by loads.  acc[s][p] receives the codes of keys
// 2p (bits 7:0) and 2p+1 (bits 15:8).
template <int D, int QPL, bool CLAMP, class LY, class QP>
__device__ __forceinline__ void sr8_pass(const QP (&qrow)[QPL], const float *k32, const int (&j)[QPL], uint32_t key0,
                                         uint32_t bh, uint64_t seed, uint32_t (&acc)[QPL][8])
{
    static_assert(D % 16 == 0, "pairs of 8-channel blocks");
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int p = 0; p < 8; ++p) acc[s][p] = 0u;
    const uint32_t s0 = (uint32_t)seed, s1 = (uint32_t)(seed >> 32);
    const float *krow = k32 + (size_t)(__lane_id() & 15) * LY::KR;
    float4 ka0, ka1, kb0, kb1, qa0[QPL], qa1[QPL], qb0[QPL], qb1[QPL];
    auto ld = [&](int c, float4 &k0, float4 &k1, float4 (&q0)[QPL], float4 (&q1)[QPL]) {
        k0 = load4(krow + (c / 4) * LY::KS);
        k1 = load4(krow + (c / 4 + 1) * LY::KS);
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            q0[s] = load4(qrow[s] + (c / 4) * LY::QS);
            q1[s] = load4(qrow[s] + (c / 4 + 1) * LY::QS);
        }
    };
    auto run = [&](int c, const float4 &k0, const float4 &k1, const float4 (&q0)[QPL], const float4 (&q1)[QPL]) {
        const uint32_t g = (uint32_t)(c / 8);
#pragma nounroll
        for (int p = 0; p < 8; ++p) {
            switch (p) {
            case 0: sr8_pair8<0, QPL, CLAMP>(k0, k1, q0, q1, j, key0, bh, g, s0, s1, acc); break;
            case 1: sr8_pair8<1, QPL, CLAMP>(k0, k1, q0, q1, j, key0, bh, g, s0, s1, acc); break;
            case 2: sr8_pair8<2, QPL, CLAMP>(k0, k1, q0, q1, j, key0, bh, g, s0, s1, acc); break;
            case 3: sr8_pair8<3, QPL, CLAMP>(k0, k1, q0, q1, j, key0, bh, g, s0, s1, acc); break;
            case 4: sr8_pair8<4, QPL, CLAMP>(k0, k1, q0, q1, j, key0, bh, g, s0, s1, acc); break;
            case 5: sr8_pair8<5, QPL, CLAMP>(k0, k1, q0, q1, j, key0, bh, g, s0, s1, acc); break;
            case 6: sr8_pair8<6, QPL, CLAMP>(k0, k1, q0, q1, j, key0, bh, g, s0, s1, acc); break;
            default: sr8_pair8<7, QPL, CLAMP>(k0, k1, q0, q1, j, key0, bh, g, s0, s1, acc); break;
            }
        }
    };
    ld(0, ka0, ka1, qa0, qa1);
    for (int c = 0; c < D - 16; c += 16) {
        dpp_guard_fenced();
        ld(c + 8, kb0, kb1, qb0, qb1);
        run(c, ka0, ka1, qa0, qa1);
        ld(c + 16, ka0, ka1, qa0, qa1);
        run(c + 8, kb0, kb1, qb0, qb1);
    }
    ld(D - 8, kb0, kb1, qb0, qb1);
    dpp_guard_fenced();
    run(D - 16, ka0, ka1, qa0, qa1);
    run(D - 8, kb0, kb1, qb0, qb1);
}

// sr8_pass without saturation first; if any lane of the wave overflowed (a
// NaN code at the end of a chain), the chunk again with the clamp.  sat[s]
// receives the keys of slot s whose accumulation saturated (as emu8_chunk).
template <int D, int QPL, class LY, class QP>
__device__ __forceinline__ void sr8_chunk_bc(const QP (&qrow)[QPL], const float *k32, const int (&j)[QPL],
                                             uint32_t key0, uint32_t bh, uint64_t seed, uint32_t (&acc)[QPL][8],
                                             uint32_t (&sat)[QPL])
{
    sr8_pass<D, QPL, false, LY>(qrow, k32, j, key0, bh, seed, acc);
    uint32_t nan = 0;
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        sat[s] = 0u;
#pragma unroll
        for (int p = 0; p < 8; ++p) nan |= e4m3_nan_bits(acc[s][p]);
    }
    if (wave_any(nan != 0)) {
        nan_keys<QPL>(acc, sat);
        sr8_pass<D, QPL, true, LY>(qrow, k32, j, key0, bh, seed, acc);
    }
}

} // namespace lamp
