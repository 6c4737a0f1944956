// lamp_loops.h -- the two logit loops of the LampAttention forward pass.
//
// Both loops give each lane QPL query rows and accumulate over the D channels
// of a group of NKEY <= 16 keys.  Lane l of every 16-lane row of the wave
// holds the key value of key (l mod NKEY) for the current channel; the FMA
// reads it through a DPP row broadcast (row_newbcast:i hands lane i of each
// row to all 16 lanes of that row), so every lane multiplies its own query
// value by the value of key i without scalar registers or LDS.  Keys and
// queries are fp32 and arrive with ordinary vector loads one 4-channel group
// ahead of their use.  A DPP read of a VGPR written by a VALU instruction less
// than two instructions earlier is a hardware hazard; the key registers are
// only written by loads, and the build scans the generated code for the
// pattern (see build.py).
#pragma once
#include <utility>

#include "lamp_device.h"

namespace lamp {

// acc + bcast_i(kv) * q with one rounding (v_fmac_f32 is a fused multiply-add).
template <int I>
__device__ __forceinline__ float fmac_bc(float acc, float kv, float q)
{
    asm("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf" : "+v"(acc) : "v"(kv), "v"(q), "n"(I));
    return acc;
}

// Two code words of two accumulators each advanced by one channel in a single
// statement: word a holds the codes of keys I0, I1 of query value qa, word b
// those of keys J0, J1 of qb; each pair is decoded, the FMAs read the keys by
// row broadcast, and the results are rounded to e4m3 into bits [15:0] of the
// word (bits [31:16] kept; no saturation, see pk_e4m3).  The decoded values go
// to four fixed registers that the statement declares clobbered, so the two
// chains interleave with no wait state between the statements of one chain
// that the compiler, not seeing into the assembly, would otherwise insert
// after every separate asm statement.
template <int I0, int I1, int J0, int J1>
__device__ __forceinline__ void emu8_words(uint32_t &a, uint32_t &b, float kv, float qa, float qb)
{
    asm("v_cvt_pk_f32_fp8 v[248:249], %0\n\t"
        "v_cvt_pk_f32_fp8 v[250:251], %1\n\t"
        "v_fmac_f32_dpp v248, %2, %3 row_newbcast:%5 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp v249, %2, %3 row_newbcast:%6 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp v250, %2, %4 row_newbcast:%7 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp v251, %2, %4 row_newbcast:%8 row_mask:0xf bank_mask:0xf\n\t"
        "v_cvt_pk_fp8_f32 %0, v248, v249\n\t"
        "v_cvt_pk_fp8_f32 %1, v250, v251"
        : "+v"(a), "+v"(b)
        : "v"(kv), "v"(qa), "v"(qb), "n"(I0), "n"(I1), "n"(J0), "n"(J1)
        : "v248", "v249", "v250", "v251");
}

// One channel of all eight code words of both query rows (16 keys) in a
// single statement: the body of emu8_words for word pairs 0..7.  One
// statement per channel keeps the compiler from placing a wait state between
// the word pairs, which it does after every separate statement.
#define LAMP_E8W(A, B, K0, K1)                                                          \
    "v_cvt_pk_f32_fp8 v[248:249], " A "\n\t"                                           \
    "v_cvt_pk_f32_fp8 v[250:251], " B "\n\t"                                           \
    "v_fmac_f32_dpp v248, %16, %17 row_newbcast:" #K0 " row_mask:0xf bank_mask:0xf\n\t" \
    "v_fmac_f32_dpp v249, %16, %17 row_newbcast:" #K1 " row_mask:0xf bank_mask:0xf\n\t" \
    "v_fmac_f32_dpp v250, %16, %18 row_newbcast:" #K0 " row_mask:0xf bank_mask:0xf\n\t" \
    "v_fmac_f32_dpp v251, %16, %18 row_newbcast:" #K1 " row_mask:0xf bank_mask:0xf\n\t" \
    "v_cvt_pk_fp8_f32 " A ", v248, v249\n\t"                                            \
    "v_cvt_pk_fp8_f32 " B ", v250, v251\n\t"

__device__ __forceinline__ void emu8_words8(uint32_t (&a)[8], uint32_t (&b)[8], float kv, float qa, float qb)
{
    asm(LAMP_E8W("%0", "%8", 0, 1) LAMP_E8W("%1", "%9", 2, 3) LAMP_E8W("%2", "%10", 4, 5)
        LAMP_E8W("%3", "%11", 6, 7) LAMP_E8W("%4", "%12", 8, 9) LAMP_E8W("%5", "%13", 10, 11)
        LAMP_E8W("%6", "%14", 12, 13) LAMP_E8W("%7", "%15", 14, 15)
        : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(a[4]), "+v"(a[5]), "+v"(a[6]), "+v"(a[7]),
          "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]), "+v"(b[4]), "+v"(b[5]), "+v"(b[6]), "+v"(b[7])
        : "v"(kv), "v"(qa), "v"(qb)
        : "v248", "v249", "v250", "v251");
}
#undef LAMP_E8W

// The compact register layout (Sec. 3.3, "Register layout": four 8-bit
// accumulators per 32-bit register): one channel of both query rows' 16
// codes held four per word -- keys 4w, 4w+1 in bits [15:0] of word w, keys
// 4w+2, 4w+3 in bits [31:16] -- in a single statement.  The high halves are
// decoded with an SDWA word select and written back with op_sel, so the
// instructions are those of emu8_words8.
#define LAMP_E8H(A, B, K0, K1, K2, K3)                                                  \
    "v_cvt_pk_f32_fp8 v[248:249], " A "\n\t"                                           \
    "v_cvt_pk_f32_fp8 v[250:251], " B "\n\t"                                           \
    "v_fmac_f32_dpp v248, %8, %9 row_newbcast:" #K0 " row_mask:0xf bank_mask:0xf\n\t"   \
    "v_fmac_f32_dpp v249, %8, %9 row_newbcast:" #K1 " row_mask:0xf bank_mask:0xf\n\t"   \
    "v_fmac_f32_dpp v250, %8, %10 row_newbcast:" #K0 " row_mask:0xf bank_mask:0xf\n\t"  \
    "v_fmac_f32_dpp v251, %8, %10 row_newbcast:" #K1 " row_mask:0xf bank_mask:0xf\n\t"  \
    "v_cvt_pk_fp8_f32 " A ", v248, v249\n\t"                                            \
    "v_cvt_pk_fp8_f32 " B ", v250, v251\n\t"                                            \
    "v_cvt_pk_f32_fp8_sdwa v[248:249], " A " src0_sel:WORD_1\n\t"                       \
    "v_cvt_pk_f32_fp8_sdwa v[250:251], " B " src0_sel:WORD_1\n\t"                       \
    "v_fmac_f32_dpp v248, %8, %9 row_newbcast:" #K2 " row_mask:0xf bank_mask:0xf\n\t"   \
    "v_fmac_f32_dpp v249, %8, %9 row_newbcast:" #K3 " row_mask:0xf bank_mask:0xf\n\t"   \
    "v_fmac_f32_dpp v250, %8, %10 row_newbcast:" #K2 " row_mask:0xf bank_mask:0xf\n\t"  \
    "v_fmac_f32_dpp v251, %8, %10 row_newbcast:" #K3 " row_mask:0xf bank_mask:0xf\n\t"  \
    "v_cvt_pk_fp8_f32 " A ", v248, v249 op_sel:[0,0,1]\n\t"                             \
    "v_cvt_pk_fp8_f32 " B ", v250, v251 op_sel:[0,0,1]\n\t"

__device__ __forceinline__ void emu8_quads4(uint32_t (&a)[4], uint32_t (&b)[4], float kv, float qa, float qb)
{
    asm(LAMP_E8H("%0", "%4", 0, 1, 2, 3) LAMP_E8H("%1", "%5", 4, 5, 6, 7) LAMP_E8H("%2", "%6", 8, 9, 10, 11)
        LAMP_E8H("%3", "%7", 12, 13, 14, 15)
        : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3])
        : "v"(kv), "v"(qa), "v"(qb)
        : "v248", "v249", "v250", "v251");
}
#undef LAMP_E8H

// One channel of the 16-bit accumulation of one query row for NKEY keys in
// a single statement: acc[i] += bcast_i(kv) * q, i = 0..NKEY-1.
#define LAMP_F16(I, ACC) "v_fmac_f32_dpp " ACC ", %[k], %[q] row_newbcast:" #I " row_mask:0xf bank_mask:0xf\n\t"
template <int NKEY>
__device__ __forceinline__ void fmac16_row(float (&acc)[NKEY], float kv, float q)
{
    static_assert(NKEY == 4 || NKEY == 8 || NKEY == 12 || NKEY == 16, "4, 8, 12 or 16 keys");
    if constexpr (NKEY == 4) {
        asm(LAMP_F16(0, "%0") LAMP_F16(1, "%1") LAMP_F16(2, "%2") LAMP_F16(3, "%3")
            : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3])
            : [k] "v"(kv), [q] "v"(q));
    } else if constexpr (NKEY == 8) {
        asm(LAMP_F16(0, "%0") LAMP_F16(1, "%1") LAMP_F16(2, "%2") LAMP_F16(3, "%3")
            LAMP_F16(4, "%4") LAMP_F16(5, "%5") LAMP_F16(6, "%6") LAMP_F16(7, "%7")
            : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]), "+v"(acc[6]),
              "+v"(acc[7])
            : [k] "v"(kv), [q] "v"(q));
    } else if constexpr (NKEY == 12) {
        asm(LAMP_F16(0, "%0") LAMP_F16(1, "%1") LAMP_F16(2, "%2") LAMP_F16(3, "%3")
            LAMP_F16(4, "%4") LAMP_F16(5, "%5") LAMP_F16(6, "%6") LAMP_F16(7, "%7")
            LAMP_F16(8, "%8") LAMP_F16(9, "%9") LAMP_F16(10, "%10") LAMP_F16(11, "%11")
            : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]), "+v"(acc[6]),
              "+v"(acc[7]), "+v"(acc[8]), "+v"(acc[9]), "+v"(acc[10]), "+v"(acc[11])
            : [k] "v"(kv), [q] "v"(q));
    } else {
        asm(LAMP_F16(0, "%0") LAMP_F16(1, "%1") LAMP_F16(2, "%2") LAMP_F16(3, "%3")
            LAMP_F16(4, "%4") LAMP_F16(5, "%5") LAMP_F16(6, "%6") LAMP_F16(7, "%7")
            LAMP_F16(8, "%8") LAMP_F16(9, "%9") LAMP_F16(10, "%10") LAMP_F16(11, "%11")
            LAMP_F16(12, "%12") LAMP_F16(13, "%13") LAMP_F16(14, "%14") LAMP_F16(15, "%15")
            : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]), "+v"(acc[6]),
              "+v"(acc[7]), "+v"(acc[8]), "+v"(acc[9]), "+v"(acc[10]), "+v"(acc[11]), "+v"(acc[12]),
              "+v"(acc[13]), "+v"(acc[14]), "+v"(acc[15])
            : [k] "v"(kv), [q] "v"(q));
    }
}
#undef LAMP_F16

// Where the loops find the fp32 queries and keys.  Row layout ([row][D]): the
// 4-channel group g of a row is at offset 4g and consecutive keys are D apart.
// Grouped layout (the pipelined kernel): queries in blocks of 64 rows and keys
// in blocks of 16, each block stored [group][row][4], so that one 4-channel
// group of a block is contiguous: group g of a query row is at 256g, of a key
// row at 64g, and consecutive keys of a block are 4 apart.
// WORDS selects the two-word 8-bit statement (emu8_words) for two query rows
// per lane: its four fixed temporaries sit at the top of the register file,
// so it is only for kernels that use the whole file anyway (the pipelined
// kernel at 128 rows per block, two waves per SIMD).
template <int QS_, int KS_, int KR_, bool WORDS_>
struct Lay {
    static constexpr int QS = QS_, KS = KS_, KR = KR_;   // query / key group stride, key row stride
    static constexpr bool WORDS = WORDS_;
};
template <int D>
using RowLay = Lay<4, 4, D, false>;
using GrpLay = Lay<256, 64, 4, true>;

// Two wait states that nothing is scheduled across.  The register allocator
// may copy a loaded key register with a VALU move where a loop is entered or
// left (to line up the loop-carried buffers); placed at the top of every loop
// over channel groups and after it, this keeps each DPP read of a key at least
// two wait states behind such a copy.  The build check verifies the result.
__device__ __forceinline__ void dpp_guard()
{
    asm volatile("s_nop 1");
}

// dpp_guard with a scheduling barrier after it, for loops whose first
// broadcast FMAs the scheduler would otherwise hoist above the wait states
// (the FMAs are side-effect-free inline assembly and may move across them).
__device__ __forceinline__ void dpp_guard_fenced()
{
    asm volatile("s_nop 1");
    __builtin_amdgcn_sched_barrier(0);
}

// Query rows come either from global memory (const float *) or from LDS
// (lds_cfptr, so that the loads are ds_read_b128 rather than flat loads).
typedef const __attribute__((address_space(3))) float *lds_cfptr;

__device__ __forceinline__ float4 load4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
typedef float f32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 load4(lds_cfptr p)
{
    const f32x4_t v = *reinterpret_cast<const __attribute__((address_space(3))) f32x4_t *>(p);
    return make_float4(v.x, v.y, v.z, v.w);
}

// Loads of a 4-channel group: this lane's key row and query rows.
template <int QPL, class LY, class QP>
__device__ __forceinline__ void load_group(const float *krow, const QP (&qrow)[QPL], int c, float4 &k4,
                                           float4 (&q4)[QPL])
{
    k4 = *reinterpret_cast<const float4 *>(krow + (c / 4) * LY::KS);
#pragma unroll
    for (int s = 0; s < QPL; ++s) q4[s] = load4(qrow[s] + (c / 4) * LY::QS);
}

__device__ __forceinline__ float f4_at(const float4 &v, int i)
{
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// One channel of the 8-bit accumulation for key pair (2P, 2P+1) of every
// slot: acc <- RN_e4m3(RN32(q * k + acc)).
template <int QPL, bool SAT, int P>
__device__ __forceinline__ void emu8_pair(float kv, const float (&q)[QPL], uint32_t (&acc)[QPL][8])
{
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        const float2 a = unpk_e4m3(acc[s][P]);
        const float x = fmac_bc<2 * P>(a.x, kv, q[s]);
        const float y = fmac_bc<2 * P + 1>(a.y, kv, q[s]);
        acc[s][P] = SAT ? pk_e4m3_sat(x, y, acc[s][P]) : pk_e4m3(x, y, acc[s][P]);
    }
}

// One channel of the non-saturating pass over every word: with WORDS and two
// query rows per lane, the two rows of a word index in one statement
// (emu8_words); otherwise one pair at a time (emu8_pair).
template <int QPL, bool SAT, bool WORDS, int... P>
__device__ __forceinline__ void emu8_channel(float kv, const float (&q)[QPL], uint32_t (&acc)[QPL][8],
                                             std::integer_sequence<int, P...>)
{
    if constexpr (!SAT && WORDS && QPL == 2 && sizeof...(P) == 8)
        emu8_words8(acc[0], acc[1], kv, q[0], q[1]);
    else if constexpr (!SAT && WORDS && QPL == 2)
        (emu8_words<2 * P, 2 * P + 1, 2 * P, 2 * P + 1>(acc[0][P], acc[1][P], kv, q[0], q[1]), ...);
    else (emu8_pair<QPL, SAT, P>(kv, q, acc), ...);
}

// Y8 of one 16-key chunk for QPL query rows of this lane (Sec. 4.1:
// acc <- RN_e4m3(RN32(q_tilde * k + acc)), channels ascending, from +0).
// k32 points at the chunk's first key (layout LY); qrow[s] at the fp32
// pre-scaled query row of slot s.  acc[s][p] receives the codes of keys 2p,
// 2p+1 in bits [15:0].
template <int D, int QPL, bool SAT, class LY = RowLay<D>, class QP>
__device__ __forceinline__ void emu8_pass(const QP (&qrow)[QPL], const float *k32, uint32_t (&acc)[QPL][8])
{
    static_assert(D % 8 == 0, "channels in pairs of 4-channel groups");
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int p = 0; p < 8; ++p) acc[s][p] = 0u;
    const float *krow = k32 + (size_t)(__lane_id() & 15) * LY::KR;
    // Two alternating load buffers: the key registers feeding the DPP
    // broadcast are only ever written by vector loads, never copied.
    float4 ka, kb, qa[QPL], qb[QPL];
    auto run = [&](const float4 &k4, const float4 (&q4)[QPL]) {
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            float q[QPL];
#pragma unroll
            for (int s = 0; s < QPL; ++s) q[s] = f4_at(q4[s], cc);
            emu8_channel<QPL, SAT, LY::WORDS>(f4_at(k4, cc), q, acc, std::make_integer_sequence<int, 8>());
        }
    };
    // steady state, then the last pair of groups without further loads (the
    // offsets stay affine in c, so they fold into the loads' immediates)
    load_group<QPL, LY>(krow, qrow, 0, ka, qa);
    for (int c = 0; c < D - 8; c += 8) {
        dpp_guard();
        load_group<QPL, LY>(krow, qrow, c + 4, kb, qb);
        run(ka, qa);
        load_group<QPL, LY>(krow, qrow, c + 8, ka, qa);
        run(kb, qb);
    }
    load_group<QPL, LY>(krow, qrow, D - 4, kb, qb);
    dpp_guard();
    run(ka, qa);
    run(kb, qb);
}

// Keys whose 8-bit code is a NaN after the non-saturating pass, one bit per
// key (bit i: key i of the 16, codes of keys 2p and 2p+1 in word p).  Such a
// chain overflowed in some step, which is exactly when the saturating
// recursion clamps to +-448: the two recursions agree up to that step.
template <int QPL>
__device__ __forceinline__ void nan_keys(const uint32_t (&acc)[QPL][8], uint32_t (&sat)[QPL])
{
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        uint32_t m = 0;
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            const uint32_t r = e4m3_nan_bits(acc[s][p]);
            m |= ((r >> 7) & 1u) << (2 * p);
            m |= ((r >> 15) & 1u) << (2 * p + 1);
        }
        sat[s] = m;
    }
}

// The fast pass uses the non-saturating conversion; if any lane of the wave
// overflowed somewhere (a NaN code at the end of a chain), the chunk is
// recomputed with the saturating conversion.  sat[s] receives the keys of
// slot s whose accumulation saturated (nan_keys), 0 when none did.
template <int D, int QPL, class LY = RowLay<D>, class QP>
__device__ __forceinline__ void emu8_chunk(const QP (&qrow)[QPL], const float *k32, uint32_t (&acc)[QPL][8],
                                           uint32_t (&sat)[QPL])
{
    emu8_pass<D, QPL, false, LY>(qrow, k32, acc);
    uint32_t nan = 0;
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        sat[s] = 0u;
#pragma unroll
        for (int p = 0; p < 8; ++p) nan |= e4m3_nan_bits(acc[s][p]);
    }
    if (wave_any(nan != 0)) {
        nan_keys<QPL>(acc, sat);
        emu8_pass<D, QPL, true, LY>(qrow, k32, acc);
    }
}

template <int D, int QPL, class LY = RowLay<D>, class QP>
__device__ __forceinline__ void emu8_chunk(const QP (&qrow)[QPL], const float *k32, uint32_t (&acc)[QPL][8])
{
    uint32_t sat[QPL];
    emu8_chunk<D, QPL, LY>(qrow, k32, acc, sat);
}

// One channel of the 16-bit accumulation for every key and slot.
template <int QPL, int NKEY, int... I>
__device__ __forceinline__ void rec16_channel(float kv, const float (&q)[QPL], float (&acc)[QPL][NKEY],
                                              std::integer_sequence<int, I...>);

// ---- the SIM profile (Sec. 4.1): FP32 range, 3 / 11 mantissa bits, no saturation
// Words of 16-bit logits for NKEY keys: e4m11 codes two per word, or, in the
// SIM profile, FP32 patterns one per word.
template <bool SIMP>
constexpr int y16_words(int nkey)
{
    return nkey == 0 ? 1 : (SIMP ? nkey : nkey / 2);
}

// Value of the i-th 16-bit logit of a word array.
template <bool SIMP>
__device__ __forceinline__ float y16_value(const uint32_t *w, int i)
{
    if constexpr (SIMP) return __builtin_bit_cast(float, w[i]);
    else return e4m11_value((w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
}

// Two SIM 8-bit logits as their bf16 patterns (exact: 3 mantissa bits).
__device__ __forceinline__ uint32_t pack_sim8(float a, float b)
{
    return (__builtin_bit_cast(uint32_t, a) >> 16) | (__builtin_bit_cast(uint32_t, b) & 0xFFFF0000u);
}

// One channel of the SIM 8-bit accumulation for every key and slot:
// acc <- RN_3(RN32(q * k + acc)).
template <int QPL, int... I>
__device__ __forceinline__ void emu8s_channel(float kv, const float (&q)[QPL], float (&acc)[QPL][16],
                                              std::integer_sequence<int, I...>)
{
#pragma unroll
    for (int s = 0; s < QPL; ++s) ((acc[s][I] = rn_sim<3>(fmac_bc<I>(acc[s][I], kv, q[s]))), ...);
}

// Y8 of one 16-key chunk in the SIM profile (as emu8_pass); codes[s][p]
// receives the bf16 patterns of keys 2p (bits [15:0]) and 2p+1.
template <int D, int QPL, class LY = RowLay<D>, class QP>
__device__ __forceinline__ void emu8s_pass(const QP (&qrow)[QPL], const float *k32, uint32_t (&codes)[QPL][8])
{
    static_assert(D % 8 == 0, "channels in pairs of 4-channel groups");
    float acc[QPL][16];
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[s][i] = 0.0f;
    const float *krow = k32 + (size_t)(__lane_id() & 15) * LY::KR;
    float4 ka, kb, qa[QPL], qb[QPL];
    auto run = [&](const float4 &k4, const float4 (&q4)[QPL]) {
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            float q[QPL];
#pragma unroll
            for (int s = 0; s < QPL; ++s) q[s] = f4_at(q4[s], cc);
            emu8s_channel<QPL>(f4_at(k4, cc), q, acc, std::make_integer_sequence<int, 16>());
        }
    };
    load_group<QPL, LY>(krow, qrow, 0, ka, qa);
    for (int c = 0; c < D - 8; c += 8) {
        dpp_guard_fenced();
        load_group<QPL, LY>(krow, qrow, c + 4, kb, qb);
        run(ka, qa);
        load_group<QPL, LY>(krow, qrow, c + 8, ka, qa);
        run(kb, qb);
    }
    load_group<QPL, LY>(krow, qrow, D - 4, kb, qb);
    dpp_guard_fenced();
    run(ka, qa);
    run(kb, qb);
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int p = 0; p < 8; ++p) codes[s][p] = pack_sim8(acc[s][2 * p], acc[s][2 * p + 1]);
}

// Y8 of a 16-key chunk in either profile (sat as in emu8_chunk; 0 in the
// SIM profile, which does not saturate).
template <int D, int QPL, bool SIMP, class LY = RowLay<D>, class QP>
__device__ __forceinline__ void emu8_any(const QP (&qrow)[QPL], const float *k32, uint32_t (&codes)[QPL][8],
                                         uint32_t (&sat)[QPL])
{
    if constexpr (SIMP) {
        emu8s_pass<D, QPL, LY>(qrow, k32, codes);
#pragma unroll
        for (int s = 0; s < QPL; ++s) sat[s] = 0u;
    } else {
        emu8_chunk<D, QPL, LY>(qrow, k32, codes, sat);
    }
}

// The 16-bit logits of the FP32 chains in acc, encoded: rounded once to e4m11
// (codes, two per word) or, in the SIM profile, to 11 mantissa bits (FP32
// patterns, one per word).
template <bool SIMP, int QPL, int NKEY>
__device__ __forceinline__ void encode16(const float (&acc)[QPL][NKEY], uint32_t (&c)[QPL][y16_words<SIMP>(NKEY)])
{
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        if constexpr (SIMP) {
#pragma unroll
            for (int i = 0; i < NKEY; ++i) c[s][i] = __builtin_bit_cast(uint32_t, rn_sim<11>(acc[s][i]));
        } else {
#pragma unroll
            for (int p = 0; p < NKEY / 2; ++p) {
                uint32_t x0, x1;
                (void)rn_e4m11_f32(acc[s][2 * p], &x0);
                (void)rn_e4m11_f32(acc[s][2 * p + 1], &x1);
                c[s][p] = x0 | (x1 << 16);
            }
        }
    }
}

// Two passes over the channels fused into one loop that shares the query
// loads: the 8-bit accumulation of the 16 keys at k32e (EMU; as emu8_pass,
// without saturation, then checked as in emu8_chunk) and the 16-bit
// accumulation of NKEY keys, this lane's key row being krowr (as rec16_keys).
// The forward kernel uses it to run the 8-bit logits of the next key tile
// together with the speculative 16-bit recompute of the current one.
// sat receives the saturated keys of the 8-bit chunk as in emu8_chunk.
// CMP: the 8-bit codes live four per register during the pass (emu8_quads4;
// two query rows per lane, the grouped layout); a8 receives them two per word
// as always.
template <int D, int QPL, int NKEY, bool EMU, bool SIMP, class LY = RowLay<D>, bool CMP = false, class QP>
__device__ __forceinline__ void fused_pass(const QP (&qrow)[QPL], const float *k32e, const float *krowr,
                                           uint32_t (&a8)[QPL][8], uint32_t (&c16)[QPL][y16_words<SIMP>(NKEY)],
                                           uint32_t (&sat)[QPL])
{
    static_assert(!CMP || (QPL == 2 && !SIMP && LY::WORDS), "compact words: two rows per lane, hardware formats");
    constexpr bool QUADS = CMP && EMU;
    uint32_t a8q[QPL][4];   // the compact words (QUADS)
    static_assert(EMU || NKEY > 0, "something to compute");
    static_assert(NKEY == 0 || NKEY == 4 || NKEY == 8 || NKEY == 12 || NKEY == 16, "0, 4, 8, 12 or 16 keys");
    static_assert(D % 8 == 0, "channels in pairs of 4-channel groups");
    constexpr int NA = NKEY > 0 ? NKEY : 1;
    constexpr int NE = (SIMP && EMU) ? 16 : 1;   // SIM 8-bit accumulators (values, not codes)
    float acc[QPL][NA], e8[QPL][NE];
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        sat[s] = 0u;
#pragma unroll
        for (int p = 0; p < 8; ++p) a8[s][p] = 0u;
#pragma unroll
        for (int p = 0; p < 4; ++p) a8q[s][p] = 0u;
#pragma unroll
        for (int i = 0; i < NA; ++i) acc[s][i] = 0.0f;
#pragma unroll
        for (int i = 0; i < NE; ++i) e8[s][i] = 0.0f;
    }
    const float *krowe = k32e + (size_t)(__lane_id() & 15) * LY::KR;
    // the SIM profile's loop needs the fenced guard (its schedule hoists
    // broadcast FMAs above a plain one)
    auto guard = [] {
        if constexpr (SIMP) dpp_guard_fenced();
        else dpp_guard();
    };
    float4 kea, keb, kra, krb, qa[QPL], qb[QPL];
    auto ld = [&](int c, float4 &ke, float4 &kr, float4 (&q4)[QPL]) {
        if constexpr (EMU) ke = load4(krowe + (c / 4) * LY::KS);
        if constexpr (NKEY > 0) kr = load4(krowr + (c / 4) * LY::KS);
#pragma unroll
        for (int s = 0; s < QPL; ++s) q4[s] = load4(qrow[s] + (c / 4) * LY::QS);
    };
    auto run = [&](const float4 &ke, const float4 &kr, const float4 (&q4)[QPL]) {
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            float q[QPL];
#pragma unroll
            for (int s = 0; s < QPL; ++s) q[s] = f4_at(q4[s], cc);
            if constexpr (EMU && SIMP)
                emu8s_channel<QPL>(f4_at(ke, cc), q, e8, std::make_integer_sequence<int, 16>());
            else if constexpr (QUADS)
                emu8_quads4(a8q[0], a8q[QPL - 1], f4_at(ke, cc), q[0], q[QPL - 1]);
            else if constexpr (EMU)
                emu8_channel<QPL, false, LY::WORDS>(f4_at(ke, cc), q, a8, std::make_integer_sequence<int, 8>());
            if constexpr (NKEY > 0)
                rec16_channel<QPL, NKEY>(f4_at(kr, cc), q, acc, std::make_integer_sequence<int, NKEY>());
        }
    };
    ld(0, kea, kra, qa);
    for (int c = 0; c < D - 8; c += 8) {
        guard();
        ld(c + 4, keb, krb, qb);
        run(kea, kra, qa);
        ld(c + 8, kea, kra, qa);
        run(keb, krb, qb);
    }
    ld(D - 4, keb, krb, qb);
    guard();
    run(kea, kra, qa);
    run(keb, krb, qb);
    if constexpr (EMU && SIMP) {
#pragma unroll
        for (int s = 0; s < QPL; ++s)
#pragma unroll
            for (int p = 0; p < 8; ++p) a8[s][p] = pack_sim8(e8[s][2 * p], e8[s][2 * p + 1]);
    } else if constexpr (EMU) {
        if constexpr (QUADS) {   // back to two codes per word
#pragma unroll
            for (int s = 0; s < QPL; ++s)
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    a8[s][2 * p] = a8q[s][p] & 0xFFFFu;
                    a8[s][2 * p + 1] = a8q[s][p] >> 16;
                }
        }
        uint32_t nan = 0;
#pragma unroll
        for (int s = 0; s < QPL; ++s)
#pragma unroll
            for (int p = 0; p < 8; ++p) nan |= e4m3_nan_bits(a8[s][p]);
        if (wave_any(nan != 0)) {
            nan_keys<QPL>(a8, sat);
            emu8_pass<D, QPL, true, LY>(qrow, k32e, a8);
        }
    }
    if constexpr (NKEY > 0) encode16<SIMP>(acc, c16);
}

// One channel of the 16-bit accumulation for every key and slot.
template <int QPL, int NKEY, int... I>
__device__ __forceinline__ void rec16_channel(float kv, const float (&q)[QPL], float (&acc)[QPL][NKEY],
                                              std::integer_sequence<int, I...>)
{
#pragma unroll
    for (int s = 0; s < QPL; ++s) fmac16_row<NKEY>(acc[s], kv, q[s]);
}

// Y16 of NKEY keys (NKEY in {4, 8, 12, 16}) for QPL query rows: the FP32 FMA
// chain over the channels in ascending order from +0, rounded once to e4m11
// (saturating).  krow is this lane's key row (layout LY): lane l of every
// 16-lane row supplies key (l mod 16) and must hold key (l mod NKEY) (lanes
// past NKEY duplicate the first keys and are not read).  codes[s][p] receives
// the e4m11 codes of keys 2p (bits [15:0]) and 2p+1 (SIM profile: rounded to
// 11 mantissa bits, codes[s][i] the FP32 pattern of key i).  With few keys per
// channel the loop is latency-bound, so the loads run PD 4-channel groups
// ahead in a ring of buffers written only by loads.
template <int D, int QPL, int NKEY, bool SIMP = false, class LY = RowLay<D>, class QP>
__device__ __forceinline__ void rec16_keys(const QP (&qrow)[QPL], const float *krow,
                                           uint32_t (&codes)[QPL][y16_words<SIMP>(NKEY)])
{
    static_assert(NKEY == 4 || NKEY == 8 || NKEY == 12 || NKEY == 16, "4, 8, 12 or 16 keys");
    constexpr int PD0 = NKEY <= 8 ? 4 : 2;
    constexpr int PD = (D / 4) % PD0 == 0 ? PD0 : 2;
    static_assert((D / 4) % PD == 0, "whole rings of 4-channel groups");
    float acc[QPL][NKEY];
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int i = 0; i < NKEY; ++i) acc[s][i] = 0.0f;
    float4 kb[PD], qb[PD][QPL];
    auto run = [&](int r) {
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            float q[QPL];
#pragma unroll
            for (int s = 0; s < QPL; ++s) q[s] = f4_at(qb[r][s], cc);
            rec16_channel<QPL, NKEY>(f4_at(kb[r], cc), q, acc, std::make_integer_sequence<int, NKEY>());
        }
    };
#pragma unroll
    for (int r = 0; r < PD; ++r) load_group<QPL, LY>(krow, qrow, 4 * r, kb[r], qb[r]);
    for (int c = 0; c < D - 4 * PD; c += 4 * PD) {
        dpp_guard();
#pragma unroll
        for (int r = 0; r < PD; ++r) {
            run(r);
            load_group<QPL, LY>(krow, qrow, c + 4 * (r + PD), kb[r], qb[r]);
        }
    }
    dpp_guard();
#pragma unroll
    for (int r = 0; r < PD; ++r) run(r);   // the last ring, no further loads
    encode16<SIMP>(acc, codes);
}

// Whether the 16-bit logit of one (query row, key) saturates: its FP32 FMA
// chain (channels ascending from +0, the recursion rec16_keys runs) rounds
// beyond 511.875, the largest e4m11 value, i.e. |sum| >= 511.9375 (a tie
// goes to the even 512).  Used only where a 16-bit code is at that maximum.
template <int D, class LY>
__device__ __forceinline__ bool y16_saturates(const float *qrow, const float *krow)
{
    float a = 0.0f;
#pragma unroll 4
    for (int c = 0; c < D; ++c) a = __builtin_fmaf(qrow[(c / 4) * LY::QS + c % 4], krow[(c / 4) * LY::KS + c % 4], a);
    return __builtin_fabsf(a) >= 511.9375f;
}

// Y16 of the 16 keys starting at k32 ([key][D] fp32).
template <int D, int QPL, bool SIMP = false, class LY = RowLay<D>, class QP>
__device__ __forceinline__ void rec16_chunk(const QP (&qrow)[QPL], const float *k32,
                                            uint32_t (&codes)[QPL][y16_words<SIMP>(16)])
{
    rec16_keys<D, QPL, 16, SIMP, LY>(qrow, k32 + (size_t)(__lane_id() & 15) * LY::KR, codes);
}

} // namespace lamp
