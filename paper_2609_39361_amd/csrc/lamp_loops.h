// lamp_loops.h -- the two logit loops of the LampAttention forward pass.
//
// Both loops give each lane QPL query rows and run over the D channels of a
// 16-key chunk.  The key value of (key, channel) is the same for every lane of
// a wave, so it is read with scalar loads into scalar registers and used as
// the scalar operand of the FMAs.  Scalar loads complete out of order and can
// only be waited for all at once, so they are issued in batches of two
// channels (32 values): wait for every load, issue the next batch, then run
// the arithmetic of the current batch while the next one is in flight.
#pragma once
#include "lamp_device.h"

namespace lamp {

// Every outstanding scalar/LDS load has completed; the scheduler may not move
// instructions across this point.
__device__ __forceinline__ void smem_fence()
{
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt, expcnt unchanged
    __builtin_amdgcn_sched_barrier(0);
}

__device__ __forceinline__ void kload2(float (&a)[16], float (&b)[16], kptr32_t kt, int c, int D)
{
    const int c1 = c + 1 < D ? c + 1 : D - 1;   // past the end: a harmless repeat
    const int c0 = c < D ? c : D - 1;
    kptr32_t p0 = kt + (size_t)c0 * 16, p1 = kt + (size_t)c1 * 16;
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = p0[i];
#pragma unroll
    for (int i = 0; i < 16; ++i) b[i] = p1[i];
}

// One channel of the 8-bit accumulation: acc <- RN_e4m3(RN32(q * k + acc)).
template <int QPL, bool SAT>
__device__ __forceinline__ void emu8_step(const float (&kv)[16], const float (&q)[QPL], uint32_t (&acc)[QPL][8])
{
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            float2 a = unpk_e4m3(acc[s][p]);
            float x = __builtin_fmaf(q[s], kv[2 * p], a.x);
            float y = __builtin_fmaf(q[s], kv[2 * p + 1], a.y);
            acc[s][p] = SAT ? pk_e4m3_sat(x, y, acc[s][p]) : pk_e4m3(x, y, acc[s][p]);
        }
}

// Y8 of one 16-key chunk for QPL query rows of this lane (Sec. 4.1:
// acc <- RN_e4m3(RN32(q_tilde * k + acc)), channels ascending, from +0).
// qrow[s] is the fp32 pre-scaled query row of slot s; kt the chunk's keys,
// [D][16] fp32.  acc[s][p] receives the codes of keys 2p, 2p+1 in bits [15:0].
template <int D, int QPL, bool SAT>
__device__ __forceinline__ void emu8_pass(const float *const (&qrow)[QPL], kptr32_t kt, uint32_t (&acc)[QPL][8])
{
    static_assert(D % 4 == 0, "channels in groups of 4");
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int p = 0; p < 8; ++p) acc[s][p] = 0u;
    float ka0[16], ka1[16], kb0[16], kb1[16];
    kload2(ka0, ka1, kt, 0, D);
    float4 qc[QPL];
#pragma unroll
    for (int s = 0; s < QPL; ++s) qc[s] = reinterpret_cast<const float4 *>(qrow[s])[0];
    for (int c = 0; c < D; c += 4) {
        float4 qn[QPL];
        const int cn = c + 4 < D ? c + 4 : c;
#pragma unroll
        for (int s = 0; s < QPL; ++s) qn[s] = reinterpret_cast<const float4 *>(qrow[s])[cn / 4];
        float q0[QPL], q1[QPL], q2[QPL], q3[QPL];
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            q0[s] = qc[s].x;
            q1[s] = qc[s].y;
            q2[s] = qc[s].z;
            q3[s] = qc[s].w;
        }
        smem_fence();
        kload2(kb0, kb1, kt, c + 2, D);
        __builtin_amdgcn_sched_barrier(0);
        emu8_step<QPL, SAT>(ka0, q0, acc);
        emu8_step<QPL, SAT>(ka1, q1, acc);
        smem_fence();
        kload2(ka0, ka1, kt, c + 4, D);
        __builtin_amdgcn_sched_barrier(0);
        emu8_step<QPL, SAT>(kb0, q2, acc);
        emu8_step<QPL, SAT>(kb1, q3, acc);
#pragma unroll
        for (int s = 0; s < QPL; ++s) qc[s] = qn[s];
    }
    smem_fence();   // drain the last (unused) batch
}

// The fast pass uses the non-saturating conversion; if any lane of the wave
// overflowed somewhere (a NaN code at the end of a chain), the chunk is
// recomputed with the saturating conversion.
template <int D, int QPL>
__device__ __forceinline__ void emu8_chunk(const float *const (&qrow)[QPL], const float *kt_generic,
                                           uint32_t (&acc)[QPL][8])
{
    kptr32_t kt = (kptr32_t)kt_generic;
    emu8_pass<D, QPL, false>(qrow, kt, acc);
    uint32_t nan = 0;
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int p = 0; p < 8; ++p) nan |= e4m3_nan_bits(acc[s][p]);
    if (wave_any(nan != 0)) emu8_pass<D, QPL, true>(qrow, kt, acc);
}

// One channel of the 16-bit accumulation: acc <- RN32(q * k + acc).
template <int QPL>
__device__ __forceinline__ void rec16_step(const float (&kv)[16], const float (&q)[QPL], float (&acc)[QPL][16])
{
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[s][i] = __builtin_fmaf(q[s], kv[i], acc[s][i]);
}

// Y16 of one 16-key chunk for QPL query rows: the FP32 FMA chain over the
// channels in ascending order from +0, rounded once to e4m11 (saturating).
// codes[s][p] receives the e4m11 codes of keys 2p (bits [15:0]) and 2p+1.
template <int D, int QPL>
__device__ __forceinline__ void rec16_chunk(const float *const (&qrow)[QPL], const float *kt_generic,
                                            uint32_t (&codes)[QPL][8])
{
    kptr32_t kt = (kptr32_t)kt_generic;
    float acc[QPL][16];
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[s][i] = 0.0f;
    float ka0[16], ka1[16], kb0[16], kb1[16];
    kload2(ka0, ka1, kt, 0, D);
    float4 qc[QPL];
#pragma unroll
    for (int s = 0; s < QPL; ++s) qc[s] = reinterpret_cast<const float4 *>(qrow[s])[0];
    for (int c = 0; c < D; c += 4) {
        float4 qn[QPL];
        const int cn = c + 4 < D ? c + 4 : c;
#pragma unroll
        for (int s = 0; s < QPL; ++s) qn[s] = reinterpret_cast<const float4 *>(qrow[s])[cn / 4];
        float q0[QPL], q1[QPL], q2[QPL], q3[QPL];
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            q0[s] = qc[s].x;
            q1[s] = qc[s].y;
            q2[s] = qc[s].z;
            q3[s] = qc[s].w;
        }
        smem_fence();
        kload2(kb0, kb1, kt, c + 2, D);
        __builtin_amdgcn_sched_barrier(0);
        rec16_step<QPL>(ka0, q0, acc);
        rec16_step<QPL>(ka1, q1, acc);
        smem_fence();
        kload2(ka0, ka1, kt, c + 4, D);
        __builtin_amdgcn_sched_barrier(0);
        rec16_step<QPL>(kb0, q2, acc);
        rec16_step<QPL>(kb1, q3, acc);
#pragma unroll
        for (int s = 0; s < QPL; ++s) qc[s] = qn[s];
    }
    smem_fence();
#pragma unroll
    for (int s = 0; s < QPL; ++s)
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            uint32_t c0, c1;
            (void)rn_e4m11((double)acc[s][2 * p], &c0);
            (void)rn_e4m11((double)acc[s][2 * p + 1], &c1);
            codes[s][p] = c0 | (c1 << 16);
        }
}

} // namespace lamp
