// lamp_fwd.hip -- the LampAttention forward kernel for gfx950 (paper Alg. 1),
// general form: d = 64, or 64-key sub-blocks.  (16-key sub-blocks with d >=
// 128 take the tile-pipelined kernel of lamp_fwd16.hip.)
//
// One workgroup handles one (batch, query head, query block of BQ rows) and
// walks its key tiles (KPT = BK*NK keys) in order.  Work split:
//   * every lane holds QPL = BQ/64 query rows (rows lane and lane+64), and
//     every wave keeps the running state (mu, omega) of all BQ rows -- the
//     state is small and every wave derives it from the same shared data, so
//     it stays identical across waves without extra traffic;
//   * wave w owns SPW = NK/NW consecutive key sub-blocks of each tile: it
//     computes their 8-bit logits and exponentials and publishes per-row
//     partial results in LDS;
//   * wave w owns the channel slice [w*CPW, (w+1)*CPW) of the output and
//     accumulates O^T = V^T E for that slice on the bf16 matrix cores.
// Per tile (Alg. 1 inner loop):
//   1. 8-bit logits of the own sub-blocks, column maxima m8 -> LDS;
//   2. stage 1 (Sec. 3.1, Eq. (7)): threats, sort, sequential margin tests on
//      the shared m8; a failing sub-block is recomputed in 16 bits by all
//      waves (KPW keys each) and raises mu_hat;
//   3. exponentials of the own sub-blocks against mu_hat (8-bit LUT in LDS,
//      16-bit table in global memory), written in place of the logit codes,
//      16-bit ones as exact bf16 high and low parts; partial row sums -> LDS;
//      lambda_hat, omega_hat;
//   4. stage 2 (Eq. (8)): per-sub-block costs -> LDS, feasibility of every
//      candidate recompute set evaluated identically by every wave, 16-bit
//      recompute of the chosen sub-blocks shared by all waves;
//   5. omega, mu update; O^T <- O^T diag(lambda_hat) + V^T E.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>

#include "lamp_device.h"
#include "lamp_kernels.h"
#include "lamp_loops.h"
#include "lamp_sr.h"
#include "lamp_stats.h"

#ifndef LAMP_MIN_WAVES
#define LAMP_MIN_WAVES 2   // minimum waves per SIMD requested from the register allocator
#endif

namespace lamp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

enum { PREC_LOW = 0, PREC_S1 = 1, PREC_S2 = 2, PREC_INACTIVE = 3 };

template <int D, int BQ, int BK, int NK>
struct Cfg {
    static constexpr int QPL = BQ / 64;                    // query rows per lane
    static constexpr int KPT = BK * NK;                    // keys per tile
    static constexpr int NCH = KPT / 16;                   // 16-key chunks per tile
    static constexpr int NW = NK < D / 32 ? NK : D / 32;   // waves
    static constexpr int SPW = NK / NW;                    // sub-blocks per wave
    static constexpr int CPW = D / NW;                     // output channels per wave
    static constexpr int CT = CPW / 32;                    // 32-channel MFMA tiles per wave
    static constexpr int QG = BQ / 32;                     // 32-row MFMA groups
    static constexpr int KPW = BK / NW;                    // keys per wave in a shared 16-bit recompute
    static constexpr int YP = KPT + 8;                     // LDS pitch (u16) of the code rows
    static constexpr size_t OFF_Y = 0;
    static constexpr size_t OFF_YL = OFF_Y + (size_t)BQ * YP * 2;        // low bf16 parts of E16
    static constexpr size_t OFF_LUT = OFF_YL + (size_t)BQ * YP * 2;
    static constexpr size_t OFF_M8 = OFF_LUT + 512;                       // f32 [NK][BQ]
    static constexpr size_t OFF_CM = OFF_M8 + (size_t)NK * BQ * 4;       // f32 [NK][BQ] + [2][NW][BQ]
    static constexpr size_t OFF_SP = OFF_CM + (size_t)(NK + 2 * NW) * BQ * 4;   // f64 [2][NW][BQ]
    static constexpr size_t OFF_CO = OFF_SP + (size_t)2 * NW * BQ * 8;   // f64 [NK][BQ]
    static constexpr size_t OFF_ED = OFF_CO + (size_t)NK * BQ * 8;       // f64 [EXPDOC_NK]
    static constexpr size_t OFF_ST = OFF_ED + (size_t)EXPDOC_NK * 8;     // u32 [ST_N] statistics
    static constexpr size_t OFF_PD = OFF_ST + (size_t)ST_N * 4;          // f64 [NW][BQ] pending rescale factors
    static constexpr size_t LDS = OFF_PD + (size_t)NW * BQ * 8;
    static_assert(BQ == 64 || BQ == 128, "64 or 128 query rows per block");
    static_assert(BK % 16 == 0 && NK <= 4 && NK % NW == 0, "sub-blocks of 16-key chunks, at most 4 per tile");
    static_assert(CPW % 32 == 0, "whole 32-channel tiles per wave");
    static_assert(KPW == 4 || KPW == 8 || KPW % 16 == 0, "recompute split in 4, 8 or multiples of 16 keys");
};

// SR: the 8-bit logits with stochastic rounding (lamp_sr.h) in place of
// round-to-nearest.
// OBS: the instantiation that also writes the logit observables (p.dbg_y8,
// p.dbg_y16), kept apart so that the stores do not change the register
// allocation of the others.
template <int D, int BQ, int BK, int NK, bool SR, bool OBS>
__global__ __launch_bounds__(64 * (NK < D / 32 ? NK : D / 32), LAMP_MIN_WAVES) void lamp_fwd_kernel(FwdParams p)
{
    using C = Cfg<D, BQ, BK, NK>;
    constexpr int QPL = C::QPL, KPT = C::KPT, NCH = C::NCH, NW = C::NW, SPW = C::SPW, CPW = C::CPW;
    constexpr int CT = C::CT, QG = C::QG, YP = C::YP, KPW = C::KPW;
    constexpr int CPS = BK / 16;   // chunks per sub-block

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t *ycode = reinterpret_cast<uint16_t *>(smem + C::OFF_Y);   // [BQ][YP] logit codes, then E (bf16 bits;
                                                                       // 16-bit sub-blocks: high part)
    uint16_t *ylo = reinterpret_cast<uint16_t *>(smem + C::OFF_YL);    // [BQ][YP] low bf16 part of E16
    uint16_t *lut = reinterpret_cast<uint16_t *>(smem + C::OFF_LUT);   // [256] 8-bit exp (bf16 bits)
    float *m8s = reinterpret_cast<float *>(smem + C::OFF_M8);          // [NK][BQ] 8-bit column maxima
    float *cms = reinterpret_cast<float *>(smem + C::OFF_CM);          // [NK][BQ] 16-bit column maxima (threshold 0)
    float *cmf = cms + NK * BQ;   // [2][NW][BQ] per-wave maxima of a shared recompute, by iteration parity
    double *sps = reinterpret_cast<double *>(smem + C::OFF_SP);        // [NW][BQ] partial row sums of E
    double *spf = sps + NW * BQ;                                       // [NW][BQ] the same over 8-bit sub-blocks
    double *cst_lds = reinterpret_cast<double *>(smem + C::OFF_CO);    // [NK][BQ] stage-2 costs
    double *edk = reinterpret_cast<double *>(smem + C::OFF_ED);        // exp_doc constants
    uint32_t *stl = reinterpret_cast<uint32_t *>(smem + C::OFF_ST);    // [ST_N] statistics (p.stats)
    double *pend = reinterpret_cast<double *>(smem + C::OFF_PD);        // [NW][BQ] pending factors (step 5)

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;   // w is wave-uniform
    const int nqb = p.Nq / BQ;   // query blocks per head (the last may be partial)
    const int BH = p.B * p.Hq;
    const int qb = nqb - 1 - (int)(blockIdx.x / BH);   // longest blocks first under causality
    const int bh = blockIdx.x % BH;
    const int b = bh / p.Hq, h = bh % p.Hq;
    const int hk = h / (p.Hq / p.Hkv);
    const int q0 = qb * BQ;
    const float NEG_INF = -__builtin_inff();

    // per-slot row, query index and visible key range [vlo, vhi]
    int row[QPL], vlo[QPL], vhi[QPL];
    const float *qrow[QPL];
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        row[s] = s * 64 + lane;
        const int j = q0 + row[s];
        vlo[s] = p.window > 0 ? (j - p.window + 1 > 0 ? j - p.window + 1 : 0) : 0;
        vhi[s] = p.causal ? j : p.N - 1;
        if (j >= p.N) {   // a row beyond N (partial last block): no visible key
            vlo[s] = p.N;
            vhi[s] = -1;
        }
        qrow[s] = p.qt + (((size_t)b * p.Hq + h) * p.Nq + j) * D;   // zero-padded rows, in bounds
    }
    // visible key range of the whole block
    const int bv_lo = p.window > 0 ? (q0 - p.window + 1 > 0 ? q0 - p.window + 1 : 0) : 0;
    const int bv_hi = p.causal ? (q0 + BQ - 1 < p.N - 1 ? q0 + BQ - 1 : p.N - 1) : p.N - 1;
    const int t_begin = bv_lo / KPT, t_end = bv_hi / KPT;

    const float *kt32 = p.kt32 + ((size_t)b * p.Hkv + hk) * (size_t)p.Nk * D;   // fp32 keys [Nk][D]
    const uint16_t *vtbase = p.vt + ((size_t)b * p.Hkv + hk) * (size_t)D * p.Nk;   // V^T [D][Nk]
    uint8_t *mrow = p.mask + (((size_t)b * p.Hq + h) * nqb + qb) * (size_t)(p.Nk / BK);

    for (int i = tid; i < 256; i += 64 * NW) lut[i] = p.lut8e[i];
    if (tid < EXPDOC_NK) edk[tid] = EXPDOC_K[tid];
    if (tid < ST_N) stl[tid] = 0u;
    for (int i = tid; i < NW * BQ; i += 64 * NW) pend[i] = 1.0;
    // logit observables (tests): this query block is observed (uniform)
    const bool dbg_blk = qb >= p.dbg_qb0 && qb < p.dbg_qb0 + p.dbg_nqb;
    const bool dbg8 = OBS && p.dbg_y8 != nullptr && dbg_blk, dbg16 = OBS && p.dbg_y16 != nullptr && dbg_blk;
    auto dbg_off = [&](int s) -> size_t {
        return ((((size_t)b * p.Hq + h) * p.dbg_nqb + (qb - p.dbg_qb0)) * BQ + row[s]) * (size_t)p.Nk;
    };

    float mu[QPL];     // running maxima (e4m11 or e4m3 values)
    double om[QPL];    // running sums omega
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        mu[s] = NEG_INF;
        om[s] = 0.0;
    }
    floatx16 acc[QG][CT];
#pragma unroll
    for (int g = 0; g < QG; ++g)
#pragma unroll
        for (int t = 0; t < CT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[g][t][r] = 0.0f;

    auto visible = [&](int s, int key) { return key >= vlo[s] && key <= vhi[s]; };

    // Observables of the 16-bit logits of 2*NWD keys from kc of every slot
    // (codes two per word): their codes for the tests, and the saturated ones
    // among the visible keys whose code is the largest e4m11 magnitude (the
    // FP32 chain rerun for those alone).
    auto obs16 = [&](int kc, const auto &yc) {
        constexpr int NWD = sizeof(yc[0]) / sizeof(uint32_t);   // words per slot
        if (dbg16) {
#pragma unroll
            for (int s = 0; s < QPL; ++s)
#pragma unroll
                for (int x = 0; x < NWD; ++x) {
                    const uint32_t lo = visible(s, kc + 2 * x) ? (yc[s][x] & 0xFFFFu) : 0xFFFFu;
                    const uint32_t hi = visible(s, kc + 2 * x + 1) ? (yc[s][x] >> 16) : 0xFFFFu;
                    *reinterpret_cast<uint32_t *>(p.dbg_y16 + dbg_off(s) + kc + 2 * x) = lo | (hi << 16);
                }
        }
        if (p.stats) {
            static_assert(QPL * 2 * NWD <= 32, "one bit per slot and key");
            uint32_t atmax = 0;   // bit s * 2NWD + i: slot s, key kc + i
#pragma unroll
            for (int s = 0; s < QPL; ++s)
#pragma unroll
                for (int i = 0; i < 2 * NWD; ++i) {
                    const uint32_t code = (yc[s][i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
                    atmax |= ((code & 0x7FFFu) == 0x7FFFu && visible(s, kc + i) ? 1u : 0u) << (s * 2 * NWD + i);
                }
            if (wave_any(atmax != 0u)) {
                uint32_t n = 0;
                for (uint32_t m = atmax; m; m &= m - 1) {
                    const int bit = __builtin_ctz(m);
                    const float *qr = qrow[0];
#pragma unroll
                    for (int s = 1; s < QPL; ++s) qr = bit / (2 * NWD) == s ? qrow[s] : qr;
                    n += y16_saturates<D, RowLay<D>>(qr, kt32 + (size_t)(kc + bit % (2 * NWD)) * D) ? 1u : 0u;
                }
                if (n) atomicAdd(&stl[ST_SAT16], n);
            }
        }
    };

    // 16-bit recompute of sub-block th shared by all waves: wave w takes keys
    // [key0, key0 + KPW) with key0 = k0 + th*BK + w*KPW.  For every 16-key
    // group (or the 4 / 8 keys) fn(key, nk, codes) receives the e4m11 codes.
    auto shared16 = [&](int k0, int th, auto fn) {
        const int key0 = k0 + th * BK + w * KPW;
        if (key0 > bv_hi || key0 + KPW - 1 < bv_lo) return;   // nothing visible in the block
        if constexpr (KPW >= 16) {
            for (int ch = 0; ch < KPW / 16; ++ch) {
                const int kc = key0 + ch * 16;
                uint32_t yc[QPL][8];
                rec16_keys<D, QPL, 16>(qrow, kt32 + (size_t)(kc + (lane & 15)) * D, yc);
                fn(kc, yc);
            }
        } else {
            uint32_t yc[QPL][KPW / 2];
            rec16_keys<D, QPL, KPW>(qrow, kt32 + (size_t)(key0 + (lane & 15) % KPW) * D, yc);
            fn(key0, yc);
        }
    };
    // write n = 4, 8 or 16 u16 codes (packed two per word) at row r, key offset ko
    auto put_codes = [&](uint16_t *arr, int r, int ko, const uint32_t *cw, int nw) {
        uint16_t *dst = arr + r * YP + ko;
        if (nw == 2) {
            *reinterpret_cast<uint2 *>(dst) = make_uint2(cw[0], cw[1]);
        } else {
            for (int t = 0; t < nw; t += 4)
                *reinterpret_cast<u32x4 *>(dst + 2 * t) = u32x4{cw[t], cw[t + 1], cw[t + 2], cw[t + 3]};
        }
    };

    for (int tile = t_begin; tile <= t_end; ++tile) {
        const int k0 = tile * KPT;
        __syncthreads();   // readers of ycode / ylo / LDS partials of the previous tile are done

        // ---- active sub-blocks (a visible pair anywhere in the block), uniform
        uint32_t active = 0;
#pragma unroll
        for (int th = 0; th < NK; ++th) {
            const int a = k0 + th * BK, z = a + BK - 1;
            bool any = false;
#pragma unroll
            for (int s = 0; s < QPL; ++s) any |= (a <= vhi[s] && z >= vlo[s]);
            if (wave_any(any)) active |= 1u << th;
        }
        if (active == 0) {   // no visible pair in the tile: no state change
            if (tid == 0)
                for (int th = 0; th < NK; ++th) mrow[tile * NK + th] = PREC_INACTIVE;
            continue;
        }

        // ---- 1. 8-bit logits of the own sub-blocks (unused at threshold 0)
        if (p.mode != MODE_ALL16) {
#pragma unroll
            for (int u = 0; u < SPW; ++u) {
                const int th = w * SPW + u;
                float mx[QPL];
#pragma unroll
                for (int s = 0; s < QPL; ++s) mx[s] = NEG_INF;
                if (active >> th & 1u) {
                    for (int ch = 0; ch < CPS; ++ch) {
                        const int c16 = th * CPS + ch;
                        const int ck0 = k0 + c16 * 16;
                        if (ck0 > bv_hi || ck0 + 15 < bv_lo) continue;   // nothing visible in the block
                        uint32_t a8[QPL][8], sat[QPL];
                        if constexpr (SR) {
                            int jq[QPL];
#pragma unroll
                            for (int s = 0; s < QPL; ++s) jq[s] = q0 + row[s];
                            sr8_chunk<D, QPL>(qrow, kt32 + (size_t)ck0 * D, p.seed, (uint64_t)bh, jq, ck0, a8, sat);
                        } else {
                            emu8_chunk<D, QPL>(qrow, kt32 + (size_t)ck0 * D, a8, sat);
                        }
                        auto vis16 = [&](int s) {
                            uint32_t m = 0;
#pragma unroll
                            for (int i = 0; i < 16; ++i) m |= (visible(s, ck0 + i) ? 1u : 0u) << i;
                            return m;
                        };
                        if (p.stats) {
                            uint32_t any = 0;
#pragma unroll
                            for (int s = 0; s < QPL; ++s) any |= sat[s];
                            if (wave_any(any != 0u)) {
                                uint32_t n = 0;
#pragma unroll
                                for (int s = 0; s < QPL; ++s) n += __builtin_popcount(sat[s] & vis16(s));
                                if (n) atomicAdd(&stl[ST_SAT8], n);
                            }
                        }
                        if (dbg8) {
#pragma unroll
                            for (int s = 0; s < QPL; ++s) {
                                const uint32_t vm = vis16(s);
                                uint32_t wd[4];
#pragma unroll
                                for (int q4 = 0; q4 < 4; ++q4) {
                                    uint32_t x = 0;
#pragma unroll
                                    for (int i = 0; i < 4; ++i) {
                                        const int key = 4 * q4 + i;
                                        const uint32_t code = (a8[s][key >> 1] >> (8 * (key & 1))) & 0xFFu;
                                        x |= ((vm >> key & 1u) ? code : 0xFFu) << (8 * i);
                                    }
                                    wd[q4] = x;
                                }
                                *reinterpret_cast<u32x4 *>(p.dbg_y8 + dbg_off(s) + ck0) =
                                    u32x4{wd[0], wd[1], wd[2], wd[3]};
                            }
                        }
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
                            const bool full = ck0 >= vlo[s] && ck0 + 15 <= vhi[s];
                            uint32_t packed[8];
#pragma unroll
                            for (int pp = 0; pp < 8; ++pp) {
                                const float2 yv = unpk_e4m3(a8[s][pp]);
                                const int i0 = ck0 + 2 * pp;
                                // invisible keys enter as -inf, by selection rather than branches
                                const float x0 = (full || visible(s, i0)) ? yv.x : NEG_INF;
                                const float x1 = (full || visible(s, i0 + 1)) ? yv.y : NEG_INF;
                                mx[s] = x0 > mx[s] ? x0 : mx[s];
                                mx[s] = x1 > mx[s] ? x1 : mx[s];
                                packed[pp] = (a8[s][pp] & 0xFFu) | ((a8[s][pp] & 0xFF00u) << 8);
                            }
                            u32x4 *dst = reinterpret_cast<u32x4 *>(ycode + row[s] * YP + c16 * 16);
                            dst[0] = u32x4{packed[0], packed[1], packed[2], packed[3]};
                            dst[1] = u32x4{packed[4], packed[5], packed[6], packed[7]};
                        }
                    }
                }
#pragma unroll
                for (int s = 0; s < QPL; ++s) m8s[th * BQ + row[s]] = mx[s];
            }
        }
        __syncthreads();   // m8s complete

        // ---- 2. running maximum mu_hat and stage 1
        float muh[QPL];
        float m8[NK][QPL];
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            muh[s] = mu[s];
#pragma unroll
            for (int th = 0; th < NK; ++th) m8[th][s] = (p.mode != MODE_ALL16) ? m8s[th * BQ + row[s]] : NEG_INF;
        }
        uint32_t prec16 = 0;   // stage-1 (or threshold-0) sub-blocks
        const bool stage1_off = (p.flags & LAMP_STAGE1_OFF) != 0u;   // flags are 0 outside the threshold mode
        if (p.mode == MODE_PURE8 || stage1_off) {   // running maximum over the 8-bit logits
#pragma unroll
            for (int s = 0; s < QPL; ++s)
#pragma unroll
                for (int th = 0; th < NK; ++th) muh[s] = m8[th][s] > muh[s] ? m8[th][s] : muh[s];
        } else if (p.mode == MODE_ALL16) {
            prec16 = active;
#pragma unroll
            for (int u = 0; u < SPW; ++u) {
                const int th = w * SPW + u;
                float cm[QPL];
#pragma unroll
                for (int s = 0; s < QPL; ++s) cm[s] = NEG_INF;
                if (active >> th & 1u) {
                    for (int ch = 0; ch < CPS; ++ch) {
                        const int c16 = th * CPS + ch;
                        const int ck0 = k0 + c16 * 16;
                        if (ck0 > bv_hi || ck0 + 15 < bv_lo) continue;
                        uint32_t yc[QPL][8];
                        rec16_chunk<D, QPL>(qrow, kt32 + (size_t)ck0 * D, yc);
                        obs16(ck0, yc);
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
#pragma unroll
                            for (int i = 0; i < 16; ++i) {
                                const float yv = e4m11_value((yc[s][i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
                                if (visible(s, ck0 + i)) cm[s] = yv > cm[s] ? yv : cm[s];
                            }
                            u32x4 *dst = reinterpret_cast<u32x4 *>(ycode + row[s] * YP + c16 * 16);
                            dst[0] = u32x4{yc[s][0], yc[s][1], yc[s][2], yc[s][3]};
                            dst[1] = u32x4{yc[s][4], yc[s][5], yc[s][6], yc[s][7]};
                        }
                    }
                }
#pragma unroll
                for (int s = 0; s < QPL; ++s) cms[th * BQ + row[s]] = cm[s];
            }
            __syncthreads();
#pragma unroll
            for (int s = 0; s < QPL; ++s)
#pragma unroll
                for (int th = 0; th < NK; ++th) {
                    const float c = cms[th * BQ + row[s]];
                    muh[s] = c > muh[s] ? c : muh[s];
                }
        } else {
            // threats T_theta = max_j (m8 - mu_j), exact in fp64 (+inf when mu_j = -inf)
            double T[NK];
#pragma unroll
            for (int th = 0; th < NK; ++th) {
                double t = -__builtin_inf();
#pragma unroll
                for (int s = 0; s < QPL; ++s)
                    if (m8[th][s] > NEG_INF) {
                        const double d = (double)m8[th][s] - (double)mu[s];
                        t = d > t ? d : t;
                    }
                T[th] = wave_max_f64(t);
            }
            // descending threat, ties by index; order packed 4 bits per rank
            uint32_t order = 0, taken = 0;
            int na = 0;
#pragma unroll
            for (int r = 0; r < NK; ++r) {
                int best = -1;
                double bt = 0.0;
#pragma unroll
                for (int th = 0; th < NK; ++th) {
                    const bool cand = (active >> th & 1u) && !(taken >> th & 1u);
                    if (cand && (best < 0 || T[th] > bt)) {
                        best = th;
                        bt = T[th];
                    }
                }
                if (best >= 0) {
                    order |= (uint32_t)best << (4 * na);
                    ++na;
                    taken |= 1u << best;
                }
            }
            // margin test of every sub-block against the current mu_hat:
            // mu_hat_j > fma(|mu_hat_j|, delta, m8); columns without a visible
            // entry are not tested; mu_hat = -inf fails
            auto fails = [&]() {
                uint32_t f = 0;
#pragma unroll
                for (int th = 0; th < NK; ++th) {
                    bool bad = false;
#pragma unroll
                    for (int s = 0; s < QPL; ++s)
                        if (m8[th][s] > NEG_INF) {
                            const double mh = (double)muh[s];
                            bad |= !(mh > __builtin_fma(__builtin_fabs(mh), p.delta, (double)m8[th][s]));
                        }
                    if (wave_any(bad)) f |= 1u << th;
                }
                return f;
            };
            uint32_t fail = fails();
            int pos = 0, par = 0;
            while (true) {
                while (pos < na && !(fail >> ((order >> (4 * pos)) & 15u) & 1u)) ++pos;
                if (pos >= na) break;
                const int th = (int)((order >> (4 * pos)) & 15u);
                ++pos;
                prec16 |= 1u << th;
                {   // all waves recompute the sub-block in 16 bits, KPW keys each
                    float cm[QPL];
#pragma unroll
                    for (int s = 0; s < QPL; ++s) cm[s] = NEG_INF;
                    shared16(k0, th, [&](int kc, const auto &yc) {
                        constexpr int NWD = sizeof(yc[0]) / sizeof(uint32_t);   // words per slot
                        obs16(kc, yc);
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
#pragma unroll
                            for (int i = 0; i < 2 * NWD; ++i) {
                                const float yv = e4m11_value((yc[s][i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
                                if (visible(s, kc + i)) cm[s] = yv > cm[s] ? yv : cm[s];
                            }
                            put_codes(ycode, row[s], kc - k0, yc[s], NWD);
                        }
                    });
#pragma unroll
                    for (int s = 0; s < QPL; ++s) cmf[(par * NW + w) * BQ + row[s]] = cm[s];
                }
                __syncthreads();
#pragma unroll
                for (int s = 0; s < QPL; ++s) {
#pragma unroll
                    for (int ww = 0; ww < NW; ++ww) {
                        const float c = cmf[(par * NW + ww) * BQ + row[s]];
                        muh[s] = c > muh[s] ? c : muh[s];
                    }
                }
                par ^= 1;   // the next write goes to the other half: readers of this one may lag
                if (pos < na) fail = fails();
            }
        }

        // ---- 3. exponentials of the own sub-blocks against mu_hat
        {
            double sp[QPL], spF[QPL];   // all exponentials / those of 8-bit sub-blocks
            float mu8[QPL];             // the running maximum the 8-bit shifts use
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
                sp[s] = spF[s] = 0.0;
                mu8[s] = (p.flags & LAMP_MU_TRUNC) ? trunc_e4m3(muh[s]) : muh[s];
            }
#pragma unroll
            for (int u = 0; u < SPW; ++u) {
                const int th = w * SPW + u;
                if (!(active >> th & 1u)) {
                    // inactive: zero exponentials so the P.V pass may read them
                    for (int ch = 0; ch < CPS; ++ch)
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
                            u32x4 *d = reinterpret_cast<u32x4 *>(ycode + row[s] * YP + (th * CPS + ch) * 16);
                            d[0] = u32x4{0u, 0u, 0u, 0u};
                            d[1] = u32x4{0u, 0u, 0u, 0u};
                        }
                    continue;
                }
                const bool hi16 = prec16 >> th & 1u;
                // Straight-line per 16-key chunk and row: all codes read, all
                // table indices formed (an invisible key reads the table's last
                // entry, whose exponential is 0), all table reads issued, then
                // the sums, which are exact in fp64 in any order (multiples of
                // 2^-41 below 2^9).
                auto run = [&](auto hi_c) {
                    constexpr bool HI = decltype(hi_c)::value;
                    for (int ch = 0; ch < CPS; ++ch) {
                        const int c16 = th * CPS + ch;
                        const int ck0 = k0 + c16 * 16;
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
                            u32x4 *rp = reinterpret_cast<u32x4 *>(ycode + row[s] * YP + c16 * 16);
                            u32x4 *lp = reinterpret_cast<u32x4 *>(ylo + row[s] * YP + c16 * 16);
                            const u32x4 c0 = rp[0], c1 = rp[1];
                            const uint32_t in[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
                            uint32_t eb[16];
#pragma unroll
                            for (int i = 0; i < 16; ++i) {
                                const uint32_t yc = (in[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
                                const bool vis = visible(s, ck0 + i);
                                if constexpr (HI) {
                                    const uint32_t x = ue5m11_code(shift_of(muh[s], e4m11_value(yc)));
                                    eb[i] = p.exp16[vis ? x : 65535u];
                                } else {
                                    const float y = (i & 1) ? __builtin_amdgcn_cvt_f32_fp8((int)in[i >> 1], 2)
                                                            : __builtin_amdgcn_cvt_f32_fp8((int)in[i >> 1], 0);
                                    const uint32_t x = ue5m3_code(shift_of(mu8[s], y));
                                    eb[i] = lut[vis ? x : 255u];
                                }
                            }
                            double a4[4] = {0.0, 0.0, 0.0, 0.0};
                            uint32_t eh[16], el[16];
#pragma unroll
                            for (int i = 0; i < 16; ++i) {
                                float ev;
                                if constexpr (HI) {
                                    ev = ue5m11e_value(eb[i]);
                                    split_bf16(ev, eh[i], el[i]);
                                } else {
                                    eh[i] = eb[i];
                                    el[i] = 0u;
                                    ev = bf16_value(eb[i]);
                                }
                                a4[i & 3] += (double)ev;
                            }
                            const double ts = (a4[0] + a4[1]) + (a4[2] + a4[3]);
                            sp[s] += ts;
                            if constexpr (!HI) spF[s] += ts;
                            rp[0] = u32x4{eh[0] | eh[1] << 16, eh[2] | eh[3] << 16, eh[4] | eh[5] << 16,
                                          eh[6] | eh[7] << 16};
                            rp[1] = u32x4{eh[8] | eh[9] << 16, eh[10] | eh[11] << 16, eh[12] | eh[13] << 16,
                                          eh[14] | eh[15] << 16};
                            if constexpr (HI) {
                                lp[0] = u32x4{el[0] | el[1] << 16, el[2] | el[3] << 16, el[4] | el[5] << 16,
                                              el[6] | el[7] << 16};
                                lp[1] = u32x4{el[8] | el[9] << 16, el[10] | el[11] << 16, el[12] | el[13] << 16,
                                              el[14] | el[15] << 16};
                            }
                        }
                    }
                };
                if (hi16) run(std::true_type());
                else run(std::false_type());
            }
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
                sps[w * BQ + row[s]] = sp[s];
                spf[w * BQ + row[s]] = spF[s];
            }
        }
        __syncthreads();

        // ---- 4. lambda_hat, omega_hat, stage 2
        double S[QPL], lam[QPL], omh[QPL];
        bool moved = false;   // exp_doc(0) is exactly 1: skip the exponentials when no maximum moved
#pragma unroll
        for (int s = 0; s < QPL; ++s) moved |= muh[s] != mu[s];
        moved = wave_any(moved);
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            double t = 0.0;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) t += sps[ww * BQ + row[s]];
            S[s] = t;
            if (muh[s] == NEG_INF) lam[s] = 1.0;
            else if (mu[s] == NEG_INF) lam[s] = 0.0;
            else lam[s] = moved ? exp_doc_k((double)mu[s] - (double)muh[s], [&](int i) { return edk[i]; }) : 1.0;
            omh[s] = __builtin_fma(lam[s], om[s], t);
        }
        uint32_t prec2 = 0;
        if (p.mode == MODE_LAMP) {
            const uint32_t F = active & ~prec16;
            // Quick feasibility of the empty recompute set.  Every cost term
            // E (omega_hat - E) is at most E omega_hat, so the computed xi_j
            // stays below omega_hat_j S_F,j (1 + 2^-40) (at most a few hundred
            // fp64 roundings), S_F,j being the exact mass of the 8-bit
            // sub-blocks; the computed limit is at least tau omega_hat_j^2
            // (1 - 2^-52).  S_F,j <= tau omega_hat_j (1 - 2^-38) on every row
            // therefore implies that the exact test accepts R = {} as well.
            bool need = false;
            if (F) {
#pragma unroll
                for (int s = 0; s < QPL; ++s) {
                    double sf = 0.0;
#pragma unroll
                    for (int ww = 0; ww < NW; ++ww) sf += spf[ww * BQ + row[s]];
                    need |= !(sf <= (p.tau * omh[s]) * (1.0 - 0x1p-38));
                }
                need = wave_any(need);
            }
            if (need) {
                // costs c_theta,j = sum_{i in theta, ascending} E (omega_hat - E)
#pragma unroll
                for (int u = 0; u < SPW; ++u) {
                    const int th = w * SPW + u;
                    if (!(F >> th & 1u)) continue;
#pragma unroll
                    for (int s = 0; s < QPL; ++s) {
                        double cth = 0.0;
                        for (int ch = 0; ch < CPS; ++ch) {
                            const int c16 = th * CPS + ch;
                            const u32x4 *rp = reinterpret_cast<const u32x4 *>(ycode + row[s] * YP + c16 * 16);
                            const u32x4 c0 = rp[0], c1 = rp[1];
                            const uint32_t in[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
#pragma unroll
                            for (int i = 0; i < 16; ++i) {
                                const double e = (double)bf16_value((in[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
                                const double tt = omh[s] - e;
                                const double pr = e * tt;
                                cth = cth + pr;   // invisible entries hold E = 0 and add +0
                            }
                        }
                        cst_lds[th * BQ + row[s]] = cth;
                    }
                }
                __syncthreads();
                // feasibility of every recompute set R within F, identical in every wave
                double cst[NK][QPL], lim[QPL];
#pragma unroll
                for (int s = 0; s < QPL; ++s) {
                    lim[s] = (p.tau * omh[s]) * omh[s];
#pragma unroll
                    for (int th = 0; th < NK; ++th) cst[th][s] = (F >> th & 1u) ? cst_lds[th * BQ + row[s]] : 0.0;
                }
                uint32_t feas = 0;
                for (int R = 0; R < (1 << NK); ++R) {
                    if (R & ~(int)F) continue;
                    bool bad = false;
#pragma unroll
                    for (int s = 0; s < QPL; ++s) {
                        double xi = 0.0;
#pragma unroll
                        for (int th = 0; th < NK; ++th)
                            if ((F >> th & 1u) && !(R >> th & 1)) xi = xi + cst[th][s];
                        bad |= !(xi <= lim[s]);
                    }
                    if (!wave_any(bad)) feas |= 1u << R;
                }
                // smallest recompute set first, then ascending bitmask
                int chosen = (int)F;
                bool found = false;
                for (int sz = 0; sz <= NK && !found; ++sz)
                    for (int R = 0; R < (1 << NK) && !found; ++R) {
                        if ((R & ~(int)F) || __builtin_popcount(R) != sz) continue;
                        if (feas >> R & 1u) {
                            chosen = R;
                            found = true;
                        }
                    }
                prec2 = (uint32_t)chosen;
                if (prec2) {
                    // stage-2 recompute shared by all waves: 16-bit logits and
                    // exponentials against the unchanged mu_hat
                    double ds[QPL];
#pragma unroll
                    for (int s = 0; s < QPL; ++s) ds[s] = 0.0;
                    auto s2fn = [&](int kc, const auto &yc) {
                        constexpr int NWD = sizeof(yc[0]) / sizeof(uint32_t);
                        obs16(kc, yc);
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
                            const uint16_t *src = ycode + row[s] * YP + (kc - k0);
                            uint32_t outw[NWD], outl[NWD];
#pragma unroll
                            for (int pp = 0; pp < NWD; ++pp) {
                                uint32_t res = 0, rlo = 0;
#pragma unroll
                                for (int t = 0; t < 2; ++t) {
                                    const int key = kc + 2 * pp + t;
                                    uint32_t eh = 0, el = 0;
                                    if (visible(s, key)) {
                                        const float old = bf16_value(src[2 * pp + t]);
                                        const float y = e4m11_value((yc[s][pp] >> (16 * t)) & 0xFFFFu);
                                        const float ev = ue5m11e_value(p.exp16[ue5m11_code(shift_of(muh[s], y))]);
                                        split_bf16(ev, eh, el);
                                        ds[s] = ds[s] - (double)old;
                                        ds[s] = ds[s] + (double)ev;
                                    }
                                    res |= eh << (16 * t);
                                    rlo |= el << (16 * t);
                                }
                                outw[pp] = res;
                                outl[pp] = rlo;
                            }
                            put_codes(ycode, row[s], kc - k0, outw, NWD);
                            put_codes(ylo, row[s], kc - k0, outl, NWD);
                        }
                    };
                    for (int th = 0; th < NK; ++th) {
                        if (!(prec2 >> th & 1u)) continue;
                        shared16(k0, th, s2fn);
                    }
#pragma unroll
                    for (int s = 0; s < QPL; ++s) sps[w * BQ + row[s]] = ds[s];
                    __syncthreads();
#pragma unroll
                    for (int s = 0; s < QPL; ++s) {
                        double t = S[s];
#pragma unroll
                        for (int ww = 0; ww < NW; ++ww) t += sps[ww * BQ + row[s]];   // exact
                        S[s] = t;
                    }
                }
            }
        }

        // ---- 5. state update; O^T <- O^T diag(lambda_hat) + V^T E
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            om[s] = __builtin_fma(lam[s], om[s], S[s]);
            mu[s] = muh[s];
        }
        if (tid == 0) {
#pragma unroll
            for (int th = 0; th < NK; ++th)
                mrow[tile * NK + th] = !(active >> th & 1u) ? PREC_INACTIVE
                                     : (prec16 >> th & 1u) ? PREC_S1
                                     : (prec2 >> th & 1u) ? PREC_S2 : PREC_LOW;
            if (p.stats) {
                // every recompute of this kernel is one at a time (or after
                // stage 2), except the all-16-bit mode's own sub-blocks
                const uint32_t rec = prec16 | prec2;
                stl[ST_TILES] += 1u;
                stl[ST_S1] += __builtin_popcount(prec16);
                stl[ST_S2] += __builtin_popcount(prec2);
                stl[ST_ACT] += __builtin_popcount(active);
                stl[ST_LATE] += p.mode == MODE_LAMP ? __builtin_popcount(rec) : 0;
                stl[ST_HIST + __builtin_popcount(rec)] += 1u;
            }
        }
        const uint32_t p16 = prec16 | prec2;
        const int half = lane >> 5, l32 = lane & 31;
        // V^T operands from global memory, one chunk ahead of the matrix-core
        // work (every chunk's keys lie below N, so the loads stay in bounds
        // even for chunks without a visible pair, whose products are skipped)
        auto load_v = [&](int c16, u32x4 (&a)[CT]) {
#pragma unroll
            for (int t = 0; t < CT; ++t)
                a[t] = *reinterpret_cast<const u32x4 *>(vtbase + (size_t)(w * CPW + t * 32 + l32) * p.Nk + k0 + c16 * 16 +
                                                        half * 8);
        };
        auto pv_chunk = [&](int c16, const u32x4 (&a)[CT]) {
            const int ck0 = k0 + c16 * 16;
            const int th = c16 / CPS;
            if (!(active >> th & 1u) || ck0 > bv_hi || ck0 + 15 < bv_lo) return;
            const bool hi16 = p16 >> th & 1u;
#pragma unroll
            for (int g = 0; g < QG; ++g) {
                const int off = (g * 32 + l32) * YP + c16 * 16 + half * 8;
                const bf16x8 bh = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(ycode + off));
#pragma unroll
                for (int t = 0; t < CT; ++t)
                    acc[g][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[t]), bh, acc[g][t],
                                                                        0, 0, 0);
                if (hi16) {   // E16 = hi + lo exactly
                    const bf16x8 bl = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(ylo + off));
#pragma unroll
                    for (int t = 0; t < CT; ++t)
                        acc[g][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[t]), bl,
                                                                            acc[g][t], 0, 0, 0);
                }
            }
        };
        u32x4 va[CT], vb[CT];
        load_v(0, va);
        {
            // lambda_hat of row 32g + l32 lives in lane (32g + l32) % 64, slot (32g + l32) / 64
            // A row to which the tile added no mass (S = 0: every exponential
            // underflowed against a maximum that overshoots) keeps O and omega
            // in the same ratio, but lambda_hat can lie below fp32's range
            // while omega, in fp64, stays tiny: O would underflow to 0 and
            // 0 / omega give NaN.  Such factors are held in pend (fp64) and
            // applied with the next tile that adds mass, or at the end.  Each
            // wave keeps its own copy of the rows' factors in LDS.
            float lamf[QPL];
            bool scale = false;
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
                double *pd = pend + w * BQ + row[s];
                const double pv = *pd;
                if (S[s] > 0.0) {
                    lamf[s] = (float)(lam[s] * pv);
                    if (pv != 1.0) *pd = 1.0;
                } else {
                    lamf[s] = 1.0f;
                    *pd = pv * lam[s];
                }
                scale |= lamf[s] != 1.0f;
            }
            if (wave_any(scale)) {
#pragma unroll
                for (int g = 0; g < QG; ++g) {
                    const float lg = __shfl(lamf[g / 2 < QPL ? g / 2 : 0], ((g & 1) << 5) + l32, 64);
#pragma unroll
                    for (int t = 0; t < CT; ++t)
#pragma unroll
                        for (int r = 0; r < 16; ++r) acc[g][t][r] *= lg;
                }
            }
        }
        static_assert(NCH % 2 == 0, "chunks in pairs");
        for (int c16 = 0; c16 < NCH; c16 += 2) {
            load_v(c16 + 1, vb);
            pv_chunk(c16, va);
            if (c16 + 2 < NCH) load_v(c16 + 2, va);
            pv_chunk(c16 + 1, vb);
        }
    }

    // ---- epilogue: O / omega, lse = mu + ln(omega), mask bytes of skipped tiles
    {
        const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
        for (int g = 0; g < QG; ++g) {
            const double og = __shfl(om[g / 2 < QPL ? g / 2 : 0], ((g & 1) << 5) + l32, 64);
            const double pg = pend[w * BQ + g * 32 + l32];
            const float inv = (float)(pg / og);   // pg = 1 unless the last tiles added no mass
            const int jq = q0 + g * 32 + l32;
            if (jq >= p.N) continue;   // beyond N in a partial last block
            float *orow = p.o + (((size_t)b * p.Hq + h) * p.N + jq) * D + w * CPW;
#pragma unroll
            for (int t = 0; t < CT; ++t)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    const int c = t * 32 + r4 * 8 + half * 4;
                    const float4 v4 = make_float4(acc[g][t][r4 * 4 + 0] * inv, acc[g][t][r4 * 4 + 1] * inv,
                                                  acc[g][t][r4 * 4 + 2] * inv, acc[g][t][r4 * 4 + 3] * inv);
                    *reinterpret_cast<float4 *>(orow + c) = v4;
                }
        }
        if (w == 0)
#pragma unroll
            for (int s = 0; s < QPL; ++s)
                if (q0 + row[s] < p.N)
                    p.lse[((size_t)b * p.Hq + h) * p.N + q0 + row[s]] = (float)((double)mu[s] + ::log(om[s]));
        const int ntiles = p.Nk / KPT;
        for (int t = tid; t < ntiles; t += 64 * NW)
            if (t < t_begin || t > t_end)
                for (int th = 0; th < NK; ++th) mrow[t * NK + th] = PREC_INACTIVE;
    }
    if (p.stats) flush_stats<NK>(p.stats, stl, (uint32_t)(p.Nk / BK), tid);
}

// ------------------------------------------------------------------ launcher
template <int D, int BQ, int BK, int NK, bool SR, bool OBS>
static hipError_t launch_fwd_obs(const FwdParams &p, hipStream_t s)
{
    using C = Cfg<D, BQ, BK, NK>;
    auto kern = lamp_fwd_kernel<D, BQ, BK, NK, SR, OBS>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)(p.B * p.Hq * (p.Nq / BQ)));
    hipLaunchKernelGGL(kern, grid, dim3(64 * C::NW), C::LDS, s, p);
    return hipGetLastError();
}

template <int D, int BQ, int BK, int NK, bool SR = false>
static hipError_t launch_fwd(const FwdParams &p, hipStream_t s)
{
    if (p.dbg_y8 || p.dbg_y16) return launch_fwd_obs<D, BQ, BK, NK, SR, true>(p, s);
    return launch_fwd_obs<D, BQ, BK, NK, SR, false>(p, s);
}

#define LAMP_FWD_CASE(D_, BQ_, BK_, NK_) \
    if (D == D_ && BQ == BQ_ && BK == BK_ && NK == NK_) return launch_fwd<D_, BQ_, BK_, NK_>(p, s);

bool fwd_supported(int D, int BQ, int BK, int NK)
{
    // configurations built: d in {64,128,256}, bq in {64,128}, (bk, nk) in {(16,4), (64,4)}
    return (D == 64 || D == 128 || D == 256) && (BQ == 64 || BQ == 128) && (BK == 16 || BK == 64) && NK == 4;
}

bool fwd_grouped(int D, int BQ, int BK, int NK)
{
    (void)BQ;
    return BK == 16 && NK == 4 && D >= 128;
}

hipError_t dispatch_fwd(int D, int BQ, int BK, int NK, const FwdParams &p, hipStream_t s, bool *found)
{
    // 16-key sub-blocks with d >= 128: the kernel pipelined across key tiles
    if (fwd_grouped(D, BQ, BK, NK)) return dispatch_fwd16(D, BQ, p, s, found);
    *found = true;
    LAMP_FWD_CASE(64, 64, 16, 4)
    LAMP_FWD_CASE(64, 128, 16, 4)
#define LAMP_FWD_D(D_) LAMP_FWD_CASE(D_, 64, 64, 4) LAMP_FWD_CASE(D_, 128, 64, 4)
    LAMP_FWD_D(64)
    LAMP_FWD_D(128)
    LAMP_FWD_D(256)
#undef LAMP_FWD_D
    *found = false;
    return hipSuccess;
}

hipError_t dispatch_fwd_sr(int D, int BQ, int BK, int NK, const FwdParams &p, hipStream_t s, bool *found)
{
    // 16-key sub-blocks with d >= 128: the pipelined kernel's SR instantiations
    if (fwd_grouped(D, BQ, BK, NK)) return dispatch_fwd16_sr(D, BQ, p, s, found);
    *found = true;
#define LAMP_FWD_SR(D_, BQ_, BK_)                                            \
    if (D == D_ && BQ == BQ_ && BK == BK_ && NK == 4) return launch_fwd<D_, BQ_, BK_, 4, true>(p, s);
#define LAMP_FWD_SR_D(D_) LAMP_FWD_SR(D_, 64, 16) LAMP_FWD_SR(D_, 128, 16) LAMP_FWD_SR(D_, 64, 64) LAMP_FWD_SR(D_, 128, 64)
    LAMP_FWD_SR_D(64)
    LAMP_FWD_SR_D(128)
    LAMP_FWD_SR_D(256)
#undef LAMP_FWD_SR_D
#undef LAMP_FWD_SR
    *found = false;
    return hipSuccess;
}

} // namespace lamp
