// lamp_fwd16.hip -- the LampAttention forward kernel for 16-key sub-blocks
// (b_k = 16, N_k = 4, d in {128, 256}), software-pipelined across key tiles.
//
// Work split as in the general kernel: one workgroup of 4 waves per (batch,
// query head, query block of BQ rows); every lane holds QPL = BQ/64 query rows
// and every wave the running state of all BQ rows; wave w owns sub-block w of
// every 64-key tile and the output channel slice [w*D/4, (w+1)*D/4).
//
// Pipelining.  The 8-bit logits of tile t+1 do not depend on any decision
// taken in tile t.  Stage 1 of tile t needs the 16-bit logits of the
// sub-blocks that fail the margin test against the running maximum mu after
// tile t-1 (the set F0; the test is monotone in mu_hat and mu_hat only grows,
// so every sub-block stage 1 recomputes is in F0; one that is not takes the
// one-at-a-time path).  So one fused pass over the channels computes the
// 16-bit logits of F0(t) (4 keys of each member per wave, codes kept in
// registers) together with the 8-bit logits of this wave's sub-block of tile
// t+1 (codes to the other half of a double-buffered LDS array).  Per tile:
//   A. fused pass: 16-bit logits of F0(t), 8-bit logits of tile t+1;
//      16-bit column maxima merged with LDS atomic max (exact fixed point:
//      e4m11 values are multiples of 2^-17 below 2^9);
//   B. barrier;
//   C. stage 1 of tile t (Sec. 3.1, Eq. (7)) on the column maxima;
//   D. exponentials of tile t (8-bit LUT in LDS, 16-bit table of exact bf16
//      high and low parts in global memory);
//   E. barrier; lambda_hat, omega_hat, stage 2 (Eq. (8));
//   G. state update, P.V on the bf16 matrix cores, F0(t+1);
//   I. barrier (the code buffer of tile t is reused by tile t+2).
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <climits>
#include <type_traits>

#include "lamp_device.h"
#include "lamp_kernels.h"
#include "lamp_loops.h"
#include "lamp_sr.h"
#include "lamp_stats.h"

#ifndef LAMP_MIN_WAVES
#define LAMP_MIN_WAVES 2
#endif

namespace lamp {

// Phase timer (a build with -DLAMP_PHASE_TIMER, for measurement only): every
// wave adds the shader-clock cycles it spends in each phase of the tile loop
// to phase_cycles[0..PHASE_N-1] (word PHASE_N counts the waves); read and
// cleared by lamp_phase_read.  Phases: 0 fused pass, 1 code and maxima
// emission, 2 barrier B, 3 stage 1, 4 exponentials, 5 barrier E, 6 rescale
// and stage 2, 7 P.V and the next speculative set, 8 barrier I, 9 prologue
// and epilogue.  (Not in the stochastic-rounding instantiations, which are
// compiled in a unit of their own, lamp_fwd16_sr.hip.)
#if defined(LAMP_PHASE_TIMER) && !defined(LAMP_FWD16_NO_LAUNCHERS)
__device__ unsigned long long phase_cycles[PHASE_N + 1];
#define LAMP_PH_INIT                                                              \
    __shared__ uint32_t ph_lds[4 * PHASE_N];                                      \
    if (lane < PHASE_N) ph_lds[w * PHASE_N + lane] = 0u;                          \
    uint32_t ph_t = (uint32_t)__builtin_readcyclecounter();
#define LAMP_PH(i)                                                                \
    do {                                                                          \
        const uint32_t ph_n = (uint32_t)__builtin_readcyclecounter();             \
        if (lane == 0) ph_lds[w * PHASE_N + (i)] += ph_n - ph_t;                  \
        ph_t = ph_n;                                                              \
    } while (0)
#define LAMP_PH_FLUSH                                                             \
    do {                                                                          \
        LAMP_PH(9);                                                               \
        if (lane < PHASE_N) atomicAdd(&phase_cycles[lane], (unsigned long long)ph_lds[w * PHASE_N + lane]); \
        if (lane == PHASE_N) atomicAdd(&phase_cycles[PHASE_N], 1ull);             \
    } while (0)
#else
#define LAMP_PH_INIT
#define LAMP_PH(i) ((void)0)
#define LAMP_PH_FLUSH ((void)0)
#endif

#ifndef LAMP_FWD16_NO_LAUNCHERS
hipError_t phase_read(unsigned long long *host, bool reset)
{
#ifdef LAMP_PHASE_TIMER
    hipError_t e = hipMemcpyFromSymbol(host, HIP_SYMBOL(phase_cycles), sizeof(phase_cycles));
    if (e == hipSuccess && reset) {
        static const unsigned long long zero[PHASE_N + 1] = {};
        e = hipMemcpyToSymbol(HIP_SYMBOL(phase_cycles), zero, sizeof(phase_cycles));
    }
    return e;
#else
    (void)host;
    (void)reset;
    return hipErrorNotSupported;
#endif
}
#endif

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

enum { PREC_LOW = 0, PREC_S1 = 1, PREC_S2 = 2, PREC_INACTIVE = 3 };


template <int D, int BQ>
struct Cfg16 {
    static constexpr int NK = 4, BK = 16, KPT = 64, NW = 4;
    static constexpr int QPL = BQ / 64;       // query rows per lane
    static constexpr int CPW = D / NW;        // output channels per wave
    static constexpr int CT = CPW / 32;       // 32-channel MFMA tiles per wave
    static constexpr int QG = BQ / 32;        // 32-row MFMA groups
    static constexpr int YP = KPT + 8;        // LDS pitch (u16) of the code rows
    static constexpr size_t YB = (size_t)BQ * YP * 2;
    static constexpr size_t OFF_Y = 0;                                  // u16 [2][BQ][YP]
    static constexpr size_t OFF_YL = OFF_Y + 2 * YB;                    // u16 [BQ][YP]
    static constexpr size_t OFF_LUT = OFF_YL + YB;                      // u16 [256]
    static constexpr size_t OFF_M8 = OFF_LUT + 512;                     // f32 [2][NK][BQ]
    static constexpr size_t OFF_CMI = OFF_M8 + (size_t)2 * NK * BQ * 4;  // i32 [2][NK][BQ]
    static constexpr size_t CMF = (size_t)2 * NW * BQ * 4 > (size_t)NK * BQ * 8 ? (size_t)2 * NW * BQ * 4
                                                                                  : (size_t)NK * BQ * 8;
    static constexpr size_t OFF_CMF = OFF_CMI + (size_t)2 * NK * BQ * 4;  // f32 [2][NW][BQ] | f64 [NK][BQ]
    static constexpr size_t OFF_SP = OFF_CMF + CMF;                     // f64 [2][NW][BQ]
    static constexpr size_t OFF_ED = OFF_SP + (size_t)2 * NW * BQ * 8;  // f64 [EXPDOC_NK]
    static constexpr size_t OFF_TS = OFF_ED + (size_t)EXPDOC_NK * 8;    // i32 [2][NK] sub-block threats
    static constexpr size_t OFF_ST = OFF_TS + (size_t)2 * NK * 4;       // u32 [ST_N] statistics
    static constexpr size_t OFF_PD = OFF_ST + (size_t)ST_N * 4;         // f64 [NW][BQ] pending rescale factors
    static constexpr size_t LDS = OFF_PD + (size_t)NW * BQ * 8;
    static_assert(BQ == 64 || BQ == 128, "64 or 128 query rows per block");
    static_assert(CPW % 32 == 0, "whole 32-channel tiles per wave");
};

// e4m11 / e4m3 values as exact fixed point in units of 2^-17 (|y| < 2^9).
__device__ __forceinline__ int fx_of(float y) { return (int)(y * 131072.0f); }
__device__ __forceinline__ float fx_value(int f) { return (float)f * (1.0f / 131072.0f); }

// Keys of the 16-bit column maxima merged by integer atomic max: exact fixed
// point for e4m11, the order-preserving map of the FP32 pattern in the SIM
// profile (whose values span FP32's range).
template <bool SIMP>
__device__ __forceinline__ int cm_key(float y)
{
    if constexpr (SIMP) return ord_of(y);
    else return fx_of(y);
}

// fx_of of an e4m11 code, from the code: the significand (with its implicit
// bit when normal) shifted by max(ex, 1) - 1.
__device__ __forceinline__ int e4m11_fx(uint32_t code)
{
    const uint32_t ex = (code >> 11) & 0xFu, m = code & 0x7FFu;
    const int mag = ex ? (int)((m | 0x800u) << (ex - 1u)) : (int)m;
    return (code & 0x8000u) ? -mag : mag;
}

template <bool SIMP>
__device__ __forceinline__ float cm_value(int f)
{
    if constexpr (SIMP) return ord_value(f);
    else return fx_value(f);
}

// SIM 16-bit logits in LDS: the high and low 16 bits of the FP32 patterns of
// two keys, in the code row and the low row.
__device__ __forceinline__ uint32_t pack_hi16(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t pack_lo16(uint32_t a, uint32_t b) { return (a & 0xFFFFu) | (b << 16); }

// The low bf16 parts E - hi of 8 SIM 16-bit exponentials kept as the high and
// low halves of their FP32 patterns (E has 12 significant bits, so E - hi is
// exact in fp32 and has at most 4; its bf16 truncation is exact down to 2^-133).
__device__ __forceinline__ u32x4 lo_bf16x8(const u32x4 &h, const u32x4 &l)
{
    u32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t hk = h[k], lk = l[k];
        const float g0 = __builtin_bit_cast(float, hk << 16), g1 = __builtin_bit_cast(float, hk & 0xFFFF0000u);
        const float e0 = __builtin_bit_cast(float, (hk << 16) | (lk & 0xFFFFu));
        const float e1 = __builtin_bit_cast(float, (hk & 0xFFFF0000u) | (lk >> 16));
        r[k] = (__builtin_bit_cast(uint32_t, e0 - g0) >> 16) | (__builtin_bit_cast(uint32_t, e1 - g1) & 0xFFFF0000u);
    }
    return r;
}

// Maximum of an int over the wave, returned to every lane: DPP exchanges inside
// each 16-lane row (quad swaps, then rotations by 4 and 8), then the four row
// maxima through scalar registers.
__device__ __forceinline__ int wave_max_i32(int v)
{
    int o = __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false);    // quad_perm [1,0,3,2]
    v = o > v ? o : v;
    o = __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false);        // quad_perm [2,3,0,1]
    v = o > v ? o : v;
    o = __builtin_amdgcn_update_dpp(v, v, 0x124, 0xF, 0xF, false);       // row_ror:4
    v = o > v ? o : v;
    o = __builtin_amdgcn_update_dpp(v, v, 0x128, 0xF, 0xF, false);       // row_ror:8
    v = o > v ? o : v;
    const int a = __builtin_amdgcn_readlane(v, 0), b = __builtin_amdgcn_readlane(v, 16);
    const int c = __builtin_amdgcn_readlane(v, 32), d = __builtin_amdgcn_readlane(v, 48);
    const int ab = a > b ? a : b, cd = c > d ? c : d;
    return ab > cd ? ab : cd;
}

} // namespace

// OBS: the instantiation that also writes the logit observables (p.dbg_y8,
// p.dbg_y16); the same code otherwise, kept apart so that the stores do not
// change the register allocation of the instantiations that do not.
// CMP: the compact register layout (Sec. 3.3, "Register layout"): the fused
// pass keeps the 8-bit codes four per register and computes the 16-bit logits
// of at most one speculative sub-block; when two or more are flagged (a
// "disruptive" tile) the others follow in a sequential 16-bit pass once the
// 8-bit codes are stored.  A schedule only: the results are those of the safe
// layout.
// SR: the 8-bit logits rounded stochastically (lamp_sr.h, sr8_chunk_bc) with
// the generator keyed by p.seed; they run after the fused pass, which then
// carries the speculative 16-bit logits alone.
template <int D, int BQ, int MODE, bool SIMP, bool OBS, bool CMP, bool SR = false>
__global__ __launch_bounds__(256, LAMP_MIN_WAVES) void lamp_fwd16_kernel(FwdParams p)
{
    using C = Cfg16<D, BQ>;
    constexpr int NK = C::NK, BK = C::BK, KPT = C::KPT, NW = C::NW, QPL = C::QPL, CPW = C::CPW;
    constexpr int CT = C::CT, QG = C::QG, YP = C::YP;
    constexpr int WPM = SIMP ? 4 : 2;   // words of 16-bit logits per 4 keys (SIM: FP32 patterns)

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t *ycode2 = reinterpret_cast<uint16_t *>(smem + C::OFF_Y);   // [2][BQ][YP] logit codes, then E
    uint16_t *ylo = reinterpret_cast<uint16_t *>(smem + C::OFF_YL);     // [BQ][YP] low bf16 part of E16
    uint16_t *lut = reinterpret_cast<uint16_t *>(smem + C::OFF_LUT);    // [256] 8-bit exp (bf16 bits; SIM table)
    float *m8s2 = reinterpret_cast<float *>(smem + C::OFF_M8);          // [2][NK][BQ] 8-bit column maxima
    int *cmi2 = reinterpret_cast<int *>(smem + C::OFF_CMI);             // [2][NK][BQ] 16-bit column maxima
    float *cmf = reinterpret_cast<float *>(smem + C::OFF_CMF);          // [2][NW][BQ] one-at-a-time maxima
    double *cst_lds = reinterpret_cast<double *>(smem + C::OFF_CMF);    // [NK][BQ] stage-2 costs (same space)
    double *sps = reinterpret_cast<double *>(smem + C::OFF_SP);         // [NW][BQ] partial row sums of E
    double *spf = sps + NW * BQ;                                        // [NW][BQ] over 8-bit sub-blocks
    double *edk = reinterpret_cast<double *>(smem + C::OFF_ED);         // exp_doc constants
    int *tsl = reinterpret_cast<int *>(smem + C::OFF_TS);               // [2][NK] threats of a tile
    uint32_t *stl = reinterpret_cast<uint32_t *>(smem + C::OFF_ST);    // [ST_N] statistics (p.stats)
    double *pend = reinterpret_cast<double *>(smem + C::OFF_PD);        // [NW][BQ] pending factors (G below)

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;   // w is wave-uniform
    LAMP_PH_INIT
    const int nqb = p.Nq / BQ;   // query blocks per head (the last may be partial)
    // Block order.  Workgroups are handed to the 8 XCDs round-robin (block i to
    // XCD i mod 8), each XCD with its own L2.  When the B*Hkv key/value heads
    // split evenly over the XCDs, XCD x takes the heads x, x+8, ... and runs the
    // query heads of one group next to each other, so the keys and values
    // they share stay in that XCD's L2; every XCD walks the query blocks
    // longest first (causality).  Otherwise: longest first over all heads.
    const int G = p.Hq / p.Hkv, KH = p.B * p.Hkv;
    int qb, b, h, hk;
    if (KH % 8 == 0) {
        const int x = (int)(blockIdx.x % 8u), r = (int)(blockIdx.x / 8u);
        const int per = (KH / 8) * G;             // blocks of one query-block rank on an XCD
        const int qrank = r / per, rest = r % per;
        const int j = x + 8 * (rest / G);         // key/value head, over the batch
        qb = nqb - 1 - qrank;
        b = j / p.Hkv;
        hk = j % p.Hkv;
        h = hk * G + rest % G;
    } else {
        const int BH = p.B * p.Hq;
        qb = nqb - 1 - (int)(blockIdx.x / BH);   // longest blocks first under causality
        const int bh = blockIdx.x % BH;
        b = bh / p.Hq;
        h = bh % p.Hq;
        hk = h / G;
    }
    const int q0 = qb * BQ;
    const float NEG_INF = -__builtin_inff();
    constexpr int mode = MODE;   // one instantiation per mode: only its path is compiled
    const bool stage1_off = (p.flags & LAMP_STAGE1_OFF) != 0u;   // flags are 0 outside the threshold mode
    const bool mu_trunc = (p.flags & LAMP_MU_TRUNC) != 0u;

    int row[QPL], vlo[QPL], vhi[QPL], jq[QPL];
    const float *qrow[QPL];
#pragma unroll
    for (int s = 0; s < QPL; ++s) {
        row[s] = s * 64 + lane;
        const int j = q0 + row[s];
        jq[s] = j;
        vlo[s] = p.window > 0 ? (j - p.window + 1 > 0 ? j - p.window + 1 : 0) : 0;
        vhi[s] = p.causal ? j : p.N - 1;
        if (j >= p.N) {   // a row beyond N (partial last block): no visible key
            vlo[s] = p.N;
            vhi[s] = -1;
        }
        // grouped layout: 64-row blocks stored [group][row][4] (zero-padded rows, in bounds)
        qrow[s] = p.qt + ((size_t)b * p.Hq + h) * p.Nq * D + (size_t)(j / 64) * 64 * D + (j % 64) * 4;
    }
    const int bv_lo = p.window > 0 ? (q0 - p.window + 1 > 0 ? q0 - p.window + 1 : 0) : 0;
    const int bv_hi = p.causal ? (q0 + BQ - 1 < p.N - 1 ? q0 + BQ - 1 : p.N - 1) : p.N - 1;
    const int t_begin = bv_lo / KPT, t_end = bv_hi / KPT;   // every tile in between has a visible pair

    const float *kt32 = p.kt32 + ((size_t)b * p.Hkv + hk) * (size_t)p.Nk * D;   // fp32 keys, grouped layout
    // row of key i in the grouped layout (16-key blocks stored [group][key][4])
    auto krow_of = [&](int i) { return kt32 + (size_t)(i / 16) * 16 * D + (i % 16) * 4; };
    const uint16_t *vtbase = p.vt + ((size_t)b * p.Hkv + hk) * (size_t)D * p.Nk;    // V^T [D][Nk]
    uint8_t *mrow = p.mask + (((size_t)b * p.Hq + h) * nqb + qb) * (size_t)(p.Nk / BK);

    for (int i = tid; i < 256; i += 256) lut[i] = SIMP ? p.sim8[i] : p.lut8e[i];
    if (tid < EXPDOC_NK) edk[tid] = EXPDOC_K[tid];
    for (int i = tid; i < 2 * NK * BQ; i += 256) cmi2[i] = INT_MIN;
    if (tid < ST_N) stl[tid] = 0u;
    for (int i = tid; i < NW * BQ; i += 256) pend[i] = 1.0;
    // logit observables (tests): this query block is observed (uniform)
    const bool dbg_blk = qb >= p.dbg_qb0 && qb < p.dbg_qb0 + p.dbg_nqb;
    const bool dbg8 = OBS && !SIMP && p.dbg_y8 != nullptr && dbg_blk;
    const bool dbg16 = OBS && !SIMP && p.dbg_y16 != nullptr && dbg_blk;
    auto dbg_off = [&](int s) -> size_t {
        return ((((size_t)b * p.Hq + h) * p.dbg_nqb + (qb - p.dbg_qb0)) * BQ + row[s]) * (size_t)p.Nk;
    };

    float mu[QPL];
    double om[QPL];
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
    auto ycode_of = [&](int tile) { return ycode2 + (size_t)(tile & 1) * BQ * YP; };
    auto m8s_of = [&](int tile) { return m8s2 + (size_t)(tile & 1) * NK * BQ; };
    auto cmi_of = [&](int tile) { return cmi2 + (size_t)(tile & 1) * NK * BQ; };

    // active sub-blocks of a tile (a visible pair anywhere in the block), uniform
    auto active_of = [&](int tile) {
        uint32_t a = 0;
#pragma unroll
        for (int th = 0; th < NK; ++th) {
            const int k = tile * KPT + th * BK, z = k + BK - 1;
            bool any = false;
#pragma unroll
            for (int s = 0; s < QPL; ++s) any |= (k <= vhi[s] && z >= vlo[s]);
            if (wave_any(any)) a |= 1u << th;
        }
        return a;
    };
    // does this wave's sub-block of `tile` have a visible pair (then it is emulated)?
    auto own_emulated = [&](int tile, uint32_t act) {
        const int ck0 = tile * KPT + w * BK;
        return (act >> w & 1u) && !(ck0 > bv_hi || ck0 + 15 < bv_lo);
    };
    // 8-bit codes of this wave's sub-block of `tile` into its code buffer, the
    // column maxima over visible keys into m8s (NEG_INF for a sub-block that
    // was not emulated)
    auto emit8 = [&](int tile, const uint32_t (&a8)[QPL][8], bool done, const uint32_t (&sat)[QPL]) {
        const int ck0 = tile * KPT + w * BK;
        uint16_t *yc = ycode_of(tile);
        float *m8s = m8s_of(tile);
        bool full = true;
#pragma unroll
        for (int s = 0; s < QPL; ++s) full &= ck0 >= vlo[s] && ck0 + 15 <= vhi[s];
        if constexpr (!SIMP) {
            // visible keys of the 16 in each slot (for the observables)
            auto vis16 = [&](int s) {
                uint32_t m = 0;
#pragma unroll
                for (int i = 0; i < 16; ++i) m |= (visible(s, ck0 + i) ? 1u : 0u) << i;
                return m;
            };
            if (done && p.stats) {
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
            if (done && dbg8) {
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
                    *reinterpret_cast<u32x4 *>(p.dbg_y8 + dbg_off(s) + ck0) = u32x4{wd[0], wd[1], wd[2], wd[3]};
                }
            }
        }
        // FULL: every key of the sub-block visible to every row of the wave
        // (a uniform branch), so no per-key visibility test
        auto run = [&](auto full_c) {
            constexpr bool FULL = decltype(full_c)::value;
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
                float mx = NEG_INF;
                if (done) {
                    uint32_t packed[8];
#pragma unroll
                    for (int pp = 0; pp < 8; ++pp) {
                        const float2 yv = SIMP ? make_float2(bf16_value(a8[s][pp] & 0xFFFFu),
                                                             bf16_value(a8[s][pp] >> 16))
                                               : unpk_e4m3(a8[s][pp]);
                        const int i0 = ck0 + 2 * pp;
                        // invisible keys enter as -inf, by selection rather than branches
                        const float x0 = (FULL || visible(s, i0)) ? yv.x : NEG_INF;
                        const float x1 = (FULL || visible(s, i0 + 1)) ? yv.y : NEG_INF;
                        mx = x0 > mx ? x0 : mx;
                        mx = x1 > mx ? x1 : mx;
                        packed[pp] = SIMP ? a8[s][pp] : (a8[s][pp] & 0xFFu) | ((a8[s][pp] & 0xFF00u) << 8);
                    }
                    u32x4 *dst = reinterpret_cast<u32x4 *>(yc + row[s] * YP + w * BK);
                    dst[0] = u32x4{packed[0], packed[1], packed[2], packed[3]};
                    dst[1] = u32x4{packed[4], packed[5], packed[6], packed[7]};
                }
                m8s[w * BQ + row[s]] = mx;
            }
        };
        if (!wave_any(!full)) run(std::true_type());
        else run(std::false_type());
    };
    // the margin test of every sub-block of `tile` against mu_hat (Eq. (7)):
    // mu_hat_j > fma(|mu_hat_j|, delta, m8); columns without a visible entry
    // are not tested; mu_hat = -inf fails.  m8 from LDS, identical in every wave.
    auto fails_of = [&](const float (&m8)[NK][QPL], const float (&mh)[QPL]) {
        uint32_t f = 0;
#pragma unroll
        for (int th = 0; th < NK; ++th) {
            bool bad = false;
#pragma unroll
            for (int s = 0; s < QPL; ++s)
                if (m8[th][s] > NEG_INF) {
                    const double m = (double)mh[s];
                    bad |= !(m > __builtin_fma(__builtin_fabs(m), p.delta, (double)m8[th][s]));
                }
            if (wave_any(bad)) f |= 1u << th;
        }
        return f;
    };
    auto load_m8 = [&](int tile, float (&m8)[NK][QPL]) {
        const float *m8s = m8s_of(tile);
#pragma unroll
        for (int th = 0; th < NK; ++th)
#pragma unroll
            for (int s = 0; s < QPL; ++s) m8[th][s] = m8s[th * BQ + row[s]];
    };
    // Threat of this wave's sub-block of `tile` against the running maximum mu
    // (the stage-1 ordering of Eq. (7)): T = max over rows with a visible 8-bit
    // logit of (m8 - mu), +inf where mu = -inf.  With the formats of Sec. 3.3
    // both are multiples of 2^-17 below 2^9, so T is exact as an int in those
    // units (INT_MAX for +inf, INT_MIN when no row has a visible logit).  Each
    // wave computes the threat of its own sub-block after the tile before
    // `tile` is complete, and the stage-1 test of `tile` reads all four.
    auto own_threat = [&](int tile) {
        if constexpr (!SIMP) {
            const float *m8s = m8s_of(tile);
            int tv = INT_MIN;
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
                const float m8v = m8s[w * BQ + row[s]];
                const bool vis = m8v > NEG_INF, muinf = mu[s] == NEG_INF;   // infinities never converted
                const int d = muinf ? INT_MAX : fx_of(vis ? m8v : 0.0f) - fx_of(muinf ? 0.0f : mu[s]);
                tv = (vis && d > tv) ? d : tv;
            }
            const int T = wave_max_i32(tv);
            if (lane == 0) tsl[(tile & 1) * NK + w] = T;
        }
    };
    // the set of sub-blocks whose 16-bit logits the next fused pass computes
    auto f0_of = [&](int tile, uint32_t act) -> uint32_t {
        if (mode == MODE_ALL16) return act;
        if (mode == MODE_PURE8 || stage1_off) return 0u;
        float m8[NK][QPL];
        load_m8(tile, m8);
        return fails_of(m8, mu);
    };
    // one-at-a-time 16-bit recompute of sub-block th of the tile at k0 shared
    // by all waves (4 keys each); fn(key0, codes[QPL][2]) receives the codes
    auto shared16 = [&](int k0, int th, auto fn) {
        const int key0 = k0 + th * BK + w * 4;
        if (key0 > bv_hi || key0 + 3 < bv_lo) return;   // nothing visible in the block
        uint32_t yc[QPL][WPM];
        rec16_keys<D, QPL, 4, SIMP, GrpLay>(qrow, krow_of(key0 + (lane & 3)), yc);
        fn(key0, yc);
    };
    // a 16-bit exponential from the table in global memory as bf16 high / low
    // parts (SIM: high / low halves of the FP32 pattern) and the value (the
    // 8-bit ones are formed inline in the exponential phase)
    auto e16_of = [&](float mref, float y, uint32_t &eh, uint32_t &el) -> float {
        if constexpr (SIMP) {
            const uint32_t eb = p.sim16[sim_shift_index<11, SIM16_EMIN, SIM16_EMAX>(mref, y)];
            eh = eb >> 16;
            el = eb & 0xFFFFu;
            return __builtin_bit_cast(float, eb);
        } else {
            const uint32_t hl = p.exp16hl[ue5m11_code(shift_of(mref, y))];
            eh = hl & 0xFFFFu;
            el = hl >> 16;
            return bf16_value(eh) + bf16_value(el);   // exact
        }
    };
    // Observables of the 16-bit logits of 4 keys from key0 of every slot
    // (codes two per word, as the recomputes leave them): their codes for the
    // tests, and the saturated ones among the visible keys whose code is the
    // largest e4m11 magnitude (the FP32 chain rerun for those alone).
    auto obs16 = [&](int key0, const uint32_t (&yc)[QPL][WPM]) {
        if constexpr (!SIMP) {
            if (dbg16) {
#pragma unroll
                for (int s = 0; s < QPL; ++s) {
                    uint32_t wd[2];
#pragma unroll
                    for (int x = 0; x < 2; ++x) {
                        const uint32_t lo = visible(s, key0 + 2 * x) ? (yc[s][x] & 0xFFFFu) : 0xFFFFu;
                        const uint32_t hi = visible(s, key0 + 2 * x + 1) ? (yc[s][x] >> 16) : 0xFFFFu;
                        wd[x] = lo | (hi << 16);
                    }
                    *reinterpret_cast<uint2 *>(p.dbg_y16 + dbg_off(s) + key0) = make_uint2(wd[0], wd[1]);
                }
            }
            if (p.stats) {
                uint32_t atmax = 0;   // bit 4s + i: slot s, key key0 + i
#pragma unroll
                for (int s = 0; s < QPL; ++s)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const uint32_t code = (yc[s][i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
                        atmax |= ((code & 0x7FFFu) == 0x7FFFu && visible(s, key0 + i) ? 1u : 0u) << (4 * s + i);
                    }
                if (wave_any(atmax != 0u)) {
                    uint32_t n = 0;
                    for (uint32_t m = atmax; m; m &= m - 1) {
                        const int bit = __builtin_ctz(m);
                        const float *qr = qrow[0];
#pragma unroll
                        for (int s = 1; s < QPL; ++s) qr = bit / 4 == s ? qrow[s] : qr;
                        n += y16_saturates<D, GrpLay>(qr, krow_of(key0 + bit % 4)) ? 1u : 0u;
                    }
                    if (n) atomicAdd(&stl[ST_SAT16], n);
                }
            }
        }
    };
    // SIM profile: the row sum of the tile's exponentials, keys ascending,
    // one fp64 addition at a time, from the values in LDS (hmask: the
    // sub-blocks holding 16-bit exponentials)
    auto seq_sum = [&](const uint16_t *yc, int s, uint32_t hmask) -> double {
        double tt = 0.0;
#pragma unroll
        for (int c = 0; c < NK; ++c) {
            const u32x4 *hp = reinterpret_cast<const u32x4 *>(yc + row[s] * YP + c * BK);
            const u32x4 h0 = hp[0], h1 = hp[1];
            u32x4 l0 = u32x4{0u, 0u, 0u, 0u}, l1 = l0;
            if (hmask >> c & 1u) {
                const u32x4 *lp = reinterpret_cast<const u32x4 *>(ylo + row[s] * YP + c * BK);
                l0 = lp[0];
                l1 = lp[1];
            }
            const uint32_t hw[8] = {h0[0], h0[1], h0[2], h0[3], h1[0], h1[1], h1[2], h1[3]};
            const uint32_t lw[8] = {l0[0], l0[1], l0[2], l0[3], l1[0], l1[1], l1[2], l1[3]};
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const uint32_t hb = (hw[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
                const uint32_t lb = (lw[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
                tt += (double)__builtin_bit_cast(float, (hb << 16) | lb);
            }
        }
        return tt;
    };

    // ---- prologue: 8-bit logits of the first tile, its F0
    int t = t_begin;
    uint32_t act = active_of(t);
    if (mode != MODE_ALL16) {
        const bool done = own_emulated(t, act);
        uint32_t a8[QPL][8], sat[QPL];
        if (done) {
            if constexpr (SR)
                sr8_chunk_bc<D, QPL, GrpLay>(qrow, kt32 + (size_t)(t * KPT + w * BK) * D, jq, (uint32_t)(t * KPT + w * BK),
                                             (uint32_t)(b * p.Hq + h), p.seed, a8, sat);
            else emu8_any<D, QPL, SIMP, GrpLay>(qrow, kt32 + (size_t)(t * KPT + w * BK) * D, a8, sat);
        }
        emit8(t, a8, done, sat);
    }
    __syncthreads();
    uint32_t F0 = f0_of(t, act);
    if (mode == MODE_LAMP && !stage1_off) own_threat(t);

    for (; t <= t_end; ++t) {
        const int k0 = t * KPT;
        const bool has_next = t < t_end;
        const uint32_t act_next = has_next ? active_of(t + 1) : 0u;
        uint16_t *ycode = ycode_of(t);

        // ---- A. fused pass: 16-bit logits of F0 (4 keys of each member per
        // wave), 8-bit logits of this wave's sub-block of the next tile
        uint32_t y16r[QPL][4 * WPM];   // 16-bit logits of keys th*16 + w*4 + {0..3} of the g-th member of F0
        {
            const int nf_all = __builtin_popcount(F0);
            const int nf = CMP ? (nf_all < 1 ? nf_all : 1) : nf_all;   // members in the fused pass
            const int kk = nf ? (lane & 15) % (4 * nf) : 0;
            int thg = 0;
            if (nf) {
                uint32_t m = F0;
                for (int g = 0; g < kk / 4; ++g) m &= m - 1;
                thg = __builtin_ctz(m);
            }
            const float *krowr = krow_of(k0 + thg * BK + w * 4 + (kk & 3));
            const bool emu = mode != MODE_ALL16 && has_next && own_emulated(t + 1, act_next);
            const float *k32e = kt32 + (size_t)(k0 + KPT + w * BK) * D;   // read only when emu (then below N)
            uint32_t a8[QPL][8], sat8[QPL];
            auto run = [&](auto nkey_c, auto emu_c) {
                constexpr int NKEY = decltype(nkey_c)::value;
                constexpr bool EMU = decltype(emu_c)::value;
                uint32_t c[QPL][y16_words<SIMP>(NKEY)];
                fused_pass<D, QPL, NKEY, EMU, SIMP, GrpLay, CMP>(qrow, k32e, krowr, a8, c, sat8);
                if constexpr (NKEY > 0)
#pragma unroll
                    for (int s = 0; s < QPL; ++s)
#pragma unroll
                        for (int pp = 0; pp < y16_words<SIMP>(NKEY); ++pp) y16r[s][pp] = c[s][pp];
            };
            using T_ = std::true_type;
            using F_ = std::false_type;
            using std::integral_constant;
            if (emu && !SR) {
                switch (nf) {
                case 0: run(integral_constant<int, 0>(), T_()); break;
                case 1: run(integral_constant<int, 4>(), T_()); break;
                case 2: run(integral_constant<int, 8>(), T_()); break;
                case 3: run(integral_constant<int, 12>(), T_()); break;
                default: run(integral_constant<int, 16>(), T_()); break;
                }
            } else {
                switch (nf) {
                case 0: break;
                case 1: run(integral_constant<int, 4>(), F_()); break;
                case 2: run(integral_constant<int, 8>(), F_()); break;
                case 3: run(integral_constant<int, 12>(), F_()); break;
                default: run(integral_constant<int, 16>(), F_()); break;
                }
            }
            if constexpr (SR)
                if (emu)
                    sr8_chunk_bc<D, QPL, GrpLay>(qrow, k32e, jq, (uint32_t)(k0 + KPT + w * BK), (uint32_t)(b * p.Hq + h),
                                                 p.seed, a8, sat8);
            LAMP_PH(0);
            if (has_next && mode != MODE_ALL16) emit8(t + 1, a8, emu, sat8);
            if constexpr (CMP) {
                // a disruptive tile: the other members of F0 in a sequential
                // 16-bit pass (4 keys of each per wave, as in the fused pass)
                if (nf_all >= 2) {
                    const int nr = nf_all - 1;
                    const int kb = (lane & 15) % (4 * nr);
                    uint32_t m = F0 & (F0 - 1u);   // without the member of the fused pass
                    for (int g = 0; g < kb / 4; ++g) m &= m - 1;
                    const float *krow = krow_of(k0 + __builtin_ctz(m) * BK + w * 4 + (kb & 3));
                    auto seq = [&](auto nkey_c) {
                        constexpr int NKEY = decltype(nkey_c)::value;
                        uint32_t c[QPL][y16_words<SIMP>(NKEY)];
                        rec16_keys<D, QPL, NKEY, SIMP, GrpLay>(qrow, krow, c);
#pragma unroll
                        for (int s = 0; s < QPL; ++s)
#pragma unroll
                            for (int pp = 0; pp < y16_words<SIMP>(NKEY); ++pp) y16r[s][WPM + pp] = c[s][pp];
                    };
                    switch (nr) {
                    case 1: seq(std::integral_constant<int, 4>()); break;
                    case 2: seq(std::integral_constant<int, 8>()); break;
                    default: seq(std::integral_constant<int, 12>()); break;
                    }
                }
            }
            // 16-bit column maxima over this wave's 4 keys of every member of F0
            int *cmi = cmi_of(t);
            uint32_t m = F0;
#pragma unroll
            for (int g = 0; g < NK; ++g) {
                if (!m) break;
                const int th = __builtin_ctz(m);
                m &= m - 1;
                const int key0 = k0 + th * BK + w * 4;
#pragma unroll
                for (int s = 0; s < QPL; ++s) {
                    int cm = INT_MIN;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        int f;
                        if constexpr (SIMP) f = cm_key<SIMP>(y16_value<SIMP>(&y16r[s][g * WPM], i));
                        else f = e4m11_fx((y16r[s][g * WPM + (i >> 1)] >> (16 * (i & 1))) & 0xFFFFu);
                        cm = (visible(s, key0 + i) && f > cm) ? f : cm;
                    }
                    if (cm != INT_MIN) atomicMax(&cmi[th * BQ + row[s]], cm);
                }
            }
        }
        LAMP_PH(1);
        __syncthreads();   // B: codes, m8 of the next tile and the 16-bit maxima are complete
        LAMP_PH(2);

        // ---- C. running maximum mu_hat and stage 1 of tile t
        float muh[QPL];
#pragma unroll
        for (int s = 0; s < QPL; ++s) muh[s] = mu[s];
        uint32_t prec16 = 0;   // stage-1 (or threshold-0) sub-blocks
        float cm16[NK][QPL];   // 16-bit column maxima of the members of F0
        {
            const int *cmi = cmi_of(t);
#pragma unroll
            for (int th = 0; th < NK; ++th)
#pragma unroll
                for (int s = 0; s < QPL; ++s) {
                    const int f = (F0 >> th & 1u) ? cmi[th * BQ + row[s]] : INT_MIN;
                    cm16[th][s] = f == INT_MIN ? NEG_INF : cm_value<SIMP>(f);
                }
        }
        if (mode == MODE_PURE8 || stage1_off) {   // running maximum over the 8-bit logits
            float m8[NK][QPL];
            load_m8(t, m8);
#pragma unroll
            for (int s = 0; s < QPL; ++s)
#pragma unroll
                for (int th = 0; th < NK; ++th) muh[s] = m8[th][s] > muh[s] ? m8[th][s] : muh[s];
        } else if (mode == MODE_ALL16) {
            prec16 = act;
#pragma unroll
            for (int s = 0; s < QPL; ++s)
#pragma unroll
                for (int th = 0; th < NK; ++th) muh[s] = cm16[th][s] > muh[s] ? cm16[th][s] : muh[s];
        } else {
            float m8[NK][QPL];
            load_m8(t, m8);
            // threats T_theta = max_j (m8 - mu_j) (+inf when mu_j = -inf): exact
            // ints from the four waves (own_threat), or, in the SIM profile,
            // exact in fp64
            using TT = std::conditional_t<SIMP, double, int>;
            TT T[NK];
            if constexpr (SIMP) {
#pragma unroll
                for (int th = 0; th < NK; ++th) {
                    double tv = -__builtin_inf();
#pragma unroll
                    for (int s = 0; s < QPL; ++s)
                        if (m8[th][s] > NEG_INF) {
                            const double d = (double)m8[th][s] - (double)mu[s];
                            tv = d > tv ? d : tv;
                        }
                    T[th] = wave_max_f64(tv);
                }
            } else {
#pragma unroll
                for (int th = 0; th < NK; ++th) T[th] = tsl[(t & 1) * NK + th];
            }
            // descending threat, ties by index; order packed 4 bits per rank
            uint32_t order = 0, taken = 0;
            int na = 0;
#pragma unroll
            for (int r = 0; r < NK; ++r) {
                int best = -1;
                TT bt = 0;
#pragma unroll
                for (int th = 0; th < NK; ++th) {
                    const bool cand = (act >> th & 1u) && !(taken >> th & 1u);
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
            uint32_t fail = F0;   // the test against mu_hat = mu
            int pos = 0, par = 0;
            while (true) {
                while (pos < na && !(fail >> ((order >> (4 * pos)) & 15u) & 1u)) ++pos;
                if (pos >= na) break;
                const int th = (int)((order >> (4 * pos)) & 15u);
                ++pos;
                prec16 |= 1u << th;
                if (F0 >> th & 1u) {
#pragma unroll
                    for (int s = 0; s < QPL; ++s) {
                        float c = muh[s];
#pragma unroll
                        for (int t2 = 0; t2 < NK; ++t2)
                            if (t2 == th) c = cm16[t2][s] > c ? cm16[t2][s] : c;
                        muh[s] = c;
                    }
                } else {
                    // outside F0 (not expected, see above): all waves recompute
                    // the sub-block in 16 bits, codes in place of the 8-bit ones
                    float cm[QPL];
#pragma unroll
                    for (int s = 0; s < QPL; ++s) cm[s] = NEG_INF;
                    shared16(k0, th, [&](int kc, const uint32_t (&yc)[QPL][WPM]) {
                        obs16(kc, yc);
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                const float yv = y16_value<SIMP>(yc[s], i);
                                if (visible(s, kc + i)) cm[s] = yv > cm[s] ? yv : cm[s];
                            }
                            uint2 *dst = reinterpret_cast<uint2 *>(ycode + row[s] * YP + (kc - k0));
                            if constexpr (SIMP) {
                                *dst = make_uint2(pack_hi16(yc[s][0], yc[s][1]), pack_hi16(yc[s][2], yc[s][3]));
                                *reinterpret_cast<uint2 *>(ylo + row[s] * YP + (kc - k0)) =
                                    make_uint2(pack_lo16(yc[s][0], yc[s][1]), pack_lo16(yc[s][2], yc[s][3]));
                            } else {
                                *dst = make_uint2(yc[s][0], yc[s][1]);
                            }
                        }
                    });
#pragma unroll
                    for (int s = 0; s < QPL; ++s) cmf[(par * NW + w) * BQ + row[s]] = cm[s];
                    __syncthreads();
#pragma unroll
                    for (int s = 0; s < QPL; ++s)
#pragma unroll
                        for (int ww = 0; ww < NW; ++ww) {
                            const float c = cmf[(par * NW + ww) * BQ + row[s]];
                            muh[s] = c > muh[s] ? c : muh[s];
                        }
                    par ^= 1;   // the next write goes to the other half: readers of this one may lag
                }
                if (pos < na) fail = fails_of(m8, muh);
            }
        }


        LAMP_PH(3);
        // ---- D. exponentials of tile t against mu_hat
        {
            // the 16-bit maxima buffer of tile t+1 was last read in tile t-1
            int *cmn = cmi_of(t + 1);
            for (int i = tid; i < NK * BQ; i += 256) cmn[i] = INT_MIN;

            double sp[QPL], spF[QPL];   // all exponentials / those of 8-bit sub-blocks
            float mu8[QPL];             // the running maximum the 8-bit shifts use
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
                sp[s] = spF[s] = 0.0;
                mu8[s] = mu_trunc ? (SIMP ? trunc_sim3(muh[s]) : trunc_e4m3(muh[s])) : muh[s];
            }
            const int th = w;   // own sub-block
            const int ck0 = k0 + th * BK;
            if (!(act >> th & 1u)) {
                // inactive: zero exponentials so the P.V pass may read them
#pragma unroll
                for (int s = 0; s < QPL; ++s) {
                    u32x4 *d = reinterpret_cast<u32x4 *>(ycode + row[s] * YP + th * BK);
                    d[0] = u32x4{0u, 0u, 0u, 0u};
                    d[1] = u32x4{0u, 0u, 0u, 0u};
                }
            } else if (!(prec16 >> th & 1u)) {
                // 8-bit sub-block, straight-line: all codes read, all table
                // indices formed and all table reads issued before the first is
                // used; invisible keys get E = 0 by selection.  The row sums are
                // exact in fp64 in any order (multiples of 2^-41 below 2^7), so
                // they run as four independent chains.
                bool full = true;
#pragma unroll
                for (int s = 0; s < QPL; ++s) full &= ck0 >= vlo[s] && ck0 + 15 <= vhi[s];
                auto run8 = [&](auto full_c) {
                    constexpr bool FULL = decltype(full_c)::value;
#pragma unroll
                    for (int s = 0; s < QPL; ++s) {
                        u32x4 *rp = reinterpret_cast<u32x4 *>(ycode + row[s] * YP + th * BK);
                        const u32x4 c0 = rp[0], c1 = rp[1];
                        const uint32_t in[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
                        uint32_t eb[16];
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            uint32_t x;
                            if constexpr (SIMP) {
                                x = sim_shift_index<3, SIM8_EMIN, SIM8_EMAX>(mu8[s], bf16_value((in[i >> 1] >> (16 * (i & 1))) & 0xFFFFu));
                            } else {
                                // the e4m3 code sits in the low byte of its 16-bit slot
                                const float y = (i & 1) ? __builtin_amdgcn_cvt_f32_fp8((int)in[i >> 1], 2)
                                                        : __builtin_amdgcn_cvt_f32_fp8((int)in[i >> 1], 0);
                                x = ue5m3_code(shift_of(mu8[s], y));
                            }
                            // an invisible key reads the table's last entry, whose
                            // exponential is 0 (the largest shift), so that every
                            // read is issued unconditionally
                            if constexpr (!FULL) x = visible(s, ck0 + i) ? x : (SIMP ? SIM8_N - 1 : 255u);
                            eb[i] = lut[x];
                        }
                        double a4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
                        for (int i = 0; i < 16; ++i) a4[i & 3] += (double)bf16_value(eb[i]);
                        const double ts = (a4[0] + a4[1]) + (a4[2] + a4[3]);
                        sp[s] += ts;
                        spF[s] += ts;
                        rp[0] = u32x4{eb[0] | eb[1] << 16, eb[2] | eb[3] << 16, eb[4] | eb[5] << 16, eb[6] | eb[7] << 16};
                        rp[1] = u32x4{eb[8] | eb[9] << 16, eb[10] | eb[11] << 16, eb[12] | eb[13] << 16,
                                      eb[14] | eb[15] << 16};
                    }
                };
                if (!wave_any(!full)) run8(std::true_type());
                else run8(std::false_type());
            } else if (!(F0 >> th & 1u)) {
                // a stage-1 sub-block outside F0: its one-at-a-time 16-bit codes
                // are in place (the members of F0 are done from registers below)
#pragma unroll
                for (int s = 0; s < QPL; ++s) {
                    u32x4 *rp = reinterpret_cast<u32x4 *>(ycode + row[s] * YP + th * BK);
                    u32x4 *lp = reinterpret_cast<u32x4 *>(ylo + row[s] * YP + th * BK);
                    if (ck0 > vhi[s] || ck0 + 15 < vlo[s]) {
                        rp[0] = u32x4{0u, 0u, 0u, 0u};
                        rp[1] = u32x4{0u, 0u, 0u, 0u};
                        lp[0] = u32x4{0u, 0u, 0u, 0u};
                        lp[1] = u32x4{0u, 0u, 0u, 0u};
                        continue;
                    }
                    const u32x4 c0 = rp[0], c1 = rp[1];
                    const uint32_t in[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
                    uint32_t inl[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};   // SIM: low halves of 16-bit logits
                    if (SIMP) {
                        const u32x4 l0 = lp[0], l1 = lp[1];
                        inl[0] = l0[0]; inl[1] = l0[1]; inl[2] = l0[2]; inl[3] = l0[3];
                        inl[4] = l1[0]; inl[5] = l1[1]; inl[6] = l1[2]; inl[7] = l1[3];
                    }
                    uint32_t outw[8], outl[8];
#pragma unroll
                    for (int pp = 0; pp < 8; ++pp) {
                        uint32_t res = 0, rlo = 0;
#pragma unroll
                        for (int t2 = 0; t2 < 2; ++t2) {
                            const int key = ck0 + 2 * pp + t2;
                            const uint32_t yc = (in[pp] >> (16 * t2)) & 0xFFFFu;
                            uint32_t eh = 0, el = 0;
                            float ev = 0.0f;
                            if (visible(s, key)) {
                                const float y = SIMP ? __builtin_bit_cast(float, (yc << 16) | ((inl[pp] >> (16 * t2)) & 0xFFFFu))
                                                     : e4m11_value(yc);
                                ev = e16_of(muh[s], y, eh, el);
                            }
                            sp[s] += (double)ev;
                            res |= eh << (16 * t2);
                            rlo |= el << (16 * t2);
                        }
                        outw[pp] = res;
                        outl[pp] = rlo;
                    }
                    rp[0] = u32x4{outw[0], outw[1], outw[2], outw[3]};
                    rp[1] = u32x4{outw[4], outw[5], outw[6], outw[7]};
                    lp[0] = u32x4{outl[0], outl[1], outl[2], outl[3]};
                    lp[1] = u32x4{outl[4], outl[5], outl[6], outl[7]};
                }
            }
            // 16-bit exponentials of this wave's 4 keys of every stage-1
            // sub-block of F0, from the codes held in registers: all table reads
            // of all such members issued first
            const uint32_t mine = prec16 & F0;
            if (mine) {
                int tg[NK];
                bool use[NK];
                {
                    uint32_t m = F0;
#pragma unroll
                    for (int g = 0; g < NK; ++g) {
                        tg[g] = m ? __builtin_ctz(m) : 0;
                        use[g] = m != 0u && (mine >> tg[g] & 1u);
                        m &= m - 1;
                    }
                }
#pragma unroll
                for (int g = 0; g < NK; ++g) {
                    if (!use[g]) continue;
                    // the 8 table reads of this member issued before the first is used
                    uint32_t hl[QPL][4];
#pragma unroll
                    for (int s = 0; s < QPL; ++s)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float y = y16_value<SIMP>(&y16r[s][g * WPM], i);
                            if constexpr (SIMP) hl[s][i] = p.sim16[sim_shift_index<11, SIM16_EMIN, SIM16_EMAX>(muh[s], y)];
                            else hl[s][i] = p.exp16hl[ue5m11_code(shift_of(muh[s], y))];
                        }
                    const int key0 = k0 + tg[g] * BK + w * 4;
                    if constexpr (!SIMP) {
                        if (dbg16 || p.stats) {
                            uint32_t yc[QPL][WPM];
#pragma unroll
                            for (int s = 0; s < QPL; ++s)
#pragma unroll
                                for (int x = 0; x < WPM; ++x) yc[s][x] = y16r[s][g * WPM + x];
                            obs16(key0, yc);
                        }
                    }
#pragma unroll
                    for (int s = 0; s < QPL; ++s) {
                        uint32_t eh[4], el[4];
                        double ev[4];
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const uint32_t x = hl[s][i];
                            float v;
                            if constexpr (SIMP) {
                                eh[i] = x >> 16;
                                el[i] = x & 0xFFFFu;
                                v = __builtin_bit_cast(float, x);
                            } else {
                                eh[i] = x & 0xFFFFu;
                                el[i] = x >> 16;
                                v = bf16_value(eh[i]) + bf16_value(el[i]);   // exact
                            }
                            const bool vis = visible(s, key0 + i);
                            eh[i] = vis ? eh[i] : 0u;
                            el[i] = vis ? el[i] : 0u;
                            ev[i] = vis ? (double)v : 0.0;
                        }
                        sp[s] += (ev[0] + ev[1]) + (ev[2] + ev[3]);
                        *reinterpret_cast<uint2 *>(ycode + row[s] * YP + (key0 - k0)) =
                            make_uint2(eh[0] | eh[1] << 16, eh[2] | eh[3] << 16);
                        *reinterpret_cast<uint2 *>(ylo + row[s] * YP + (key0 - k0)) =
                            make_uint2(el[0] | el[1] << 16, el[2] | el[3] << 16);
                    }
                }
            }
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
                sps[w * BQ + row[s]] = sp[s];
                spf[w * BQ + row[s]] = spF[s];
            }
        }
        LAMP_PH(4);
        __syncthreads();   // E
        LAMP_PH(5);

        // ---- lambda_hat, omega_hat, stage 2
        double S[QPL], lam[QPL], omh[QPL];
        bool moved = false;   // exp_doc(0) is exactly 1: skip the exponentials when no maximum moved
#pragma unroll
        for (int s = 0; s < QPL; ++s) moved |= muh[s] != mu[s];
        moved = wave_any(moved);
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            double tt = 0.0;
            if constexpr (SIMP) {
                tt = seq_sum(ycode, s, prec16);
            } else {
#pragma unroll
                for (int ww = 0; ww < NW; ++ww) tt += sps[ww * BQ + row[s]];
            }
            S[s] = tt;
            if (muh[s] == NEG_INF) lam[s] = 1.0;
            else if (mu[s] == NEG_INF) lam[s] = 0.0;
            else lam[s] = moved ? exp_doc_k((double)mu[s] - (double)muh[s], [&](int i) { return edk[i]; }) : 1.0;
            omh[s] = __builtin_fma(lam[s], om[s], tt);
        }
        uint32_t prec2 = 0;
        if (mode == MODE_LAMP) {
            const uint32_t F = act & ~prec16;
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
                // costs c_theta,j = sum_{i in theta, ascending} E (omega_hat - E), own sub-block
                if (F >> w & 1u) {
#pragma unroll
                    for (int s = 0; s < QPL; ++s) {
                        const u32x4 *rp = reinterpret_cast<const u32x4 *>(ycode + row[s] * YP + w * BK);
                        const u32x4 c0 = rp[0], c1 = rp[1];
                        const uint32_t in[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
                        double cth = 0.0;
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const double e = (double)bf16_value((in[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
                            const double tt = omh[s] - e;
                            const double pr = e * tt;
                            cth = cth + pr;   // invisible entries hold E = 0 and add +0
                        }
                        cst_lds[w * BQ + row[s]] = cth;
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
                    // stage-2 recompute shared by all waves (4 keys each): 16-bit
                    // logits and exponentials against the unchanged mu_hat
                    double ds[QPL];
#pragma unroll
                    for (int s = 0; s < QPL; ++s) ds[s] = 0.0;
                    auto s2fn = [&](int kc, const uint32_t (&yc)[QPL][WPM]) {
                        obs16(kc, yc);
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
                            const uint16_t *src = ycode + row[s] * YP + (kc - k0);
                            uint32_t outw[2], outl[2];
#pragma unroll
                            for (int pp = 0; pp < 2; ++pp) {
                                uint32_t res = 0, rlo = 0;
#pragma unroll
                                for (int t2 = 0; t2 < 2; ++t2) {
                                    const int key = kc + 2 * pp + t2;
                                    uint32_t eh = 0, el = 0;
                                    if (visible(s, key)) {
                                        const float old = bf16_value(src[2 * pp + t2]);
                                        const float ev = e16_of(muh[s], y16_value<SIMP>(yc[s], 2 * pp + t2), eh, el);
                                        if constexpr (!SIMP) {
                                            ds[s] = ds[s] - (double)old;
                                            ds[s] = ds[s] + (double)ev;
                                        }
                                    }
                                    res |= eh << (16 * t2);
                                    rlo |= el << (16 * t2);
                                }
                                outw[pp] = res;
                                outl[pp] = rlo;
                            }
                            *reinterpret_cast<uint2 *>(ycode + row[s] * YP + (kc - k0)) = make_uint2(outw[0], outw[1]);
                            *reinterpret_cast<uint2 *>(ylo + row[s] * YP + (kc - k0)) = make_uint2(outl[0], outl[1]);
                        }
                    };
                    // sub-blocks of R without codes from the fused pass: one batched
                    // recompute, 4 keys of each per wave (as for F0)
                    const uint32_t Rn = prec2 & ~F0;
                    uint32_t y16b[QPL][4 * WPM];
                    if (Rn) {
                        const int nr = __builtin_popcount(Rn);
                        const int kb = (lane & 15) % (4 * nr);
                        uint32_t m = Rn;
                        for (int g = 0; g < kb / 4; ++g) m &= m - 1;
                        const float *krow = krow_of(k0 + __builtin_ctz(m) * BK + w * 4 + (kb & 3));
                        auto rec = [&](auto nkey_c) {
                            constexpr int NKEY = decltype(nkey_c)::value;
                            uint32_t c[QPL][y16_words<SIMP>(NKEY)];
                            rec16_keys<D, QPL, NKEY, SIMP, GrpLay>(qrow, krow, c);
#pragma unroll
                            for (int s = 0; s < QPL; ++s)
#pragma unroll
                                for (int pp = 0; pp < y16_words<SIMP>(NKEY); ++pp) y16b[s][pp] = c[s][pp];
                        };
                        switch (nr) {
                        case 1: rec(std::integral_constant<int, 4>()); break;
                        case 2: rec(std::integral_constant<int, 8>()); break;
                        case 3: rec(std::integral_constant<int, 12>()); break;
                        default: rec(std::integral_constant<int, 16>()); break;
                        }
                    }
                    for (int th = 0; th < NK; ++th) {
                        if (!(prec2 >> th & 1u)) continue;
                        // this wave's 4 keys of sub-block th: codes from the fused pass
                        // (member of F0) or from the batch above
                        const bool inF0 = F0 >> th & 1u;
                        const int gi = __builtin_popcount((inF0 ? F0 : Rn) & ((1u << th) - 1u));
                        uint32_t yc[QPL][WPM];
#pragma unroll
                        for (int s = 0; s < QPL; ++s) {
#pragma unroll
                            for (int x = 0; x < WPM; ++x) yc[s][x] = inF0 ? y16r[s][x] : y16b[s][x];
#pragma unroll
                            for (int g = 1; g < NK; ++g)
                                if (g == gi)
#pragma unroll
                                    for (int x = 0; x < WPM; ++x)
                                        yc[s][x] = inF0 ? y16r[s][g * WPM + x] : y16b[s][g * WPM + x];
                        }
                        s2fn(k0 + th * BK + w * 4, yc);
                    }
                    if constexpr (!SIMP) {
#pragma unroll
                        for (int s = 0; s < QPL; ++s) sps[w * BQ + row[s]] = ds[s];
                    }
                    __syncthreads();
#pragma unroll
                    for (int s = 0; s < QPL; ++s) {
                        if constexpr (SIMP) {
                            S[s] = seq_sum(ycode, s, prec16 | prec2);
                        } else {
                            double tt = S[s];
#pragma unroll
                            for (int ww = 0; ww < NW; ++ww) tt += sps[ww * BQ + row[s]];   // exact
                            S[s] = tt;
                        }
                    }
                }
            }
        }

        LAMP_PH(6);
        // ---- G. state update; O^T <- O^T diag(lambda_hat) + V^T E; next F0
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
            om[s] = __builtin_fma(lam[s], om[s], S[s]);
            mu[s] = muh[s];
        }
        if (tid == 0) {
#pragma unroll
            for (int th = 0; th < NK; ++th)
                mrow[t * NK + th] = !(act >> th & 1u) ? PREC_INACTIVE
                                  : (prec16 >> th & 1u) ? PREC_S1
                                  : (prec2 >> th & 1u) ? PREC_S2 : PREC_LOW;
            if (p.stats && act) {
                const uint32_t rec = prec16 | prec2;
                stl[ST_TILES] += 1u;
                stl[ST_S1] += __builtin_popcount(prec16);
                stl[ST_S2] += __builtin_popcount(prec2);
                stl[ST_ACT] += __builtin_popcount(act);
                stl[ST_UNUSED] += __builtin_popcount(F0 & ~rec);
                stl[ST_LATE] += __builtin_popcount(rec & ~F0);
                stl[ST_HIST + __builtin_popcount(rec)] += 1u;
            }
        }
        const uint32_t p16 = prec16 | prec2;
        const int half = lane >> 5, l32 = lane & 31;
        // V^T operands from global memory, one chunk ahead of the matrix-core
        // work (every chunk's keys lie below N, so the loads stay in bounds)
        auto load_v = [&](int c16, u32x4 (&a)[CT]) {
#pragma unroll
            for (int tt = 0; tt < CT; ++tt)
                a[tt] = *reinterpret_cast<const u32x4 *>(vtbase + (size_t)(w * CPW + tt * 32 + l32) * p.Nk + k0 +
                                                         c16 * 16 + half * 8);
        };
        auto pv_chunk = [&](int c16, const u32x4 (&a)[CT]) {
            const int ck0 = k0 + c16 * 16;
            if (!(act >> c16 & 1u) || ck0 > bv_hi || ck0 + 15 < bv_lo) return;
            const bool hi16 = p16 >> c16 & 1u;
#pragma unroll
            for (int g = 0; g < QG; ++g) {
                const int off = (g * 32 + l32) * YP + c16 * 16 + half * 8;
                const bf16x8 bh = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(ycode + off));
#pragma unroll
                for (int tt = 0; tt < CT; ++tt)
                    acc[g][tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[tt]), bh,
                                                                         acc[g][tt], 0, 0, 0);
                if (hi16) {   // E16 = hi + lo exactly
                    u32x4 lw = *reinterpret_cast<const u32x4 *>(ylo + off);
                    if constexpr (SIMP) lw = lo_bf16x8(*reinterpret_cast<const u32x4 *>(ycode + off), lw);
                    const bf16x8 bl = __builtin_bit_cast(bf16x8, lw);
#pragma unroll
                    for (int tt = 0; tt < CT; ++tt)
                        acc[g][tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[tt]), bl,
                                                                             acc[g][tt], 0, 0, 0);
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
                    for (int tt = 0; tt < CT; ++tt)
#pragma unroll
                        for (int r = 0; r < 16; ++r) acc[g][tt][r] *= lg;
                }
            }
        }
        load_v(1, vb);
        pv_chunk(0, va);
        load_v(2, va);
        pv_chunk(1, vb);
        load_v(3, vb);
        pv_chunk(2, va);
        pv_chunk(3, vb);

        F0 = has_next ? f0_of(t + 1, act_next) : 0u;
        if (mode == MODE_LAMP && !stage1_off && has_next) own_threat(t + 1);
        act = act_next;
        LAMP_PH(7);
        __syncthreads();   // I: this tile's code buffer is rewritten by the pass of tile t+1
        LAMP_PH(8);
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
            for (int tt = 0; tt < CT; ++tt)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    const int c = tt * 32 + r4 * 8 + half * 4;
                    const float4 v4 = make_float4(acc[g][tt][r4 * 4 + 0] * inv, acc[g][tt][r4 * 4 + 1] * inv,
                                                  acc[g][tt][r4 * 4 + 2] * inv, acc[g][tt][r4 * 4 + 3] * inv);
                    *reinterpret_cast<float4 *>(orow + c) = v4;
                }
        }
        if (w == 0)
#pragma unroll
            for (int s = 0; s < QPL; ++s)
                if (q0 + row[s] < p.N)
                    p.lse[((size_t)b * p.Hq + h) * p.N + q0 + row[s]] = (float)((double)mu[s] + ::log(om[s]));
        const int ntiles = p.Nk / KPT;
        for (int tt = tid; tt < ntiles; tt += 256)
            if (tt < t_begin || tt > t_end)
                for (int th = 0; th < NK; ++th) mrow[tt * NK + th] = PREC_INACTIVE;
    }
    if (p.stats) flush_stats<NK>(p.stats, stl, (uint32_t)(p.Nk / BK), tid);
    LAMP_PH_FLUSH;
}

// ------------------------------------------------------------------ launcher
#ifndef LAMP_FWD16_NO_LAUNCHERS
template <int D, int BQ, int MODE, bool SIMP, bool OBS, bool CMP = false>
static hipError_t launch_fwd16_obs(const FwdParams &p, hipStream_t s)
{
    using C = Cfg16<D, BQ>;
    auto kern = lamp_fwd16_kernel<D, BQ, MODE, SIMP, OBS, CMP>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)(p.B * p.Hq * (p.Nq / BQ)));
    hipLaunchKernelGGL(kern, grid, dim3(256), C::LDS, s, p);
    return hipGetLastError();
}

template <int D, int BQ, int MODE, bool SIMP>
static hipError_t launch_fwd16_mode(const FwdParams &p, hipStream_t s)
{
    const bool obs = p.dbg_y8 || p.dbg_y16;
    // the compact layout: threshold mode, hardware formats, 128-row blocks
    if constexpr (MODE == MODE_LAMP && !SIMP && BQ == 128)
        if (p.flags & LAMP_COMPACT)
            return obs ? launch_fwd16_obs<D, BQ, MODE, SIMP, true, true>(p, s)
                       : launch_fwd16_obs<D, BQ, MODE, SIMP, false, true>(p, s);
    if constexpr (!SIMP)
        if (obs) return launch_fwd16_obs<D, BQ, MODE, SIMP, true>(p, s);
    return launch_fwd16_obs<D, BQ, MODE, SIMP, false>(p, s);
}

template <int D, int BQ, bool SIMP>
static hipError_t launch_fwd16_prof(const FwdParams &p, hipStream_t s)
{
    if (p.mode == MODE_PURE8) return launch_fwd16_mode<D, BQ, MODE_PURE8, SIMP>(p, s);
    if (p.mode == MODE_ALL16) return launch_fwd16_mode<D, BQ, MODE_ALL16, SIMP>(p, s);
    return launch_fwd16_mode<D, BQ, MODE_LAMP, SIMP>(p, s);
}

template <int D, int BQ>
static hipError_t launch_fwd16(const FwdParams &p, hipStream_t s)
{
    if (p.flags & LAMP_SIM_PROFILE) return launch_fwd16_prof<D, BQ, true>(p, s);
    return launch_fwd16_prof<D, BQ, false>(p, s);
}

hipError_t dispatch_fwd16(int D, int BQ, const FwdParams &p, hipStream_t s, bool *found)
{
    *found = true;
    if (D == 128 && BQ == 64) return launch_fwd16<128, 64>(p, s);
    if (D == 128 && BQ == 128) return launch_fwd16<128, 128>(p, s);
    if (D == 256 && BQ == 64) return launch_fwd16<256, 64>(p, s);
    if (D == 256 && BQ == 128) return launch_fwd16<256, 128>(p, s);
    *found = false;
    return hipSuccess;
}

#endif // LAMP_FWD16_NO_LAUNCHERS

} // namespace lamp
