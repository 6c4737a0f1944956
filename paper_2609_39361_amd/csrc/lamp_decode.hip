// lamp_decode.hip -- LampAttention for single query rows against a key/value
// cache: the vector form of the look-ahead (paper Sec. 2, the two-step
// procedure and the greedy knapsack of Eq. (6)), for decode.
//
// Per query row the key tiles (64 keys) are visited in order; in each tile
//   1. the maximizer c of the 8-bit logits is tested against the running
//      maximum with the safety margin (mu > fma(|mu|, delta, fl(y_c)));
//      on failure y_c is recomputed in 16 bits and mu_hat = max(mu, y16_c),
//      otherwise mu_hat = mu;
//   2. the remaining 8-bit logits are sorted by their cost E (omega_hat - E)
//      (the scaled p (1 - p) of Eq. (6)) and kept in 8 bits while the fp64
//      running sum of the sorted costs stays within tau omega_hat^2; the
//      first cost that would pass the limit and every later one are
//      recomputed in 16 bits against the same mu_hat;
//   3. omega, O and mu are updated (Sec. 2, online softmax).
//
// Three passes over a chunk of keys, each a device function (a role) that a
// workgroup runs:
//   logits     the logits of every (query row, key), which depend on no
//              decision, in 8 bits and in 16 bits (codes), and the mask code
//              of every key: one thread per key, the 4 query rows of a group
//              accumulated together, queries read from LDS (broadcast), keys
//              staged through LDS from coalesced loads of the bf16 cache (no
//              fp32 copy);
//   decisions  one wave per query row: lane i holds key i of the tile; DPP
//              reductions, a bitonic sort of the costs and the sequential sum;
//              runs of up to 8 tiles that keep the running maximum and pass
//              the knapsack's quick acceptance are evaluated together; the row
//              state (mu, omega) passes from chunk to chunk, and each chunk
//              records mu_hat and its rescale factors per tile and the mask
//              codes of the recomputed keys;
//   P.V        in parallel over 512-key pieces for all query rows of a
//              key/value head (fp32 FMAs; every exponential is exact in fp32),
//              the weights recomputed from the codes.
// dec_stage_kernel runs the decisions of one chunk, the logits of the next and
// P.V of the one before in one launch (the chunk pipeline); dec_logits_kernel,
// dec_lamp_kernel and dec_pv_kernel run one role each (the serial schedule);
// dec_reduce_kernel combines the pieces' partial outputs over the chunks.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lamp_decode.h"
#include "lamp_device.h"
#include "lamp_kernels.h"

namespace lamp {

namespace {

constexpr int TK = 64;   // keys per tile: one per lane

__device__ __forceinline__ void unpack8(const uint4 &w, float (&f)[8])
{
    const uint32_t x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = __builtin_bit_cast(float, x[i] << 16);
        f[2 * i + 1] = __builtin_bit_cast(float, x[i] & 0xFFFF0000u);
    }
}

// Wave reductions on the VALU: DPP exchanges within each row of 16 lanes
// (neighbours, pairs, half-row mirror, row mirror) leave every lane with its
// row's result; the four rows are then read out with readlane.  The DPP forms
// here are compiler builtins, so the compiler inserts any wait states they
// need.  DPP control codes: quad_perm [1,0,3,2] = 0xB1, [2,3,0,1] = 0x4E,
// row_half_mirror = 0x141, row_mirror = 0x140.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v)
{
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, 0xF, 0xF, true);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, true);
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// The value of lane (this lane xor j): within a 16-lane row by DPP (j = 1, 2
// and 8 one move: quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_ror:8; j = 4
// two: row_half_mirror then quad_perm [3,2,1,0]), across rows by a lane
// permute.  j is a constant wherever the callers' loops are unrolled.
template <int J>
__device__ __forceinline__ uint32_t xor_dpp(uint32_t v)
{
    if constexpr (J == 1) return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, true);
    if constexpr (J == 2) return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, true);
    if constexpr (J == 8) return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, true);
    const int w = __builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, true);
    return (uint32_t)__builtin_amdgcn_update_dpp(0, w, 0x1B, 0xF, 0xF, true);
}

__device__ __forceinline__ uint32_t xor_lanes(uint32_t v, int j)
{
    switch (j) {
    case 1: return xor_dpp<1>(v);
    case 2: return xor_dpp<2>(v);
    case 4: return xor_dpp<4>(v);
    case 8: return xor_dpp<8>(v);
    default: return (uint32_t)__shfl_xor((int)v, j, 64);
    }
}

__device__ __forceinline__ double xor_lanes(double v, int j)
{
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = xor_lanes((uint32_t)u, j), hi = xor_lanes((uint32_t)(u >> 32), j);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ float readlane_f32(float v, int l)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

__device__ __forceinline__ double readlane_f64(double v, int l)
{
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Inclusive prefix sum over the wave in fp64: within each 16-lane row by DPP
// row shifts of 1, 2, 4 and 8 (lanes shifted in from outside the row read 0),
// then the totals of the rows below added in.
__device__ __forceinline__ double prefix_sum_f64(double v)
{
    v += dpp_f64<0x111>(v);
    v += dpp_f64<0x112>(v);
    v += dpp_f64<0x114>(v);
    v += dpp_f64<0x118>(v);
    const double t0 = readlane_f64(v, 15), t1 = readlane_f64(v, 31), t2 = readlane_f64(v, 47);
    const int r = (int)(__lane_id() >> 4);
    const double off = (r >= 1 ? t0 : 0.0) + ((r >= 2 ? t1 : 0.0) + (r >= 3 ? t2 : 0.0));
    return v + off;
}

__device__ __forceinline__ float wave_max_f32(float v)
{
    float o;
    o = dpp_f32<0xB1>(v); v = o > v ? o : v;
    o = dpp_f32<0x4E>(v); v = o > v ? o : v;
    o = dpp_f32<0x141>(v); v = o > v ? o : v;
    o = dpp_f32<0x140>(v); v = o > v ? o : v;
    const float a = readlane_f32(v, 0), b = readlane_f32(v, 16), c = readlane_f32(v, 32), d = readlane_f32(v, 48);
    const float ab = a > b ? a : b, cd = c > d ? c : d;
    return ab > cd ? ab : cd;
}

__device__ __forceinline__ float wave_sum_f32(float v)
{
    v += dpp_f32<0xB1>(v);
    v += dpp_f32<0x4E>(v);
    v += dpp_f32<0x141>(v);
    v += dpp_f32<0x140>(v);
    return (readlane_f32(v, 0) + readlane_f32(v, 16)) + (readlane_f32(v, 32) + readlane_f32(v, 48));
}

// Sum over the wave; exact for the exponentials of the hardware formats
// (multiples of 2^-41 in [0, 1], 64 of them), so the order does not matter.
__device__ __forceinline__ double wave_sum_f64(double v)
{
    v += dpp_f64<0xB1>(v);
    v += dpp_f64<0x4E>(v);
    v += dpp_f64<0x141>(v);
    v += dpp_f64<0x140>(v);
    return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

} // namespace

// ------------------------------------------------------------------ phase 1
// The logits of every (query row, key), which depend on no decision: the
// 8-bit ones (the emulated e4m3 recursion) unless every logit is recomputed,
// and the 16-bit ones (the FP32 FMA chain over the channels in ascending
// order, rounded once to e4m11) unless none is, with the mask code of every
// key (0, or 1 when every logit is 16-bit, where visible; 3 elsewhere; the
// decisions overwrite the recomputed ones).
//
// grid (key blocks of 256 from key kb0, B * Hkv * row groups); a row group is
// 4 consecutive rows of the G*M query rows of one key/value head (row rho is
// query head hk*G + rho / M, query r = rho % M).  Thread t owns key
// kb0 + 256 blockIdx.x + t.  The keys reach LDS in stages of 64 channels with
// coalesced 16-byte loads (8 threads per 128-byte key row), so each global
// load instruction covers whole cache lines; every thread then reads its own
// row from LDS (pitch 72 bf16 against bank conflicts).  The next stage's loads
// are issued before the current stage is computed.
constexpr int P1_CH = 64, P1_PITCH = P1_CH + 8;

template <int D, int MODE, bool SAT>
__device__ __forceinline__ void dec_staged(const uint16_t *kblk, int nvalid, uint16_t *tile, const float *qs,
                                           uint32_t (&acc)[2], float (&acc16)[4])
{
    constexpr bool L8 = MODE != MODE_ALL16, L16 = MODE != MODE_PURE8 && !SAT;
    const int tid = threadIdx.x;
    acc[0] = acc[1] = 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc16[i] = 0.0f;
    // this thread's 16-byte pieces of 8 key rows (rows beyond N repeat the
    // last key, not stored), one stage of 64 channels held in registers
#define LAMP_P1_ADDR(j) (kblk + (size_t)((tid + 256 * (j)) >> 3 < nvalid ? (tid + 256 * (j)) >> 3 : nvalid - 1) * D + \
                         ((tid + 256 * (j)) & 7) * 8)
#define LAMP_P1_LOAD(c0) \
    w0 = *reinterpret_cast<const uint4 *>(LAMP_P1_ADDR(0) + (c0)); w1 = *reinterpret_cast<const uint4 *>(LAMP_P1_ADDR(1) + (c0)); \
    w2 = *reinterpret_cast<const uint4 *>(LAMP_P1_ADDR(2) + (c0)); w3 = *reinterpret_cast<const uint4 *>(LAMP_P1_ADDR(3) + (c0)); \
    w4 = *reinterpret_cast<const uint4 *>(LAMP_P1_ADDR(4) + (c0)); w5 = *reinterpret_cast<const uint4 *>(LAMP_P1_ADDR(5) + (c0)); \
    w6 = *reinterpret_cast<const uint4 *>(LAMP_P1_ADDR(6) + (c0)); w7 = *reinterpret_cast<const uint4 *>(LAMP_P1_ADDR(7) + (c0));
#define LAMP_P1_STORE(j, w) *reinterpret_cast<uint4 *>(tile + (((tid + 256 * (j)) >> 3) * P1_PITCH) + ((tid + 256 * (j)) & 7) * 8) = (w);
    uint4 w0, w1, w2, w3, w4, w5, w6, w7;
    LAMP_P1_LOAD(0)
#pragma clang loop unroll(full)
    for (int c0 = 0; c0 < D; c0 += P1_CH) {
        __syncthreads();   // the previous stage is no longer read
        LAMP_P1_STORE(0, w0) LAMP_P1_STORE(1, w1) LAMP_P1_STORE(2, w2) LAMP_P1_STORE(3, w3)
        LAMP_P1_STORE(4, w4) LAMP_P1_STORE(5, w5) LAMP_P1_STORE(6, w6) LAMP_P1_STORE(7, w7)
        __syncthreads();
        if (c0 + P1_CH < D) {
            LAMP_P1_LOAD(c0 + P1_CH)
        }
#pragma unroll 2
        for (int c = 0; c < P1_CH; c += 8) {
            float kf[8];
            unpack8(*reinterpret_cast<const uint4 *>(tile + tid * P1_PITCH + c), kf);
            // the 4 rows' queries for these 8 channels: broadcast LDS reads
            float qv[4][8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float4 a = *reinterpret_cast<const float4 *>(qs + i * D + c0 + c);
                const float4 b = *reinterpret_cast<const float4 *>(qs + i * D + c0 + c + 4);
                qv[i][0] = a.x; qv[i][1] = a.y; qv[i][2] = a.z; qv[i][3] = a.w;
                qv[i][4] = b.x; qv[i][5] = b.y; qv[i][6] = b.z; qv[i][7] = b.w;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                if (L8) {
                    const float2 a = unpk_e4m3(acc[0]);
                    const float x = __builtin_fmaf(qv[0][j], kf[j], a.x);
                    const float y = __builtin_fmaf(qv[1][j], kf[j], a.y);
                    acc[0] = SAT ? pk_e4m3_sat(x, y, acc[0]) : pk_e4m3(x, y, acc[0]);
                    const float2 bb = unpk_e4m3(acc[1]);
                    const float z = __builtin_fmaf(qv[2][j], kf[j], bb.x);
                    const float u = __builtin_fmaf(qv[3][j], kf[j], bb.y);
                    acc[1] = SAT ? pk_e4m3_sat(z, u, acc[1]) : pk_e4m3(z, u, acc[1]);
                }
                if (L16) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc16[i] = __builtin_fmaf(qv[i][j], kf[j], acc16[i]);
                }
            }
        }
    }
}

#undef LAMP_P1_ADDR
#undef LAMP_P1_LOAD
#undef LAMP_P1_STORE

template <int D>
struct LogitsLds {
    uint16_t tile[256 * P1_PITCH];
    float qs[4 * D];   // the group's 4 pre-scaled query rows
};

// Workgroup (bx, by) of the logit pass over the launch's key chunk: keys
// ka + 256 bx .., row group by % ngroups of key/value head by / ngroups.
template <int D, int MODE>
__device__ __forceinline__ void dec_logits_role(const DecParams &p, LogitsLds<D> &sm, int bx, int by)
{
    uint16_t *tile = sm.tile;
    float *qs = sm.qs;
    const int G = p.Hq / p.Hkv;
    const int rows = G * p.M, ngroups = (rows + 3) / 4;
    const int grp = by % ngroups;
    const int bhk = by / ngroups;
    const int b = bhk / p.Hkv, hk = bhk % p.Hkv;
    const int key0 = p.ka + bx * 256;
    const int key = key0 + (int)threadIdx.x;
    const int nvalid = p.N - key0 < 256 ? p.N - key0 : 256;
    const uint16_t *kblk = p.k + (((size_t)b * p.Hkv + hk) * p.N + key0) * D;
    size_t qrow[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        int rho = grp * 4 + i;
        rho = rho < rows ? rho : rows - 1;   // a partial group repeats its last row (not stored)
        const int h = hk * G + rho / p.M, r = rho % p.M;
        qrow[i] = ((size_t)b * p.Hq + h) * p.M + r;
    }
    // the group's queries scaled in fp32 (the same product as the forward
    // pass's prepass: bf16 value times RN32(1/sqrt(d)))
    for (int x = (int)threadIdx.x; x < 4 * D; x += 256) qs[x] = bf16_value(p.q[qrow[x / D] * D + x % D]) * p.qscale;
    __syncthreads();
    uint32_t acc[2];
    float acc16[4];
    dec_staged<D, MODE, false>(kblk, nvalid, tile, qs, acc, acc16);
    // an overflow somewhere gives a NaN code at the end of its 8-bit chain:
    // the workgroup re-runs those chains with the saturating conversion
    if (MODE != MODE_ALL16 && __syncthreads_or((e4m3_nan_bits(acc[0]) | e4m3_nan_bits(acc[1])) != 0u)) {
        float unused[4];
        dec_staged<D, MODE, true>(kblk, nvalid, tile, qs, acc, unused);
    }
    if (key >= p.Np || key >= p.kz) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rho = grp * 4 + i;
        if (rho >= rows) continue;
        const int P = p.N - p.M + rho % p.M;
        const int vlo = p.window > 0 ? (P - p.window + 1 > 0 ? P - p.window + 1 : 0) : 0;
        const int vhi = p.causal ? P : p.N - 1;
        const size_t at = qrow[i] * (size_t)p.Np + key;
        if (key < p.N) {
            if (MODE != MODE_ALL16) p.y8[at] = (uint8_t)(acc[i >> 1] >> (8 * (i & 1)));
            if (MODE != MODE_PURE8) {
                uint32_t code;
                (void)rn_e4m11((double)acc16[i], &code);
                p.y16[at] = (uint16_t)code;
            }
        }
        p.mask[at] = key >= vlo && key <= vhi ? (MODE == MODE_ALL16 ? 1 : 0) : 3;
    }
}

// ------------------------------------------------------------------ phase 2
// The decisions of one query row, one wave per row, lane i holding key i of a
// tile.  Nothing in the output feeds a decision, so the decisions record only
// what they fixed: per visited tile mu_hat and the factor f_t = (prod of
// lambda_hat of the later tiles) / omega that turns the tile's exponentials
// into the final weights of P.V (O = sum_t f_t sum_{i in t} E_i v_i), both
// with the R = G*M query rows of a key/value head interleaved (mu
// [b][hk][tile][rho], f likewise); and per recomputed key its mask code (1 or
// 2), handed to a sink.  P.V recomputes each weight from the mask code, the
// 8-bit or 16-bit logit code and mu_hat, with the same tables.
//
// No global store is issued per tile (on gfx950 a wait for a load also waits
// for every earlier store of the wave, so a store in the tile loop would cost
// a store round trip at the next load): mu_hat and lambda_hat of 64 tiles at
// a time are held one per lane and written when the window is complete.
template <int MODE>
struct RowDecider {
    const DecParams *p;
    const uint16_t *lut;   // LDS: ue5m3 shift code -> bf16 bits of the exponential
    const double *edk;     // LDS: the exp_doc constants
    double *frow;          // lambda_hat, then the P.V factor, of this row's tiles (stride RR)
    float *murow;          // mu_hat of this row's tiles (stride RR)
    int64_t row;
    int lane, vlo, vhi, t_begin, t_end, RR;
    int tc_lo, tc_hi;      // this row's tiles in the launch's key chunk
    int t_rec;             // the tile after the last one recorded
    float mu;
    double om;
    float w_mu;            // mu_hat and lambda_hat of tile tc_lo + 64 wcur + lane
    double w_lam;
    int wcur;

    __device__ __forceinline__ void start(const DecParams &pp, const uint16_t *lut_, const double *edk_, int64_t row_,
                                          int lane_)
    {
        p = &pp;
        lut = lut_;
        edk = edk_;
        lane = lane_;
        row = row_;
        const int r = (int)(row % pp.M);
        const int h = (int)((row / pp.M) % pp.Hq);
        const int b = (int)(row / ((int64_t)pp.M * pp.Hq));
        const int G = pp.Hq / pp.Hkv, hk = h / G;
        RR = G * pp.M;
        const int rho = (h - hk * G) * pp.M + r;   // this row's slot among the rows of the head
        const int P = pp.N - pp.M + r;              // the query's position
        vlo = pp.window > 0 ? (P - pp.window + 1 > 0 ? P - pp.window + 1 : 0) : 0;
        vhi = pp.causal ? P : pp.N - 1;
        t_begin = vlo / TK;
        t_end = vhi / TK;
        tc_lo = t_begin > pp.ka / TK ? t_begin : pp.ka / TK;
        tc_hi = t_end < pp.kz / TK - 1 ? t_end : pp.kz / TK - 1;
        t_rec = tc_lo;
        const int ntiles = pp.Np / TK;
        frow = pp.f + ((size_t)b * pp.Hkv + hk) * (size_t)ntiles * RR + rho;
        murow = pp.mut + ((size_t)b * pp.Hkv + hk) * (size_t)ntiles * RR + rho;
        // the state the earlier chunks left (the first starts empty)
        mu = pp.chunk > 0 ? pp.mu_st[row] : -__builtin_inff();
        om = pp.chunk > 0 ? pp.om_st[row] : 0.0;
        w_mu = 0.0f;
        w_lam = 0.0;
        wcur = 0;
    }

    __device__ __forceinline__ void flush_window()
    {
        const int tt = tc_lo + 64 * wcur + lane;
        if (tt < t_rec) {
            frow[(size_t)tt * RR] = w_lam;
            murow[(size_t)tt * RR] = w_mu;
        }
    }

    __device__ __forceinline__ void record_tile(int tt, float muh, double lam)
    {
        if ((tt - tc_lo) >> 6 != wcur) {
            flush_window();
            wcur = (tt - tc_lo) >> 6;
        }
        if (lane == ((tt - tc_lo) & 63)) {
            w_mu = muh;
            w_lam = lam;
        }
        t_rec = tt + 1;
    }

    __device__ __forceinline__ float e_of(float muh, float yy, bool high) const
    {
        if (high) {
            const uint32_t hl = p->exp16hl[ue5m11_code(shift_of(muh, yy))];
            return bf16_value(hl & 0xFFFFu) + bf16_value(hl >> 16);   // exact
        }
        return bf16_value(lut[ue5m3_code(shift_of(muh, yy))]);
    }

    // One tile exactly as the procedure states it: look-ahead test on the
    // maximizer, exponentials, rescale, knapsack, update.  code: this lane's
    // 8-bit logit code; y16_of(): this lane's 16-bit logit; sink(key, prec)
    // is called by the lanes of the recomputed keys (mask code 1 or 2; in the
    // threshold mode only).
    template <class Y16, class Sink>
    __device__ __forceinline__ void tile_exact(int t, uint32_t code, Y16 y16_of, Sink sink)
    {
        const float NEG_INF = -__builtin_inff();
        const int key = t * TK + lane;
        const bool vis = key >= vlo && key <= vhi;   // vhi < N
        float y = NEG_INF;   // this key's logit in the precision chosen for it
        uint8_t prec = vis ? 0 : 3;
        bool have16 = false;
        float y16 = 0.0f;
        float muh;
        if (MODE == MODE_ALL16) {
            y16 = y16_of();
            have16 = true;
            y = vis ? y16 : NEG_INF;
            prec = vis ? 1 : 3;
            const float mx = wave_max_f32(y);
            muh = mx > mu ? mx : mu;
        } else {
            y = vis ? e4m3_value(code) : NEG_INF;
            const float mx = wave_max_f32(y);
            if (MODE == MODE_PURE8) {
                muh = mx > mu ? mx : mu;
            } else {
                const double m = (double)mu;
                if (m > __builtin_fma(__builtin_fabs(m), p->delta, (double)mx)) {
                    muh = mu;
                } else {
                    // the first lane holding the maximum; all visible lanes
                    // compute their 16-bit logit (the issue cost of one lane's)
                    const uint64_t at = __ballot(vis && y == mx);
                    const int c = __builtin_ctzll(at);
                    y16 = y16_of();
                    have16 = true;
                    const float yc = __shfl(y16, c, 64);
                    muh = yc > mu ? yc : mu;
                    if (lane == c) {
                        y = y16;
                        prec = 1;
                    }
                }
            }
        }
        float e = vis ? e_of(muh, y, prec == 1) : 0.0f;
        const double lam = mu == NEG_INF ? 0.0
                         : (mu == muh ? 1.0 : exp_doc_k((double)mu - (double)muh, [&](int i) { return edk[i]; }));
        const double S = wave_sum_f64((double)e);
        const double omh = __builtin_fma(lam, om, S);
        double S2 = S;
        if (MODE == MODE_LAMP) {
            const bool cand = prec == 0;
            const double ec = cand ? (double)e : 0.0;
            // quick acceptance of the empty recompute set: every cost is at
            // most E omega_hat, and the fp64 sorted sum stays below
            // omega_hat S_F (1 + 2^-45), so S_F <= tau omega_hat (1 - 2^-38)
            // implies that the exact greedy keeps every logit.  S_F is bounded
            // from an fp32 sum of its 64 non-negative terms (relative error
            // below 2^-17).
            const double SF = (double)wave_sum_f32(cand ? e : 0.0f) * (1.0 + 0x1p-17);
            if (!(SF <= (p->tau * omh) * (1.0 - 0x1p-38))) {
                const double tt = omh - ec;
                double kap = cand ? ec * tt : __builtin_inf();
                int idx = lane;
                // bitonic sort of (cost, lane) ascending over the wave
#pragma unroll
                for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
                    for (int j = k >> 1; j >= 1; j >>= 1) {
                        const double ok = xor_lanes(kap, j);
                        const int oi = (int)xor_lanes((uint32_t)idx, j);
                        const bool mine_less = kap < ok || (kap == ok && idx < oi);
                        const bool up = (lane & k) == 0;
                        const bool lower = (lane & j) == 0;
                        const bool keep = (lower == up) ? mine_less : !mine_less;
                        if (!keep) {
                            kap = ok;
                            idx = oi;
                        }
                    }
                }
                // the greedy: sorted costs summed one at a time in fp64, in
                // straight-line code on values read out of their lanes (the
                // index of the first cost that is infinite or would pass the
                // limit is the count kept; the sum after it is not used)
                const double lim = (p->tau * omh) * omh;
                // First from a prefix scan of the sorted costs (any
                // association), whose sums differ from the sequential ones
                // by less than 70 units of 2^-53 of the prefix: the
                // sequential sum is monotone, so the crossing is the scan's
                // when neither neighbour of it lies within 2^-44 of the limit
                // (infinite costs, last in the order, fail either way).
                int nkeep = 64;
                {
                    const double sc = prefix_sum_f64(kap);
                    const uint64_t okb = __ballot(kap != __builtin_inf() && sc <= lim);
                    const int n = okb == ~0ull ? 64 : __builtin_ctzll(~okb);
                    const bool near = (lane == n - 1 || lane == n) && kap != __builtin_inf() &&
                                      __builtin_fabs(sc - lim) <= 0x1p-44 * sc;
                    nkeep = wave_any(near) ? -1 : n;
                }
                if (nkeep < 0) {   // too close to call: the greedy itself
                    double xi = 0.0;
                    nkeep = 64;
#pragma unroll
                    for (int i = 0; i < 64; ++i) {
                        const double kk = readlane_f64(kap, i);
                        const double nx = xi + kk;
                        const bool ok = kk != __builtin_inf() && nx <= lim;
                        nkeep = (nkeep == 64 && !ok) ? i : nkeep;
                        xi = nx;
                    }
                }
                // sorted position -> key lane: each sorted slot sends its
                // recompute flag to the lane of its key (idx is a permutation)
                const int rflag = __builtin_amdgcn_ds_permute(idx << 2, (lane >= nkeep && kap != __builtin_inf()) ? 1 : 0);
                const uint64_t rbits = __ballot(rflag != 0);
                if (rbits) {
                    if (!have16) {
                        y16 = y16_of();
                        have16 = true;
                    }
                    if (rbits >> lane & 1ull) {
                        prec = 2;
                        y = y16;
                        e = e_of(muh, y, true);
                    }
                    S2 = wave_sum_f64((double)e);
                }
            }
        }
        om = __builtin_fma(lam, om, S2);
        mu = muh;
        record_tile(t, muh, lam);
        if (MODE == MODE_LAMP) sink(key, prec, prec == 1 || prec == 2);
    }

    // Runs of tiles in which nothing changes precision.  Once mu is finite, a
    // tile whose maximizer passes the look-ahead test against mu (pure 8-bit
    // mode: whose maximum does not exceed mu) keeps mu_hat = mu and lambda_hat
    // = 1, so its exponentials and sum depend on mu alone; the knapsack then
    // keeps all its logits when the quick acceptance holds against omega_hat
    // = omega + S.  Up to CH tiles are evaluated together on that assumption,
    // 64/CH lanes per tile and CH keys per lane (CH reductions at once over
    // groups of lanes); the omega chain is then replayed tile by tile in the
    // same order and rounding as in tile_exact, and the tiles up to the first
    // one where a test fails are committed.  Returns the number committed;
    // the caller passes the next tile to tile_exact.  Every committed value
    // equals what tile_exact would have produced: the maximum and the fp64
    // sum of the exponentials are exact in any order, and the fp32 sum only
    // feeds a bound that holds in any order (a tile the bound does not accept
    // here goes through the exact path, whose greedy then decides).
    // words(j, sub): the CH 8-bit codes of keys CH*sub .. CH*sub + CH-1 of
    // tile t + j, one per byte (j < nt).
    template <int CH, class Words>
    __device__ __forceinline__ int run(int t, int nt, Words words)
    {
        static_assert(CH == 4 || CH == 8, "runs of 4 or 8 tiles");
        constexpr int LPT = TK / CH;   // lanes per tile
        const float NEG_INF = -__builtin_inff();
        const int jl = lane / LPT, sub = lane % LPT;
        const int tj = t + jl;
        const bool in = jl < nt;
        const uint64_t cw = in ? words(jl, sub) : 0ull;
        const int key0 = tj * TK + CH * sub;
        float mxl = NEG_INF, sf = 0.0f;
        double sl = 0.0;
#pragma unroll
        for (int k = 0; k < CH; ++k) {
            const int key = key0 + k;
            const bool vis = in && key >= vlo && key <= vhi;
            const uint8_t code = (uint8_t)(cw >> (8 * k));
            const float y = vis ? e4m3_value(code) : NEG_INF;
            mxl = y > mxl ? y : mxl;
            const float e = vis ? bf16_value(lut[ue5m3_code(shift_of(mu, y))]) : 0.0f;
            sl += (double)e;
            sf += e;
        }
        // reductions over the lanes of each tile (quad neighbours, quad
        // pairs, half-row mirror, and for 16 lanes the row mirror)
        {
            float o;
            o = dpp_f32<0xB1>(mxl); mxl = o > mxl ? o : mxl;
            o = dpp_f32<0x4E>(mxl); mxl = o > mxl ? o : mxl;
            o = dpp_f32<0x141>(mxl); mxl = o > mxl ? o : mxl;
            if (LPT == 16) { o = dpp_f32<0x140>(mxl); mxl = o > mxl ? o : mxl; }
            sl += dpp_f64<0xB1>(sl);
            sl += dpp_f64<0x4E>(sl);
            sl += dpp_f64<0x141>(sl);
            if (LPT == 16) sl += dpp_f64<0x140>(sl);
            if (MODE == MODE_LAMP) {
                sf += dpp_f32<0xB1>(sf);
                sf += dpp_f32<0x4E>(sf);
                sf += dpp_f32<0x141>(sf);
                if (LPT == 16) sf += dpp_f32<0x140>(sf);
            }
        }
        // the look-ahead test of every tile at once (lane LPT j holds tile j's
        // maximum), then the omega chain and the quick acceptance tile by tile
        // up to the first failure, without branches
        const double m = (double)mu;
        const bool passl = MODE == MODE_PURE8 ? !(mxl > mu) : m > __builtin_fma(__builtin_fabs(m), p->delta, (double)mxl);
        constexpr uint64_t heads = LPT == 8 ? 0x0101010101010101ull : 0x0001000100010001ull;
        const uint64_t fails = ~__ballot(passl) & heads & (nt < CH ? (1ull << (LPT * nt)) - 1ull : ~0ull);
        int jc = fails ? __builtin_ctzll(fails) / LPT : nt;   // tiles committed
        double omv = om;
#pragma unroll
        for (int j = 0; j < CH; ++j) {
            const double omh = __builtin_fma(1.0, omv, readlane_f64(sl, LPT * j));
            bool ok = true;
            if (MODE == MODE_LAMP) {
                const double SF = (double)readlane_f32(sf, LPT * j) * (1.0 + 0x1p-17);
                ok = SF <= (p->tau * omh) * (1.0 - 0x1p-38);
            }
            jc = (j < jc && !ok) ? j : jc;
            omv = j < jc ? omh : omv;
        }
        om = omv;
#pragma unroll
        for (int j = 0; j < CH; ++j)
            if (j < jc) record_tile(t + j, mu, 1.0);
        return jc;
    }

    // After the chunk's last tile: the outstanding window, the row state for
    // the next chunk, and the P.V factors within the chunk, g_t = the product
    // of lambda_hat over the chunk's later tiles, from its last tile backwards
    // in runs of 64 (lane j: tile t_rec - 1 - 64c - j), with their product
    // over the whole chunk (the reduction over the chunks scales each chunk's
    // partial output by the product over the later chunks, divided by the
    // final omega).  After the last chunk also lse.
    __device__ __forceinline__ void finish(float *lse)
    {
        flush_window();
        __threadfence_block();   // the rescale factors written above, read back by every lane below
        double carry = 1.0;
        for (int t0 = t_rec - 1; t0 >= tc_lo; t0 -= 64) {
            const int tt = t0 - lane;
            const double lam = tt >= tc_lo ? frow[(size_t)tt * RR] : 1.0;
            double incl = lam;   // inclusive product over lanes 0..j
#pragma unroll
            for (int m = 1; m < 64; m <<= 1) {
                const double o = __shfl_up(incl, m, 64);
                if (lane >= m) incl *= o;
            }
            double excl = __shfl_up(incl, 1, 64);
            if (lane == 0) excl = 1.0;
            if (tt >= tc_lo) frow[(size_t)tt * RR] = carry * excl;
            carry *= __shfl(incl, 63, 64);
        }
        if (lane == 0) {
            p->lam_c[row * p->nchunks + p->chunk] = carry;
            p->mu_st[row] = mu;
            p->om_st[row] = om;
            if (p->chunk == p->nchunks - 1) *lse = (float)((double)mu + ::log(om));
        }
    }
};

// The split form's decisions: one wave per query row over the codes phase 1
// wrote.  The 8-bit logits' mask codes (0, or 3 where invisible) were written
// with the codes by phase 1 (the all-16-bit mode: 1 where visible); this
// kernel writes 3 over the tiles no key of which is visible and the codes of
// the recomputed keys.  The recomputed keys are collected in LDS and written
// at the end of the row (or when the list is full).
constexpr int REC_CAP = 256;   // recomputed keys held in LDS per wave

template <int MODE>
struct DecideLds {
    uint8_t cbuf[4][MODE != MODE_ALL16 ? 32 * TK : 1];    // per wave: rings of two
    uint16_t hbuf[4][MODE != MODE_PURE8 ? 32 * TK : 1];   // blocks of 16 tiles' codes
    int rec_key[4][MODE == MODE_LAMP ? REC_CAP : 1];
    uint8_t rec_code[4][MODE == MODE_LAMP ? REC_CAP : 1];
    uint16_t lut[256];
    double edk[EXPDOC_NK];
};

// Workgroup bx of the decisions over the launch's key chunk: query rows
// 4 bx .. 4 bx + 3, one wave each.
template <int D, int MODE>
__device__ __forceinline__ void dec_decide_role(const DecParams &p, DecideLds<MODE> &sm, int bx)
{
    uint16_t *lut = sm.lut;
    double *edk = sm.edk;
    auto &cbuf = sm.cbuf;
    auto &hbuf = sm.hbuf;
    auto &rec_key = sm.rec_key;
    auto &rec_code = sm.rec_code;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    for (int i = tid; i < 256; i += 256) lut[i] = p.lut8e[i];
    if (tid < EXPDOC_NK) edk[tid] = EXPDOC_K[tid];
    __syncthreads();

    const int64_t nrows = (int64_t)p.B * p.Hq * p.M;
    const int64_t row = (int64_t)bx * 4 + wv;
    if (row >= nrows) return;   // whole wave
    // the decisions are bound by the latency of their dependent chains: a
    // higher wave priority lets them issue as soon as they are ready beside
    // the other key chunks' logit and P.V workgroups
    __builtin_amdgcn_s_setprio(2);
    RowDecider<MODE> d;
    d.start(p, lut, edk, row, lane);
    // this launch's tiles of the row (t_begin, t_end: the chunk's part of the
    // visible range)
    const int t_begin = d.tc_lo, t_end = d.tc_hi;
    const int ntiles = p.Np / TK;
    const uint8_t *y8row = p.y8 + row * (size_t)p.Np;
    const uint16_t *y16row = p.y16 + row * (size_t)p.Np;
    uint8_t *mrow = p.mask + row * (size_t)p.Np;

    // the chunk's tiles without a visible key (phase 1 wrote the same code
    // for those it covers; the first chunk also covers the keys before kb0)
    {
        const int lo = p.chunk == 0 ? 0 : p.ka / TK, hi = p.chunk == p.nchunks - 1 ? ntiles : p.kz / TK;
        for (int t = lo + lane; t < hi; t += 64)
            if (t < d.t_begin || t > d.t_end)
                for (int i = 0; i < TK; ++i) mrow[t * TK + i] = 3;
    }

    // recomputed keys of this row (LDS list)
    int nrec = 0;
    auto flush_rec = [&]() {
        for (int i = lane; i < nrec; i += 64) mrow[rec_key[wv][i]] = rec_code[wv][i];
        nrec = 0;
    };
    auto sink = [&](int key, uint8_t prec, bool recd) {
        const uint64_t rb = __ballot(recd);
        if (rb) {
            if (nrec + 64 > REC_CAP) flush_rec();
            if (recd) {
                const int pos = nrec + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(rb >> 32),
                                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)rb, 0u));
                rec_key[wv][pos] = key;
                rec_code[wv][pos] = prec;
            }
            nrec += __builtin_popcountll(rb);
        }
    };

    // The logit codes arrive 16 tiles (a block) at a time: per lane keys
    // 16 lane .. 16 lane + 15 of the block (one 16-byte load of 8-bit codes,
    // two of 16-bit codes), held in registers one block ahead and passed
    // through this wave's LDS rings of two blocks, so no load is waited for
    // inside the tile loop.
    uint8_t *cb = cbuf[wv];
    uint16_t *hb = hbuf[wv];
    uint4 nxt8 = make_uint4(0u, 0u, 0u, 0u), nxt16a = nxt8, nxt16b = nxt8;
    auto load_block = [&](int kb) {
        const int tb = t_begin + 16 * kb;
        const int k = tb * TK + 16 * lane;
        const bool ok = tb <= t_end && k + 16 <= p.Np;
        if (MODE != MODE_ALL16) nxt8 = ok ? *reinterpret_cast<const uint4 *>(y8row + k) : make_uint4(0u, 0u, 0u, 0u);
        if (MODE != MODE_PURE8) {
            nxt16a = ok ? *reinterpret_cast<const uint4 *>(y16row + k) : make_uint4(0u, 0u, 0u, 0u);
            nxt16b = ok ? *reinterpret_cast<const uint4 *>(y16row + k + 8) : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    load_block(0);
    int kn = 0;   // blocks below kn are in the rings; the registers hold block kn
    // make the codes of every tile up to t_hi readable (LDS operations of a
    // wave stay in order; the ring slot written held a block two behind)
    auto ensure = [&](int t_hi) {
        while ((t_hi - t_begin) >> 4 >= kn) {
            if (MODE != MODE_ALL16) *reinterpret_cast<uint4 *>(cb + (kn & 1) * 16 * TK + 16 * lane) = nxt8;
            if (MODE != MODE_PURE8) {
                *reinterpret_cast<uint4 *>(hb + (kn & 1) * 16 * TK + 16 * lane) = nxt16a;
                *reinterpret_cast<uint4 *>(hb + (kn & 1) * 16 * TK + 16 * lane + 8) = nxt16b;
            }
            ++kn;
            load_block(kn);
        }
    };
    auto exact = [&](int t) {
        const uint32_t code = MODE != MODE_ALL16 ? cb[((t - t_begin) & 31) * TK + lane] : 0u;
        d.tile_exact(t, code, [&]() { return e4m11_value(hb[((t - t_begin) & 31) * TK + lane]); }, sink);
    };
    constexpr int CH = 8;
    int t = t_begin;
    while (t <= t_end) {
        if (MODE == MODE_ALL16 || d.mu == -__builtin_inff()) {
            ensure(t);
            exact(t);
            ++t;
            continue;
        }
        const int nt = t_end - t + 1 < CH ? t_end - t + 1 : CH;
        ensure(t + nt - 1);
        const int jc = d.template run<CH>(t, nt, [&](int j, int sub) -> uint64_t {
            const uint2 w = *reinterpret_cast<const uint2 *>(cb + ((t + j - t_begin) & 31) * TK + CH * sub);
            return ((uint64_t)w.y << 32) | w.x;
        });
        t += jc;
        if (jc < nt) {
            exact(t);
            ++t;
        }
    }
    if (MODE == MODE_LAMP) flush_rec();
    d.finish(p.lse + row);
}

// ------------------------------------------------------------------ phase 3
// P.V: one workgroup per (piece of PV_CHUNK keys of the launch's key chunk,
// b, key/value head) for NR of the R = G*M query rows of the head.  The
// piece's weights E g_t of those rows are first formed in LDS: E from the
// key's mask code and logit (the 8-bit code through the ue5m3 table, or the
// recomputed 16-bit logit through the ue5m11 table) against the tile's
// mu_hat, the same computation as in the decisions, and g_t the tile's factor
// within its chunk; then the main loop issues one 16-byte load of V (8
// channels of one key) per lane and key, one step ahead of its arithmetic
// (the first step before the weights), feeding 8 FMAs per query row, and
// reads the key's weights from LDS (one broadcast read).  Partial outputs per
// piece go to a workspace; the reduce kernel combines them over the chunks.
constexpr int PV_CHUNK = DEC_PV_KEYS, PV_ROWS = 16;

template <int D, int NR>
struct PvLds {
    float wl[PV_CHUNK][NR];
    float red[4][NR][D];
    uint16_t lut[256];
};

// Workgroup (bx, by) of P.V over the launch's key chunk: keys ka + 512 bx ..,
// key/value head by, its query rows rg0 .. rg0 + NR - 1.
template <int D, int NR>
__device__ __forceinline__ void dec_pv_role(const DecParams &p, PvLds<D, NR> &sm, int bx, int by, int rg0)
{
    constexpr int CC = D / 8, KG = 256 / CC;   // channel chunks; keys per step over the workgroup
    auto &wl = sm.wl;
    auto &red = sm.red;
    uint16_t *lut = sm.lut;
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
    const int cc = tid % CC, kg = tid / CC;
    const int chunk = bx;
    const int bhk = by;
    const int b = bhk / p.Hkv, hk = bhk % p.Hkv;
    const int G = p.Hq / p.Hkv, RR = G * p.M;
    const int ntiles = p.Np / TK;
    const int k0 = p.ka + chunk * PV_CHUNK;
    const int k_end = k0 + PV_CHUNK < p.N ? k0 + PV_CHUNK : p.N;
    const int pvc = (k0 - p.kb0) / PV_CHUNK;   // this piece among the call's
    for (int i = tid; i < 256; i += 256) lut[i] = p.lut8e[i];
    // U keys of V per step and lane (8 channels each), the first step's loads
    // issued before the weights are formed and every later step's one step
    // ahead of its arithmetic (keys past the chunk read a valid row and have
    // weight 0)
    constexpr int U = 4, STEPS = PV_CHUNK / (U * KG);
    const uint16_t *vbase = p.v + (size_t)bhk * p.N * D + cc * 8;
    uint4 vbuf[2][U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int key = k0 + kg + u * KG;
        vbuf[0][u] = *reinterpret_cast<const uint4 *>(vbase + (size_t)(key < k_end ? key : k_end - 1) * D);
    }
    __syncthreads();
    // the weights, 8 per thread at a time with all their loads issued together
    // (consecutive threads: consecutive keys of one row)
    constexpr int EB = 8;
    for (int x0 = tid; x0 < PV_CHUNK * NR; x0 += 256 * EB) {
        uint32_t mc[EB], c8[EB];
        float muv[EB];
        double fv[EB];
        size_t at[EB];
#pragma unroll
        for (int e = 0; e < EB; ++e) {
            const int x = x0 + 256 * e;
            const int i = x / PV_CHUNK, kl = x % PV_CHUNK;
            const int key = k0 + kl, rho = rg0 + i;
            const bool valid = x < PV_CHUNK * NR && key < k_end && rho < RR;
            const int64_t rid = ((int64_t)b * p.Hq + hk * G + rho / p.M) * p.M + rho % p.M;
            at[e] = (size_t)rid * p.Np + key;
            const size_t tat = ((size_t)bhk * ntiles + key / TK) * RR + rho;
            mc[e] = valid ? p.mask[at[e]] : 3u;
            c8[e] = valid ? p.y8[at[e]] : 0u;
            muv[e] = valid ? p.mut[tat] : 0.0f;
            fv[e] = valid ? p.f[tat] : 0.0;
        }
#pragma unroll
        for (int e = 0; e < EB; ++e) {
            const int x = x0 + 256 * e;
            if (x >= PV_CHUNK * NR) break;
            float wgt = 0.0f;
            if (mc[e] != 3u) {
                float ev;
                if (mc[e] == 0u) {
                    ev = bf16_value(lut[ue5m3_code(shift_of(muv[e], e4m3_value(c8[e])))]);
                } else {
                    const uint32_t hl = p.exp16hl[ue5m11_code(shift_of(muv[e], e4m11_value(p.y16[at[e]])))];
                    ev = bf16_value(hl & 0xFFFFu) + bf16_value(hl >> 16);   // exact
                }
                wgt = ev * (float)fv[e];
            }
            wl[x % PV_CHUNK][x / PV_CHUNK] = wgt;
        }
    }
    __syncthreads();
    float acc[NR][8];
#pragma unroll
    for (int i = 0; i < NR; ++i)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[i][c] = 0.0f;
#pragma clang loop unroll(full)
    for (int st = 0; st < STEPS; ++st) {
        if (st + 1 < STEPS) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int key = k0 + kg + (st + 1) * U * KG + u * KG;
                vbuf[(st + 1) & 1][u] = *reinterpret_cast<const uint4 *>(vbase + (size_t)(key < k_end ? key : k_end - 1) * D);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float vf[8];
            unpack8(vbuf[st & 1][u], vf);
            const int kl = kg + st * U * KG + u * KG;
#pragma unroll
            for (int i = 0; i < NR; ++i) {
                const float wgt = wl[kl][i];
#pragma unroll
                for (int c = 0; c < 8; ++c) acc[i][c] = __builtin_fmaf(wgt, vf[c], acc[i][c]);
            }
        }
    }
    // lanes with the same channel chunk: add over the key groups of the wave,
    // then over the 4 waves through LDS
#pragma unroll
    for (int m = CC; m < 64; m <<= 1)
#pragma unroll
        for (int i = 0; i < NR; ++i)
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[i][c] += __shfl_xor(acc[i][c], m, 64);
    if (lane < CC)
#pragma unroll
        for (int i = 0; i < NR; ++i)
#pragma unroll
            for (int c = 0; c < 8; ++c) red[w][i][cc * 8 + c] = acc[i][c];
    __syncthreads();
    const int nch = (p.N - p.kb0 + PV_CHUNK - 1) / PV_CHUNK;
    for (int x = tid; x < NR * D; x += 256) {
        const int i = x / D, c = x % D;
        const int rho = rg0 + i;
        if (rho >= RR) continue;
        const float v = red[0][i][c] + red[1][i][c] + red[2][i][c] + red[3][i][c];
        const int64_t rid = ((int64_t)b * p.Hq + hk * G + rho / p.M) * p.M + rho % p.M;
        p.part[((size_t)rid * nch + pvc) * D + c] = v;
    }
}

// ------------------------------------------------------------------ kernels
template <int D, int MODE>
__global__ __launch_bounds__(256) void dec_logits_kernel(DecParams p)
{
    __shared__ __align__(16) LogitsLds<D> sm;
    dec_logits_role<D, MODE>(p, sm, (int)blockIdx.x, (int)blockIdx.y);
}

template <int D, int MODE>
__global__ __launch_bounds__(256) void dec_lamp_kernel(DecParams p)
{
    __shared__ __align__(16) DecideLds<MODE> sm;
    dec_decide_role<D, MODE>(p, sm, (int)blockIdx.x);
}

template <int D, int NR>
__global__ __launch_bounds__(256) void dec_pv_kernel(DecParams p, int rg0)
{
    __shared__ __align__(16) PvLds<D, NR> sm;
    dec_pv_role<D, NR>(p, sm, (int)blockIdx.x, (int)blockIdx.y, rg0);
}

// One stage of the key-chunk pipeline: the decisions of chunk c - 1, the
// logits of chunk c and P.V of chunk c - 2 in one launch (each part may be
// empty; pd, pl, pp carry the chunks).  Stages run in order on one stream, so
// every part finds what it reads complete; within a stage the three overlap:
// the decisions (bound by the latency of their reductions, at a higher wave
// priority) take the first nd workgroups, then the logit workgroups (bound by
// the VALU) and the P.V ones (bound by HBM) are interleaved in proportion.
// The workgroups share one LDS buffer laid out per part.
template <int D, int MODE, int NR>
__global__ __launch_bounds__(256) void dec_stage_kernel(DecParams pd, DecParams pl, DecParams pp, int nd, int nl_x,
                                                        int nl, int np_x, int np)
{
    constexpr size_t A = sizeof(LogitsLds<D>), B = sizeof(DecideLds<MODE>), C = sizeof(PvLds<D, NR>);
    constexpr size_t AB = A > B ? A : B, ABC = AB > C ? AB : C;
    __shared__ __align__(16) unsigned char buf[ABC];
    const int bid = (int)blockIdx.x;
    if (bid < nd) {
        dec_decide_role<D, MODE>(pd, *reinterpret_cast<DecideLds<MODE> *>(buf), bid);
        return;
    }
    // the r-th of the other workgroups: logits when floor((r + 1) nl / T)
    // passes floor(r nl / T) (their index), P.V otherwise
    const int64_t r = bid - nd, T = (int64_t)nl + np;
    const int64_t il = r * nl / T;
    if ((r + 1) * nl / T > il) {
        dec_logits_role<D, MODE>(pl, *reinterpret_cast<LogitsLds<D> *>(buf), (int)(il % nl_x), (int)(il / nl_x));
    } else {
        const int64_t ip = r - il;
        const int per = np_x * pp.B * pp.Hkv;   // workgroups per group of NR rows
        const int rg = (int)(ip / per), rem = (int)(ip % per);
        dec_pv_role<D, NR>(pp, *reinterpret_cast<PvLds<D, NR> *>(buf), rem % np_x, rem / np_x, rg * NR);
    }
}

// ------------------------------------------------------------------ phase 4
// O = sum over the key chunks c of F_c times the sum of chunk c's partial
// outputs, F_c = (product of the later chunks' lambda_hat products) / omega.
// Thread x: channels 4 (x % (D/4)) .. + 3 of row x / (D/4), the pieces of a
// chunk read four at a time.
template <int D>
__global__ __launch_bounds__(256) void dec_reduce_kernel(DecParams p)
{
    constexpr int Q = D / 4;
    const int64_t nrows = (int64_t)p.B * p.Hq * p.M;
    const int nch = (p.N - p.kb0 + PV_CHUNK - 1) / PV_CHUNK, per = p.ck / PV_CHUNK;
    const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (x >= nrows * Q) return;
    const int64_t row = x / Q;
    const int c4 = (int)(x % Q) * 4;
    const float4 *part = reinterpret_cast<const float4 *>(p.part + row * nch * D + c4);
    double fc = 1.0 / p.om_st[row];
    float4 s = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int cc = p.nchunks - 1; cc >= 0; --cc) {
        const int a = cc * per, z = (cc + 1) * per < nch ? (cc + 1) * per : nch;
        float4 sc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll 4
        for (int ch = a; ch < z; ++ch) {
            const float4 v = part[(size_t)ch * (D / 4)];
            sc.x += v.x;
            sc.y += v.y;
            sc.z += v.z;
            sc.w += v.w;
        }
        const float f = (float)fc;
        s.x += f * sc.x;
        s.y += f * sc.y;
        s.z += f * sc.z;
        s.w += f * sc.w;
        fc *= p.lam_c[row * p.nchunks + cc];
    }
    float *o = p.o + row * D + c4;
    if (((uintptr_t)p.o & 15u) == 0u) {
        *reinterpret_cast<float4 *>(o) = s;
    } else {
        o[0] = s.x;
        o[1] = s.y;
        o[2] = s.z;
        o[3] = s.w;
    }
}

// ------------------------------------------------------------------ launchers
template <int D>
static hipError_t dec_logits_d(const DecParams &p, hipStream_t s)
{
    const int G = p.Hq / p.Hkv, ngroups = (G * p.M + 3) / 4;
    const int kend = p.kz < p.N ? p.kz : p.N;
    dim3 g((unsigned)((kend - p.ka + 255) / 256), (unsigned)(p.B * p.Hkv * ngroups));
    if (p.mode == MODE_PURE8) hipLaunchKernelGGL((dec_logits_kernel<D, MODE_PURE8>), g, dim3(256), 0, s, p);
    else if (p.mode == MODE_ALL16) hipLaunchKernelGGL((dec_logits_kernel<D, MODE_ALL16>), g, dim3(256), 0, s, p);
    else hipLaunchKernelGGL((dec_logits_kernel<D, MODE_LAMP>), g, dim3(256), 0, s, p);
    return hipGetLastError();
}

template <int D>
static hipError_t dec_decide_d(const DecParams &p, hipStream_t s)
{
    const int64_t nrows = (int64_t)p.B * p.Hq * p.M;
    dim3 g((unsigned)((nrows + 3) / 4));
    if (p.mode == MODE_PURE8) hipLaunchKernelGGL((dec_lamp_kernel<D, MODE_PURE8>), g, dim3(256), 0, s, p);
    else if (p.mode == MODE_ALL16) hipLaunchKernelGGL((dec_lamp_kernel<D, MODE_ALL16>), g, dim3(256), 0, s, p);
    else hipLaunchKernelGGL((dec_lamp_kernel<D, MODE_LAMP>), g, dim3(256), 0, s, p);
    return hipGetLastError();
}

template <int D>
static hipError_t dec_pv_d(const DecParams &p, hipStream_t s)
{
    const int rows = (p.Hq / p.Hkv) * p.M;
    const int kend = p.kz < p.N ? p.kz : p.N;
    dim3 g((unsigned)((kend - p.ka + PV_CHUNK - 1) / PV_CHUNK), (unsigned)(p.B * p.Hkv));
    for (int rg0 = 0; rg0 < rows; rg0 += PV_ROWS) {
        const int nr = rows - rg0;
        if (nr <= 4) hipLaunchKernelGGL((dec_pv_kernel<D, 4>), g, dim3(256), 0, s, p, rg0);
        else if (nr <= 8) hipLaunchKernelGGL((dec_pv_kernel<D, 8>), g, dim3(256), 0, s, p, rg0);
        else hipLaunchKernelGGL((dec_pv_kernel<D, PV_ROWS>), g, dim3(256), 0, s, p, rg0);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int D>
static hipError_t dec_reduce_d(const DecParams &p, hipStream_t s)
{
    const int64_t nrows = (int64_t)p.B * p.Hq * p.M;
    hipLaunchKernelGGL(dec_reduce_kernel<D>, dim3((unsigned)((nrows * (D / 4) + 255) / 256)), dim3(256), 0, s, p);
    return hipGetLastError();
}

// One pipeline stage (dec_stage_kernel); a null part is empty.
template <int D, int MODE, int NR>
static hipError_t dec_stage_dmn(const DecParams *pd, const DecParams *pl, const DecParams *pp, hipStream_t s)
{
    const DecParams &any = pd ? *pd : pl ? *pl : *pp;
    const int G = any.Hq / any.Hkv, rows = G * any.M, ngroups = (rows + 3) / 4;
    const int64_t nrows = (int64_t)any.B * any.Hq * any.M;
    const int nd = pd ? (int)((nrows + 3) / 4) : 0;
    int nl_x = 1, nl = 0, np_x = 1, np = 0;
    if (pl) {
        const int kend = pl->kz < pl->N ? pl->kz : pl->N;
        nl_x = (kend - pl->ka + 255) / 256;
        nl = nl_x * pl->B * pl->Hkv * ngroups;
    }
    if (pp) {
        const int kend = pp->kz < pp->N ? pp->kz : pp->N;
        np_x = (kend - pp->ka + PV_CHUNK - 1) / PV_CHUNK;
        np = np_x * pp->B * pp->Hkv * ((rows + NR - 1) / NR);
    }
    const DecParams &d0 = pd ? *pd : any, &l0 = pl ? *pl : any, &p0 = pp ? *pp : any;
    hipLaunchKernelGGL((dec_stage_kernel<D, MODE, NR>), dim3((unsigned)(nd + nl + np)), dim3(256), 0, s, d0, l0, p0, nd,
                       nl_x, nl, np_x, np);
    return hipGetLastError();
}

template <int D, int MODE>
static hipError_t dec_stage_dm(const DecParams *pd, const DecParams *pl, const DecParams *pp, hipStream_t s)
{
    const DecParams &any = pd ? *pd : pl ? *pl : *pp;
    if ((any.Hq / any.Hkv) * any.M <= 4) return dec_stage_dmn<D, MODE, 4>(pd, pl, pp, s);
    return dec_stage_dmn<D, MODE, 8>(pd, pl, pp, s);
}

template <int D>
static hipError_t dec_stage_d(const DecParams *pd, const DecParams *pl, const DecParams *pp, hipStream_t s)
{
    const DecParams &any = pd ? *pd : pl ? *pl : *pp;
    if (any.mode == MODE_PURE8) return dec_stage_dm<D, MODE_PURE8>(pd, pl, pp, s);
    if (any.mode == MODE_ALL16) return dec_stage_dm<D, MODE_ALL16>(pd, pl, pp, s);
    return dec_stage_dm<D, MODE_LAMP>(pd, pl, pp, s);
}

#define LAMP_DEC_BY_D(fn, ...)                                  \
    if (D == 64) return fn<64>(__VA_ARGS__);                    \
    if (D == 128) return fn<128>(__VA_ARGS__);                  \
    if (D == 256) return fn<256>(__VA_ARGS__);                  \
    return hipErrorInvalidValue;

hipError_t launch_dec_logits(int D, const DecParams &p, hipStream_t s) { LAMP_DEC_BY_D(dec_logits_d, p, s) }
hipError_t launch_dec_decide(int D, const DecParams &p, hipStream_t s) { LAMP_DEC_BY_D(dec_decide_d, p, s) }
hipError_t launch_dec_pv(int D, const DecParams &p, hipStream_t s) { LAMP_DEC_BY_D(dec_pv_d, p, s) }
hipError_t launch_dec_reduce(int D, const DecParams &p, hipStream_t s) { LAMP_DEC_BY_D(dec_reduce_d, p, s) }
hipError_t launch_dec_stage(int D, const DecParams *pd, const DecParams *pl, const DecParams *pp, hipStream_t s)
{
    if (!pd && !pl && !pp) return hipSuccess;
    LAMP_DEC_BY_D(dec_stage_d, pd, pl, pp, s)
}

#undef LAMP_DEC_BY_D

} // namespace lamp
