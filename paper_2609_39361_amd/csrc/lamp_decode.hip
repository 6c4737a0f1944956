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
// Four kernels:
//   dec_logits8_kernel  the 8-bit logits of every (query row, key), which
//                       depend on no decision: one thread per key, the 4 query
//                       rows of a group accumulated together, queries read
//                       from LDS (broadcast), keys staged through LDS from
//                       coalesced loads of the bf16 cache (no fp32 copy);
//   dec_lamp_kernel     the decisions, one wave per query row: lane i holds
//                       key i of the tile; DPP reductions, a bitonic sort of
//                       the costs and the sequential sum; it writes the
//                       exponentials and per-tile rescale factors;
//   dec_pv_kernel       P.V in parallel over key chunks for all query rows of
//                       a key/value head (fp32 FMAs; every exponential is
//                       exact in fp32);
//   dec_reduce_kernel   the sum of the chunks' partial outputs.
#include <hip/hip_runtime.h>
#include <stdint.h>

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

// 16-bit logit of this lane's key: the FP32 FMA chain over the channels in
// ascending order from +0, rounded once to e4m11 (saturating).  The key row's
// loads are all issued before the chain starts: the decision loop waits for
// this recompute, so its cost is one memory round trip, not one per group.
template <int D>
__device__ __forceinline__ float dec16_chain(const uint16_t *krow, kptr32_t q)
{
    uint4 kw[D / 8];
#pragma unroll
    for (int g = 0; g < D / 8; ++g) kw[g] = *reinterpret_cast<const uint4 *>(krow + 8 * g);
    float acc = 0.0f;
#pragma unroll
    for (int g = 0; g < D / 8; ++g) {
        float kf[8];
        unpack8(kw[g], kf);
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = __builtin_fmaf(q[8 * g + j], kf[j], acc);
    }
    uint32_t code;
    return rn_e4m11((double)acc, &code);
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
// grid (key blocks of 256 from key kb0, B * Hkv * row groups); a row group is
// 4 consecutive rows of the G*M query rows of one key/value head (row rho is
// query head hk*G + rho / M, query r = rho % M).  Thread t owns key
// kb0 + 256 blockIdx.x + t.  The keys reach LDS in stages of 64 channels with
// coalesced 16-byte loads (8 threads per 128-byte key row), so each global
// load instruction covers whole cache lines; every thread then reads its own
// row from LDS (pitch 72 bf16 against bank conflicts).
constexpr int P1_CH = 64, P1_PITCH = P1_CH + 8;

template <int D, bool SAT>
__device__ __forceinline__ void dec8_staged(const uint16_t *kblk, int nvalid, uint16_t *tile, const float *qs,
                                            uint32_t (&acc)[2])
{
    const int tid = threadIdx.x;
    acc[0] = acc[1] = 0u;
    for (int c0 = 0; c0 < D; c0 += P1_CH) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int x = tid + 256 * j, key = x >> 3, part = x & 7;
            const int kc = key < nvalid ? key : nvalid - 1;   // rows beyond N repeat the last key (not stored)
            const uint4 w = *reinterpret_cast<const uint4 *>(kblk + (size_t)kc * D + c0 + part * 8);
            *reinterpret_cast<uint4 *>(tile + key * P1_PITCH + part * 8) = w;
        }
        __syncthreads();
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
                const float2 a = unpk_e4m3(acc[0]);
                const float x = __builtin_fmaf(qv[0][j], kf[j], a.x);
                const float y = __builtin_fmaf(qv[1][j], kf[j], a.y);
                acc[0] = SAT ? pk_e4m3_sat(x, y, acc[0]) : pk_e4m3(x, y, acc[0]);
                const float2 bb = unpk_e4m3(acc[1]);
                const float z = __builtin_fmaf(qv[2][j], kf[j], bb.x);
                const float u = __builtin_fmaf(qv[3][j], kf[j], bb.y);
                acc[1] = SAT ? pk_e4m3_sat(z, u, acc[1]) : pk_e4m3(z, u, acc[1]);
            }
        }
        __syncthreads();   // the tile is overwritten by the next stage
    }
}

template <int D>
__global__ __launch_bounds__(256) void dec_logits8_kernel(DecParams p)
{
    __shared__ __align__(16) uint16_t tile[256 * P1_PITCH];
    __shared__ __align__(16) float qs[4 * D];   // the group's 4 pre-scaled query rows
    const int G = p.Hq / p.Hkv;
    const int rows = G * p.M, ngroups = (rows + 3) / 4;
    const int grp = (int)(blockIdx.y % (unsigned)ngroups);
    const int bhk = (int)(blockIdx.y / (unsigned)ngroups);
    const int b = bhk / p.Hkv, hk = bhk % p.Hkv;
    const int key0 = p.kb0 + (int)blockIdx.x * 256;
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
    for (int x = (int)threadIdx.x; x < 4 * D; x += 256) qs[x] = p.qt[qrow[x / D] * D + x % D];
    __syncthreads();
    uint32_t acc[2];
    dec8_staged<D, false>(kblk, nvalid, tile, qs, acc);
    // an overflow somewhere gives a NaN code at the end of its chain: the
    // workgroup re-runs its chains with the saturating conversion
    if (__syncthreads_or((e4m3_nan_bits(acc[0]) | e4m3_nan_bits(acc[1])) != 0u))
        dec8_staged<D, true>(kblk, nvalid, tile, qs, acc);
    if (key >= p.N) return;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        if (grp * 4 + i < rows) p.y8[qrow[i] * (size_t)p.Np + key] = (uint8_t)(acc[i >> 1] >> (8 * (i & 1)));
}

// ------------------------------------------------------------------ phase 2
// The decisions, one wave per query row.  The output does not feed any
// decision, so this kernel writes the exponentials of every visible key (and
// 0 for invisible keys of the visited tiles) and, per visited tile, the
// factor f_t = (prod of lambda_hat of the later tiles) / omega that turns them
// into the final weights of P.V: O = sum_t f_t sum_{i in t} E_i v_i.  Both are
// stored with the R = G*M query rows of a key/value head interleaved
// (e [b][hk][key][rho], f [b][hk][tile][rho]) for the P.V kernel.
template <int D, int MODE>
__global__ __launch_bounds__(256) void dec_lamp_kernel(DecParams p)
{
    __shared__ uint16_t lut[256];
    __shared__ double edk[EXPDOC_NK];
    __shared__ __align__(16) uint8_t cbuf[4][16 * TK];   // per wave: the codes of 16 tiles
    const int tid = threadIdx.x, lane = tid & 63;
    for (int i = tid; i < 256; i += 256) lut[i] = p.lut8e[i];
    if (tid < EXPDOC_NK) edk[tid] = EXPDOC_K[tid];
    __syncthreads();

    const int64_t nrows = (int64_t)p.B * p.Hq * p.M;
    const int64_t row = (int64_t)blockIdx.x * 4 + (tid >> 6);
    if (row >= nrows) return;   // whole wave
    const int r = (int)(row % p.M);
    const int h = (int)((row / p.M) % p.Hq);
    const int b = (int)(row / ((int64_t)p.M * p.Hq));
    const int G = p.Hq / p.Hkv, hk = h / G;
    const int RR = G * p.M, rho = (h - hk * G) * p.M + r;   // rows of the head, this row's slot
    const int P = p.N - p.M + r;   // the query's position
    const int vlo = p.window > 0 ? (P - p.window + 1 > 0 ? P - p.window + 1 : 0) : 0;
    const int vhi = p.causal ? P : p.N - 1;
    const int t_begin = vlo / TK, t_end = vhi / TK;
    const int ntiles = p.Np / TK;
    const kptr32_t qv = (kptr32_t)(p.qt + row * D);
    const uint16_t *kbase = p.k + ((size_t)b * p.Hkv + hk) * (size_t)p.N * D;
    const uint8_t *y8row = p.y8 + row * (size_t)p.Np;
    float *erow = p.e + ((size_t)b * p.Hkv + hk) * (size_t)p.Np * RR + rho;          // stride RR per key
    double *frow = p.f + ((size_t)b * p.Hkv + hk) * (size_t)ntiles * RR + rho;       // stride RR per tile
    uint8_t *mrow = p.mask + row * (size_t)p.Np;
    const float NEG_INF = -__builtin_inff();
    float mu = NEG_INF;
    double om = 0.0;

    // tiles without a visible key
    for (int t = lane; t < ntiles; t += 64)
        if (t < t_begin || t > t_end)
            for (int i = 0; i < TK; ++i) mrow[t * TK + i] = 3;

    // The 8-bit logit codes arrive 16 tiles at a time: one 16-byte load per
    // lane (keys 16 lane .. 16 lane + 15 of the block), held in registers one
    // block ahead and passed through this wave's LDS buffer, so no global load
    // is waited for inside the tile loop (on gfx950 a wait for a load also
    // waits for every earlier store of the wave).
    uint8_t *cb = cbuf[tid >> 6];
    auto load_block = [&](int tb) -> uint4 {
        const int k = tb * TK + 16 * lane;
        return (MODE != MODE_ALL16 && tb <= t_end && k + 16 <= p.Np) ? *reinterpret_cast<const uint4 *>(y8row + k)
                                                                      : make_uint4(0u, 0u, 0u, 0u);
    };
    uint4 nxt = load_block(t_begin);
    for (int t = t_begin; t <= t_end; ++t) {
        const int key = t * TK + lane;
        const bool vis = key >= vlo && key <= vhi;   // vhi < N
        const int tb = (t - t_begin) & 15;
        if (MODE != MODE_ALL16 && tb == 0) {
            *reinterpret_cast<uint4 *>(cb + 16 * lane) = nxt;   // LDS operations of a wave stay in order
            nxt = load_block(t + 16);
        }
        const uint8_t code = MODE != MODE_ALL16 ? cb[tb * TK + lane] : (uint8_t)0;
        const int keyc = key < p.N ? key : p.N - 1;
        const uint16_t *krow = kbase + (size_t)keyc * D;
        float y = NEG_INF;   // this key's logit in the precision chosen for it
        uint8_t prec = vis ? 0 : 3;
        bool have16 = false;
        float y16 = 0.0f;
        float muh;
        if (MODE == MODE_ALL16) {
            y16 = dec16_chain<D>(krow, qv);
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
                if (m > __builtin_fma(__builtin_fabs(m), p.delta, (double)mx)) {
                    muh = mu;
                } else {
                    // the first lane holding the maximum; all visible lanes
                    // compute their 16-bit logit (the issue cost of one lane's)
                    const uint64_t at = __ballot(vis && y == mx);
                    const int c = __builtin_ctzll(at);
                    y16 = dec16_chain<D>(krow, qv);
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
        auto e_of = [&](float yy, bool high) -> float {
            if (high) {
                const uint32_t hl = p.exp16hl[ue5m11_code(shift_of(muh, yy))];
                return bf16_value(hl & 0xFFFFu) + bf16_value(hl >> 16);   // exact
            }
            return bf16_value(lut[ue5m3_code(shift_of(muh, yy))]);
        };
        float e = vis ? e_of(y, prec == 1) : 0.0f;
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
            if (!(SF <= (p.tau * omh) * (1.0 - 0x1p-38))) {
                const double tt = omh - ec;
                double kap = cand ? ec * tt : __builtin_inf();
                int idx = lane;
                // bitonic sort of (cost, lane) ascending over the wave
#pragma unroll
                for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
                    for (int j = k >> 1; j >= 1; j >>= 1) {
                        const double ok = __shfl_xor(kap, j, 64);
                        const int oi = __shfl_xor(idx, j, 64);
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
                const double lim = (p.tau * omh) * omh;
                double xi = 0.0;
                int nkeep = 64;
#pragma unroll
                for (int i = 0; i < 64; ++i) {
                    const double kk = readlane_f64(kap, i);
                    const double nx = xi + kk;
                    const bool ok = kk != __builtin_inf() && nx <= lim;
                    nkeep = (nkeep == 64 && !ok) ? i : nkeep;
                    xi = nx;
                }
                // sorted position -> key lane: each sorted slot sends its
                // recompute flag to the lane of its key (idx is a permutation)
                const int rflag = __builtin_amdgcn_ds_permute(idx << 2, (lane >= nkeep && kap != __builtin_inf()) ? 1 : 0);
                const uint64_t rbits = __ballot(rflag != 0);
                if (rbits) {
                    if (!have16) {
                        y16 = dec16_chain<D>(krow, qv);
                        have16 = true;
                    }
                    if (rbits >> lane & 1ull) {
                        prec = 2;
                        y = y16;
                        e = e_of(y, true);
                    }
                    S2 = wave_sum_f64((double)e);
                }
            }
        }
        om = __builtin_fma(lam, om, S2);
        mu = muh;
        erow[(size_t)key * RR] = e;
        mrow[key] = prec;
        if (lane == 0) frow[(size_t)t * RR] = lam;
    }
    if (lane == 0) p.lse[row] = (float)((double)mu + ::log(om));
    __threadfence_block();   // lane 0's rescale factors, read back by every lane below
    // f_t = (prod over the later visited tiles of lambda_hat) / omega, from the
    // last tile backwards in chunks of 64 (lane j: tile t_end - 64c - j)
    double carry = 1.0 / om;
    for (int t0 = t_end; t0 >= t_begin; t0 -= 64) {
        const int t = t0 - lane;
        const double lam = t >= t_begin ? frow[(size_t)t * RR] : 1.0;
        double incl = lam;   // inclusive product over lanes 0..j
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) {
            const double o = __shfl_up(incl, m, 64);
            if (lane >= m) incl *= o;
        }
        double excl = __shfl_up(incl, 1, 64);
        if (lane == 0) excl = 1.0;
        if (t >= t_begin) frow[(size_t)t * RR] = carry * excl;
        carry *= __shfl(incl, 63, 64);
    }
}

// ------------------------------------------------------------------ phase 3
// P.V: one workgroup per (chunk of PV_CHUNK keys from key kb0, b, key/value
// head) for NR of the R = G*M query rows of the head.  The chunk's weights
// E f_t of those rows are first gathered into LDS (coalesced), so the main
// loop issues one 16-byte load of V (8 channels of one key) per lane and key,
// feeding 8 FMAs per query row, and reads the key's weights from LDS (one
// broadcast read).  Partial outputs per chunk go to a workspace; phase 4 adds
// them up.
constexpr int PV_CHUNK = 512, PV_ROWS = 16;

template <int D, int NR>
__global__ __launch_bounds__(256) void dec_pv_kernel(DecParams p, int rg0)
{
    constexpr int CC = D / 8, KG = 256 / CC;   // channel chunks; keys per step over the workgroup
    __shared__ __align__(16) float wl[PV_CHUNK][NR];
    __shared__ float red[4][NR][D];
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
    const int cc = tid % CC, kg = tid / CC;
    const int chunk = (int)blockIdx.x;
    const int bhk = (int)blockIdx.y;
    const int b = bhk / p.Hkv, hk = bhk % p.Hkv;
    const int G = p.Hq / p.Hkv, RR = G * p.M;
    const int ntiles = p.Np / TK;
    const int k0 = p.kb0 + chunk * PV_CHUNK;
    const int k_end = k0 + PV_CHUNK < p.N ? k0 + PV_CHUNK : p.N;
    for (int x = tid; x < PV_CHUNK * NR; x += 256) {
        const int kl = x / NR, i = x % NR;
        const int key = k0 + kl, rho = rg0 + i;
        float wgt = 0.0f;
        if (key < k_end && rho < RR) {
            const int P = p.N - p.M + rho % p.M;
            const int vlo = p.window > 0 ? (P - p.window + 1 > 0 ? P - p.window + 1 : 0) : 0;
            const int vhi = p.causal ? P : p.N - 1;
            if (key >= vlo && key <= vhi)
                wgt = p.e[((size_t)bhk * p.Np + key) * RR + rho] *
                      (float)p.f[((size_t)bhk * ntiles + key / TK) * RR + rho];
        }
        wl[kl][i] = wgt;
    }
    __syncthreads();
    float acc[NR][8];
#pragma unroll
    for (int i = 0; i < NR; ++i)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[i][c] = 0.0f;
    const uint16_t *vbase = p.v + (size_t)bhk * p.N * D + cc * 8;
    // U keys per iteration, their loads issued before any arithmetic (keys
    // past the chunk read a valid row and have weight 0)
    constexpr int U = 4;
    for (int kl0 = kg; kl0 < PV_CHUNK; kl0 += U * KG) {
        uint4 vw[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int key = k0 + kl0 + u * KG;
            vw[u] = *reinterpret_cast<const uint4 *>(vbase + (size_t)(key < k_end ? key : k_end - 1) * D);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float vf[8];
            unpack8(vw[u], vf);
            const int kl = kl0 + u * KG;
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
        p.part[((size_t)rid * nch + chunk) * D + c] = v;
    }
}

// ------------------------------------------------------------------ phase 4
// O = sum over the key chunks of the partial outputs.
template <int D>
__global__ __launch_bounds__(256) void dec_reduce_kernel(DecParams p)
{
    const int64_t nrows = (int64_t)p.B * p.Hq * p.M;
    const int nch = (p.N - p.kb0 + PV_CHUNK - 1) / PV_CHUNK;
    const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (x >= nrows * D) return;
    const int64_t row = x / D;
    const int c = (int)(x % D);
    float s = 0.0f;
    for (int ch = 0; ch < nch; ++ch) s += p.part[(row * nch + ch) * D + c];
    p.o[x] = s;
}

// ------------------------------------------------------------------ launchers
template <int D>
static hipError_t launch_decode_d(const DecParams &p, hipStream_t s)
{
    if (p.mode != MODE_ALL16) {   // the all-16-bit mode reads no 8-bit logit
        const int G = p.Hq / p.Hkv, ngroups = (G * p.M + 3) / 4;
        dim3 g1((unsigned)((p.N - p.kb0 + 255) / 256), (unsigned)(p.B * p.Hkv * ngroups));
        hipLaunchKernelGGL(dec_logits8_kernel<D>, g1, dim3(256), 0, s, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t nrows = (int64_t)p.B * p.Hq * p.M;
    dim3 g2((unsigned)((nrows + 3) / 4));
    if (p.mode == MODE_PURE8) hipLaunchKernelGGL((dec_lamp_kernel<D, MODE_PURE8>), g2, dim3(256), 0, s, p);
    else if (p.mode == MODE_ALL16) hipLaunchKernelGGL((dec_lamp_kernel<D, MODE_ALL16>), g2, dim3(256), 0, s, p);
    else hipLaunchKernelGGL((dec_lamp_kernel<D, MODE_LAMP>), g2, dim3(256), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int rows = (p.Hq / p.Hkv) * p.M;
    dim3 g3((unsigned)((p.N - p.kb0 + PV_CHUNK - 1) / PV_CHUNK), (unsigned)(p.B * p.Hkv));
    for (int rg0 = 0; rg0 < rows; rg0 += PV_ROWS) {
        const int nr = rows - rg0;
        if (nr <= 4) hipLaunchKernelGGL((dec_pv_kernel<D, 4>), g3, dim3(256), 0, s, p, rg0);
        else if (nr <= 8) hipLaunchKernelGGL((dec_pv_kernel<D, 8>), g3, dim3(256), 0, s, p, rg0);
        else hipLaunchKernelGGL((dec_pv_kernel<D, PV_ROWS>), g3, dim3(256), 0, s, p, rg0);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(dec_reduce_kernel<D>, dim3((unsigned)((nrows * D + 255) / 256)), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_decode(int D, const DecParams &p, hipStream_t s)
{
    if (D == 64) return launch_decode_d<64>(p, s);
    if (D == 128) return launch_decode_d<128>(p, s);
    return launch_decode_d<256>(p, s);
}

} // namespace lamp
