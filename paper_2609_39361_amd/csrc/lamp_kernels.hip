// lamp_kernels.hip -- HIP kernels of the LampAttention forward pass for gfx950.
//
// One workgroup handles one (batch, query head, query block of BQ rows) and
// walks the key tiles of KPT = BK*NK keys in order (paper Alg. 1, outer
// loops).  Each 64-lane wave owns 64 query rows, one row per lane, and keeps
// that row's running state (mu, omega) and its output accumulator O^T in
// matrix-core accumulators.  Per tile:
//   1. the 8-bit logits of the tile: per lane, 16 keys at a time, one fp32 FMA
//      per multiply-add with the key value read from scalar registers (every
//      lane of a wave uses the same key), the running sums rounded to e4m3
//      after every step with the packed hardware conversion;
//   2. stage 1 (Sec. 3.1, Eq. (7)): per sub-block column maxima and threats,
//      reduced over the block through LDS, sorted, then tested sequentially;
//      a failing sub-block is recomputed in 16 bits (fp64 accumulation
//      rounded to e4m11) and raises mu_hat;
//   3. exponentials against mu_hat: the 8-bit ones from a 256-entry LUT in
//      LDS, the 16-bit ones from a 65536-entry table;
//   4. lambda_hat = exp(mu - mu_hat), omega_hat, and stage 2 (Eq. (8)):
//      per-sub-block costs, feasibility of every candidate recompute set
//      reduced over the block, recompute of the chosen set;
//   5. O^T <- O^T diag(lambda_hat) + V^T E on the bf16 matrix cores (the
//      8-bit exponentials are exact in bf16, a 16-bit one is split into two
//      bf16 terms).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lamp_device.h"
#include "lamp_kernels.h"

namespace lamp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ prepass
// q_tilde = RN32(q * s), fp32 [B][Hq][N][D].
__global__ void prescale_q_kernel(const uint16_t *__restrict__ q, float *__restrict__ qt, float s, size_t n)
{
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    size_t stride = (size_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) qt[i] = bf16_value(q[i]) * s;
}

// K regrouped per 16 keys, channel-major: kt[B][Hkv][N/16][D][16], fp32 and
// fp64, so that one scalar load brings 16 (resp. 8) keys of one channel.
__global__ void regroup_k_kernel(const uint16_t *__restrict__ k, float *__restrict__ kt32,
                                 double *__restrict__ kt64, int D, size_t n)
{
    size_t o = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    size_t stride = (size_t)gridDim.x * blockDim.x;
    for (; o < n; o += stride) {
        size_t kk = o & 15;
        size_t c = (o >> 4) % (size_t)D;
        size_t grp = (o >> 4) / (size_t)D;       // (b*Hkv + h) * N/16 + key group
        float v = bf16_value(k[(grp * 16 + kk) * (size_t)D + c]);
        kt32[o] = v;
        kt64[o] = (double)v;
    }
}

// ------------------------------------------------------------------ tables
// Exponential tables: E = RN(exp(-s)) for every shift code s, correctly
// rounded (Sec. 3.3 LUT exp; Sec. 4.1 exponentials correctly rounded).  exp
// is evaluated with exp_doc (error below 2^-50 relative); an entry whose
// enclosure straddles a rounding midpoint is counted in *ambiguous and the
// library refuses to run.
__device__ __forceinline__ double rn_grid(double y, int mbits, int emin)
{
    int e = __builtin_amdgcn_frexp_exp(y) - 1;
    int qe = (e > emin ? e : emin) - mbits;
    double c = __builtin_amdgcn_ldexp(1.5, 52 + qe);
    return (y + c) - c;
}

__device__ __forceinline__ uint32_t grid_code(double r, int mbits, int emin, int bias)
{
    if (r < __builtin_amdgcn_ldexp(1.0, emin))
        return (uint32_t)(r * __builtin_amdgcn_ldexp(1.0, mbits - emin));
    uint32_t hi = (uint32_t)(__builtin_bit_cast(uint64_t, r) >> 32);
    uint32_t ex = (hi >> 20) - 1023u + (uint32_t)bias;
    return (ex << mbits) | ((hi >> (20 - mbits)) & ((1u << mbits) - 1u));
}

__device__ __forceinline__ double grid_value(uint32_t c, int mbits, int bias)
{
    uint32_t ex = c >> mbits, m = c & ((1u << mbits) - 1u);
    if (ex == 0) return __builtin_amdgcn_ldexp((double)m, 1 - bias - mbits);
    return __builtin_amdgcn_ldexp((double)((1u << mbits) | m), (int)ex - bias - mbits);
}

__global__ void build_tables_kernel(uint8_t *__restrict__ lut8, uint16_t *__restrict__ lut8e,
                                    uint16_t *__restrict__ exp16, unsigned *__restrict__ ambiguous)
{
    unsigned c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= 65536u + 256u) return;
    bool small = c >= 65536u;
    unsigned code = small ? c - 65536u : c;
    int mb = small ? 3 : 11;
    double s = grid_value(code, mb, 15);
    double y = exp_doc(-s);
    double lo = y * (1.0 - 0x1p-48), hi = y * (1.0 + 0x1p-48);
    double r = rn_grid(y, mb, -30);
    if (rn_grid(lo, mb, -30) != r || rn_grid(hi, mb, -30) != r) atomicAdd(ambiguous, 1u);
    uint32_t e = grid_code(r, mb, -30, 31);
    if (small) {
        lut8[code] = (uint8_t)e;
        lut8e[code] = (uint16_t)bf16_bits((float)r);   // E8 is exact in bf16
    } else {
        exp16[code] = (uint16_t)e;
    }
}

// ------------------------------------------------------------------ 8-bit emulation
// Accumulate NC chunks of 16 keys for this lane's query over channels
// [c0, c0 + 8): acc[g][p] holds the e4m3 codes of keys 2p, 2p+1 of chunk g.
// kt points at the regrouped K of chunk 0 (uniform across the wave; chunk g
// is g*D*16 floats further); qv holds the lane's 8 pre-scaled query values.
// SAT selects the saturating conversion.
template <int D, int NC, bool SAT>
__device__ __forceinline__ void emulate8(kptr32_t kt, int c0, const float (&qv)[8], uint32_t (&acc)[NC][8])
{
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
        const float q = qv[cc];
#pragma unroll
        for (int g = 0; g < NC; ++g) {
            kptr32_t kp = kt + ((size_t)g * D + (c0 + cc)) * 16;
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                float2 a = unpk_e4m3(acc[g][p]);
                float x = __builtin_fmaf(q, kp[2 * p], a.x);
                float y = __builtin_fmaf(q, kp[2 * p + 1], a.y);
                acc[g][p] = SAT ? pk_e4m3_sat(x, y, acc[g][p]) : pk_e4m3(x, y, acc[g][p]);
            }
        }
    }
}

template <int D, int NC, bool SAT>
__device__ __forceinline__ void logits8_pass(const float *__restrict__ qrow, kptr32_t kt, uint32_t (&acc)[NC][8])
{
#pragma unroll
    for (int g = 0; g < NC; ++g)
#pragma unroll
        for (int p = 0; p < 8; ++p) acc[g][p] = 0u;
    const float4 *q4 = reinterpret_cast<const float4 *>(qrow);
    float4 a = q4[0], b = q4[1];
    for (int c0 = 0; c0 < D; c0 += 8) {
        float qv[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        if (c0 + 8 < D) {
            a = q4[(c0 + 8) / 4];
            b = q4[(c0 + 8) / 4 + 1];
        }
        emulate8<D, NC, SAT>(kt, c0, qv, acc);
    }
}

// Y8 codes of NC consecutive 16-key chunks for the lane's query row qrow
// (Sec. 4.1: acc <- RN_e4m3(RN32(q_tilde * k + acc)), channels ascending).
// The fast pass uses the non-saturating conversion; if any lane of the wave
// overflowed somewhere (a NaN code at the end), the chunks are recomputed
// with the saturating conversion.
template <int D, int NC>
__device__ __forceinline__ void logits8_chunks(const float *__restrict__ qrow, const float *kt_generic,
                                               uint32_t (&acc)[NC][8])
{
    kptr32_t kt = (kptr32_t)kt_generic;
    logits8_pass<D, NC, false>(qrow, kt, acc);
    uint32_t nan = 0;
#pragma unroll
    for (int g = 0; g < NC; ++g)
#pragma unroll
        for (int p = 0; p < 8; ++p) nan |= e4m3_nan_bits(acc[g][p]);
    if (wave_any(nan != 0)) logits8_pass<D, NC, true>(qrow, kt, acc);
}

// ------------------------------------------------------------------ 16-bit logits
// Y16 for 16 keys (one regrouped chunk) of the lane's query: the fp64 FMA
// chain over channels in ascending order, rounded once to e4m11.  kt64 is
// uniform; every product of an fp32 query value and a bf16 key is exact.
template <int D>
__device__ __forceinline__ void logits16_chunk(const float *__restrict__ qrow, const double *kt64_generic,
                                               float (&val)[16], uint32_t (&code)[16])
{
    kptr64_t kt64 = (kptr64_t)kt64_generic;
    double acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.0;
    const float4 *q4 = reinterpret_cast<const float4 *>(qrow);
    for (int c0 = 0; c0 < D; c0 += 4) {
        float4 qq = q4[c0 / 4];
        float qs[4] = {qq.x, qq.y, qq.z, qq.w};
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            double qd = (double)qs[cc];
            kptr64_t kp = kt64 + (size_t)(c0 + cc) * 16;
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[i] = __builtin_fma(qd, kp[i], acc[i]);
        }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) val[i] = rn_e4m11(acc[i], &code[i]);
}

// ------------------------------------------------------------------ logits entry kernels
// One wave: 64 rows x (16*NC) keys.  grid.x = B*Hq*ceil(nrows/64), grid.y = N/(16*NC).
template <int D, int NC>
__global__ __launch_bounds__(64) void logits8_kernel(LogitsParams p)
{
    const int lane = threadIdx.x;
    const int nrg = (p.nrows + 63) / 64;
    const int bh = blockIdx.x / nrg;
    const int rg = blockIdx.x % nrg;
    const int b = bh / p.Hq, h = bh % p.Hq;
    const int hk = h / (p.Hq / p.Hkv);
    const int r = rg * 64 + lane;
    const int rr = r < p.nrows ? r : p.nrows - 1;
    const int j = p.row0 + rr;
    const int key0 = blockIdx.y * 16 * NC;
    const float *qrow = p.qt + (((size_t)b * p.Hq + h) * p.N + j) * D;
    const float *kt = p.kt32 + (((size_t)b * p.Hkv + hk) * (p.N / 16) + key0 / 16) * (size_t)D * 16;
    uint32_t acc[NC][8];
    logits8_chunks<D, NC>(qrow, kt, acc);
    if (r >= p.nrows) return;
    uint8_t *out = p.y8 + (((size_t)b * p.Hq + h) * p.nrows + r) * p.N + key0;
#pragma unroll
    for (int g = 0; g < NC; ++g)
#pragma unroll
        for (int pp = 0; pp < 8; ++pp)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                int i = key0 + g * 16 + 2 * pp + t;
                bool vis = !(p.causal && i > j) && !(p.window > 0 && i <= j - p.window);
                out[g * 16 + 2 * pp + t] = vis ? (uint8_t)(acc[g][pp] >> (8 * t)) : (uint8_t)0xFF;
            }
}

template <int D>
__global__ __launch_bounds__(64) void logits16_kernel(LogitsParams p)
{
    const int lane = threadIdx.x;
    const int nrg = (p.nrows + 63) / 64;
    const int bh = blockIdx.x / nrg;
    const int rg = blockIdx.x % nrg;
    const int b = bh / p.Hq, h = bh % p.Hq;
    const int hk = h / (p.Hq / p.Hkv);
    const int r = rg * 64 + lane;
    const int rr = r < p.nrows ? r : p.nrows - 1;
    const int j = p.row0 + rr;
    const int key0 = blockIdx.y * 16;
    const float *qrow = p.qt + (((size_t)b * p.Hq + h) * p.N + j) * D;
    const double *kt = p.kt64 + (((size_t)b * p.Hkv + hk) * (p.N / 16) + key0 / 16) * (size_t)D * 16;
    float val[16];
    uint32_t code[16];
    logits16_chunk<D>(qrow, kt, val, code);
    if (r >= p.nrows) return;
    uint16_t *out = p.y16 + (((size_t)b * p.Hq + h) * p.nrows + r) * p.N + key0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        int key = key0 + i;
        bool vis = !(p.causal && key > j) && !(p.window > 0 && key <= j - p.window);
        out[i] = vis ? (uint16_t)code[i] : (uint16_t)0xFFFF;
    }
}

// ------------------------------------------------------------------ self tests
// e4m3 codes of fp32 values by the emulator's sequence: the non-saturating
// conversion, then the saturating one where the first gave NaN.  raw (may be
// null) receives the non-saturating codes.
__global__ void selftest_e4m3_kernel(const float *__restrict__ in, uint8_t *__restrict__ out,
                                     uint8_t *__restrict__ raw, size_t n)
{
    size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 2;
    if (i >= n) return;
    float a = in[i], b = (i + 1 < n) ? in[i + 1] : 0.0f;
    uint32_t r = pk_e4m3(a, b);
    uint32_t f = e4m3_nan_bits(r) ? pk_e4m3_sat(a, b) : r;
    out[i] = (uint8_t)f;
    if (raw) raw[i] = (uint8_t)r;
    if (i + 1 < n) {
        out[i + 1] = (uint8_t)(f >> 8);
        if (raw) raw[i + 1] = (uint8_t)(r >> 8);
    }
}

__global__ void selftest_exp_doc_kernel(const double *__restrict__ x, double *__restrict__ y, size_t n)
{
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) y[i] = exp_doc(x[i]);
}

// ------------------------------------------------------------------ the forward kernel
enum { PREC_LOW = 0, PREC_S1 = 1, PREC_S2 = 2, PREC_INACTIVE = 3 };

template <int D, int BQ, int BK, int NK>
struct FwdCfg {
    static constexpr int KPT = BK * NK;          // keys per tile
    static constexpr int NCH = KPT / 16;         // 16-key chunks per tile
    static constexpr int NW = BQ / 64;           // waves per workgroup
    static constexpr int NC = NCH < 4 ? NCH : 4; // chunks emulated together
    static constexpr int YP = KPT + 8;           // LDS row pitch (u16) of codes
    static constexpr int VP = KPT + 8;           // LDS row pitch (u16) of V^T
    static constexpr int CT = D / 32;            // 32-channel MFMA tiles
    static constexpr size_t LDS_Y = (size_t)BQ * YP * 2;
    static constexpr size_t LDS_V = (size_t)D * VP * 2;
    static constexpr size_t LDS_LUT = 512;
    static constexpr size_t LDS_X = (size_t)NW * 256;
    static constexpr size_t LDS = LDS_Y + LDS_V + LDS_LUT + LDS_X;
    static_assert(KPT % 16 == 0 && NCH % NC == 0, "tile must be a multiple of 64 keys or below");
    static_assert(NK <= 4, "at most 4 sub-blocks per tile");
};

// Per-wave exchange record in LDS (stage decisions are block-wide).
struct Xch {
    double thr[4];          // per sub-block threat partial (stage 1)
    uint32_t act, fail;     // sub-block bit masks
    uint32_t feas;          // stage-2 feasibility, bit R of the candidates
};

template <int D, int BQ, int BK, int NK>
__global__ __launch_bounds__(BQ, 1) void lamp_fwd_kernel(FwdParams p)
{
    using C = FwdCfg<D, BQ, BK, NK>;
    constexpr int KPT = C::KPT, NCH = C::NCH, NW = C::NW, NC = C::NC, YP = C::YP, VP = C::VP, CT = C::CT;

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t *ycode = reinterpret_cast<uint16_t *>(smem);                       // [BQ][YP]
    uint16_t *vt = reinterpret_cast<uint16_t *>(smem + C::LDS_Y);              // [D][VP]
    uint16_t *lut = reinterpret_cast<uint16_t *>(smem + C::LDS_Y + C::LDS_V);  // [256]
    Xch *xch = reinterpret_cast<Xch *>(smem + C::LDS_Y + C::LDS_V + C::LDS_LUT);

    const int tid = threadIdx.x;
    const int w = tid >> 6, lane = tid & 63;
    const int nqb = p.N / BQ;
    const int BH = p.B * p.Hq;
    const int qb = nqb - 1 - (int)(blockIdx.x / BH);   // longest blocks first under causality
    const int bh = blockIdx.x % BH;
    const int b = bh / p.Hq, h = bh % p.Hq;
    const int hk = h / (p.Hq / p.Hkv);
    const int q0 = qb * BQ;
    const int row = w * 64 + lane;                      // row within the block
    const int j = q0 + row;                             // this lane's query
    const int wj_lo = q0 + w * 64, wj_hi = wj_lo + 63;  // the wave's queries
    // visible key range of this lane and of the wave
    const int vlo = p.window > 0 ? (j - p.window + 1 > 0 ? j - p.window + 1 : 0) : 0;
    const int vhi = p.causal ? j : p.N - 1;
    const int wv_lo = p.window > 0 ? (wj_lo - p.window + 1 > 0 ? wj_lo - p.window + 1 : 0) : 0;
    const int wv_hi = p.causal ? wj_hi : p.N - 1;
    const int bv_lo = p.window > 0 ? (q0 - p.window + 1 > 0 ? q0 - p.window + 1 : 0) : 0;
    const int bv_hi = p.causal ? q0 + BQ - 1 : p.N - 1;
    const int t_begin = bv_lo / KPT, t_end = bv_hi / KPT;

    const float *qrow = p.qt + (((size_t)b * p.Hq + h) * p.N + j) * D;
    const float *kt32 = p.kt32 + ((size_t)b * p.Hkv + hk) * (size_t)(p.N / 16) * D * 16;
    const double *kt64 = p.kt64 + ((size_t)b * p.Hkv + hk) * (size_t)(p.N / 16) * D * 16;
    const uint16_t *vbase = p.v + ((size_t)b * p.Hkv + hk) * (size_t)p.N * D;
    uint16_t *myrow = ycode + row * YP;

    for (int i = tid; i < 256; i += BQ) lut[i] = p.lut8e[i];

    float mu = -__builtin_inff();   // running maximum (an e4m11 or e4m3 value)
    double om = 0.0;                // running sum omega
    floatx16 acc[2][CT];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int t = 0; t < CT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[g][t][r] = 0.0f;

    uint8_t *mrow = p.mask + (((size_t)b * p.Hq + h) * nqb + qb) * (size_t)(p.N / BK);

    for (int tile = t_begin; tile <= t_end; ++tile) {
        const int k0 = tile * KPT;
        __syncthreads();   // previous tile's readers of vt / ycode are done
        // ---- stage V^T of the tile into LDS: vt[c][i] = v[k0 + i][c]; each
        // work item packs two consecutive keys of 8 channels into 8 dwords
        for (int e = tid; e < (KPT / 2) * (D / 8); e += BQ) {
            const int i = 2 * (e % (KPT / 2)), c8 = (e / (KPT / 2)) * 8;
            const u32x4 r0 = *reinterpret_cast<const u32x4 *>(vbase + (size_t)(k0 + i) * D + c8);
            const u32x4 r1 = *reinterpret_cast<const u32x4 *>(vbase + (size_t)(k0 + i + 1) * D + c8);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                *reinterpret_cast<uint32_t *>(vt + (c8 + 2 * t) * VP + i) = (r0[t] & 0xFFFFu) | (r1[t] << 16);
                *reinterpret_cast<uint32_t *>(vt + (c8 + 2 * t + 1) * VP + i) = (r0[t] >> 16) | (r1[t] & 0xFFFF0000u);
            }
        }

        // ---- per-lane activity of each sub-block (visibility only)
        uint32_t act_lane = 0;
#pragma unroll
        for (int th = 0; th < NK; ++th) {
            int a = k0 + th * BK, z = a + BK - 1;
            if (a <= vhi && z >= vlo) act_lane |= 1u << th;
        }
        float m8[NK];
#pragma unroll
        for (int th = 0; th < NK; ++th) m8[th] = -__builtin_inff();

        // ---- 1. the 8-bit logits of the tile (skipped at threshold 0)
        if (p.mode != MODE_ALL16) {
            for (int cg = 0; cg < NCH; cg += NC) {
                const int ck0 = k0 + cg * 16, ck1 = ck0 + NC * 16 - 1;
                if (ck0 > wv_hi || ck1 < wv_lo) continue;          // nothing visible to the wave
                uint32_t a8[NC][8];
                logits8_chunks<D, NC>(qrow, kt32 + (size_t)(ck0 / 16) * D * 16, a8);
                const bool full = ck1 <= vhi && ck0 >= vlo;
#pragma unroll
                for (int g = 0; g < NC; ++g) {
                    const int th = ((cg + g) * 16) / BK;
                    float mx = -__builtin_inff();
                    uint32_t packed[8];
#pragma unroll
                    for (int pp = 0; pp < 8; ++pp) {
                        float2 yv = unpk_e4m3(a8[g][pp]);
                        int i0 = ck0 + g * 16 + 2 * pp;
                        bool v0 = full || (i0 >= vlo && i0 <= vhi);
                        bool v1 = full || (i0 + 1 >= vlo && i0 + 1 <= vhi);
                        if (v0) mx = yv.x > mx ? yv.x : mx;
                        if (v1) mx = yv.y > mx ? yv.y : mx;
                        packed[pp] = (a8[g][pp] & 0xFFu) | ((a8[g][pp] & 0xFF00u) << 8);
                    }
#pragma unroll
                    for (int t = 0; t < NK; ++t)
                        if (t == th) m8[t] = mx > m8[t] ? mx : m8[t];
                    u32x4 *dst = reinterpret_cast<u32x4 *>(myrow + (cg + g) * 16);
                    dst[0] = u32x4{packed[0], packed[1], packed[2], packed[3]};
                    dst[1] = u32x4{packed[4], packed[5], packed[6], packed[7]};
                }
            }
        }

        // ---- 2. stage decisions
        uint32_t prec16 = 0;      // sub-blocks whose logits are 16-bit (stage 1)
        float muh = mu;
        uint32_t active;
        {
            // threats and first fail set; exchanged once for all modes
            double thr[NK];
#pragma unroll
            for (int th = 0; th < NK; ++th) {
                double t = (m8[th] > -__builtin_inff()) ? (double)m8[th] - (double)mu : -__builtin_inf();
                thr[th] = wave_max_f64(t);
            }
            uint32_t fail_lane = 0;
#pragma unroll
            for (int th = 0; th < NK; ++th) {
                if (m8[th] > -__builtin_inff()) {
                    double mh = (double)muh;
                    if (!(mh > __builtin_fma(__builtin_fabs(mh), p.delta, (double)m8[th]))) fail_lane |= 1u << th;
                }
            }
            uint32_t act_w = 0, fail_w = 0;
#pragma unroll
            for (int th = 0; th < NK; ++th) {
                if (wave_any(act_lane >> th & 1u)) act_w |= 1u << th;
                if (wave_any(fail_lane >> th & 1u)) fail_w |= 1u << th;
            }
            if (lane == 0) {
#pragma unroll
                for (int th = 0; th < NK; ++th) xch[w].thr[th] = thr[th];
                xch[w].act = act_w;
                xch[w].fail = fail_w;
            }
            __syncthreads();
            double T[NK];
            uint32_t fail = 0;
            active = 0;
#pragma unroll
            for (int th = 0; th < NK; ++th) T[th] = -__builtin_inf();
            for (int ww = 0; ww < NW; ++ww) {
#pragma unroll
                for (int th = 0; th < NK; ++th) T[th] = xch[ww].thr[th] > T[th] ? xch[ww].thr[th] : T[th];
                active |= xch[ww].act;
                fail |= xch[ww].fail;
            }
            if (active == 0) {           // tile without a visible pair: no state change (uniform)
                if (tid == 0)
                    for (int th = 0; th < NK; ++th) mrow[tile * NK + th] = PREC_INACTIVE;
                continue;
            }

            if (p.mode == MODE_PURE8) {
#pragma unroll
                for (int th = 0; th < NK; ++th) muh = m8[th] > muh ? m8[th] : muh;
            } else {
                // sort active sub-blocks by threat, descending, ties by
                // index; the order is packed 4 bits per rank
                uint32_t order = 0, taken = 0;
                int na = 0;
#pragma unroll
                for (int r = 0; r < NK; ++r) {
                    int best = -1;
                    double bt = 0.0;
#pragma unroll
                    for (int th = 0; th < NK; ++th) {
                        bool cand = (active >> th & 1u) && !(taken >> th & 1u);
                        if (cand && (best < 0 || T[th] > bt)) { best = th; bt = T[th]; }
                    }
                    if (best >= 0) {
                        order |= (uint32_t)best << (4 * na);
                        ++na;
                        taken |= 1u << best;
                    }
                }
                if (p.mode == MODE_ALL16) fail = active;
                int pos = 0;
                while (true) {
                    while (pos < na && !(fail >> ((order >> (4 * pos)) & 15u) & 1u)) ++pos;
                    if (pos >= na) break;
                    const int th = (int)((order >> (4 * pos)) & 15u);
                    ++pos;
                    prec16 |= 1u << th;
                    // recompute sub-block th in 16 bits for this wave's rows
                    for (int ch = 0; ch < BK / 16; ++ch) {
                        const int c16 = th * (BK / 16) + ch;
                        const int ck0 = k0 + c16 * 16;
                        if (ck0 > wv_hi || ck0 + 15 < wv_lo) continue;
                        float val[16];
                        uint32_t code[16];
                        logits16_chunk<D>(qrow, kt64 + (size_t)(ck0 / 16) * D * 16, val, code);
                        uint32_t packed[8];
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            int key = ck0 + i;
                            if (key >= vlo && key <= vhi) muh = val[i] > muh ? val[i] : muh;
                        }
#pragma unroll
                        for (int pp = 0; pp < 8; ++pp) packed[pp] = code[2 * pp] | (code[2 * pp + 1] << 16);
                        u32x4 *dst = reinterpret_cast<u32x4 *>(myrow + c16 * 16);
                        dst[0] = u32x4{packed[0], packed[1], packed[2], packed[3]};
                        dst[1] = u32x4{packed[4], packed[5], packed[6], packed[7]};
                    }
                    if (p.mode == MODE_ALL16 || pos >= na) continue;
                    // re-test the remaining sub-blocks against the raised mu_hat
                    uint32_t fl = 0;
                    for (int a = pos; a < na; ++a) {
                        const int t2 = (int)((order >> (4 * a)) & 15u);
                        float m = -__builtin_inff();
#pragma unroll
                        for (int th2 = 0; th2 < NK; ++th2)
                            if (th2 == t2) m = m8[th2];
                        if (m > -__builtin_inff()) {
                            double mh = (double)muh;
                            if (!(mh > __builtin_fma(__builtin_fabs(mh), p.delta, (double)m))) fl |= 1u << t2;
                        }
                    }
                    uint32_t fw = 0;
                    for (int th2 = 0; th2 < NK; ++th2)
                        if (wave_any(fl >> th2 & 1u)) fw |= 1u << th2;
                    __syncthreads();
                    if (lane == 0) xch[w].fail = fw;
                    __syncthreads();
                    fail = 0;
                    for (int ww = 0; ww < NW; ++ww) fail |= xch[ww].fail;
                }
            }
        }

        // ---- 3. exponentials of the tile against mu_hat; S = sum E (exact in fp64)
        double S = 0.0;
        for (int c16 = 0; c16 < NCH; ++c16) {
            const int ck0 = k0 + c16 * 16;
            const int th = (c16 * 16) / BK;
            u32x4 *rowp = reinterpret_cast<u32x4 *>(myrow + c16 * 16);
            if (!(active >> th & 1u) || ck0 > vhi || ck0 + 15 < vlo) {
                rowp[0] = u32x4{0u, 0u, 0u, 0u};
                rowp[1] = u32x4{0u, 0u, 0u, 0u};
                continue;
            }
            const bool hi16 = prec16 >> th & 1u;
            u32x4 c0 = rowp[0], c1 = rowp[1];
            uint32_t in[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
            uint32_t outw[8];
#pragma unroll
            for (int pp = 0; pp < 8; ++pp) {
                uint32_t res = 0;
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    int key = ck0 + 2 * pp + t;
                    uint32_t yc = (in[pp] >> (16 * t)) & 0xFFFFu;
                    uint32_t ec = 0;
                    float ev = 0.0f;
                    if (key >= vlo && key <= vhi) {
                        if (hi16) {
                            float x = shift_of(muh, e4m11_value(yc));
                            ec = p.exp16[ue5m11_code(x)];
                            ev = ue5m11e_value(ec);
                        } else {
                            float x = shift_of(muh, e4m3_value(yc));
                            ec = lut[ue5m3_code(x)];
                            ev = bf16_value(ec);
                        }
                    }
                    S += (double)ev;
                    res |= ec << (16 * t);
                }
                outw[pp] = res;
            }
            rowp[0] = u32x4{outw[0], outw[1], outw[2], outw[3]};
            rowp[1] = u32x4{outw[4], outw[5], outw[6], outw[7]};
        }

        // ---- 4. lambda_hat, omega_hat; stage 2
        double lam;
        if (muh == -__builtin_inff()) lam = 1.0;
        else if (mu == -__builtin_inff()) lam = 0.0;
        else lam = exp_doc((double)mu - (double)muh);
        const double omh = __builtin_fma(lam, om, S);
        uint32_t prec2 = 0;     // stage-2 sub-blocks
        if (p.mode == MODE_LAMP) {
            const uint32_t F = active & ~prec16;
            if (F) {
                double cost[NK];
#pragma unroll
                for (int th = 0; th < NK; ++th) cost[th] = 0.0;
#pragma unroll
                for (int th = 0; th < NK; ++th) {
                    if (!(F >> th & 1u)) continue;
                    for (int ch = 0; ch < BK / 16; ++ch) {
                        const int c16 = th * (BK / 16) + ch;
                        const int ck0 = k0 + c16 * 16;
                        if (ck0 > vhi || ck0 + 15 < vlo) continue;
                        const u32x4 *rowp = reinterpret_cast<const u32x4 *>(myrow + c16 * 16);
                        u32x4 c0 = rowp[0], c1 = rowp[1];
                        uint32_t in[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
                        double cth = cost[th];
#pragma unroll
                        for (int pp = 0; pp < 8; ++pp)
#pragma unroll
                            for (int t = 0; t < 2; ++t) {
                                int key = ck0 + 2 * pp + t;
                                if (key < vlo || key > vhi) continue;
                                double e = (double)bf16_value((in[pp] >> (16 * t)) & 0xFFFFu);
                                double tt = omh - e;
                                double pr = e * tt;
                                cth = cth + pr;
                            }
                        cost[th] = cth;
                    }
                }
                // feasibility of every candidate recompute set R within F
                const double lim = (p.tau * omh) * omh;
                uint32_t feas = 0;
                for (int R = 0; R < (1 << NK); ++R) {
                    if (R & ~(int)F) continue;
                    double xi = 0.0;
#pragma unroll
                    for (int th = 0; th < NK; ++th)
                        if ((F >> th & 1u) && !(R >> th & 1)) xi = xi + cost[th];
                    bool bad = !(xi <= lim);
                    if (!wave_any(bad)) feas |= 1u << R;
                }
                __syncthreads();
                if (lane == 0) xch[w].feas = feas;
                __syncthreads();
                for (int ww = 0; ww < NW; ++ww) feas &= xch[ww].feas;
                // smallest recompute set first, then ascending bitmask
                int chosen = (int)F;
                bool found = false;
                for (int sz = 0; sz <= NK && !found; ++sz)
                    for (int R = 0; R < (1 << NK) && !found; ++R) {
                        if ((R & ~(int)F) || __builtin_popcount(R) != sz) continue;
                        if (feas >> R & 1u) { chosen = R; found = true; }
                    }
                prec2 = (uint32_t)chosen;
                // stage-2 recompute: 16-bit logits and exponentials, mu_hat unchanged
                for (int th = 0; th < NK; ++th) {
                    if (!(prec2 >> th & 1u)) continue;
                    for (int ch = 0; ch < BK / 16; ++ch) {
                        const int c16 = th * (BK / 16) + ch;
                        const int ck0 = k0 + c16 * 16;
                        if (ck0 > wv_hi || ck0 + 15 < wv_lo) continue;
                        float val[16];
                        uint32_t code[16];
                        logits16_chunk<D>(qrow, kt64 + (size_t)(ck0 / 16) * D * 16, val, code);
                        u32x4 *rowp = reinterpret_cast<u32x4 *>(myrow + c16 * 16);
                        u32x4 c0 = rowp[0], c1 = rowp[1];
                        uint32_t in[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
                        uint32_t outw[8];
#pragma unroll
                        for (int pp = 0; pp < 8; ++pp) {
                            uint32_t res = 0;
#pragma unroll
                            for (int t = 0; t < 2; ++t) {
                                int key = ck0 + 2 * pp + t;
                                uint32_t ec = 0;
                                if (key >= vlo && key <= vhi) {
                                    float old = bf16_value((in[pp] >> (16 * t)) & 0xFFFFu);
                                    float x = shift_of(muh, val[2 * pp + t]);
                                    ec = p.exp16[ue5m11_code(x)];
                                    S = S - (double)old;
                                    S = S + (double)ue5m11e_value(ec);
                                }
                                res |= ec << (16 * t);
                            }
                            outw[pp] = res;
                        }
                        rowp[0] = u32x4{outw[0], outw[1], outw[2], outw[3]};
                        rowp[1] = u32x4{outw[4], outw[5], outw[6], outw[7]};
                    }
                }
            }
        }
        om = __builtin_fma(lam, om, S);
        mu = muh;
        if (tid == 0) {
#pragma unroll
            for (int th = 0; th < NK; ++th)
                mrow[tile * NK + th] = !(active >> th & 1u) ? PREC_INACTIVE
                                     : (prec16 >> th & 1u) ? PREC_S1
                                     : (prec2 >> th & 1u) ? PREC_S2 : PREC_LOW;
        }
        const uint32_t prec_any16 = prec16 | prec2;

        // ---- 5. O^T <- O^T diag(lambda_hat) + V^T E on the matrix cores
        __syncthreads();   // vt complete
        {
            const float lamf = (float)lam;
            if (wave_any(lamf != 1.0f)) {
                const float l0 = __shfl(lamf, lane & 31, 64);
                const float l1 = __shfl(lamf, 32 + (lane & 31), 64);
#pragma unroll
                for (int t = 0; t < CT; ++t)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        acc[0][t][r] *= l0;
                        acc[1][t][r] *= l1;
                    }
            }
        }
        const int half = lane >> 5, l32 = lane & 31;
        for (int c16 = 0; c16 < NCH; ++c16) {
            const int ck0 = k0 + c16 * 16;
            if (ck0 > wv_hi || ck0 + 15 < wv_lo) continue;
            const int th = (c16 * 16) / BK;
            if (!(active >> th & 1u)) continue;
            const bool hi16 = prec_any16 >> th & 1u;
            bf16x8 bh[2], bl[2];
#pragma unroll
            for (int g = 0; g < 2; ++g) {
                const u32x4 e = *reinterpret_cast<const u32x4 *>(ycode + (w * 64 + g * 32 + l32) * YP + c16 * 16 + half * 8);
                if (!hi16) {
                    bh[g] = __builtin_bit_cast(bf16x8, e);
                } else {
                    u32x4 hw, lw;
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        float e0 = ue5m11e_value(e[t] & 0xFFFFu), e1 = ue5m11e_value(e[t] >> 16);
                        uint32_t h0 = bf16_bits(e0), h1 = bf16_bits(e1);
                        float r0 = e0 - bf16_value(h0), r1 = e1 - bf16_value(h1);
                        hw[t] = h0 | (h1 << 16);
                        lw[t] = bf16_bits(r0) | (bf16_bits(r1) << 16);
                    }
                    bh[g] = __builtin_bit_cast(bf16x8, hw);
                    bl[g] = __builtin_bit_cast(bf16x8, lw);
                }
            }
#pragma unroll
            for (int t = 0; t < CT; ++t) {
                const u32x4 av = *reinterpret_cast<const u32x4 *>(vt + (t * 32 + l32) * VP + c16 * 16 + half * 8);
                const bf16x8 a = __builtin_bit_cast(bf16x8, av);
#pragma unroll
                for (int g = 0; g < 2; ++g) {
                    acc[g][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bh[g], acc[g][t], 0, 0, 0);
                    if (hi16) acc[g][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bl[g], acc[g][t], 0, 0, 0);
                }
            }
        }
    }

    // ---- epilogue: O / omega, lse = mu + ln(omega), mask bytes of skipped tiles
    {
        const int half = lane >> 5, l32 = lane & 31;
        const double om0 = __shfl(om, l32, 64), om1 = __shfl(om, 32 + l32, 64);
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            const float inv = (float)(1.0 / (g ? om1 : om0));
            const int jq = q0 + w * 64 + g * 32 + l32;
            float *orow = p.o + (((size_t)b * p.Hq + h) * p.N + jq) * D;
#pragma unroll
            for (int t = 0; t < CT; ++t)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    const int c = t * 32 + r4 * 8 + half * 4;
                    float4 v4 = make_float4(acc[g][t][r4 * 4 + 0] * inv, acc[g][t][r4 * 4 + 1] * inv,
                                            acc[g][t][r4 * 4 + 2] * inv, acc[g][t][r4 * 4 + 3] * inv);
                    *reinterpret_cast<float4 *>(orow + c) = v4;
                }
        }
        p.lse[((size_t)b * p.Hq + h) * p.N + j] = (float)((double)mu + ::log(om));
        const int ntiles = p.N / KPT;
        for (int t = tid; t < ntiles; t += BQ)
            if (t < t_begin || t > t_end)
                for (int th = 0; th < NK; ++th) mrow[t * NK + th] = PREC_INACTIVE;
    }
}

// ------------------------------------------------------------------ launchers
template <int D, int BQ, int BK, int NK>
static hipError_t launch_fwd(const FwdParams &p, hipStream_t s)
{
    using C = FwdCfg<D, BQ, BK, NK>;
    auto kern = lamp_fwd_kernel<D, BQ, BK, NK>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)(p.B * p.Hq * (p.N / BQ)));
    hipLaunchKernelGGL(kern, grid, dim3(BQ), C::LDS, s, p);
    return hipGetLastError();
}

#define LAMP_FWD_CASE(D_, BQ_, BK_, NK_) \
    if (D == D_ && BQ == BQ_ && BK == BK_ && NK == NK_) return launch_fwd<D_, BQ_, BK_, NK_>(p, s);

hipError_t dispatch_fwd(int D, int BQ, int BK, int NK, const FwdParams &p, hipStream_t s, bool *found)
{
    *found = true;
    // configurations built: d in {64,128,256}, bq in {64,128}, (bk, nk) in
    // {(16,4), (64,4)}
#define LAMP_FWD_D(D_)                                                           \
    LAMP_FWD_CASE(D_, 64, 16, 4) LAMP_FWD_CASE(D_, 128, 16, 4)                     \
    LAMP_FWD_CASE(D_, 64, 64, 4) LAMP_FWD_CASE(D_, 128, 64, 4)
    LAMP_FWD_D(64)
    LAMP_FWD_D(128)
    LAMP_FWD_D(256)
#undef LAMP_FWD_D
    *found = false;
    return hipSuccess;
}

hipError_t launch_prepass(const uint16_t *q, const uint16_t *k, float *qt, float *kt32, double *kt64,
                          int B, int Hq, int Hkv, int N, int D, float scale, hipStream_t s)
{
    size_t nq = (size_t)B * Hq * N * D, nk = (size_t)B * Hkv * N * D;
    unsigned gq = (unsigned)((nq + 255) / 256 < 65536 ? (nq + 255) / 256 : 65536);
    unsigned gk = (unsigned)((nk + 255) / 256 < 65536 ? (nk + 255) / 256 : 65536);
    hipLaunchKernelGGL(prescale_q_kernel, dim3(gq), dim3(256), 0, s, q, qt, scale, nq);
    hipLaunchKernelGGL(regroup_k_kernel, dim3(gk), dim3(256), 0, s, k, kt32, kt64, D, nk);
    return hipGetLastError();
}

hipError_t launch_logits8(const LogitsParams &p, int D, hipStream_t s)
{
    const unsigned gx = (unsigned)(p.B * p.Hq * ((p.nrows + 63) / 64));
    if (p.N % 64 == 0) {
        dim3 grid(gx, (unsigned)(p.N / 64));
        if (D == 64) hipLaunchKernelGGL((logits8_kernel<64, 4>), grid, dim3(64), 0, s, p);
        else if (D == 128) hipLaunchKernelGGL((logits8_kernel<128, 4>), grid, dim3(64), 0, s, p);
        else hipLaunchKernelGGL((logits8_kernel<256, 4>), grid, dim3(64), 0, s, p);
    } else {
        dim3 grid(gx, (unsigned)(p.N / 16));
        if (D == 64) hipLaunchKernelGGL((logits8_kernel<64, 1>), grid, dim3(64), 0, s, p);
        else if (D == 128) hipLaunchKernelGGL((logits8_kernel<128, 1>), grid, dim3(64), 0, s, p);
        else hipLaunchKernelGGL((logits8_kernel<256, 1>), grid, dim3(64), 0, s, p);
    }
    return hipGetLastError();
}

hipError_t launch_logits16(const LogitsParams &p, int D, hipStream_t s)
{
    dim3 grid((unsigned)(p.B * p.Hq * ((p.nrows + 63) / 64)), (unsigned)(p.N / 16));
    if (D == 64) hipLaunchKernelGGL(logits16_kernel<64>, grid, dim3(64), 0, s, p);
    else if (D == 128) hipLaunchKernelGGL(logits16_kernel<128>, grid, dim3(64), 0, s, p);
    else hipLaunchKernelGGL(logits16_kernel<256>, grid, dim3(64), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_build_tables(uint8_t *lut8, uint16_t *lut8e, uint16_t *exp16, unsigned *ambiguous, hipStream_t s)
{
    hipLaunchKernelGGL(build_tables_kernel, dim3((65536 + 256 + 255) / 256), dim3(256), 0, s, lut8, lut8e, exp16,
                       ambiguous);
    return hipGetLastError();
}

hipError_t launch_selftest_e4m3(const float *in, uint8_t *out, uint8_t *raw, size_t n, hipStream_t s)
{
    size_t pairs = (n + 1) / 2;
    hipLaunchKernelGGL(selftest_e4m3_kernel, dim3((unsigned)((pairs + 255) / 256)), dim3(256), 0, s, in, out, raw, n);
    return hipGetLastError();
}

hipError_t launch_selftest_exp_doc(const double *x, double *y, size_t n, hipStream_t s)
{
    hipLaunchKernelGGL(selftest_exp_doc_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x, y, n);
    return hipGetLastError();
}

} // namespace lamp
