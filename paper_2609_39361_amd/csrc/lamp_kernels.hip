// lamp_kernels.hip -- auxiliary HIP kernels of liblamp.so for gfx950: the
// prepass (pre-scaled Q, K in fp32), the exponential
// tables, the stand-alone logit kernels and the self tests.  The forward
// kernel is in lamp_fwd.hip, the logit loops in lamp_loops.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lamp_device.h"
#include "lamp_kernels.h"
#include "lamp_loops.h"
#include "lamp_sr.h"

namespace lamp {

static_assert(SIM8_ENTRIES == SIM8_N && SIM16_TABLE == SIM16_N && SIM8_N <= SIM8_TABLE, "SIM table sizes");

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ prepass
// One thread per 4 channels of one row of one head.  u (below rows * D/4)
// indexes the float4 groups of a head's output in storage order: the row
// layout (blk = 0) stores [rows][D]; the grouped layout stores blocks of blk
// rows, each [D/4][blk][4], so that one 4-channel group of a block is
// contiguous.  Returns the row j and group g of u.
__device__ __forceinline__ void rg_of(int u, int G, int blk, int &j, int &g)
{
    if (blk == 0) {
        j = u / G;
        g = u % G;
        return;
    }
    const int per = blk * G, r = u % per;
    j = (u / per) * blk + r % blk;
    g = r / blk;
}

// 4 bf16 values (8 bytes) as fp32, times s (s = 1: exact conversion)
__device__ __forceinline__ float4 bf16x4_scaled(const uint2 w, float s)
{
    return make_float4(bf16_value(w.x & 0xFFFFu) * s, bf16_value(w.x >> 16) * s, bf16_value(w.y & 0xFFFFu) * s,
                       bf16_value(w.y >> 16) * s);
}

// Nonzero iff one of the bf16 values in a word has an all-ones exponent
// (an infinity or a NaN).
__device__ __forceinline__ uint32_t bf16_nonfinite(uint32_t w)
{
    return ((w & 0x7F80u) == 0x7F80u) | ((w & 0x7F800000u) == 0x7F800000u);
}

// Or `bit` into *bad once per wave if any lane saw a non-finite value.
__device__ __forceinline__ void flag_nonfinite(unsigned *bad, bool seen, unsigned bit)
{
    if (__ballot(seen) != 0ull && __lane_id() == (unsigned)__builtin_ctzll(__ballot(seen))) atomicOr(bad, bit);
}

// Pre-scaled queries q~ = RN32(q * s), rows padded with zeros from N to Nq:
// qt [BH][Nq][D] from q [BH][N][D] (grouped layout: blk = 64).  Grid: x over
// the float4 groups of a head, y over heads (both grid-stride).
// With bad (may be null), bit `bit` is or-ed into *bad if an element of q is
// not finite.
__global__ void prescale_q_kernel(const uint16_t *__restrict__ q, float *__restrict__ qt, float s, int N, int Nq,
                                  int D, int BH, int blk, unsigned *bad, unsigned bit)
{
    const int G = D / 4, n4 = Nq * G;
    bool seen = false;
    for (int bh = blockIdx.y; bh < BH; bh += gridDim.y)
        for (int u = blockIdx.x * blockDim.x + threadIdx.x; u < n4; u += gridDim.x * blockDim.x) {
            int j, g;
            rg_of(u, G, blk, j, g);
            const uint2 w = j < N ? *reinterpret_cast<const uint2 *>(q + ((size_t)bh * N + j) * D + 4 * g)
                                  : make_uint2(0u, 0u);
            seen |= (bf16_nonfinite(w.x) | bf16_nonfinite(w.y)) != 0u;
            reinterpret_cast<float4 *>(qt + (size_t)bh * Nq * D)[u] = bf16x4_scaled(w, s);
        }
    if (bad) flag_nonfinite(bad, seen, bit);
}

// K in fp32 (bf16 -> fp32 is exact), rows padded with zeros from N to Nk:
// k32 [BH][Nk][D] from k [BH][N][D] (grouped layout: blk = 16).
__global__ void convert_k_kernel(const uint16_t *__restrict__ k, float *__restrict__ k32, int N, int Nk, int D,
                                 int BH, int blk, unsigned *bad)
{
    const int G = D / 4, n4 = Nk * G;
    bool seen = false;
    for (int bh = blockIdx.y; bh < BH; bh += gridDim.y)
        for (int u = blockIdx.x * blockDim.x + threadIdx.x; u < n4; u += gridDim.x * blockDim.x) {
            int j, g;
            rg_of(u, G, blk, j, g);
            const uint2 w = j < N ? *reinterpret_cast<const uint2 *>(k + ((size_t)bh * N + j) * D + 4 * g)
                                  : make_uint2(0u, 0u);
            seen |= (bf16_nonfinite(w.x) | bf16_nonfinite(w.y)) != 0u;
            reinterpret_cast<float4 *>(k32 + (size_t)bh * Nk * D)[u] = bf16x4_scaled(w, 1.0f);
        }
    if (bad) flag_nonfinite(bad, seen, 2u);
}

// V^T [B*Hkv][D][Nk] from V [B*Hkv][N][D] (bf16), keys padded with zeros
// from N to Nk: 64x64 tiles through LDS.  grid (Nk/64, D/64, B*Hkv); Nk and
// D are multiples of 64.
__global__ __launch_bounds__(256) void transpose_v_kernel(const uint16_t *__restrict__ v, uint16_t *__restrict__ vt,
                                                          int N, int Nk, int D, unsigned *bad)
{
    __shared__ uint16_t tile[64][66];
    const size_t bh = blockIdx.z;
    const int n0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
    const uint16_t *src = v + bh * (size_t)N * D;
    uint16_t *dst = vt + bh * (size_t)D * Nk;
    bool seen = false;
    for (int e = threadIdx.x; e < 64 * 64; e += 256) {
        const int r = e / 64, c = e % 64;
        const uint16_t x = n0 + r < N ? src[(size_t)(n0 + r) * D + c0 + c] : (uint16_t)0;
        seen |= (x & 0x7F80u) == 0x7F80u;
        tile[r][c] = x;
    }
    if (bad) flag_nonfinite(bad, seen, 4u);
    __syncthreads();
    for (int e = threadIdx.x; e < 64 * 64; e += 256) {
        const int c = e / 64, r = e % 64;
        dst[(size_t)(c0 + c) * Nk + n0 + r] = tile[r][c];
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
                                    uint16_t *__restrict__ exp16, uint32_t *__restrict__ exp16hl,
                                    unsigned *__restrict__ ambiguous)
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
        uint32_t eh, el;   // the same value as exact bf16 high and low parts, for P.V
        split_bf16((float)r, eh, el);
        exp16hl[code] = eh | (el << 16);
    }
}

// Exponential tables of the SIM profile (layout in lamp_device.h): entry
// ((e - EMIN) << P) | m is RN_P(exp(-s)), s = (2^P + m) 2^(e-P), rounded to P
// mantissa bits in FP32's exponent range (quantum 2^(-126-P) below 2^-126);
// the same enclosure check as above.  sim8 holds 256 entries, those past
// SIM8_N being 0.
__global__ void build_sim_tables_kernel(uint16_t *__restrict__ sim8, uint32_t *__restrict__ sim16,
                                        unsigned *__restrict__ ambiguous)
{
    unsigned c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= (unsigned)SIM16_N + (unsigned)SIM8_TABLE) return;
    const bool small = c >= (unsigned)SIM16_N;
    const unsigned idx = small ? c - (unsigned)SIM16_N : c;
    if (small && idx >= (unsigned)SIM8_N) {   // padding of the 256-entry copy
        sim8[idx] = 0;
        return;
    }
    const int P = small ? 3 : 11;
    const int e = (small ? SIM8_EMIN : SIM16_EMIN) + (int)(idx >> P);
    const double s = __builtin_amdgcn_ldexp((double)((1u << P) | (idx & ((1u << P) - 1u))), e - P);
    const double y = exp_doc(-s);
    const double lo = y * (1.0 - 0x1p-48), hi = y * (1.0 + 0x1p-48);
    const double r = rn_grid(y, P, -126);
    if (rn_grid(lo, P, -126) != r || rn_grid(hi, P, -126) != r) atomicAdd(ambiguous, 1u);
    if (small) sim8[idx] = (uint16_t)bf16_bits((float)r);   // 4 significant bits: exact in bf16
    else sim16[idx] = __builtin_bit_cast(uint32_t, (float)r);
}

// ------------------------------------------------------------------ logits entry kernels
// One wave: 64 rows x (16*NC) keys.  grid.x = B*Hq*ceil(nrows/64), grid.y = N/(16*NC).
template <int D, int NC, bool SR>
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
    const float *qrow[1] = {p.qt + (((size_t)b * p.Hq + h) * p.N + j) * D};
    for (int g = 0; g < NC; ++g) {
        const int key0 = (blockIdx.y * NC + g) * 16;
        const float *kt = p.kt32 + (((size_t)b * p.Hkv + hk) * p.N + key0) * (size_t)D;
        uint32_t acc[1][8], sat[1];
        if constexpr (SR) {
            const int jq[1] = {j};
            sr8_chunk<D, 1>(qrow, kt, p.seed, (uint64_t)bh, jq, key0, acc, sat);
        } else {
            emu8_chunk<D, 1>(qrow, kt, acc);
        }
        if (r < p.nrows) {
            uint8_t *out = p.y8 + (((size_t)b * p.Hq + h) * p.nrows + r) * p.N + key0;
#pragma unroll
            for (int pp = 0; pp < 8; ++pp)
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const int i = key0 + 2 * pp + t;
                    const bool vis = !(p.causal && i > j) && !(p.window > 0 && i <= j - p.window);
                    out[2 * pp + t] = vis ? (uint8_t)(acc[0][pp] >> (8 * t)) : (uint8_t)0xFF;
                }
        }
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
    const float *qrow[1] = {p.qt + (((size_t)b * p.Hq + h) * p.N + j) * D};
    const float *kt = p.kt32 + (((size_t)b * p.Hkv + hk) * p.N + key0) * (size_t)D;
    uint32_t codes[1][8];
    rec16_chunk<D, 1>(qrow, kt, codes);
    if (r >= p.nrows) return;
    uint16_t *out = p.y16 + (((size_t)b * p.Hq + h) * p.nrows + r) * p.N + key0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int key = key0 + i;
        const bool vis = !(p.causal && key > j) && !(p.window > 0 && key <= j - p.window);
        out[i] = vis ? (uint16_t)(codes[0][i >> 1] >> (16 * (i & 1))) : (uint16_t)0xFFFF;
    }
}

// SIM profile logit values: one wave, 64 rows x 16 keys.
template <int D, bool HIGH>
__global__ __launch_bounds__(64) void logits_sim_kernel(LogitsParams p)
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
    const float *qrow[1] = {p.qt + (((size_t)b * p.Hq + h) * p.N + j) * D};
    const float *kt = p.kt32 + (((size_t)b * p.Hkv + hk) * p.N + key0) * (size_t)D;
    float val[16];
    if constexpr (HIGH) {
        uint32_t w[1][16];
        rec16_chunk<D, 1, true>(qrow, kt, w);
#pragma unroll
        for (int i = 0; i < 16; ++i) val[i] = __builtin_bit_cast(float, w[0][i]);
    } else {
        uint32_t w[1][8];
        emu8s_pass<D, 1>(qrow, kt, w);
#pragma unroll
        for (int i = 0; i < 16; ++i) val[i] = bf16_value((w[0][i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
    }
    if (r >= p.nrows) return;
    float *out = p.ysim + (((size_t)b * p.Hq + h) * p.nrows + r) * p.N + key0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int key = key0 + i;
        const bool vis = !(p.causal && key > j) && !(p.window > 0 && key <= j - p.window);
        out[i] = vis ? val[i] : __builtin_nanf("");
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

// ------------------------------------------------------------------ launchers
// Grid of the prepass kernels: 256-thread blocks over one head's float4
// groups (x), heads (y); both capped, the kernels stride over the rest.
static dim3 prepass_grid(int BH, int rows, int D)
{
    const long n4 = (long)rows * (D / 4);
    const long gx = (n4 + 255) / 256;
    return dim3((unsigned)(gx < 4096 ? (gx > 0 ? gx : 1) : 4096), (unsigned)(BH < 65535 ? (BH > 0 ? BH : 1) : 65535));
}

hipError_t launch_prepass(const uint16_t *q, const uint16_t *k, float *qt, float *kt32, int B, int Hq, int Hkv,
                          int N, int Nq, int Nk, int D, float scale, hipStream_t s, bool grouped, unsigned *bad)
{
    hipLaunchKernelGGL(prescale_q_kernel, prepass_grid(B * Hq, Nq, D), dim3(256), 0, s, q, qt, scale, N, Nq, D, B * Hq,
                       grouped ? 64 : 0, bad, 1u);
    hipLaunchKernelGGL(convert_k_kernel, prepass_grid(B * Hkv, Nk, D), dim3(256), 0, s, k, kt32, N, Nk, D, B * Hkv,
                       grouped ? 16 : 0, bad);
    return hipGetLastError();
}

hipError_t launch_prescale_q(const uint16_t *q, float *qt, int BH, int rows, int D, float scale, hipStream_t s)
{
    hipLaunchKernelGGL(prescale_q_kernel, prepass_grid(BH, rows, D), dim3(256), 0, s, q, qt, scale, rows, rows, D, BH, 0,
                       (unsigned *)nullptr, 0u);
    return hipGetLastError();
}

hipError_t launch_transpose_v(const uint16_t *v, uint16_t *vt, int B, int Hkv, int N, int Nk, int D, hipStream_t s,
                              unsigned *bad)
{
    hipLaunchKernelGGL(transpose_v_kernel, dim3((unsigned)(Nk / 64), (unsigned)(D / 64), (unsigned)(B * Hkv)),
                       dim3(256), 0, s, v, vt, N, Nk, D, bad);
    return hipGetLastError();
}

template <bool SR>
static void launch_logits8_t(const LogitsParams &p, int D, hipStream_t s)
{
    const unsigned gx = (unsigned)(p.B * p.Hq * ((p.nrows + 63) / 64));
    if (p.N % 64 == 0) {
        dim3 grid(gx, (unsigned)(p.N / 64));
        if (D == 64) hipLaunchKernelGGL((logits8_kernel<64, 4, SR>), grid, dim3(64), 0, s, p);
        else if (D == 128) hipLaunchKernelGGL((logits8_kernel<128, 4, SR>), grid, dim3(64), 0, s, p);
        else hipLaunchKernelGGL((logits8_kernel<256, 4, SR>), grid, dim3(64), 0, s, p);
    } else {
        dim3 grid(gx, (unsigned)(p.N / 16));
        if (D == 64) hipLaunchKernelGGL((logits8_kernel<64, 1, SR>), grid, dim3(64), 0, s, p);
        else if (D == 128) hipLaunchKernelGGL((logits8_kernel<128, 1, SR>), grid, dim3(64), 0, s, p);
        else hipLaunchKernelGGL((logits8_kernel<256, 1, SR>), grid, dim3(64), 0, s, p);
    }
}

hipError_t launch_logits8(const LogitsParams &p, int D, hipStream_t s, bool sr)
{
    if (sr) launch_logits8_t<true>(p, D, s);
    else launch_logits8_t<false>(p, D, s);
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

hipError_t launch_logits_sim(const LogitsParams &p, int D, int high, hipStream_t s)
{
    dim3 grid((unsigned)(p.B * p.Hq * ((p.nrows + 63) / 64)), (unsigned)(p.N / 16));
    if (high) {
        if (D == 64) hipLaunchKernelGGL((logits_sim_kernel<64, true>), grid, dim3(64), 0, s, p);
        else if (D == 128) hipLaunchKernelGGL((logits_sim_kernel<128, true>), grid, dim3(64), 0, s, p);
        else hipLaunchKernelGGL((logits_sim_kernel<256, true>), grid, dim3(64), 0, s, p);
    } else {
        if (D == 64) hipLaunchKernelGGL((logits_sim_kernel<64, false>), grid, dim3(64), 0, s, p);
        else if (D == 128) hipLaunchKernelGGL((logits_sim_kernel<128, false>), grid, dim3(64), 0, s, p);
        else hipLaunchKernelGGL((logits_sim_kernel<256, false>), grid, dim3(64), 0, s, p);
    }
    return hipGetLastError();
}

hipError_t launch_build_sim_tables(uint16_t *sim8, uint32_t *sim16, unsigned *ambiguous, hipStream_t s)
{
    hipLaunchKernelGGL(build_sim_tables_kernel, dim3((SIM16_N + SIM8_TABLE + 255) / 256), dim3(256), 0, s, sim8, sim16,
                       ambiguous);
    return hipGetLastError();
}

hipError_t launch_build_tables(uint8_t *lut8, uint16_t *lut8e, uint16_t *exp16, uint32_t *exp16hl, unsigned *ambiguous,
                              hipStream_t s)
{
    hipLaunchKernelGGL(build_tables_kernel, dim3((65536 + 256 + 255) / 256), dim3(256), 0, s, lut8, lut8e, exp16,
                       exp16hl, ambiguous);
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
