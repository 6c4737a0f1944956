// lamp_rates.hip -- issue rates, measured on the device, of the VALU
// instructions the logit loops are made of.
//
// The forward kernel is bound by VALU issue, and not every instruction it
// issues takes one issue slot: on gfx950 a plain fp32 FMA on VGPR operands
// issues faster than one that reads its key through a DPP broadcast, and the
// packed fp32 -> e4m3 conversion takes about two slots.  The published VALU
// peak therefore overstates what the emulated 8-bit accumulation can reach.
// These kernels time each instruction kind (16 independent chains per lane,
// 8 waves per SIMD, so that issue and not latency binds) and the complete
// emulated step of the 8-bit loop (decode a code pair, two broadcast FMAs,
// round the pair back), giving the instruction-mix floor the benchmark sets
// beside the measured kernel time.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lamp_kernels.h"

namespace lamp {

namespace {

#define LAMP_REP16(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15)

// plain fp32 FMA, VGPR operands
__global__ __launch_bounds__(256) void rate_fmac_kernel(float *out, int iters, float q)
{
    float a[16];
    const float k = (float)threadIdx.x * 1e-3f;
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = (float)i * 1e-3f;
    for (int it = 0; it < iters; ++it) {
#define LAMP_F(i) asm volatile("v_fmac_f32 %0, %1, %2" : "+v"(a[i]) : "v"(k), "v"(q));
        LAMP_REP16(LAMP_F)
#undef LAMP_F
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += a[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// fp32 FMA reading its first operand through a DPP row broadcast (the key feed
// of the logit loops); the wait states keep the broadcast source away from
// the VALU write that produced it
__global__ __launch_bounds__(256) void rate_fmac_dpp_kernel(float *out, int iters, float q)
{
    float a[16];
    const float k = (float)threadIdx.x * 1e-3f;
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = (float)i * 1e-3f;
    asm volatile("s_nop 4");
    for (int it = 0; it < iters; ++it) {
#define LAMP_F(i) \
    asm volatile("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf" : "+v"(a[i]) : "v"(k), "v"(q), "n"(i));
        LAMP_REP16(LAMP_F)
#undef LAMP_F
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += a[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// packed e4m3 -> fp32 decode of a code pair
__global__ __launch_bounds__(256) void rate_decode_kernel(float *out, int iters, float q)
{
    typedef float f2 __attribute__((ext_vector_type(2)));
    f2 a[16];
    const uint32_t c = threadIdx.x * 0x01010101u;
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = f2{q, q};
    for (int it = 0; it < iters; ++it) {
#define LAMP_F(i) asm volatile("v_cvt_pk_f32_fp8 %0, %1" : "=v"(a[i]) : "v"(c));
        LAMP_REP16(LAMP_F)
#undef LAMP_F
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += a[i][0] + a[i][1];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// packed fp32 -> e4m3 rounding of a value pair
__global__ __launch_bounds__(256) void rate_encode_kernel(float *out, int iters, float q)
{
    uint32_t a[16];
    const float x = (float)threadIdx.x * 1e-3f;
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = (uint32_t)i;
    for (int it = 0; it < iters; ++it) {
#define LAMP_F(i) asm volatile("v_cvt_pk_fp8_f32 %0, %1, %2" : "+v"(a[i]) : "v"(x), "v"(q));
        LAMP_REP16(LAMP_F)
#undef LAMP_F
    }
    uint32_t s = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += a[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = (float)s;
}

// the emulated step of the 8-bit loop: two multiply-adds (decode, two
// broadcast FMAs, round back), on two fixed temporaries
__global__ __launch_bounds__(256) void rate_step_kernel(float *out, int iters, float q)
{
    uint32_t a[16];
    const float k = (float)threadIdx.x * 1e-3f;
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = (uint32_t)i * 0x0101u;
    asm volatile("s_nop 4");
    for (int it = 0; it < iters; ++it) {
#define LAMP_F(i)                                                                        \
    asm volatile("v_cvt_pk_f32_fp8 v[40:41], %0\n\t"                                     \
                 "v_fmac_f32_dpp v40, %1, %2 row_newbcast:0 row_mask:0xf bank_mask:0xf\n\t" \
                 "v_fmac_f32_dpp v41, %1, %2 row_newbcast:1 row_mask:0xf bank_mask:0xf\n\t" \
                 "v_cvt_pk_fp8_f32 %0, v40, v41"                                         \
                 : "+v"(a[i])                                                            \
                 : "v"(k), "v"(q)                                                        \
                 : "v40", "v41");
        LAMP_REP16(LAMP_F)
#undef LAMP_F
    }
    uint32_t s = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += a[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = (float)s;
}

// the emulated step of the SIM profile's 8-bit loop: one broadcast FMA and
// the round-to-nearest-even of the FP32 pattern to 3 mantissa bits (last kept
// bit extracted, one 3-input add, one mask), per multiply-add
__global__ __launch_bounds__(256) void rate_step_sim_kernel(float *out, int iters, float q)
{
    float a[16];
    const float k = (float)threadIdx.x * 1e-3f;
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = (float)i * 1e-3f;
    asm volatile("s_nop 4");
    for (int it = 0; it < iters; ++it) {
#define LAMP_F(i)                                                                                     \
    asm volatile("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf\n\t"           \
                 "v_bfe_u32 v40, %0, 20, 1\n\t"                                                      \
                 "v_add3_u32 %0, %0, v40, %4\n\t"                                                    \
                 "v_and_b32 %0, %5, %0"                                                              \
                 : "+v"(a[i])                                                                        \
                 : "v"(k), "v"(q), "n"(i), "v"(0x7FFFFu), "v"(0xFFF00000u)                           \
                 : "v40");
        LAMP_REP16(LAMP_F)
#undef LAMP_F
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += a[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

#undef LAMP_REP16

} // namespace

hipError_t measure_issue_rates(double *ns, hipStream_t s)
{
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const int blocks = cus * 8, threads = 256, iters = 4096;   // 8 waves per SIMD
    float *out = nullptr;
    e = hipMalloc(&out, (size_t)blocks * threads * sizeof(float));
    if (e != hipSuccess) return e;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    void (*kern[RATE_N])(float *, int, float) = {rate_fmac_kernel, rate_fmac_dpp_kernel, rate_decode_kernel,
                                                 rate_encode_kernel, rate_step_kernel, rate_step_sim_kernel};
    if ((e = hipEventCreate(&e0)) == hipSuccess && (e = hipEventCreate(&e1)) == hipSuccess) {
        // instructions (steps for the last two kinds) per SIMD of one launch
        const double per_simd = (double)blocks * (threads / 64) * iters * 16 / ((double)cus * 4);
        for (int i = 0; i < RATE_N && e == hipSuccess; ++i) {
            hipLaunchKernelGGL(kern[i], dim3(blocks), dim3(threads), 0, s, out, 64, 1.0f);   // warm-up
            if ((e = hipEventRecord(e0, s)) != hipSuccess) break;
            hipLaunchKernelGGL(kern[i], dim3(blocks), dim3(threads), 0, s, out, iters, 1.0f);
            if ((e = hipEventRecord(e1, s)) != hipSuccess) break;
            if ((e = hipEventSynchronize(e1)) != hipSuccess) break;
            float ms = 0.0f;
            if ((e = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess) break;
            ns[i] = (double)ms * 1e6 / per_simd;
        }
    }
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    const hipError_t ef = hipFree(out);
    return e != hipSuccess ? e : ef;
}

} // namespace lamp
