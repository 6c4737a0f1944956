// lamp_fwd16_sr.hip -- the pipelined forward kernel (lamp_fwd16.hip) with the
// 8-bit logits rounded stochastically (lamp_sr.h), in a translation unit of
// its own so that its instantiations compile beside the others.  Built for
// the threshold and pure 8-bit modes in the formats of Sec. 3.3 (the all-16-bit
// mode computes no 8-bit logit and runs the kernel without SR).
#define LAMP_FWD16_NO_LAUNCHERS
#include "lamp_fwd16.hip"

namespace lamp {

template <int D, int BQ, int MODE, bool OBS>
static hipError_t launch_fwd16_sr_obs(const FwdParams &p, hipStream_t s)
{
    using C = Cfg16<D, BQ>;
    auto kern = lamp_fwd16_kernel<D, BQ, MODE, false, OBS, false, true>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)(p.B * p.Hq * (p.Nq / BQ)));
    hipLaunchKernelGGL(kern, grid, dim3(256), C::LDS, s, p);
    return hipGetLastError();
}

template <int D, int BQ, int MODE>
static hipError_t launch_fwd16_sr_mode(const FwdParams &p, hipStream_t s)
{
    if (p.dbg_y8 || p.dbg_y16) return launch_fwd16_sr_obs<D, BQ, MODE, true>(p, s);
    return launch_fwd16_sr_obs<D, BQ, MODE, false>(p, s);
}

template <int D, int BQ>
static hipError_t launch_fwd16_sr(const FwdParams &p, hipStream_t s)
{
    if (p.mode == MODE_PURE8) return launch_fwd16_sr_mode<D, BQ, MODE_PURE8>(p, s);
    return launch_fwd16_sr_mode<D, BQ, MODE_LAMP>(p, s);
}

hipError_t dispatch_fwd16_sr(int D, int BQ, const FwdParams &p, hipStream_t s, bool *found)
{
    *found = true;
    if (D == 128 && BQ == 64) return launch_fwd16_sr<128, 64>(p, s);
    if (D == 128 && BQ == 128) return launch_fwd16_sr<128, 128>(p, s);
    if (D == 256 && BQ == 64) return launch_fwd16_sr<256, 64>(p, s);
    if (D == 256 && BQ == 128) return launch_fwd16_sr<256, 128>(p, s);
    *found = false;
    return hipSuccess;
}

} // namespace lamp
