// lamp_kernels.h -- kernel parameter blocks and launchers (library-internal).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "lamp.h"

namespace lamp {

enum { MODE_LAMP = 0, MODE_PURE8 = 1, MODE_ALL16 = 2 };

// Sizes of the SIM profile's exponential tables (layout in lamp_device.h):
// the 8-bit one padded to 256 entries for the forward kernel's LDS copy.
constexpr int SIM8_ENTRIES = 112, SIM8_TABLE = 256, SIM16_TABLE = 45056;

struct FwdParams {
    const float *qt;          // [B][Hq][Nq][D] pre-scaled queries, fp32 (row or grouped layout, see launch_prepass)
    const float *kt32;        // [B][Hkv][Nk][D] keys, fp32 (row or grouped layout)
    const uint16_t *vt;       // [B][Hkv][D][Nk] bf16, V transposed
    const uint16_t *exp16;    // ue5m11 shift code -> ue5m11 exp code
    const uint32_t *exp16hl;  // ue5m11 shift code -> bf16 high | low << 16 of the ue5m11 exp
    const uint16_t *lut8e;    // ue5m3 shift code -> bf16 bits of the ue5m3 exp
    const uint16_t *sim8;     // SIM profile: 8-bit exp table (bf16 bits), lamp_device.h layout
    const uint32_t *sim16;    // SIM profile: 16-bit exp table (FP32 patterns)
    float *o;                 // [B][Hq][N][D]
    float *lse;               // [B][Hq][N]
    uint8_t *mask;            // [B][Hq][N/BQ][N/BK]
    int B, Hq, Hkv, N;        // N: sequence length (visibility, O / lse rows)
    int Nq, Nk;               // padded lengths: rows of qt, keys of kt32 / vt (whole blocks / tiles)
    int causal, window, mode;
    unsigned flags;           // LAMP_SIM_PROFILE; LAMP_STAGE1_OFF | LAMP_MU_TRUNC in the threshold mode
    double delta, tau;
    uint64_t seed;            // key of the stochastic-rounding generator (dispatch_fwd_sr)
    uint64_t *stats;          // LAMP_STATS_WORDS(NK) counters added to, or null
    uint8_t *dbg_y8;          // [B][Hq][dbg_nqb*BQ][Nk] 8-bit codes of the observed query blocks, or null
    uint16_t *dbg_y16;        // the same for the 16-bit codes of recomputed sub-blocks, or null
    int dbg_qb0, dbg_nqb;     // observed query blocks of every (b, h)
};

struct LogitsParams {
    const float *qt;
    const float *kt32;
    uint8_t *y8;
    uint16_t *y16;
    float *ysim;              // SIM profile logit values
    int B, Hq, Hkv, N, causal, window, row0, nrows;
    uint64_t seed;            // stochastic rounding of the 8-bit logits (launch_logits8, sr)
};

// The fixed scratch of lamp_attn_fwd_noalloc (lamp_noalloc.hip): its size,
// and its device address on the current device.
constexpr size_t NOALLOC_SCRATCH_BYTES = LAMP_NOALLOC_SCRATCH_BYTES;
hipError_t noalloc_scratch_address(void **ptr);

// Phase timer of the pipelined kernel (a -DLAMP_PHASE_TIMER build): PHASE_N
// cycle sums and the number of waves; hipErrorNotSupported otherwise.
constexpr int PHASE_N = 10;
hipError_t phase_read(unsigned long long *host, bool reset);
hipError_t launch_prescale_q(const uint16_t *q, float *qt, int BH, int rows, int D, float scale, hipStream_t s);
bool fwd_supported(int D, int BQ, int BK, int NK);
hipError_t dispatch_fwd16(int D, int BQ, const FwdParams &p, hipStream_t s, bool *found);
hipError_t dispatch_fwd16_sr(int D, int BQ, const FwdParams &p, hipStream_t s, bool *found);
hipError_t dispatch_fwd(int D, int BQ, int BK, int NK, const FwdParams &p, hipStream_t s, bool *found);
// the general kernel with stochastically rounded 8-bit logits (row layout)
hipError_t dispatch_fwd_sr(int D, int BQ, int BK, int NK, const FwdParams &p, hipStream_t s, bool *found);
// bad (may be null): bit 2 is or-ed into *bad if a V element is not finite.
hipError_t launch_transpose_v(const uint16_t *v, uint16_t *vt, int B, int Hkv, int N, int Nk, int D, hipStream_t s,
                              unsigned *bad = nullptr);

// Issue rates of the logit loops' instructions (lamp_rates.hip): ns per
// wave-instruction (per emulated step for RATE_STEP) per SIMD, into ns[RATE_N].
enum { RATE_FMAC = 0, RATE_FMAC_DPP = 1, RATE_DECODE = 2, RATE_ENCODE = 3, RATE_STEP = 4, RATE_STEP_SIM = 5, RATE_N = 6 };
hipError_t measure_issue_rates(double *ns, hipStream_t s);
// grouped: the layout of the pipelined kernel (queries in 64-row and keys in
// 16-row blocks, each block stored [D/4][rows][4]); otherwise [rows][D].
// bad (may be null): bit 0 (q) or bit 1 (k) is or-ed into *bad if an element
// is not finite.
hipError_t launch_prepass(const uint16_t *q, const uint16_t *k, float *qt, float *kt32, int B, int Hq, int Hkv,
                          int N, int Nq, int Nk, int D, float scale, hipStream_t s, bool grouped = false,
                          unsigned *bad = nullptr);
// whether dispatch_fwd runs the pipelined kernel (which reads the grouped layout)
bool fwd_grouped(int D, int BQ, int BK, int NK);
hipError_t launch_logits8(const LogitsParams &p, int D, hipStream_t s, bool sr = false);
hipError_t launch_logits16(const LogitsParams &p, int D, hipStream_t s);
hipError_t launch_logits_sim(const LogitsParams &p, int D, int high, hipStream_t s);
hipError_t launch_build_sim_tables(uint16_t *sim8, uint32_t *sim16, unsigned *ambiguous, hipStream_t s);
hipError_t launch_build_tables(uint8_t *lut8, uint16_t *lut8e, uint16_t *exp16, uint32_t *exp16hl, unsigned *ambiguous,
                              hipStream_t s);
hipError_t launch_selftest_e4m3(const float *in, uint8_t *out, uint8_t *raw, size_t n, hipStream_t s);
hipError_t launch_selftest_exp_doc(const double *x, double *y, size_t n, hipStream_t s);

} // namespace lamp
