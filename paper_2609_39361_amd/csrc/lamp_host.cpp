// lamp_host.cpp -- the C ABI of liblamp.so (declared in include/lamp.h):
// argument validation, per-device tables and workspace, kernel launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "lamp.h"
#include "lamp_kernels.h"

namespace {

thread_local char g_err[512] = "";

int fail(int status, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return status;
}

#define HIP_TRY(expr)                                                                              \
    do {                                                                                           \
        hipError_t e_ = (expr);                                                                    \
        if (e_ != hipSuccess) return fail(LAMP_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_));  \
    } while (0)

struct DeviceState {
    bool ready = false;
    uint8_t *lut8 = nullptr;
    uint16_t *lut8e = nullptr;
    uint16_t *exp16 = nullptr;
    uint32_t *exp16hl = nullptr;
    uint16_t *sim8 = nullptr;    // SIM profile tables
    uint32_t *sim16 = nullptr;
    void *ws = nullptr;
    size_t ws_bytes = 0;
    void *dws = nullptr;         // decode workspace: pre-scaled queries, 8-bit logit codes
    size_t dws_bytes = 0;
};

std::mutex g_mu;
std::vector<DeviceState> g_dev;

// Kernel timing (lamp_timing_enable / lamp_timing_read): event triples
// around the prepass and the forward kernel of each lamp_attn_fwd call.
struct TimedCall {
    hipEvent_t e[3];
};
std::mutex g_tmu;
bool g_timing = false;
std::vector<TimedCall> g_timed;

DeviceState *state_of(int dev)
{
    if (dev < 0) return nullptr;
    if ((size_t)dev >= g_dev.size()) g_dev.resize((size_t)dev + 1);
    return &g_dev[(size_t)dev];
}

// Build the exponential tables of the current device (lock held).
int init_locked(int dev)
{
    DeviceState *st = state_of(dev);
    if (st->ready) return LAMP_OK;
    HIP_TRY(hipMalloc(&st->lut8, 256));
    HIP_TRY(hipMalloc(&st->lut8e, 256 * sizeof(uint16_t)));
    HIP_TRY(hipMalloc(&st->exp16, 65536 * sizeof(uint16_t)));
    HIP_TRY(hipMalloc(&st->exp16hl, 65536 * sizeof(uint32_t)));
    unsigned *amb = nullptr;
    HIP_TRY(hipMalloc(&amb, sizeof(unsigned)));
    HIP_TRY(hipMemset(amb, 0, sizeof(unsigned)));
    HIP_TRY(hipMalloc(&st->sim8, lamp::SIM8_TABLE * sizeof(uint16_t)));
    HIP_TRY(hipMalloc(&st->sim16, lamp::SIM16_TABLE * sizeof(uint32_t)));
    HIP_TRY(lamp::launch_build_tables(st->lut8, st->lut8e, st->exp16, st->exp16hl, amb, nullptr));
    HIP_TRY(lamp::launch_build_sim_tables(st->sim8, st->sim16, amb, nullptr));
    unsigned h_amb = 0;
    HIP_TRY(hipMemcpy(&h_amb, amb, sizeof(unsigned), hipMemcpyDeviceToHost));
    HIP_TRY(hipFree(amb));
    if (h_amb != 0) return fail(LAMP_ERR_INIT, "%u exponential table entries could not be rounded with certainty", h_amb);
    st->ready = true;
    return LAMP_OK;
}

int current_device(int *dev)
{
    HIP_TRY(hipGetDevice(dev));
    return LAMP_OK;
}

// Scale applied to Q before accumulation, RN32(1/sqrt(d)).
float scale_of(int d)
{
    switch (d) {
    case 64: return 0.125f;
    case 256: return 0.0625f;
    case 128: {
        uint32_t b = 0x3DB504F3u;   // RN32(1/sqrt(128))
        float f;
        std::memcpy(&f, &b, 4);
        return f;
    }
    default: return 0.0f;
    }
}

struct Workspace {
    float *qt;
    float *kt32;
    uint16_t *vt;   // only when asked for (the forward pass)
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Grow-only workspace for the pre-scaled Q (Nq rows per head), the fp32 K
// and (with_vt) the transposed V (Nk keys per head) (lock held).
int workspace_locked(int dev, int B, int Hq, int Hkv, int Nq, int Nk, int d, Workspace *w, bool with_vt = false)
{
    DeviceState *st = state_of(dev);
    size_t nq = (size_t)B * Hq * Nq * d, nk = (size_t)B * Hkv * Nk * d;
    size_t bq = align256(nq * 4), bk32 = align256(nk * 4), bvt = with_vt ? align256(nk * 2) : 0;
    size_t need = bq + bk32 + bvt;
    if (need > st->ws_bytes) {
        if (st->ws) {
            HIP_TRY(hipDeviceSynchronize());
            HIP_TRY(hipFree(st->ws));
            st->ws = nullptr;
            st->ws_bytes = 0;
        }
        HIP_TRY(hipMalloc(&st->ws, need));
        st->ws_bytes = need;
    }
    char *base = static_cast<char *>(st->ws);
    w->qt = reinterpret_cast<float *>(base);
    w->kt32 = reinterpret_cast<float *>(base + bq);
    w->vt = with_vt ? reinterpret_cast<uint16_t *>(base + bq + bk32) : nullptr;
    return LAMP_OK;
}

// rows: query rows per (b, h) to compute (N for the prefill form; M for the
// decode form, whose query pointer may be null when M = 0).
int check_common(const void *q, const void *k, int B, int Hq, int Hkv, int N, int d, int causal, int window,
                 int rows = -1)
{
    if (rows < 0) rows = N;
    if ((B > 0 && N > 0 && rows > 0) && (!q || !k)) return fail(LAMP_ERR_INVALID_ARG, "null input pointer");
    if (B < 0 || Hq <= 0 || Hkv <= 0 || N < 0 || d <= 0)
        return fail(LAMP_ERR_INVALID_ARG, "invalid sizes (B=%d Hq=%d Hkv=%d N=%d d=%d)", B, Hq, Hkv, N, d);
    if (Hq % Hkv) return fail(LAMP_ERR_INVALID_ARG, "Hq=%d is not a multiple of Hkv=%d", Hq, Hkv);
    if (causal != 0 && causal != 1) return fail(LAMP_ERR_INVALID_ARG, "causal must be 0 or 1");
    if (window < 0) return fail(LAMP_ERR_INVALID_ARG, "window must be >= 0");
    if (window > 0 && !causal) return fail(LAMP_ERR_INVALID_ARG, "a sliding window requires causal=1");
    if (d != 64 && d != 128 && d != 256) return fail(LAMP_ERR_UNSUPPORTED, "head dimension %d not built (64, 128, 256)", d);
    if (N > (1 << 20)) return fail(LAMP_ERR_UNSUPPORTED, "N=%d above 2^20", N);
    if ((size_t)B * Hq * (size_t)N > (size_t)1 << 31) return fail(LAMP_ERR_UNSUPPORTED, "B*Hq*N above 2^31");
    return LAMP_OK;
}

} // namespace

extern "C" {

const char *lamp_status_str(int s)
{
    switch (s) {
    case LAMP_OK: return "ok";
    case LAMP_ERR_INVALID_ARG: return "invalid argument";
    case LAMP_ERR_UNSUPPORTED: return "unsupported configuration";
    case LAMP_ERR_HIP: return "HIP runtime error";
    case LAMP_ERR_INIT: return "device table initialisation failed";
    default: return "unknown status";
    }
}

const char *lamp_last_error(void) { return g_err; }

int lamp_init(int device)
{
    std::lock_guard<std::mutex> lk(g_mu);
    int prev = 0;
    HIP_TRY(hipGetDevice(&prev));
    HIP_TRY(hipSetDevice(device));
    int rc = init_locked(device);
    HIP_TRY(hipSetDevice(prev));
    return rc;
}

void lamp_shutdown(void)
{
    std::lock_guard<std::mutex> lk(g_mu);
    int prev = 0;
    if (hipGetDevice(&prev) != hipSuccess) return;
    for (size_t i = 0; i < g_dev.size(); ++i) {
        DeviceState &st = g_dev[i];
        if (!st.ready && !st.ws && !st.dws) continue;
        if (hipSetDevice((int)i) != hipSuccess) continue;
        (void)hipDeviceSynchronize();
        (void)hipFree(st.lut8);
        (void)hipFree(st.lut8e);
        (void)hipFree(st.exp16);
        (void)hipFree(st.exp16hl);
        (void)hipFree(st.sim8);
        (void)hipFree(st.sim16);
        (void)hipFree(st.ws);
        (void)hipFree(st.dws);
        st = DeviceState();
    }
    (void)hipSetDevice(prev);
}

// The forward pass; sr: the 8-bit logits rounded stochastically with `seed`.
static int fwd_impl(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int N, int d,
                    int causal, int window, int bq, int bk, int nk, double delta, double tau, unsigned flags, bool sr,
                    uint64_t seed, float *o, float *lse, uint8_t *mask, void *stream)
{
    int rc = check_common(q, k, B, Hq, Hkv, N, d, causal, window);
    if (rc) return rc;
    if ((B > 0 && N > 0) && (!v || !o || !lse || !mask))
        return fail(LAMP_ERR_INVALID_ARG, "null pointer among v, o, lse, mask");
    if (!(delta >= 0.0) || std::isinf(delta)) return fail(LAMP_ERR_INVALID_ARG, "delta must be finite and >= 0");
    if (!(tau >= 0.0)) return fail(LAMP_ERR_INVALID_ARG, "tau must be >= 0 (or +inf)");
    if (flags & ~(unsigned)(LAMP_STAGE1_OFF | LAMP_MU_TRUNC | LAMP_SIM_PROFILE))
        return fail(LAMP_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
    if (bq <= 0 || bk <= 0 || nk <= 0) return fail(LAMP_ERR_INVALID_ARG, "block sizes must be positive");
    if (!lamp::fwd_supported(d, bq, bk, nk))
        return fail(LAMP_ERR_UNSUPPORTED, "block sizes (bq=%d, bk=%d, nk=%d) not built for d=%d", bq, bk, nk, d);
    if (sr && (flags & LAMP_SIM_PROFILE))
        return fail(LAMP_ERR_UNSUPPORTED, "stochastic rounding is built for the formats of Sec. 3.3, not the SIM profile");
    if ((flags & LAMP_SIM_PROFILE) && !(bk == 16 && nk == 4 && (d == 128 || d == 256)))
        return fail(LAMP_ERR_UNSUPPORTED, "the SIM profile is built for bk=16, nk=4, d in {128, 256} (bk=%d, nk=%d, d=%d)",
                    bk, nk, d);
    if (B == 0 || N == 0) return LAMP_OK;   // nothing to compute
    // the workspace holds whole query blocks and whole key tiles (zero padded)
    const int Nq = (N + bq - 1) / bq * bq, Nk = (N + bk * nk - 1) / (bk * nk) * (bk * nk);
    int dev = 0;
    rc = current_device(&dev);
    if (rc) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    lamp::FwdParams p{};
    Workspace w{};
    {
        std::lock_guard<std::mutex> lk(g_mu);
        rc = init_locked(dev);
        if (rc) return rc;
        rc = workspace_locked(dev, B, Hq, Hkv, Nq, Nk, d, &w, true);
        if (rc) return rc;
        DeviceState *st = state_of(dev);
        p.exp16 = st->exp16;
        p.exp16hl = st->exp16hl;
        p.lut8e = st->lut8e;
        p.sim8 = st->sim8;
        p.sim16 = st->sim16;
    }
    p.qt = w.qt;
    p.kt32 = w.kt32;
    p.vt = w.vt;
    p.o = o;
    p.lse = lse;
    p.mask = mask;
    p.B = B;
    p.Hq = Hq;
    p.Hkv = Hkv;
    p.N = N;
    p.Nq = Nq;
    p.Nk = Nk;
    p.causal = causal;
    p.window = window;
    p.delta = delta;
    p.tau = tau;
    p.mode = std::isinf(tau) ? lamp::MODE_PURE8 : (tau == 0.0 ? lamp::MODE_ALL16 : lamp::MODE_LAMP);
    p.flags = p.mode == lamp::MODE_LAMP ? flags : (flags & (unsigned)LAMP_SIM_PROFILE);
    p.seed = seed;
    // the all-16-bit mode computes no 8-bit logit: the rounding mode does not matter there
    const bool use_sr = sr && p.mode != lamp::MODE_ALL16;
    bool timed = false;
    TimedCall tc{};
    {
        std::lock_guard<std::mutex> lk(g_tmu);
        timed = g_timing;
    }
    if (timed) {
        for (int i = 0; i < 3; ++i) HIP_TRY(hipEventCreate(&tc.e[i]));
        HIP_TRY(hipEventRecord(tc.e[0], s));
    }
    HIP_TRY(lamp::launch_prepass(q, k, w.qt, w.kt32, B, Hq, Hkv, N, Nq, Nk, d, scale_of(d), s,
                                 !use_sr && lamp::fwd_grouped(d, bq, bk, nk)));
    HIP_TRY(lamp::launch_transpose_v(v, w.vt, B, Hkv, N, Nk, d, s));
    if (timed) HIP_TRY(hipEventRecord(tc.e[1], s));
    bool found = false;
    if (use_sr) HIP_TRY(lamp::dispatch_fwd_sr(d, bq, bk, nk, p, s, &found));
    else HIP_TRY(lamp::dispatch_fwd(d, bq, bk, nk, p, s, &found));
    if (!found)
        return fail(LAMP_ERR_UNSUPPORTED, "block sizes (bq=%d, bk=%d, nk=%d) not built for d=%d", bq, bk, nk, d);
    if (timed) {
        HIP_TRY(hipEventRecord(tc.e[2], s));
        std::lock_guard<std::mutex> lk(g_tmu);
        g_timed.push_back(tc);
    }
    return LAMP_OK;
}

int lamp_attn_fwd(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int N, int d,
                  int causal, int window, int bq, int bk, int nk, double delta, double tau, unsigned flags, float *o,
                  float *lse, uint8_t *mask, void *stream)
{
    return fwd_impl(q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, delta, tau, flags, false, 0, o, lse, mask,
                    stream);
}

int lamp_attn_fwd_sr(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int N, int d,
                     int causal, int window, int bq, int bk, int nk, double delta, double tau, unsigned flags,
                     uint64_t seed, float *o, float *lse, uint8_t *mask, void *stream)
{
    return fwd_impl(q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, delta, tau, flags, true, seed, o, lse, mask,
                    stream);
}

int lamp_attn_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int M, int N,
                     int d, int causal, int window, int tk, double delta, double tau, unsigned flags, float *o,
                     float *lse, uint8_t *mask, void *stream)
{
    if (M < 0 || M > N) return fail(LAMP_ERR_INVALID_ARG, "M=%d query rows must lie in [0, N=%d]", M, N);
    int rc = check_common(q, k, B, Hq, Hkv, N, d, causal, window, M);
    if (rc) return rc;
    if ((B > 0 && M > 0) && (!q || !k || !v || !o || !lse || !mask))
        return fail(LAMP_ERR_INVALID_ARG, "null pointer among q, k, v, o, lse, mask");
    if (!(delta >= 0.0) || std::isinf(delta)) return fail(LAMP_ERR_INVALID_ARG, "delta must be finite and >= 0");
    if (!(tau >= 0.0)) return fail(LAMP_ERR_INVALID_ARG, "tau must be >= 0 (or +inf)");
    if (flags) return fail(LAMP_ERR_INVALID_ARG, "unknown flags 0x%x (the decode form takes none)", flags);
    if (tk != 64) return fail(LAMP_ERR_UNSUPPORTED, "keys per update tk=%d not built (64)", tk);
    if (B == 0 || M == 0) return LAMP_OK;   // nothing to compute
    const int Np = (N + 63) / 64 * 64, nch = (N + 511) / 512;   // key chunks of the P.V pass
    const size_t nrows = (size_t)B * Hq * M;
    const size_t bq = align256(nrows * d * 4), by8 = align256(nrows * Np);
    const size_t be = align256(nrows * Np * 4), bf = align256(nrows * (Np / 64) * 8);
    const size_t bpart = align256(nrows * nch * d * 4), need = bq + by8 + be + bf + bpart;
    int dev = 0;
    rc = current_device(&dev);
    if (rc) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    lamp::DecParams p{};
    {
        std::lock_guard<std::mutex> lk(g_mu);
        rc = init_locked(dev);
        if (rc) return rc;
        DeviceState *st = state_of(dev);
        if (need > st->dws_bytes) {
            if (st->dws) {
                HIP_TRY(hipDeviceSynchronize());
                HIP_TRY(hipFree(st->dws));
                st->dws = nullptr;
                st->dws_bytes = 0;
            }
            HIP_TRY(hipMalloc(&st->dws, need));
            st->dws_bytes = need;
        }
        char *base = static_cast<char *>(st->dws);
        p.qt = reinterpret_cast<float *>(base);
        p.y8 = reinterpret_cast<uint8_t *>(base + bq);
        p.e = reinterpret_cast<float *>(base + bq + by8);
        p.f = reinterpret_cast<double *>(base + bq + by8 + be);
        p.part = reinterpret_cast<float *>(base + bq + by8 + be + bf);
        p.lut8e = st->lut8e;
        p.exp16hl = st->exp16hl;
    }
    p.k = k;
    p.v = v;
    p.o = o;
    p.lse = lse;
    p.mask = mask;
    p.B = B;
    p.Hq = Hq;
    p.Hkv = Hkv;
    p.M = M;
    p.N = N;
    p.Np = Np;
    const int first = window > 0 ? N - M - window + 1 : 0;
    p.kb0 = first > 0 ? first / 64 * 64 : 0;
    p.causal = causal;
    p.window = window;
    p.delta = delta;
    p.tau = tau;
    p.mode = std::isinf(tau) ? lamp::MODE_PURE8 : (tau == 0.0 ? lamp::MODE_ALL16 : lamp::MODE_LAMP);
    bool timed = false;
    TimedCall tc{};
    {
        std::lock_guard<std::mutex> lk(g_tmu);
        timed = g_timing;
    }
    if (timed) {
        for (int i = 0; i < 3; ++i) HIP_TRY(hipEventCreate(&tc.e[i]));
        HIP_TRY(hipEventRecord(tc.e[0], s));
    }
    HIP_TRY(lamp::launch_prescale_q(q, const_cast<float *>(p.qt), B * Hq, M, d, scale_of(d), s));
    if (timed) HIP_TRY(hipEventRecord(tc.e[1], s));
    HIP_TRY(lamp::launch_decode(d, p, s));
    if (timed) {
        HIP_TRY(hipEventRecord(tc.e[2], s));
        std::lock_guard<std::mutex> lk(g_tmu);
        g_timed.push_back(tc);
    }
    return LAMP_OK;
}

int lamp_issue_rates(double *ns_per_simd, void *stream)
{
    if (!ns_per_simd) return fail(LAMP_ERR_INVALID_ARG, "null output pointer");
    HIP_TRY(lamp::measure_issue_rates(ns_per_simd, static_cast<hipStream_t>(stream)));
    return LAMP_OK;
}

int lamp_timing_enable(int on)
{
    std::lock_guard<std::mutex> lk(g_tmu);
    g_timing = on != 0;
    return LAMP_OK;
}

int lamp_timing_read(int *launches, double *fwd_ms, double *prepass_ms)
{
    std::vector<TimedCall> calls;
    {
        std::lock_guard<std::mutex> lk(g_tmu);
        calls.swap(g_timed);
    }
    double tf = 0.0, tp = 0.0;
    int rc = LAMP_OK;
    for (TimedCall &c : calls) {
        float a = 0.f, b = 0.f;
        if (rc == LAMP_OK) {
            hipError_t e = hipEventSynchronize(c.e[2]);
            if (e == hipSuccess) e = hipEventElapsedTime(&a, c.e[0], c.e[1]);
            if (e == hipSuccess) e = hipEventElapsedTime(&b, c.e[1], c.e[2]);
            if (e != hipSuccess) rc = fail(LAMP_ERR_HIP, "kernel timing events: %s", hipGetErrorString(e));
        }
        tp += a;
        tf += b;
        for (int i = 0; i < 3; ++i) (void)hipEventDestroy(c.e[i]);
    }
    if (launches) *launches = (int)calls.size();
    if (fwd_ms) *fwd_ms = tf;
    if (prepass_ms) *prepass_ms = tp;
    return rc;
}

static int logits_common(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                         int window, int row0, int nrows, void *out, lamp::LogitsParams *p, Workspace *w)
{
    int rc = check_common(q, k, B, Hq, Hkv, N, d, causal, window);
    if (rc) return rc;
    if (!out) return fail(LAMP_ERR_INVALID_ARG, "null output pointer");
    if (B == 0 || N == 0 || N % 16) return fail(LAMP_ERR_UNSUPPORTED, "N=%d is not a positive multiple of 16 (B=%d)", N, B);
    if (row0 < 0 || nrows <= 0 || row0 + nrows > N) return fail(LAMP_ERR_INVALID_ARG, "row range outside [0, N)");
    int dev = 0;
    rc = current_device(&dev);
    if (rc) return rc;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        rc = init_locked(dev);
        if (rc) return rc;
        rc = workspace_locked(dev, B, Hq, Hkv, N, N, d, w);
        if (rc) return rc;
    }
    *p = lamp::LogitsParams{};
    p->qt = w->qt;
    p->kt32 = w->kt32;
    p->B = B;
    p->Hq = Hq;
    p->Hkv = Hkv;
    p->N = N;
    p->causal = causal;
    p->window = window;
    p->row0 = row0;
    p->nrows = nrows;
    return LAMP_OK;
}

int lamp_attn_logits8(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                      int window, int row0, int nrows, uint8_t *y8, void *stream)
{
    lamp::LogitsParams p;
    Workspace w;
    int rc = logits_common(q, k, B, Hq, Hkv, N, d, causal, window, row0, nrows, y8, &p, &w);
    if (rc) return rc;
    p.y8 = y8;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(lamp::launch_prepass(q, k, w.qt, w.kt32, B, Hq, Hkv, N, N, N, d, scale_of(d), s));
    HIP_TRY(lamp::launch_logits8(p, d, s));
    return LAMP_OK;
}

int lamp_attn_logits8_sr(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                         int window, int row0, int nrows, uint64_t seed, uint8_t *y8, void *stream)
{
    lamp::LogitsParams p;
    Workspace w;
    int rc = logits_common(q, k, B, Hq, Hkv, N, d, causal, window, row0, nrows, y8, &p, &w);
    if (rc) return rc;
    p.y8 = y8;
    p.seed = seed;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(lamp::launch_prepass(q, k, w.qt, w.kt32, B, Hq, Hkv, N, N, N, d, scale_of(d), s));
    HIP_TRY(lamp::launch_logits8(p, d, s, true));
    return LAMP_OK;
}

int lamp_attn_logits16(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                       int window, int row0, int nrows, uint16_t *y16, void *stream)
{
    lamp::LogitsParams p;
    Workspace w;
    int rc = logits_common(q, k, B, Hq, Hkv, N, d, causal, window, row0, nrows, y16, &p, &w);
    if (rc) return rc;
    p.y16 = y16;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(lamp::launch_prepass(q, k, w.qt, w.kt32, B, Hq, Hkv, N, N, N, d, scale_of(d), s));
    HIP_TRY(lamp::launch_logits16(p, d, s));
    return LAMP_OK;
}

int lamp_attn_logits_sim(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv, int N, int d, int causal,
                         int window, int row0, int nrows, int high, float *y, void *stream)
{
    lamp::LogitsParams p;
    Workspace w;
    int rc = logits_common(q, k, B, Hq, Hkv, N, d, causal, window, row0, nrows, y, &p, &w);
    if (rc) return rc;
    p.ysim = y;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(lamp::launch_prepass(q, k, w.qt, w.kt32, B, Hq, Hkv, N, N, N, d, scale_of(d), s));
    HIP_TRY(lamp::launch_logits_sim(p, d, high != 0, s));
    return LAMP_OK;
}

int lamp_selftest_e4m3(const float *in, uint8_t *out, uint8_t *raw, size_t n, void *stream)
{
    if (!in || !out) return fail(LAMP_ERR_INVALID_ARG, "null pointer");
    if (n == 0) return LAMP_OK;
    HIP_TRY(lamp::launch_selftest_e4m3(in, out, raw, n, static_cast<hipStream_t>(stream)));
    return LAMP_OK;
}

int lamp_selftest_exp_doc(const double *x, double *y, size_t n, void *stream)
{
    if (!x || !y) return fail(LAMP_ERR_INVALID_ARG, "null pointer");
    if (n == 0) return LAMP_OK;
    HIP_TRY(lamp::launch_selftest_exp_doc(x, y, n, static_cast<hipStream_t>(stream)));
    return LAMP_OK;
}

int lamp_get_tables(int device, uint8_t *lut8, uint16_t *exp16)
{
    int rc = lamp_init(device);
    if (rc) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    int prev = 0;
    HIP_TRY(hipGetDevice(&prev));
    HIP_TRY(hipSetDevice(device));
    DeviceState *st = state_of(device);
    if (lut8) HIP_TRY(hipMemcpy(lut8, st->lut8, 256, hipMemcpyDeviceToHost));
    if (exp16) HIP_TRY(hipMemcpy(exp16, st->exp16, 65536 * sizeof(uint16_t), hipMemcpyDeviceToHost));
    HIP_TRY(hipSetDevice(prev));
    return LAMP_OK;
}

int lamp_get_exp16_parts(int device, uint32_t *parts)
{
    if (!parts) return fail(LAMP_ERR_INVALID_ARG, "null pointer");
    int rc = lamp_init(device);
    if (rc) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    int prev = 0;
    HIP_TRY(hipGetDevice(&prev));
    HIP_TRY(hipSetDevice(device));
    HIP_TRY(hipMemcpy(parts, state_of(device)->exp16hl, 65536 * sizeof(uint32_t), hipMemcpyDeviceToHost));
    HIP_TRY(hipSetDevice(prev));
    return LAMP_OK;
}

int lamp_get_sim_tables(int device, uint16_t *sim8, uint32_t *sim16)
{
    int rc = lamp_init(device);
    if (rc) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    int prev = 0;
    HIP_TRY(hipGetDevice(&prev));
    HIP_TRY(hipSetDevice(device));
    DeviceState *st = state_of(device);
    hipError_t e = hipSuccess;
    if (sim8) e = hipMemcpy(sim8, st->sim8, lamp::SIM8_ENTRIES * sizeof(uint16_t), hipMemcpyDeviceToHost);
    if (e == hipSuccess && sim16) e = hipMemcpy(sim16, st->sim16, lamp::SIM16_TABLE * sizeof(uint32_t), hipMemcpyDeviceToHost);
    (void)hipSetDevice(prev);
    if (e != hipSuccess) return fail(LAMP_ERR_HIP, "lamp_get_sim_tables: %s", hipGetErrorString(e));
    return LAMP_OK;
}

} // extern "C"
