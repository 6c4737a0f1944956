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
#include "lamp_decode.h"
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
    void *ws = nullptr;          // the library's workspace of this device (grow-only)
    size_t ws_bytes = 0;
    std::vector<void *> retired; // outgrown workspaces, freed by lamp_reserve / lamp_shutdown
    void *scratch = nullptr;     // device address of this device's fixed scratch (lamp_attn_fwd_noalloc)
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
    // this device's copy of the fixed scratch (the device is current here)
    HIP_TRY(lamp::noalloc_scratch_address(&st->scratch));
    if (!st->scratch) return fail(LAMP_ERR_INIT, "no device address for the fixed scratch");
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
    unsigned *flag;   // non-finite input flag (LAMP_CHECK_FINITE)
    float *qt;
    float *kt32;
    uint16_t *vt;     // only when asked for (the forward pass)
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Byte sizes of the prepass workspace: a 256-byte header (the check flag),
// the pre-scaled Q (Nq rows per head), the fp32 K and (with_vt) the
// transposed V (Nk keys per head).
struct WsLayout {
    size_t qt, k32, vt, total;
};

WsLayout ws_layout(int B, int Hq, int Hkv, int64_t Nq, int64_t Nk, int d, bool with_vt)
{
    const size_t nq = (size_t)B * Hq * Nq * d, nk = (size_t)B * Hkv * Nk * d;
    WsLayout l;
    l.qt = align256(nq * 4);
    l.k32 = align256(nk * 4);
    l.vt = with_vt ? align256(nk * 2) : 0;
    l.total = 256 + l.qt + l.k32 + l.vt;
    return l;
}

void carve(void *base, const WsLayout &l, Workspace *w)
{
    char *c = static_cast<char *>(base);
    w->flag = reinterpret_cast<unsigned *>(c);
    w->qt = reinterpret_cast<float *>(c + 256);
    w->kt32 = reinterpret_cast<float *>(c + 256 + l.qt);
    w->vt = l.vt ? reinterpret_cast<uint16_t *>(c + 256 + l.qt + l.k32) : nullptr;
}

bool capturing(hipStream_t s)
{
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    return hipStreamIsCapturing(s, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone;
}

// The library's workspace of `dev` with at least `need` bytes (lock held).  A
// workspace that is too small is retired, not freed: launches already queued
// may still read it; lamp_reserve and lamp_shutdown free retired ones after
// waiting for the device.  Growth is refused while `s` is being captured.
int library_ws_locked(int dev, size_t need, hipStream_t s, void **base)
{
    DeviceState *st = state_of(dev);
    if (need > st->ws_bytes) {
        if (capturing(s))
            return fail(LAMP_ERR_WORKSPACE, "the library workspace holds %zu bytes, the call needs %zu, and the stream "
                        "is being captured (reserve it with lamp_reserve or pass a workspace)", st->ws_bytes, need);
        size_t grow = st->ws_bytes + st->ws_bytes / 2;
        size_t bytes = align256(need > grow ? need : grow);
        void *p = nullptr;
        HIP_TRY(hipMalloc(&p, bytes));
        if (st->ws) st->retired.push_back(st->ws);
        st->ws = p;
        st->ws_bytes = bytes;
    }
    *base = st->ws;
    return LAMP_OK;
}

// The workspace of a call: the caller's (extra->workspace) or the library's.
int call_ws(int dev, const lamp_fwd_extra *extra, size_t need, hipStream_t s, void **base)
{
    if (extra && extra->workspace) {
        if ((reinterpret_cast<uintptr_t>(extra->workspace) & 255u) != 0)
            return fail(LAMP_ERR_INVALID_ARG, "workspace not aligned to 256 bytes");
        if (extra->workspace_bytes < need)
            return fail(LAMP_ERR_WORKSPACE, "workspace of %zu bytes, the call needs %zu", extra->workspace_bytes, need);
        *base = extra->workspace;
        return LAMP_OK;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    return library_ws_locked(dev, need, s, base);
}

// Free the retired workspaces of every device (lock held, after a device sync).
void free_retired_locked(DeviceState *st)
{
    for (void *p : st->retired) (void)hipFree(p);
    st->retired.clear();
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

// The sizes check_common accepts (d built, N and B*Hq*N within the limits):
// the workspace sizes of these cannot overflow.
bool sizes_built(int B, int Hq, int N, int d)
{
    return (d == 64 || d == 128 || d == 256) && N <= (1 << 20) && (size_t)B * Hq * (size_t)N <= (size_t)1 << 31;
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
    case LAMP_ERR_INIT: return "device tables not built";
    case LAMP_ERR_NONFINITE_INPUT: return "non-finite input";
    case LAMP_ERR_WORKSPACE: return "workspace too small";
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
        if (!st.ready && !st.ws && st.retired.empty()) continue;
        if (hipSetDevice((int)i) != hipSuccess) continue;
        (void)hipDeviceSynchronize();
        (void)hipFree(st.lut8);
        (void)hipFree(st.lut8e);
        (void)hipFree(st.exp16);
        (void)hipFree(st.exp16hl);
        (void)hipFree(st.sim8);
        (void)hipFree(st.sim16);
        (void)hipFree(st.ws);
        free_retired_locked(&st);
        st = DeviceState();
    }
    (void)hipSetDevice(prev);
}

static size_t fwd_ws_bytes(int B, int Hq, int Hkv, int N, int bq, int bk, int nk, int d)
{
    // the workspace holds whole query blocks and whole key tiles (zero padded)
    const int64_t T = (int64_t)bk * nk;
    const int64_t Nq = ((int64_t)N + bq - 1) / bq * bq, Nk = ((int64_t)N + T - 1) / T * T;
    return ws_layout(B, Hq, Hkv, Nq, Nk, d, true).total;
}

// The forward pass; sr: the 8-bit logits rounded stochastically with `seed`.
// fixed: the allocation-free entry point, whose workspace is the device's
// fixed scratch (the tables must already exist; nothing is allocated).
static int fwd_impl(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int N, int d,
                    int causal, int window, int bq, int bk, int nk, double delta, double tau, unsigned flags, bool sr,
                    uint64_t seed, float *o, float *lse, uint8_t *mask, const lamp_fwd_extra *extra, void *stream,
                    bool fixed = false)
{
    int rc = check_common(q, k, B, Hq, Hkv, N, d, causal, window);
    if (rc) return rc;
    if ((B > 0 && N > 0) && (!v || !o || !lse || !mask))
        return fail(LAMP_ERR_INVALID_ARG, "null pointer among v, o, lse, mask");
    if (!(delta >= 0.0) || std::isinf(delta)) return fail(LAMP_ERR_INVALID_ARG, "delta must be finite and >= 0");
    if (!(tau >= 0.0)) return fail(LAMP_ERR_INVALID_ARG, "tau must be >= 0 (or +inf)");
    if (flags & ~(unsigned)(LAMP_STAGE1_OFF | LAMP_MU_TRUNC | LAMP_SIM_PROFILE | LAMP_CHECK_FINITE | LAMP_COMPACT))
        return fail(LAMP_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
    if (bq <= 0 || bk <= 0 || nk <= 0) return fail(LAMP_ERR_INVALID_ARG, "block sizes must be positive");
    if (!lamp::fwd_supported(d, bq, bk, nk))
        return fail(LAMP_ERR_UNSUPPORTED, "block sizes (bq=%d, bk=%d, nk=%d) not built for d=%d", bq, bk, nk, d);
    if (sr && (flags & LAMP_SIM_PROFILE))
        return fail(LAMP_ERR_UNSUPPORTED, "stochastic rounding is built for the formats of Sec. 3.3, not the SIM profile");
    if ((flags & LAMP_SIM_PROFILE) && !(bk == 16 && nk == 4 && (d == 128 || d == 256)))
        return fail(LAMP_ERR_UNSUPPORTED, "the SIM profile is built for bk=16, nk=4, d in {128, 256} (bk=%d, nk=%d, d=%d)",
                    bk, nk, d);
    const bool dbg = extra && (extra->dbg_y8 || extra->dbg_y16);
    const int nqb_all = (N + bq - 1) / bq;
    if (dbg) {
        if (flags & LAMP_SIM_PROFILE)
            return fail(LAMP_ERR_UNSUPPORTED, "the logit observables are built for the formats of Sec. 3.3");
        if (extra->dbg_qb0 < 0 || extra->dbg_nqb <= 0 || extra->dbg_qb0 > nqb_all - extra->dbg_nqb)
            return fail(LAMP_ERR_INVALID_ARG, "observed query blocks [%d, %d + %d) outside [0, %d)", extra->dbg_qb0,
                        extra->dbg_qb0, extra->dbg_nqb, nqb_all);
    }
    if (B == 0 || N == 0) return LAMP_OK;   // nothing to compute
    const int Nq = nqb_all * bq, Nk = (N + bk * nk - 1) / (bk * nk) * (bk * nk);
    const bool check = (flags & LAMP_CHECK_FINITE) != 0u;
    flags &= ~(unsigned)LAMP_CHECK_FINITE;
    int dev = 0;
    rc = current_device(&dev);
    if (rc) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (check && capturing(s))
        return fail(LAMP_ERR_INVALID_ARG, "LAMP_CHECK_FINITE waits for the stream, which is being captured");
    lamp::FwdParams p{};
    void *ws_fixed = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        if (fixed && ((size_t)dev >= g_dev.size() || !g_dev[(size_t)dev].ready))
            return fail(LAMP_ERR_INIT, "device %d is not initialised (call lamp_init first)", dev);
        DeviceState *st = state_of(dev);
        if (fixed) {
            ws_fixed = st->scratch;
        } else {
            rc = init_locked(dev);
            if (rc) return rc;
        }
        p.exp16 = st->exp16;
        p.exp16hl = st->exp16hl;
        p.lut8e = st->lut8e;
        p.sim8 = st->sim8;
        p.sim16 = st->sim16;
    }
    const WsLayout lay = ws_layout(B, Hq, Hkv, Nq, Nk, d, true);
    void *base = nullptr;
    if (fixed) {
        if (lay.total > lamp::NOALLOC_SCRATCH_BYTES)
            return fail(LAMP_ERR_WORKSPACE, "the call needs %zu bytes of workspace, above the fixed scratch of %zu",
                        lay.total, lamp::NOALLOC_SCRATCH_BYTES);
        base = ws_fixed;
    } else {
        rc = call_ws(dev, extra, lay.total, s, &base);
        if (rc) return rc;
    }
    Workspace w{};
    carve(base, lay, &w);
    p.qt = w.qt;
    p.kt32 = w.kt32;
    p.vt = w.vt;
    p.o = o;
    p.lse = lse;
    p.mask = mask;
    p.stats = extra ? extra->stats : nullptr;
    if (dbg) {
        p.dbg_y8 = extra->dbg_y8;
        p.dbg_y16 = extra->dbg_y16;
        p.dbg_qb0 = extra->dbg_qb0;
        p.dbg_nqb = extra->dbg_nqb;
        const size_t n = (size_t)B * Hq * extra->dbg_nqb * bq * Nk;
        if (p.dbg_y8) HIP_TRY(hipMemsetAsync(p.dbg_y8, 0xFF, n, s));
        if (p.dbg_y16) HIP_TRY(hipMemsetAsync(p.dbg_y16, 0xFF, n * sizeof(uint16_t), s));
    }
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
    if (sr) p.flags &= ~(unsigned)LAMP_COMPACT;   // a schedule of the pipelined kernel only
    p.seed = seed;
    // the all-16-bit mode computes no 8-bit logit: the rounding mode does not matter there
    const bool use_sr = sr && p.mode != lamp::MODE_ALL16;
    bool timed = false;
    TimedCall tc{};
    if (!fixed) {   // the allocation-free entry point creates no events
        std::lock_guard<std::mutex> lk(g_tmu);
        timed = g_timing;
    }
    if (timed) {
        for (int i = 0; i < 3; ++i) HIP_TRY(hipEventCreate(&tc.e[i]));
        HIP_TRY(hipEventRecord(tc.e[0], s));
    }
    unsigned *bad = nullptr;
    if (check) {
        bad = w.flag;
        HIP_TRY(hipMemsetAsync(bad, 0, sizeof(unsigned), s));
    }
    HIP_TRY(lamp::launch_prepass(q, k, w.qt, w.kt32, B, Hq, Hkv, N, Nq, Nk, d, scale_of(d), s,
                                 lamp::fwd_grouped(d, bq, bk, nk), bad));
    HIP_TRY(lamp::launch_transpose_v(v, w.vt, B, Hkv, N, Nk, d, s, bad));
    if (check) {
        unsigned h_bad = 0;
        HIP_TRY(hipMemcpyAsync(&h_bad, bad, sizeof(unsigned), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
        if (h_bad) {
            if (timed)
                for (int i = 0; i < 3; ++i) (void)hipEventDestroy(tc.e[i]);
            return fail(LAMP_ERR_NONFINITE_INPUT, "a NaN or an infinity among the elements of%s%s%s",
                        (h_bad & 1u) ? " q" : "", (h_bad & 2u) ? " k" : "", (h_bad & 4u) ? " v" : "");
        }
    }
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
                  float *lse, uint8_t *mask, const lamp_fwd_extra *extra, void *stream)
{
    return fwd_impl(q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, delta, tau, flags, false, 0, o, lse, mask,
                    extra, stream);
}

int lamp_attn_fwd_noalloc(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int N,
                          int d, int causal, int window, int bq, int bk, int nk, double delta, double tau,
                          unsigned flags, float *o, float *lse, uint8_t *mask, const lamp_fwd_extra *extra,
                          void *stream)
{
    if (extra && extra->workspace)
        return fail(LAMP_ERR_INVALID_ARG, "lamp_attn_fwd_noalloc takes no workspace (it uses its fixed scratch)");
    if (flags & LAMP_CHECK_FINITE)
        return fail(LAMP_ERR_UNSUPPORTED, "LAMP_CHECK_FINITE reads a flag back to the host; use lamp_attn_fwd");
    return fwd_impl(q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, delta, tau, flags, false, 0, o, lse, mask,
                    extra, stream, true);
}

int lamp_attn_fwd_sr(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int N, int d,
                     int causal, int window, int bq, int bk, int nk, double delta, double tau, unsigned flags,
                     uint64_t seed, float *o, float *lse, uint8_t *mask, const lamp_fwd_extra *extra, void *stream)
{
    return fwd_impl(q, k, v, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, delta, tau, flags, true, seed, o, lse, mask,
                    extra, stream);
}

size_t lamp_attn_fwd_workspace_size(int B, int Hq, int Hkv, int N, int d, int bq, int bk, int nk)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || N < 0 || d <= 0 || bq <= 0 || bk <= 0 || nk <= 0) return 0;
    if (B == 0 || N == 0) return 0;
    if (!sizes_built(B, Hq, N, d) || !lamp::fwd_supported(d, bq, bk, nk)) return 0;
    return fwd_ws_bytes(B, Hq, Hkv, N, bq, bk, nk, d);
}

int lamp_reserve(int device, size_t bytes)
{
    std::lock_guard<std::mutex> lk(g_mu);
    int prev = 0;
    HIP_TRY(hipGetDevice(&prev));
    HIP_TRY(hipSetDevice(device));
    DeviceState *st = state_of(device);
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) {
        free_retired_locked(st);
        void *base = nullptr;
        int rc = library_ws_locked(device, align256(bytes), nullptr, &base);
        (void)hipSetDevice(prev);
        return rc;
    }
    (void)hipSetDevice(prev);
    return fail(LAMP_ERR_HIP, "lamp_reserve: %s", hipGetErrorString(e));
}

// Byte sizes of the decode workspace: 8-bit and 16-bit logit codes, per-tile
// factors and mu_hat, partial outputs of the P.V pieces, and per row the
// state carried between key chunks and each chunk's product of rescale
// factors.
struct DecLayout {
    size_t y8, y16, f, mu, part, mu_st, om_st, lam_c, total;
};

static DecLayout dec_layout(int B, int Hq, int M, int N, int d)
{
    const int64_t Np = ((int64_t)N + 63) / 64 * 64;
    const int64_t nch = ((int64_t)N + lamp::DEC_PV_KEYS - 1) / lamp::DEC_PV_KEYS;   // pieces of the P.V pass
    const size_t nrows = (size_t)B * Hq * M;
    DecLayout l;
    l.y8 = align256(nrows * Np);
    l.y16 = align256(nrows * Np * 2);
    l.f = align256(nrows * (Np / 64) * 8);
    l.mu = align256(nrows * (Np / 64) * 4);
    l.part = align256(nrows * nch * d * 4);
    l.mu_st = align256(nrows * 4);
    l.om_st = align256(nrows * 8);
    l.lam_c = align256(nrows * lamp::DEC_MAX_CHUNKS * 8);
    l.total = l.y8 + l.y16 + l.f + l.mu + l.part + l.mu_st + l.om_st + l.lam_c;
    return l;
}

// The decode form's key chunks: about DEC_CHUNKS chunks of a multiple of
// DEC_PV_KEYS keys (one when the keys from kb0 are at most 2048); the last
// ends at Np.
static constexpr int DEC_CHUNKS = 2;
static int64_t round_pv(int64_t x)
{
    return (x + lamp::DEC_PV_KEYS - 1) / lamp::DEC_PV_KEYS * lamp::DEC_PV_KEYS;
}
static void dec_chunks(int N, int kb0, int *ck, int *nchunks)
{
    const int64_t span = (int64_t)N - kb0;
    if (span <= 2048) {
        *ck = (int)round_pv(span);
        *nchunks = 1;
        return;
    }
    *ck = (int)round_pv((span + DEC_CHUNKS - 1) / DEC_CHUNKS);
    *nchunks = (int)((span + *ck - 1) / *ck);
}

size_t lamp_attn_decode_workspace_size(int B, int Hq, int Hkv, int M, int N, int d)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || M < 0 || M > N || d <= 0) return 0;
    if (B == 0 || M == 0) return 0;
    if (!sizes_built(B, Hq, N, d)) return 0;
    return dec_layout(B, Hq, M, N, d).total;
}

int lamp_attn_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B, int Hq, int Hkv, int M, int N,
                     int d, int causal, int window, int tk, double delta, double tau, unsigned flags, float *o,
                     float *lse, uint8_t *mask, const lamp_fwd_extra *extra, void *stream)
{
    if (M < 0 || M > N) return fail(LAMP_ERR_INVALID_ARG, "M=%d query rows must lie in [0, N=%d]", M, N);
    int rc = check_common(q, k, B, Hq, Hkv, N, d, causal, window, M);
    if (rc) return rc;
    if ((B > 0 && M > 0) && (!q || !k || !v || !o || !lse || !mask))
        return fail(LAMP_ERR_INVALID_ARG, "null pointer among q, k, v, o, lse, mask");
    if (!(delta >= 0.0) || std::isinf(delta)) return fail(LAMP_ERR_INVALID_ARG, "delta must be finite and >= 0");
    if (!(tau >= 0.0)) return fail(LAMP_ERR_INVALID_ARG, "tau must be >= 0 (or +inf)");
    if (flags & ~(unsigned)LAMP_DECODE_SERIAL)
        return fail(LAMP_ERR_INVALID_ARG, "unknown flags 0x%x (the decode form takes LAMP_DECODE_SERIAL)", flags);
    if (tk != 64) return fail(LAMP_ERR_UNSUPPORTED, "keys per update tk=%d not built (64)", tk);
    if (extra && (extra->stats || extra->dbg_y8 || extra->dbg_y16))
        return fail(LAMP_ERR_UNSUPPORTED, "the decode form takes a workspace only (no stats, no logit observables)");
    if (B == 0 || M == 0) return LAMP_OK;   // nothing to compute
    const int Np = (N + 63) / 64 * 64;
    const DecLayout lay = dec_layout(B, Hq, M, N, d);
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
        p.lut8e = st->lut8e;
        p.exp16hl = st->exp16hl;
    }
    void *wsb = nullptr;
    rc = call_ws(dev, extra, lay.total, s, &wsb);
    if (rc) return rc;
    {
        char *base = static_cast<char *>(wsb);
        p.y8 = reinterpret_cast<uint8_t *>(base);
        p.y16 = reinterpret_cast<uint16_t *>(base + lay.y8);
        p.f = reinterpret_cast<double *>(base + lay.y8 + lay.y16);
        p.mut = reinterpret_cast<float *>(base + lay.y8 + lay.y16 + lay.f);
        size_t off = lay.y8 + lay.y16 + lay.f + lay.mu;
        p.part = reinterpret_cast<float *>(base + off);
        off += lay.part;
        p.mu_st = reinterpret_cast<float *>(base + off);
        off += lay.mu_st;
        p.om_st = reinterpret_cast<double *>(base + off);
        off += lay.om_st;
        p.lam_c = reinterpret_cast<double *>(base + off);
    }
    p.q = q;
    p.qscale = scale_of(d);
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
    if (timed) HIP_TRY(hipEventRecord(tc.e[1], s));   // no prepass: the logits scale the queries
    auto chunk_of = [&](int c) {
        lamp::DecParams pc = p;
        pc.chunk = c;
        pc.ka = p.kb0 + c * p.ck;
        pc.kz = c == p.nchunks - 1 ? Np : pc.ka + p.ck;
        return pc;
    };
    if (flags & LAMP_DECODE_SERIAL) {
        // one key chunk, the passes one after another
        p.ck = (int)round_pv(N - p.kb0);
        p.nchunks = 1;
        const lamp::DecParams pc = chunk_of(0);
        HIP_TRY(lamp::launch_dec_logits(d, pc, s));
        HIP_TRY(lamp::launch_dec_decide(d, pc, s));
        HIP_TRY(lamp::launch_dec_pv(d, pc, s));
    } else if ((Hq / Hkv) * M <= lamp::DEC_STAGE_MAX_ROWS) {
        // the key chunks in a pipeline of stage launches on `s`: stage g
        // runs the logits of chunk g (bound by the VALU), the decisions of
        // chunk g - 1 (bound by latency; they take the chunks in order, each
        // continuing the row state of the one before) and P.V of chunk g - 2
        // (bound by HBM) side by side
        dec_chunks(N, p.kb0, &p.ck, &p.nchunks);
        for (int g = 0; g < p.nchunks + 2; ++g) {
            lamp::DecParams pl, pd, pp;
            const bool hl = g < p.nchunks, hd = g >= 1 && g - 1 < p.nchunks, hp = g >= 2;
            if (hl) pl = chunk_of(g);
            if (hd) pd = chunk_of(g - 1);
            if (hp) pp = chunk_of(g - 2);
            HIP_TRY(lamp::launch_dec_stage(d, hd ? &pd : nullptr, hl ? &pl : nullptr, hp ? &pp : nullptr, s));
        }
    } else {
        // more query rows per key/value head than a stage holds: the chunks
        // one after another
        dec_chunks(N, p.kb0, &p.ck, &p.nchunks);
        for (int c = 0; c < p.nchunks; ++c) {
            const lamp::DecParams pc = chunk_of(c);
            HIP_TRY(lamp::launch_dec_logits(d, pc, s));
            HIP_TRY(lamp::launch_dec_decide(d, pc, s));
            HIP_TRY(lamp::launch_dec_pv(d, pc, s));
        }
    }
    HIP_TRY(lamp::launch_dec_reduce(d, p, s));
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

int lamp_phase_read(uint64_t *cycles, int reset)
{
    if (!cycles) return fail(LAMP_ERR_INVALID_ARG, "null pointer");
    unsigned long long h[lamp::PHASE_N + 1];
    const hipError_t e = lamp::phase_read(h, reset != 0);
    if (e == hipErrorNotSupported)
        return fail(LAMP_ERR_UNSUPPORTED, "this library was built without the phase timer (LAMP_PHASE_TIMER)");
    if (e != hipSuccess) return fail(LAMP_ERR_HIP, "lamp_phase_read: %s", hipGetErrorString(e));
    for (int i = 0; i <= lamp::PHASE_N; ++i) cycles[i] = h[i];
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
                         int window, int row0, int nrows, void *out, lamp::LogitsParams *p, Workspace *w,
                         void *stream)
{
    int rc = check_common(q, k, B, Hq, Hkv, N, d, causal, window);
    if (rc) return rc;
    if (!out) return fail(LAMP_ERR_INVALID_ARG, "null output pointer");
    if (B == 0 || N == 0 || N % 16) return fail(LAMP_ERR_UNSUPPORTED, "N=%d is not a positive multiple of 16 (B=%d)", N, B);
    if (row0 < 0 || nrows <= 0 || nrows > N - row0) return fail(LAMP_ERR_INVALID_ARG, "row range outside [0, N)");
    int dev = 0;
    rc = current_device(&dev);
    if (rc) return rc;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        rc = init_locked(dev);
        if (rc) return rc;
        const WsLayout lay = ws_layout(B, Hq, Hkv, N, N, d, false);
        void *base = nullptr;
        rc = library_ws_locked(dev, lay.total, static_cast<hipStream_t>(stream), &base);
        if (rc) return rc;
        carve(base, lay, w);
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
    int rc = logits_common(q, k, B, Hq, Hkv, N, d, causal, window, row0, nrows, y8, &p, &w, stream);
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
    int rc = logits_common(q, k, B, Hq, Hkv, N, d, causal, window, row0, nrows, y8, &p, &w, stream);
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
    int rc = logits_common(q, k, B, Hq, Hkv, N, d, causal, window, row0, nrows, y16, &p, &w, stream);
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
    if (high != 0 && high != 1) return fail(LAMP_ERR_INVALID_ARG, "high must be 0 or 1");
    lamp::LogitsParams p;
    Workspace w;
    int rc = logits_common(q, k, B, Hq, Hkv, N, d, causal, window, row0, nrows, y, &p, &w, stream);
    if (rc) return rc;
    p.ysim = y;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(lamp::launch_prepass(q, k, w.qt, w.kt32, B, Hq, Hkv, N, N, N, d, scale_of(d), s));
    HIP_TRY(lamp::launch_logits_sim(p, d, high, s));
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
