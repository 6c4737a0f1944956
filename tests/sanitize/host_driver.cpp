// A driver for the host side of liblamp under AddressSanitizer and
// UndefinedBehaviourSanitizer (test infrastructure; built host-only and run
// by tests/test_sanitize.py, on a machine with or without a GPU: every call
// here either fails its argument checks before touching a device or fails
// cleanly in the HIP runtime when there is none).  Any sanitizer report
// aborts; a return code that differs from the expected one is counted and
// makes the exit status 1.
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>

#include "lamp.h"

static int failures = 0;

static void expect(int rc, int want, const char *what)
{
    if (rc != want) {
        std::fprintf(stderr, "%s: got %d (%s), want %d\n", what, rc, lamp_last_error(), want);
        ++failures;
    }
    // the message buffer is a C string whatever happened
    (void)std::strlen(lamp_last_error());
}

static void expect_any_error(int rc, const char *what)
{
    if (rc == LAMP_OK) {
        std::fprintf(stderr, "%s: succeeded without a device\n", what);
        ++failures;
    }
    (void)std::strlen(lamp_last_error());
}

int main()
{
    uint16_t buf16[64] = {0};
    float buf32[64] = {0};
    uint8_t buf8[64] = {0};
    const uint16_t *q = buf16, *k = buf16, *v = buf16;
    float *o = buf32, *lse = buf32;
    uint8_t *mask = buf8;
    const double inf = std::numeric_limits<double>::infinity(), nan = std::nan("");
    const int E = LAMP_ERR_INVALID_ARG, U = LAMP_ERR_UNSUPPORTED;

    for (int s = -2; s < 10; ++s) (void)std::strlen(lamp_status_str(s));
    (void)std::strlen(lamp_status_str(INT_MIN));
    (void)std::strlen(lamp_status_str(INT_MAX));

    // sizes, flags and thresholds the forward pass refuses
    struct Case { int B, Hq, Hkv, N, d, causal, window, bq, bk, nk; double delta, tau; unsigned flags; int want; };
    const Case cases[] = {
        {1, 3, 2, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {-1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 0, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 0, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, -5, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, 256, 0, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, 256, 96, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, U},
        {1, 2, 1, 256, 128, 2, 0, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, 256, 128, 1, -1, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, 256, 128, 0, 16, 128, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 128, 16, 4, -1.0, 0.5, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 128, 16, 4, inf, 0.5, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 128, 16, 4, nan, 0.5, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, -1.0, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, nan, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 32, E},
        {1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0x80000000u, E},
        {1, 2, 1, 256, 128, 1, 0, 0, 16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 128, -16, 4, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 128, 16, 0, 0x1p-8, 0.5, 0, E},
        {1, 2, 1, 256, 128, 1, 0, 32, 16, 4, 0x1p-8, 0.5, 0, U},
        {1, 2, 1, 256, 128, 1, 0, INT_MAX, INT_MAX, INT_MAX, 0x1p-8, 0.5, 0, U},
        {1, 2, 1, 256, 128, 1, 0, 128, 64, 4, 0x1p-8, 0.5, 4, U},
        {1, 2, 1, 256, 64, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 4, U},
        {1, 1, 1, (1 << 20) + 1, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, U},
        {1, 1, 1, INT_MAX, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, U},
        {4096, 1024, 1, 1 << 20, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, U},
        {INT_MAX, INT_MAX, 1, 1 << 20, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, U},
    };
    for (const Case &c : cases) {
        char what[160];
        std::snprintf(what, sizeof what, "fwd B=%d Hq=%d Hkv=%d N=%d d=%d causal=%d window=%d bq=%d bk=%d nk=%d flags=%u",
                      c.B, c.Hq, c.Hkv, c.N, c.d, c.causal, c.window, c.bq, c.bk, c.nk, c.flags);
        expect(lamp_attn_fwd(q, k, v, c.B, c.Hq, c.Hkv, c.N, c.d, c.causal, c.window, c.bq, c.bk, c.nk, c.delta,
                             c.tau, c.flags, o, lse, mask, nullptr, nullptr), c.want, what);
        expect(lamp_attn_fwd_noalloc(q, k, v, c.B, c.Hq, c.Hkv, c.N, c.d, c.causal, c.window, c.bq, c.bk, c.nk,
                                     c.delta, c.tau, c.flags, o, lse, mask, nullptr, nullptr), c.want, what);
        if (!(c.flags & LAMP_SIM_PROFILE))
            expect(lamp_attn_fwd_sr(q, k, v, c.B, c.Hq, c.Hkv, c.N, c.d, c.causal, c.window, c.bq, c.bk, c.nk,
                                    c.delta, c.tau, c.flags, ~0ull, o, lse, mask, nullptr, nullptr), c.want, what);
        (void)lamp_attn_fwd_workspace_size(c.B, c.Hq, c.Hkv, c.N, c.d, c.bq, c.bk, c.nk);
    }
    // null pointers
    expect(lamp_attn_fwd(nullptr, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, o, lse, mask, nullptr,
                         nullptr), E, "fwd null q");
    expect(lamp_attn_fwd(q, k, nullptr, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, o, lse, mask, nullptr,
                         nullptr), E, "fwd null v");
    expect(lamp_attn_fwd(q, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, o, lse, nullptr, nullptr,
                         nullptr), E, "fwd null mask");
    expect(lamp_attn_fwd_sr(q, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, LAMP_SIM_PROFILE, 1, o, lse,
                            mask, nullptr, nullptr), U, "fwd_sr SIM");

    // the optional arguments
    uint64_t stats[16];
    lamp_fwd_extra ex;
    std::memset(&ex, 0, sizeof ex);
    ex.dbg_y8 = buf8;
    ex.dbg_qb0 = 1;
    ex.dbg_nqb = 2;
    expect(lamp_attn_fwd(q, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, o, lse, mask, &ex, nullptr), E,
           "observed blocks outside");
    ex.dbg_qb0 = INT_MAX;
    ex.dbg_nqb = INT_MAX;
    expect(lamp_attn_fwd(q, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, o, lse, mask, &ex, nullptr), E,
           "observed blocks at INT_MAX");
    ex.dbg_qb0 = -1;
    ex.dbg_nqb = 1;
    expect(lamp_attn_fwd(q, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, o, lse, mask, &ex, nullptr), E,
           "observed blocks negative");
    ex.dbg_qb0 = 0;
    ex.dbg_nqb = 2;
    expect(lamp_attn_fwd(q, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, LAMP_SIM_PROFILE, o, lse, mask,
                         &ex, nullptr), U, "observables with SIM");
    lamp_fwd_extra ws;
    std::memset(&ws, 0, sizeof ws);
    ws.workspace = buf8;
    ws.workspace_bytes = 64;
    expect(lamp_attn_fwd_noalloc(q, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, 0, o, lse, mask, &ws,
                                 nullptr), E, "noalloc with a workspace");
    expect(lamp_attn_fwd_noalloc(q, k, v, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 0x1p-8, 0.5, LAMP_CHECK_FINITE, o, lse,
                                 mask, nullptr, nullptr), U, "noalloc with the finite check");
    lamp_fwd_extra st;
    std::memset(&st, 0, sizeof st);
    st.stats = stats;

    // the decode form: (B, Hq, Hkv, M, N, d, causal, window, tk)
    expect(lamp_attn_decode(q, k, v, 1, 4, 1, 1, 256, 128, 1, 0, 32, 0x1p-8, 0.5, 0, o, lse, mask, nullptr, nullptr),
           U, "decode tk");
    expect(lamp_attn_decode(q, k, v, 1, 4, 1, 1, 256, 128, 1, 0, 64, 0x1p-8, 0.5, 4, o, lse, mask, nullptr, nullptr),
           E, "decode flags");
    expect(lamp_attn_decode(q, k, v, 1, 4, 1, 300, 256, 128, 1, 0, 64, 0x1p-8, 0.5, 0, o, lse, mask, nullptr,
                            nullptr), E, "decode M > N");
    expect(lamp_attn_decode(q, k, v, 1, 4, 1, -1, 256, 128, 1, 0, 64, 0x1p-8, 0.5, 0, o, lse, mask, nullptr,
                            nullptr), E, "decode M < 0");
    expect(lamp_attn_decode(q, k, v, 1, 4, 1, 1, 256, 96, 1, 0, 64, 0x1p-8, 0.5, 0, o, lse, mask, nullptr, nullptr),
           U, "decode d");
    expect(lamp_attn_decode(q, k, v, 1, 4, 1, 1, 256, 128, 1, 0, 64, 0x1p-8, -1.0, 0, o, lse, mask, nullptr,
                            nullptr), E, "decode tau");
    expect(lamp_attn_decode(q, k, v, 1, 4, 1, 1, 256, 128, 1, 0, 64, 0x1p-8, 0.5, 0, o, lse, mask, &st, nullptr), U,
           "decode stats");
    expect(lamp_attn_decode(q, k, v, 1, 4, 1, 1, INT_MAX, 128, 1, 0, 64, 0x1p-8, 0.5, 0, o, lse, mask, nullptr,
                            nullptr), U, "decode N = INT_MAX");

    // the logit entry points
    expect(lamp_attn_logits8(q, k, 1, 2, 1, 250, 128, 1, 0, 0, 16, buf8, nullptr), U, "logits8 N % 16");
    expect(lamp_attn_logits8(q, k, 1, 2, 1, 256, 128, 1, 0, 250, 16, buf8, nullptr), E, "logits8 rows");
    expect(lamp_attn_logits8(q, k, 1, 2, 1, 256, 128, 1, 0, INT_MAX, INT_MAX, buf8, nullptr), E, "logits8 INT_MAX");
    expect(lamp_attn_logits8(q, k, 1, 2, 1, 256, 128, 1, 0, -1, 16, buf8, nullptr), E, "logits8 row0 < 0");
    expect(lamp_attn_logits8_sr(q, k, 1, 2, 1, 256, 96, 1, 0, 0, 16, 5, buf8, nullptr), U, "logits8_sr d");
    expect(lamp_attn_logits16(q, k, 1, 2, 1, 256, 128, 1, 0, 0, 16, nullptr, nullptr), E, "logits16 null");
    expect(lamp_attn_logits_sim(q, k, 1, 2, 1, 256, 128, 1, 0, 0, 16, 2, buf32, nullptr), E, "logits_sim high");

    // workspace sizes at the extremes (no arithmetic may overflow)
    const int ext[] = {INT_MIN, -1, 0, 1, 16, 128, 1 << 20, INT_MAX};
    for (int a : ext)
        for (int b : ext) {
            (void)lamp_attn_fwd_workspace_size(a, b, 1, b, 128, 128, 16, 4);
            (void)lamp_attn_fwd_workspace_size(1, 1, 1, a, b, a, b, a);
            (void)lamp_attn_fwd_workspace_size(a, a, a, b, 256, 1, 1, 1);
            (void)lamp_attn_decode_workspace_size(a, b, 1, 1, b, 128);
            (void)lamp_attn_decode_workspace_size(1, 1, 1, a, b, 256);
            (void)lamp_attn_decode_workspace_size(a, a, a, b, b, b);
        }

    // host-only bookkeeping and null outputs
    expect(lamp_issue_rates(nullptr, nullptr), E, "issue rates null");
    expect(lamp_timing_enable(1), LAMP_OK, "timing enable");
    expect(lamp_timing_enable(0), LAMP_OK, "timing disable");
    int launches = -1;
    double fwd_ms = -1, pre_ms = -1;
    expect(lamp_timing_read(&launches, &fwd_ms, &pre_ms), LAMP_OK, "timing read");
    expect(lamp_timing_read(nullptr, nullptr, nullptr), LAMP_OK, "timing read nulls");
    if (launches != 0 || fwd_ms != 0.0 || pre_ms != 0.0) {
        std::fprintf(stderr, "timing read without calls: %d %g %g\n", launches, fwd_ms, pre_ms);
        ++failures;
    }
    (void)lamp_phase_read(nullptr, 0);
    expect(lamp_selftest_e4m3(nullptr, nullptr, nullptr, 16, nullptr), E, "selftest e4m3 null");
    expect(lamp_selftest_exp_doc(nullptr, nullptr, 16, nullptr), E, "selftest exp null");

    // calls that pass every argument check: without a device they fail in
    // the HIP runtime; with one they may run (all pointers here are host
    // pointers, so nothing is launched: only the status is looked at)
    expect_any_error(lamp_init(-1), "init device -1");
    expect_any_error(lamp_init(INT_MAX), "init device INT_MAX");
    expect_any_error(lamp_reserve(-1, 1 << 20), "reserve device -1");
    expect_any_error(lamp_get_tables(-1, buf8, buf16), "tables device -1");
    lamp_shutdown();
    lamp_shutdown();

    if (failures) {
        std::fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    std::printf("host driver: all calls clean\n");
    return 0;
}
