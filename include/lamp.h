/*
 * lamp.h -- C ABI of liblamp.so, the MI355X (gfx950) LampAttention forward pass.
 *
 * LampAttention (look-ahead mixed-precision FlashAttention) computes every
 * QK^T logit with 8-bit (e4m3) accumulation, flags the numerically sensitive
 * (query block x key sub-block) sub-blocks in two stages -- a running-maximum
 * look-ahead with a safety margin, then a block-LAMP knapsack on an analytical
 * round-off bound -- recomputes only those in 16 bits (e4m11), and finishes
 * with the online-softmax rescale and the P.V accumulation.  Paper: Sec. 3.1
 * (block LAMP, Eqs. (7) and (8)), Sec. 3.2 (Algorithm 1), Sec. 3.3 (formats).
 *
 * Conventions shared by every entry point:
 *   - Pointers named q, k, v, o, lse, mask, y8, y16 are DEVICE pointers to
 *     memory the caller owns; the library never frees or retains them.
 *   - Tensors are dense row-major: q [B][Hq][N][d], k and v [B][Hkv][N][d]
 *     (bf16 bit patterns, uint16_t), o [B][Hq][N][d] fp32, lse [B][Hq][N]
 *     fp32, mask [B][Hq][ceil(N/bq)][ceil(N/(bk*nk))*nk] uint8.  Query head h reads kv head
 *     h / (Hq/Hkv) (grouped-query attention).
 *   - Visibility: key i is visible to query j unless causal and i > j, or
 *     window > 0 and i <= j - window (window requires causal).
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream).  Results are valid after the stream has been synchronised.
 *   - Every function returns a lamp_status; nothing aborts or throws across
 *     the ABI.  lamp_last_error() describes the last failure of the calling
 *     thread.
 *   - Inputs are assumed finite.  A non-finite q, k or v element gives
 *     unspecified results unless the call asks for the check
 *     (LAMP_CHECK_FINITE), which then returns LAMP_ERR_NONFINITE_INPUT.
 */
#ifndef LAMP_H
#define LAMP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    LAMP_OK = 0,
    LAMP_ERR_INVALID_ARG = 1,   /* null pointer, negative size, bad parameter */
    LAMP_ERR_UNSUPPORTED = 2,   /* valid but not built: shape or block sizes */
    LAMP_ERR_HIP = 3,           /* a HIP runtime call failed */
    LAMP_ERR_INIT = 4,          /* device tables could not be built (or, for
                                   lamp_attn_fwd_noalloc, were not built yet) */
    LAMP_ERR_NONFINITE_INPUT = 5,  /* LAMP_CHECK_FINITE found a NaN or an infinity in q, k or v */
    LAMP_ERR_WORKSPACE = 6      /* the workspace is too small and may not grow now */
} lamp_status;

/* Optional arguments of the forward entry points (defined below). */
struct lamp_fwd_extra;

/* Mask codes, one byte per (query block, key sub-block). */
enum {
    LAMP_MASK_LOW = 0,      /* kept in 8 bits */
    LAMP_MASK_STAGE1 = 1,   /* recomputed in 16 bits by the running-max test, Eq. (7) */
    LAMP_MASK_STAGE2 = 2,   /* recomputed in 16 bits by the block-LAMP knapsack, Eq. (8) */
    LAMP_MASK_INACTIVE = 3  /* no visible (query, key) pair: never computed */
};

/*
 * lamp_attn_fwd -- the LampAttention forward pass (Algorithm 1).
 *
 * Inputs q, k, v: bf16, layouts above.  bq = queries per block (b_q), bk =
 * keys per sub-block (b_k), nk = sub-blocks per key tile (N_k); the paper's
 * tiles hold bq queries x bk*nk keys.  delta >= 0: safety margin of Eq. (7).
 * tau >= 0: threshold of Eq. (8); tau = +INFINITY is the pure 8-bit path (no
 * recomputation, the paper's 8-bit baseline) and tau = 0 recomputes every
 * active sub-block (16-bit FlashAttention in the paper's formats).
 * flags: 0, or LAMP_STAGE1_OFF and/or LAMP_MU_TRUNC (below), which apply for
 * 0 < tau < +INFINITY (the two end modes ignore them), and/or
 * LAMP_SIM_PROFILE, which applies in every mode; other bits are
 * LAMP_ERR_INVALID_ARG.
 *
 * Outputs: o (normalised attention output), lse (mu + ln omega per query row,
 * natural log), mask (codes above).  Every mask byte of the rows is written.
 *
 * Built configurations (LAMP_ERR_UNSUPPORTED otherwise): d in {64, 128, 256};
 * bq in {64, 128}; (bk, nk) in {(16, 4), (64, 4)}; N <= 2^20; with
 * LAMP_SIM_PROFILE only (bk, nk) = (16, 4) and d in {128, 256}, the tiling of
 * the paper's simulation (Sec. 4.1: 128 queries x 64 keys in 4 sub-blocks).  N need not be a
 * multiple of the block sizes: keys at or beyond N are invisible and the last
 * query block is partial (its missing rows take part in no test).  The mask
 * then holds ceil(N/bq) query blocks of ceil(N/(bk*nk))*nk sub-blocks, codes
 * of sub-blocks beyond N being 3.  B = 0 or N = 0 returns LAMP_OK and writes
 * nothing.
 *
 * extra: NULL, or the optional outputs and the workspace (lamp_fwd_extra
 * below).
 *
 * Workspace.  A call needs lamp_attn_fwd_workspace_size(...) bytes of device
 * memory for the prepass (the pre-scaled Q and K in fp32, V transposed) and a
 * check flag.  With extra->workspace set, the call uses that memory and
 * allocates nothing; calls on distinct workspaces may overlap.  Otherwise it
 * uses the library's per-device workspace: when that is too small the call
 * allocates a larger one (never while `stream` is being captured into a graph:
 * then LAMP_ERR_WORKSPACE) and keeps the old one until lamp_reserve or
 * lamp_shutdown, so launches still in flight never see memory freed;
 * lamp_reserve sizes it ahead of time.  Calls that overlap on one device
 * without their own workspace race on the library's.
 *
 * The first call on a device builds the library's exponential tables (or
 * lamp_init, ahead of time).
 */
int lamp_attn_fwd(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                  int B, int Hq, int Hkv, int N, int d,
                  int causal, int window, int bq, int bk, int nk,
                  double delta, double tau, unsigned flags,
                  float *o, float *lse, uint8_t *mask,
                  const struct lamp_fwd_extra *extra, void *stream);

/*
 * Optional arguments of the forward entry points (lamp_attn_fwd,
 * lamp_attn_fwd_sr, lamp_attn_fwd_noalloc; lamp_attn_decode takes only the
 * workspace).  A zero-initialised struct asks for nothing.
 *
 * stats: DEVICE pointer to LAMP_STATS_WORDS(nk) uint64_t counters that the
 *   call ADDS to (the caller zeroes them); word meanings below.
 * dbg_y8, dbg_y16, dbg_qb0, dbg_nqb: observables of the forward kernel for
 *   the query blocks [dbg_qb0, dbg_qb0 + dbg_nqb) of every (b, h), for tests.
 *   With Nt = ceil(N/(bk*nk))*bk*nk keys and rows r = (qb - dbg_qb0)*bq + i:
 *   dbg_y8 (DEVICE, uint8 [B][Hq][dbg_nqb*bq][Nt]) receives the e4m3 code of
 *   every visible pair's 8-bit logit as the forward kernel computed it (Alg. 1,
 *   low-precision accumulation), 0xFF elsewhere and everywhere at tau = 0;
 *   dbg_y16 (DEVICE, uint16 [B][Hq][dbg_nqb*bq][Nt]) receives the e4m11 code
 *   of every visible pair's 16-bit logit in the sub-blocks recomputed in 16
 *   bits (mask codes 1 and 2), 0xFFFF elsewhere.  Either pointer may be NULL.
 *   Rows at or beyond N hold 0xFF / 0xFFFF.  Not with LAMP_SIM_PROFILE
 *   (LAMP_ERR_UNSUPPORTED).  The arrays are filled with hipMemsetAsync on
 *   `stream` first.
 * workspace, workspace_bytes: DEVICE memory for the prepass (above), aligned
 *   to 256 bytes, at least the size the workspace-size call gives; the
 *   library writes it and does not retain it after the stream has passed the
 *   call.
 */
typedef struct lamp_fwd_extra {
    uint64_t *stats;
    uint8_t *dbg_y8;
    uint16_t *dbg_y16;
    int dbg_qb0;
    int dbg_nqb;
    void *workspace;
    size_t workspace_bytes;
} lamp_fwd_extra;

/*
 * Statistics words (lamp_fwd_extra.stats), summed over every query block of
 * the call.  Words 0-5 and the histogram follow from the definition of the
 * method (the CPU reference counts them the same way); words 6 and 7 describe
 * the forward kernel's speculative schedule.
 *   LAMP_STAT_TILES     (query block, key tile) pairs with an active sub-block
 *   LAMP_STAT_STAGE1    sub-blocks recomputed by the first stage (mask code 1;
 *                       every active sub-block at tau = 0)
 *   LAMP_STAT_STAGE2    sub-blocks recomputed by the second stage (code 2)
 *   LAMP_STAT_INACTIVE  sub-blocks without a visible pair (code 3)
 *   LAMP_STAT_SAT8      visible 8-bit logits whose accumulation was clamped to
 *                       +-448 in some step (Sec. 3.3 assumes QK-Norm so that
 *                       this never happens): round-to-nearest gave a value
 *                       beyond 448, or, with stochastic rounding, |t| > 448;
 *                       0 in the SIM profile, which does not saturate
 *   LAMP_STAT_SAT16     16-bit logits of recomputed sub-blocks (visible pairs)
 *                       whose rounding to e4m11 was clamped to +-511.875; 0
 *                       in the SIM profile
 *   LAMP_STAT_SPEC_UNUSED  sub-blocks whose 16-bit logits the kernel computed
 *                       speculatively but did not use
 *   LAMP_STAT_LATE16    sub-blocks recomputed in 16 bits outside the
 *                       speculative batch (one at a time or after stage 2)
 *   LAMP_STAT_HIST + c  key tiles (with an active sub-block) in which c of the
 *                       nk sub-blocks were recomputed in 16 bits, c = 0..nk
 */
enum {
    LAMP_STAT_TILES = 0,
    LAMP_STAT_STAGE1 = 1,
    LAMP_STAT_STAGE2 = 2,
    LAMP_STAT_INACTIVE = 3,
    LAMP_STAT_SAT8 = 4,
    LAMP_STAT_SAT16 = 5,
    LAMP_STAT_SPEC_UNUSED = 6,
    LAMP_STAT_LATE16 = 7,
    LAMP_STAT_HIST = 8
};
#define LAMP_STATS_WORDS(nk) (LAMP_STAT_HIST + (nk) + 1)

/* Bytes of workspace lamp_attn_fwd / lamp_attn_fwd_sr need for these sizes
 * (0 for sizes or block sizes they refuse; B = 0 or N = 0 needs none). */
size_t lamp_attn_fwd_workspace_size(int B, int Hq, int Hkv, int N, int d, int bq, int bk, int nk);

/* Bytes of workspace lamp_attn_decode needs (0 for sizes it refuses). */
size_t lamp_attn_decode_workspace_size(int B, int Hq, int Hkv, int M, int N, int d);

/*
 * lamp_reserve -- grow the library's own workspace of `device` to at least
 * `bytes` now, so that later calls without a workspace of their own never
 * allocate.  Synchronous: waits for the device, then frees the workspaces
 * earlier growth retired.  The workspace never shrinks.
 */
int lamp_reserve(int device, size_t bytes);

/*
 * lamp_attn_fwd_noalloc -- lamp_attn_fwd for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, outputs and results as
 * lamp_attn_fwd; it calls no hipMalloc, hipFree or other allocating routine.
 *
 * Its workspace is a fixed scratch of 256 MiB (LAMP_NOALLOC_SCRATCH_BYTES)
 * that the library holds on every device it runs on from load until the
 * process ends; its device address is taken once per device by lamp_init,
 * which must have been called for the current device (LAMP_ERR_INIT
 * otherwise).  A call whose workspace (lamp_attn_fwd_workspace_size) exceeds
 * the scratch returns LAMP_ERR_WORKSPACE: e.g. the Qwen3-8B-shaped 8K prefill
 * (176 MiB) fits, four such sequences do not.  extra->workspace must be NULL
 * (LAMP_ERR_INVALID_ARG) and LAMP_CHECK_FINITE is refused
 * (LAMP_ERR_UNSUPPORTED); statistics and observables are allowed; kernel
 * timing (lamp_timing_enable) does not record these calls.  Every call on a
 * device shares that device's scratch, which keeps the last call's contents:
 * calls that overlap on one device (other streams, other threads) race.
 */
#define LAMP_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
int lamp_attn_fwd_noalloc(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                          int B, int Hq, int Hkv, int N, int d,
                          int causal, int window, int bq, int bk, int nk,
                          double delta, double tau, unsigned flags,
                          float *o, float *lse, uint8_t *mask,
                          const struct lamp_fwd_extra *extra, void *stream);

/* Variants of Algorithm 1 (flags of lamp_attn_fwd). */
enum {
    /* The first stage disabled (the paper's appendix on first-stage
     * recomputation): mu_hat is the running maximum of the 8-bit logits and
     * the second stage alone chooses the 16-bit sub-blocks. */
    LAMP_STAGE1_OFF = 1,
    /* The 8-bit shifts use mu_hat truncated (toward zero) to e4m3, saturating
     * at 448 (Sec. 3.3: the running maxima may be rounded to e4m3 for the
     * low-precision shifts by dropping the low mantissa bits); with
     * LAMP_SIM_PROFILE, truncated to 3 mantissa bits, without saturation. */
    LAMP_MU_TRUNC = 2,
    /* The "SIM" precision profile (Sec. 4.1, the numerics of the paper's own
     * simulation) in place of the formats of Sec. 3.3: the 8-bit and 16-bit
     * numbers are FP32 values with 3 and 11 stored mantissa bits, FP32's
     * exponent range and gradual underflow, round-to-nearest-even, no
     * saturation (an overflow gives an infinity, as in FP32).  The 8-bit
     * logits round to 3 bits after every FP32 FMA; the 16-bit logits are the
     * FP32 FMA chain rounded once to 11 bits; each shift is the exact
     * difference max(0, mu_hat - y) rounded once to 3 or 11 bits; each
     * exponential is exp(-shift) correctly rounded to 3 or 11 bits; the row
     * sum of a tile's exponentials is the fp64 sum over keys in ascending
     * order.  Logits are assumed finite. */
    LAMP_SIM_PROFILE = 4,
    /* Check q, k and v for NaN and infinity in the prepass (which reads every
     * element anyway) and return LAMP_ERR_NONFINITE_INPUT without running the
     * forward kernel if one is found.  The call then waits for its prepass on
     * `stream` (it is synchronous), and refuses a stream being captured into a
     * graph (LAMP_ERR_INVALID_ARG).  Applies in every mode. */
    LAMP_CHECK_FINITE = 8,
    /* The compact register layout of Sec. 3.3 ("Register layout") as the
     * kernel's schedule: 8-bit accumulators four per 32-bit register, room
     * for one 16-bit sub-block in the fused 8-bit pass, and a sequential
     * 16-bit pass for "disruptive" tiles where two or more sub-blocks are
     * flagged.  Results are bit-identical to the default (safe) layout.
     * Applies to the pipelined kernel (b_k = 16, N_k = 4, d >= 128) at
     * b_q = 128 in the threshold mode with the formats of Sec. 3.3; the flag
     * has no effect elsewhere. */
    LAMP_COMPACT = 16
};

/*
 * lamp_attn_fwd_sr -- lamp_attn_fwd with the 8-bit accumulation rounded
 * stochastically instead of to nearest (Sec. 3.3, "Floating-point formats":
 * stochastic rounding as the remedy for the swamping of e4m3 accumulation).
 *
 * Each FP32 FMA result t of the 8-bit recursion goes to one of its two e4m3
 * neighbours: with a = min(|t|, 448), lo the e4m3 number next to a toward
 * zero and u its spacing, to lo + u when floor(2^20 (a - lo) / u) + r >= 2^20,
 * else to lo, with the sign of t.  r is a 20-bit field of the output of
 * Philox4x64-10 (Salmon et al., SC 2011) under key (seed, 0) at counter
 * (j, i, b*Hq + h, c / 12) -- query row j, key i, query head h of batch b,
 * channel c: with m = c mod 12, bits [20 (m mod 3), 20 (m mod 3) + 20) of
 * output word m / 3.  The numbers depend on the logit and the channel alone, so the
 * result does not depend on the block sizes, and the 8-bit logits are those
 * of lamp_attn_logits8_sr with the same seed.  Everything else is as in
 * lamp_attn_fwd (the 16-bit logits keep round-to-nearest; tau = 0 computes
 * no 8-bit logit and equals lamp_attn_fwd).
 *
 * Arguments, layouts, outputs, extra and workspace as lamp_attn_fwd; flags: 0,
 * LAMP_STAGE1_OFF, LAMP_MU_TRUNC and/or LAMP_CHECK_FINITE (LAMP_COMPACT is
 * accepted and has no effect here); LAMP_SIM_PROFILE gives
 * LAMP_ERR_UNSUPPORTED.  Built for the configurations lamp_attn_fwd lists for
 * the formats of Sec. 3.3.  The generator costs some hundred VALU operations
 * per 8 multiply-adds: expect this pass to run far slower than
 * lamp_attn_fwd.
 */
int lamp_attn_fwd_sr(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                     int B, int Hq, int Hkv, int N, int d,
                     int causal, int window, int bq, int bk, int nk,
                     double delta, double tau, unsigned flags, uint64_t seed,
                     float *o, float *lse, uint8_t *mask,
                     const struct lamp_fwd_extra *extra, void *stream);

/*
 * lamp_attn_decode -- LampAttention for query rows against a key/value cache
 * in the vector form of the look-ahead (Sec. 2: the two-step procedure and the
 * greedy knapsack of Eq. (6)), e.g. one new token per sequence (decode).
 *
 * q [B][Hq][M][d]: M query rows per (b, h) at positions N-M .. N-1; k, v
 * [B][Hkv][N][d]: the cache (bf16, 16-byte aligned).  Each row visits its key
 * tiles of tk keys in order; in each tile the maximizer c of the 8-bit logits
 * passes if mu > fma(|mu|, delta, fl(y_c)) (mu_hat = mu), otherwise y_c is
 * recomputed in 16 bits and mu_hat = max(mu, y16_c); the other 8-bit logits
 * are sorted by E (omega_hat - E) ascending (ties by key) and kept while the
 * fp64 running sum stays within (tau omega_hat) omega_hat, the rest being
 * recomputed in 16 bits against the same mu_hat.  tau = +INFINITY keeps every
 * logit in 8 bits, tau = 0 recomputes them all.
 *
 * Outputs: o [B][Hq][M][d] fp32, lse [B][Hq][M] fp32, mask
 * [B][Hq][M][ceil(N/tk)*tk] uint8, one code per key (0 8-bit, 1 the maximizer
 * recomputed by the look-ahead test -- every key at tau = 0 --, 2 recomputed
 * by the knapsack, 3 invisible).  Built: tk = 64, d in {64, 128, 256};
 * flags: 0 or LAMP_DECODE_SERIAL.  By default the keys from the first one
 * any row sees are taken in 2 chunks of a multiple of 512 keys (one when
 * there are at most 2048): the decisions visit the chunks in order,
 * carrying each row's running maximum and sum, and with at most 8 query rows
 * per key/value head the logits of chunk c + 1, the decisions of chunk c and
 * P.V of chunk c - 1 run side by side in one launch.  B = 0 or M = 0 returns
 * LAMP_OK and writes nothing.  The
 * workspace (the 8-bit and 16-bit logit codes, per-tile mu_hat and rescale
 * factors, partial outputs, the row state between key chunks:
 * lamp_attn_decode_workspace_size bytes) comes from extra->workspace or from
 * the library's per-device workspace, as for lamp_attn_fwd; extra->stats and
 * the dbg pointers must be NULL (LAMP_ERR_UNSUPPORTED).
 */
/* Flags of lamp_attn_decode. */
enum {
    /* One key chunk and the three passes (logits, decisions, P.V) one after
     * another, instead of the default pipeline of key chunks (below); the
     * same masks and lse, O equal up to the order of its final sums. */
    LAMP_DECODE_SERIAL = 256
};

int lamp_attn_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                     int B, int Hq, int Hkv, int M, int N, int d,
                     int causal, int window, int tk, double delta, double tau, unsigned flags,
                     float *o, float *lse, uint8_t *mask,
                     const struct lamp_fwd_extra *extra, void *stream);

/*
 * lamp_attn_logits8 -- the 8-bit logits alone (Alg. 1, first accumulation;
 * Sec. 4.1 recursive FMA summation rounded to e4m3 after every step).
 * Writes the e4m3 codes of rows [row0, row0 + nrows) of every (b, h):
 * y8 [B][Hq][nrows][N]; invisible entries hold 0xFF.  d in {64, 128, 256},
 * N a multiple of 16, 0 <= row0, row0 + nrows <= N.
 */
int lamp_attn_logits8(const uint16_t *q, const uint16_t *k,
                      int B, int Hq, int Hkv, int N, int d, int causal, int window,
                      int row0, int nrows, uint8_t *y8, void *stream);

/*
 * lamp_attn_logits8_sr -- lamp_attn_logits8 with the stochastic rounding of
 * lamp_attn_fwd_sr (same seed, same numbers).  Same arguments and layout.
 */
int lamp_attn_logits8_sr(const uint16_t *q, const uint16_t *k,
                         int B, int Hq, int Hkv, int N, int d, int causal, int window,
                         int row0, int nrows, uint64_t seed, uint8_t *y8, void *stream);

/*
 * lamp_attn_logits16 -- the 16-bit logits of the recompute steps (Alg. 1):
 * the dot product of the pre-scaled query and the key accumulated by FP32
 * FMAs in ascending channel order, rounded once to e4m11 (saturating).  Codes
 * [B][Hq][nrows][N] uint16; invisible entries hold 0xFFFF.
 */
int lamp_attn_logits16(const uint16_t *q, const uint16_t *k,
                       int B, int Hq, int Hkv, int N, int d, int causal, int window,
                       int row0, int nrows, uint16_t *y16, void *stream);

/*
 * lamp_attn_logits_sim -- the logits of the SIM profile (LAMP_SIM_PROFILE):
 * high = 0 the 8-bit recursion (FP32 FMA, then 3 mantissa bits, every step),
 * high = 1 the 16-bit one (FP32 FMA chain, then 11 mantissa bits once); any
 * other value is LAMP_ERR_INVALID_ARG.
 * Values y [B][Hq][nrows][N] fp32 (device); invisible entries hold a NaN.
 * d in {64, 128, 256}, N a multiple of 16, 0 <= row0, row0 + nrows <= N.
 */
int lamp_attn_logits_sim(const uint16_t *q, const uint16_t *k,
                         int B, int Hq, int Hkv, int N, int d, int causal, int window,
                         int row0, int nrows, int high, float *y, void *stream);

/*
 * Kernel timing, for measurement.  While enabled (lamp_timing_enable(1)),
 * each lamp_attn_fwd call records three HIP events on its own stream: before
 * the prepass (query scaling, key conversion), between it and the forward
 * kernel, and after the forward kernel.  lamp_timing_read waits for the
 * events of every call recorded since the previous read, stores the number
 * of calls and the summed durations (milliseconds) of the forward kernel and
 * of the prepass (any output pointer may be NULL), destroys the events and
 * forgets the calls.  Calls made while disabled record nothing.
 */
int lamp_timing_enable(int on);
int lamp_timing_read(int *launches, double *fwd_ms, double *prepass_ms);

/*
 * Issue rates of the VALU instructions the logit loops are made of, measured
 * on the current device, for the benchmark's instruction-mix floor of the
 * forward kernel (which is bound by VALU issue).  ns_per_simd (HOST memory,
 * 6 entries) receives the nanoseconds one SIMD spends per wave-instruction
 * of: [0] an fp32 FMA on VGPR operands, [1] an fp32 FMA reading its first
 * operand through a DPP row broadcast, [2] a packed e4m3 -> fp32 decode,
 * [3] a packed fp32 -> e4m3 rounding, [4] per emulated step of the 8-bit
 * loop (decode, two broadcast FMAs, rounding: two multiply-adds per lane),
 * and [5] per emulated step of the SIM profile's 8-bit loop (a broadcast FMA
 * and the 3-instruction rounding of the FP32 pattern: one multiply-add).
 * Each kind runs 16 independent chains per lane at 8 waves per SIMD.  The
 * call allocates a small device buffer, runs on `stream` and waits for it;
 * it takes a few milliseconds.
 */
int lamp_issue_rates(double *ns_per_simd, void *stream);

/*
 * lamp_phase_read -- the phase timer of the pipelined forward kernel, in a
 * library built for measurement with -DLAMP_PHASE_TIMER (liblamp_phase.so;
 * LAMP_ERR_UNSUPPORTED in the normal build).  cycles (HOST memory, 11
 * entries) receives the shader-clock cycles all waves of the launches since
 * the last reset spent in each phase of the tile loop -- [0] the fused
 * 8-bit/16-bit pass, [1] code and maxima emission, [2] barrier B, [3] stage
 * 1, [4] exponentials, [5] barrier E, [6] rescale and stage 2, [7] P.V and
 * the next speculative set, [8] barrier I, [9] prologue and epilogue -- and
 * [10] the number of waves.  reset != 0 clears the sums.  Synchronous.
 */
int lamp_phase_read(uint64_t *cycles, int reset);

/* Build the device tables of `device` now (otherwise done by the first call). */
int lamp_init(int device);

/* Release every device table and workspace the library holds (waits for
 * every device the library used). */
void lamp_shutdown(void);

/*
 * Diagnostics used by the test suite.
 *
 * lamp_selftest_e4m3: e4m3 codes of fp32 values, in[n] -> out[n] (device
 * pointers), by the same rounding sequence as the 8-bit accumulation (the
 * hardware conversion, saturating at +-448); raw (device, may be NULL)
 * receives the codes of the non-saturating hardware conversion alone.
 * lamp_selftest_exp_doc: the fp64 exponential used for the rescale factor
 * exp(mu - mu_hat), x[n] -> y[n] (device pointers).
 * lamp_get_tables: copies the device exponential tables to HOST memory:
 * lut8[256] (ue5m3 shift code -> ue5m3 exp code) and exp16[65536] (ue5m11
 * shift code -> ue5m11 exp code); either pointer may be NULL.
 * lamp_get_exp16_parts: copies to HOST memory parts[65536], the same 16-bit
 * exponentials as exact bf16 pairs (bits of the high part in [15:0], of the
 * low part in [31:16]; high = the fp32 value with its low 16 bits cleared,
 * low = value - high), the form the forward pass feeds to the matrix cores.
 * lamp_get_sim_tables: copies to HOST memory the exponential tables of the
 * SIM profile: sim8[112] (bf16 bits) and sim16[45056] (FP32 patterns), entry
 * ((e - emin) << p) | m holding RN_p(exp(-s)) for the shift
 * s = (2^p + m) 2^(e - p), p = 3 with e in [-6, 7], p = 11 with e in
 * [-14, 7]; either pointer may be NULL.
 */
int lamp_selftest_e4m3(const float *in, uint8_t *out, uint8_t *raw, size_t n, void *stream);
int lamp_selftest_exp_doc(const double *x, double *y, size_t n, void *stream);
int lamp_get_tables(int device, uint8_t *lut8, uint16_t *exp16);
int lamp_get_exp16_parts(int device, uint32_t *parts);
int lamp_get_sim_tables(int device, uint16_t *sim8, uint32_t *sim16);

const char *lamp_status_str(int status);
const char *lamp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* LAMP_H */
