// lamp_decode.h -- the decode form's parameter block and launchers
// (library-internal; lamp_decode.hip, lamp_host.cpp).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lamp {

// Decode form (vector LAMP, Sec. 2): M query rows per (b, h) at positions
// N-M .. N-1 against a bf16 key/value cache of N keys.
struct DecParams {
    const uint16_t *q;        // [B][Hq][M][D] bf16 queries
    float qscale;             // their scale, RN32(1/sqrt(D)) (applied in fp32 as the logits read them)
    const uint16_t *k, *v;    // [B][Hkv][N][D] bf16 cache
    uint8_t *y8;              // [B][Hq][M][Np] 8-bit logit codes (workspace)
    uint16_t *y16;            // [B][Hq][M][Np] e4m11 codes of the 16-bit logits (workspace)
    float *mut;               // [B][Hkv][Np/64][G*M] mu_hat per visited tile (workspace)
    double *f;                // [B][Hkv][Np/64][G*M] lambda_hat per tile, then its P.V factor within its key chunk (workspace)
    float *part;              // [B][Hq][M][ceil(N/DEC_PV_KEYS)][D] partial outputs of the P.V pieces (workspace)
    const uint16_t *lut8e;    // ue5m3 shift code -> bf16 bits of the ue5m3 exp
    const uint32_t *exp16hl;  // ue5m11 shift code -> bf16 high | low << 16 of the ue5m11 exp
    float *o, *lse;           // [B][Hq][M][D], [B][Hq][M]
    uint8_t *mask;            // [B][Hq][M][Np] one code per key
    int B, Hq, Hkv, M, N;
    int Np;                   // keys rounded up to whole tiles of 64
    int kb0;                  // first key any row can see (a multiple of 64)
    int causal, window, mode;
    double delta, tau;
    // Key chunks: the call's keys from kb0 in chunks of ck (a multiple of
    // DEC_PV_KEYS); a launch covers keys [ka, kz) of chunk `chunk` of nchunks (the last
    // one ends at Np).  The decisions carry the row state from chunk to chunk.
    int ka, kz, chunk, nchunks, ck;
    float *mu_st;             // [B][Hq][M] running maximum after the chunks decided so far (workspace)
    double *om_st;            // [B][Hq][M] running sum likewise
    double *lam_c;            // [B][Hq][M][nchunks] product of lambda_hat over each chunk's tiles (workspace)
};

// Key chunks of the decode form: at most this many per call; their length
// is a multiple of the keys of one P.V workgroup.
constexpr int DEC_MAX_CHUNKS = 8;
constexpr int DEC_PV_KEYS = 512;

// The decode form's kernels for one key chunk (p.ka, p.kz, p.chunk): the
// logits, the decisions (in chunk order: each continues the row state of the
// previous chunk), and P.V; then, once every chunk is through, the reduction
// over the chunks.  launch_dec_stage runs the decisions of one chunk, the
// logits of a later one and P.V of an earlier one in one launch (null: none;
// rows per key/value head at most 8).
constexpr int DEC_STAGE_MAX_ROWS = 8;
hipError_t launch_dec_logits(int D, const DecParams &p, hipStream_t s);
hipError_t launch_dec_decide(int D, const DecParams &p, hipStream_t s);
hipError_t launch_dec_pv(int D, const DecParams &p, hipStream_t s);
hipError_t launch_dec_reduce(int D, const DecParams &p, hipStream_t s);
hipError_t launch_dec_stage(int D, const DecParams *pd, const DecParams *pl, const DecParams *pp, hipStream_t s);

} // namespace lamp
