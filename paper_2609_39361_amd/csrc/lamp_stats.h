// lamp_stats.h -- the statistics words of the forward kernels (lamp.h,
// LAMP_STAT_*): per-workgroup counters kept in LDS and added to the caller's
// words once at the end.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lamp.h"

namespace lamp {

// Statistics of one workgroup in LDS (flushed to the LAMP_STAT_* words at the
// end): tiles with an active sub-block, stage-1 and stage-2 sub-blocks,
// active sub-blocks, speculative 16-bit sub-blocks not used, 16-bit
// sub-blocks recomputed outside the speculative batch, saturated 8-bit and
// 16-bit logits, then the histogram of recomputed sub-blocks per tile.
enum { ST_TILES = 0, ST_S1, ST_S2, ST_ACT, ST_UNUSED, ST_LATE, ST_SAT8, ST_SAT16, ST_HIST, ST_N = ST_HIST + 8 };

// Add a workgroup's statistics (stl, in LDS) to the LAMP_STAT_* words; nsub:
// sub-blocks of one query block's mask row.  Called by every thread.
template <int NK>
__device__ __forceinline__ void flush_stats(uint64_t *stats, const uint32_t *stl, uint32_t nsub, int tid)
{
    __syncthreads();
    if (tid != 0) return;
    auto add = [&](int word, uint32_t v) {
        if (v) atomicAdd(reinterpret_cast<unsigned long long *>(stats + word), (unsigned long long)v);
    };
    add(LAMP_STAT_TILES, stl[ST_TILES]);
    add(LAMP_STAT_STAGE1, stl[ST_S1]);
    add(LAMP_STAT_STAGE2, stl[ST_S2]);
    add(LAMP_STAT_INACTIVE, nsub - stl[ST_ACT]);
    add(LAMP_STAT_SAT8, stl[ST_SAT8]);
    add(LAMP_STAT_SAT16, stl[ST_SAT16]);
    add(LAMP_STAT_SPEC_UNUSED, stl[ST_UNUSED]);
    add(LAMP_STAT_LATE16, stl[ST_LATE]);
    for (int c = 0; c <= NK; ++c) add(LAMP_STAT_HIST + c, stl[ST_HIST + c]);
}

} // namespace lamp
