// Per-stage constants of a validated template for the split kernel (gfx950,
// one wavefront per template, lane s = stage s).
#pragma once

#include "device_common.h"

namespace heddle {

// Per-lane (lane = stage s) decoded record and stage constants.
template <class V> struct StageInfo {
    int S;                   // uniform
    int prow;                // offset of the stage's time-prefix row
    int lrow;                // offset of the stage's memory-limit rows (in-flight count 1)
    V p2p;                   // outbound p2p (ns, or fixed point for fp32)
};

// Per-stage constants of a template that passed validation (one wavefront
// per template, lane s = stage s): the stage's time-prefix row (GPU type, TP,
// all-to-all variant), its memory-limit rows, its outbound p2p.
template <class V, bool F32>
__device__ StageInfo<V> stage_info(const DevProfile &P, const PriceArgs &A, int S, uint32_t rec_in, int lane)
{
    StageInfo<V> x;
    const int N = P.n_types;
    x.S = S;
    const bool act = lane < S;
    const uint32_t rec = act ? rec_in : 0u;
    const int g = rec & 0xFF;
    const int gn = __builtin_amdgcn_update_dpp(g, g, kDppWaveShl1, 0xF, 0xF, false);   // next stage's type
    // unsigned 32-bit offsets from uniform table bases; lanes past S read entry 0
    const uint2 rows = P.stage_tab[rec & 0xFFFFu];
    const int64_t p2p = F32 ? P.p2p_fx[(uint32_t)(g * N + gn)] : P.p2p_ns[(uint32_t)(g * N + gn)];
    x.prow = (int)rows.x;
    x.lrow = (int)rows.y;
    x.p2p = lane < S - 1 ? (V)p2p : (V)0;
    return x;
}

}  // namespace heddle
