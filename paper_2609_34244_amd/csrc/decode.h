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
    const int R = P.L + 1, N = P.n_types;
    x.S = S;
    const bool act = lane < S;
    const uint32_t rec = act ? rec_in : 0u;
    const int g = rec & 0xFF;
    const int l2tp = (rec >> 8) & 15, l2ep = (rec >> 12) & 15;
    const int tp = 1 << l2tp, ep = 1 << l2ep;
    const int ki = nibble(P.tp_index, l2tp), ei = nibble(P.ep_index, l2ep);
    const int gn = __builtin_amdgcn_update_dpp(g, g, kDppWaveShl1, 0xF, 0xF, false);   // next stage's type
    // unsigned 32-bit offsets from uniform table bases
    const int node = P.node_size[(uint32_t)g];
    const int64_t p2p = F32 ? P.p2p_fx[(uint32_t)(g * N + gn)] : P.p2p_ns[(uint32_t)(g * N + gn)];
    x.prow = act ? ((g * P.n_tp + ki) * 3 + a2a_variant(ep, tp, node)) * R : 0;
    x.lrow = act ? ((g * P.n_tp + ki) * P.n_ep + ei) * P.n_f * 2 * P.lim_stride : 0;
    x.p2p = lane < S - 1 ? (V)p2p : (V)0;
    return x;
}

}  // namespace heddle
