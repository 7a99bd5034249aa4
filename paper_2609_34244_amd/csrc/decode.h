// Template decode and validation shared by the pricing kernels (gfx950,
// one wavefront per template, lane s = stage s).
#pragma once

#include "device_common.h"

namespace heddle {

// Per-lane (lane = stage s) decoded record and stage constants.
template <class V> struct StageInfo {
    int status;              // uniform: HEDDLE_S_* of the template (0 if valid)
    int S, D;                // uniform
    int prow;                // offset of the stage's time-prefix row
    int lrow;                // offset of the stage's memory-limit rows (in-flight count 1)
    V p2p;                   // outbound p2p (ns, or fixed point for fp32)
};

// Template decode and validation (feasibility masks of section 5.1, exact
// profile match of section 5.2). All per-lane table reads are issued at once
// on clamped indices; the checks then run in status order over all stages.
// `cnt` is a per-wavefront LDS array with one counter per GPU type.
template <class V, bool F32>
__device__ StageInfo<V> decode(const DevProfile &P, const PriceArgs &A, int S, uint32_t rec_in, int lane,
                               uint32_t *cnt)
{
    StageInfo<V> x;
    const int L = P.L, R = L + 1, N = P.n_types;
    x.S = S;
    x.status = 0;
    x.D = 1;
    x.prow = x.lrow = 0;
    x.p2p = 0;
    const bool act = lane < x.S && lane < A.s_max;
    const uint32_t rec = act ? rec_in : 0u;
    const int g = rec & 0xFF;
    const int l2tp = (rec >> 8) & 15, l2ep = (rec >> 12) & 15;
    const int dpv = (int)(rec >> 16);
    const int tp = 1 << l2tp, ep = 1 << l2ep;
    const int ki = nibble(P.tp_index, l2tp), ei = nibble(P.ep_index, l2ep);
    const int gc = g < N ? g : N - 1;                          // clamped for speculative reads
    const int gn = __builtin_amdgcn_update_dpp(gc, gc, kDppWaveShl1, 0xF, 0xF, false);   // next stage's type
    const int node = P.node_size[gc];
    const int prof = P.profiled[gc * P.n_tp + ki];
    const int ngpu = P.n_gpus[gc];
    const int64_t p2p = F32 ? P.p2p_fx[gc * N + gn] : P.p2p_ns[gc * N + gn];

    if (x.S < 1 || x.S > A.s_max || x.S > L) { x.status = HEDDLE_S_BAD_SHAPE; return x; }
    if (ballot(act && g >= N)) { x.status = HEDDLE_S_BAD_TYPE; return x; }
    if (ballot(act && (!((P.tp_present >> l2tp) & 1) || tp > node))) { x.status = HEDDLE_S_BAD_TP; return x; }
    if (ballot(act && !prof)) { x.status = HEDDLE_S_UNPROFILED; return x; }
    x.D = rl32(dpv, 0);
    if (ballot(act && (dpv < 1 || dpv != x.D))) { x.status = HEDDLE_S_BAD_DP; return x; }
    if (ballot(act && (!((P.ep_present >> l2ep) & 1) || ((uint32_t)x.D % (uint32_t)ep) != 0))) {
        x.status = HEDDLE_S_BAD_EP;
        return x;
    }
    // GPUs of this lane's type used by the template: sum of TP over its stages
    // (times D below), accumulated with LDS atomics
    wave_sync();
    if (act) cnt[g] = 0;
    wave_sync();
    if (act) atomicAdd(&cnt[g], (uint32_t)tp);
    wave_sync();
    const uint32_t used = act ? cnt[g] : 0u;
    if (ballot(act && (int64_t)used * x.D > ngpu)) { x.status = HEDDLE_S_OVERSUBSCRIBED; return x; }

    if (act) {
        x.prow = ((g * P.n_tp + ki) * 3 + a2a_variant(ep, tp, node)) * R;
        x.lrow = ((g * P.n_tp + ki) * P.n_ep + ei) * P.n_f * 2 * P.lim_stride;
        x.p2p = lane < x.S - 1 ? (V)p2p : (V)0;
    }
    return x;
}

}  // namespace heddle
