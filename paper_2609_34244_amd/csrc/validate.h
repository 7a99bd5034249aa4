// Template validation with one lane per template, shared by the kernels that
// map templates to lanes (gfx950).
#pragma once

#include "device_common.h"

namespace heddle {

// Validation in status order (section 5.1 feasibility masks, section 5.2
// exact profile match), one lane over its own stages; cnt is the lane's
// column of per-type GPU counters (all zero on entry and on exit), cs words
// apart.
__device__ __forceinline__ int validate_lane(const DevProfile &P, const PriceArgs &A, int S, const uint32_t *rec,
                                             uint32_t *cnt, int cs = 64)
{
    if (S < 1 || S > A.s_max || S > P.L) return HEDDLE_S_BAD_SHAPE;
    const int N = P.n_types;
    const int D = (int)(rec[0] >> 16);
    bool b_type = false, b_tp = false, b_prof = false, b_dp = false, b_ep = false;
    for (int s = 0; s < S; s++) {
        const uint32_t r = rec[s];
        const int g = r & 0xFF, l2tp = (r >> 8) & 15, l2ep = (r >> 12) & 15, dpv = (int)(r >> 16);
        const int gc = g < N ? g : N - 1;                      // clamped for the table reads
        const int ki = nibble(P.tp_index, l2tp);
        b_type |= g >= N;
        b_tp |= !((P.tp_present >> l2tp) & 1) || (1 << l2tp) > P.node_size[gc];
        b_prof |= !P.profiled[gc * P.n_tp + ki];
        b_dp |= dpv < 1 || dpv != D;
        b_ep |= !((P.ep_present >> l2ep) & 1) || ((uint32_t)D % (1u << l2ep)) != 0;
    }
    if (b_type) return HEDDLE_S_BAD_TYPE;
    if (b_tp) return HEDDLE_S_BAD_TP;
    if (b_prof) return HEDDLE_S_UNPROFILED;
    if (b_dp) return HEDDLE_S_BAD_DP;
    if (b_ep) return HEDDLE_S_BAD_EP;
    // GPUs of each type: sum of TP over the stages of that type, times D
    for (int s = 0; s < S; s++) cnt[(rec[s] & 0xFF) * cs] += 1u << ((rec[s] >> 8) & 15);
    bool over = false;
    for (int s = 0; s < S; s++) {
        const int g = rec[s] & 0xFF;
        over |= (int64_t)cnt[g * cs] * D > P.n_gpus[g];
    }
    for (int s = 0; s < S; s++) cnt[(rec[s] & 0xFF) * cs] = 0;
    return over ? HEDDLE_S_OVERSUBSCRIBED : HEDDLE_S_OK;
}

}  // namespace heddle
