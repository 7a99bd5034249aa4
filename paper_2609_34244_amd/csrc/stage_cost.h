// Cost of one pipeline stage holding layers [i, j) under the profile-based
// cost model (Heddle, arXiv 2609.34244, section 5.2): stage time (layer
// costs with the all-to-all of MoE layers, plus the outbound p2p), per-GPU
// memory with min(S - s, M_p) micro-batches of activations in flight, and
// gradient synchronisation (ring all-reduce of dense gradients over the D
// replicas and of expert gradients over D / EP). Shared by every kernel that
// evaluates a split, so they price identically.
#pragma once

#include "device_common.h"

namespace heddle {

struct StageCost {
    uint64_t T;        // stage time: ns, or fixed point (2^fx_exp) for fp32, not rounded
    int64_t mem;       // per-GPU bytes
    int64_t g;         // gradient synchronisation, ns
    bool fits;         // mem <= the GPU's memory
};

// rec: the stage's packed record; g_next: the next stage's GPU type (ignored
// for the last stage). The record must have passed validation.
template <bool F32>
__device__ __forceinline__ StageCost stage_cost(const DevProfile &P, uint32_t rec, int g_next, int s, int S,
                                                int i, int j, int D, int64_t Mp)
{
    const int R = P.L + 1, N = P.n_types;
    const int g = rec & 0xFF, l2tp = (rec >> 8) & 15, l2ep = (rec >> 12) & 15;
    const int tp = 1 << l2tp, ep = 1 << l2ep;
    const int ki = nibble(P.tp_index, l2tp), ei = nibble(P.ep_index, l2ep);
    const int node = P.node_size[g];
    const uint64_t *prow = P.rows64[F32 ? 1 : 0] + ((size_t)(g * P.n_tp + ki) * 3 + a2a_variant(ep, tp, node)) * R;
    int64_t p2p = 0;
    if (s + 1 < S) p2p = F32 ? P.p2p_fx[g * N + g_next] : P.p2p_ns[g * N + g_next];
    StageCost c;
    c.T = prow[j] - prow[i] + (uint64_t)p2p;
    const int srow = (ki * P.n_ep + ei) * R, arow = ki * R;
    const longlong2 sx_i = P.pair_sx[srow + i], sx_j = P.pair_sx[srow + j];   // {state, expert grad}
    const longlong2 ag_i = P.pair_ag[arow + i], ag_j = P.pair_ag[arow + j];   // {activations, dense grad}
    const int64_t f = (int64_t)(S - s) < Mp ? (int64_t)(S - s) : Mp;
    c.mem = (sx_j.x - sx_i.x) + f * (ag_j.x - ag_i.x);
    c.fits = c.mem <= P.mem_cap[g];
    const int64_t bw = (int64_t)tp * D <= node ? P.intra_bw[g] : P.link_bw[g * N + g];
    c.g = allreduce_ns(ag_j.y - ag_i.y, D, bw) +
          allreduce_ns(sx_j.y - sx_i.y, (int64_t)((uint32_t)D / (uint32_t)ep), bw);
    return c;
}

// 1F1B iteration time (section 5.3) from the bottleneck B, the sum of stage
// times and the largest synchronisation; fp32: B and every stage time are
// already rounded (exact integers with 24 significant bits), the largest
// synchronisation is rounded here and the total once more by the caller.
template <bool F32>
__device__ __forceinline__ uint64_t iteration_time(const DevProfile &P, int64_t Mp, uint64_t B, uint64_t sumT,
                                                   int64_t maxg)
{
    const uint64_t maxg_v = F32 ? rne24((uint64_t)maxg) << (-P.fx_exp) : (uint64_t)maxg;
    return (uint64_t)(Mp - 1) * B + sumT + maxg_v;
}

}  // namespace heddle
