// Expert tiling on gfx950 (Heddle, arXiv 2609.34244, section 5.3, expert
// tiling paragraph), as a pass over priced plans.
//
// A stage of TP k and DP D spans W = k * D GPUs; its expert layout is EP e x
// ETP t x EDP W / (e t). The layouts priced for a stage: e from the EP list,
// t a profiled TP degree of the stage's GPU type no larger than its node (ETP
// stays within one node like TP, while an EP group may span nodes), e t
// dividing W. Under a layout an
// MoE layer costs its profiled time at TP k with the experts' part at ETP k
// replaced by the experts' part at ETP t scaled to the stage's tokens per GPU
// (ceil(x_t * t / k); a per-(type, TP, ETP) prefix table), plus one
// all-to-all at intra-node bandwidth if the e t GPUs of an EP group fit one
// node, else at the same-type inter-node link; memory holds the dense state
// at TP k, the expert state at ETP t divided by e and the in-flight
// activations; synchronisation all-reduces the dense gradients over D
// replicas and the expert gradients (ETP t, divided by e) over the EDP
// replicas. A stage's layout reaches no other stage, and with every stage at
// its fastest fitting layout under a bound G on the synchronisation term both
// (M-1) max t and sum t are as small as G allows, so the best layouts for the
// whole 1F1B iteration are found by trying every synchronisation value of a
// fitting layout as G: the smallest iteration time wins, then the smallest G;
// per stage the fastest layout wins, then the smaller synchronisation, then
// the first in (EP list, TP list) order.
//
// Mapping: one wavefront per plan (grid-stride). Lanes are (stage, layout)
// slots while the layouts are priced (time, synchronisation and memory into
// LDS; time all ones when the layout is not allowed or does not fit); then
// lanes are stages, each keeping in place the layouts that no other layout of
// its stage beats in both time and synchronisation (only those can be chosen,
// and only their synchronisation values need to be tried as bounds); then
// lanes are the kept layouts as thresholds G, each pricing the plan under its
// G from the kept table (broadcast reads); a wavefront minimum of (iteration
// time, G) decides, and lanes as stages write the layouts back.
#include <cstring>

#include "exact_math.h"
#include "heddle_internal.h"
#include "device_common.h"

namespace heddle {

constexpr uint64_t kNoLayout = ~0ull;

// per-stage constants of the layout pricing, one LDS record per stage
struct StageK {
    int64_t W, cap, bw, T0, n_moe, dstate, act_b, inflight, g_dense;
    int32_t g, ki, node, i0, j0, pad;
};

__device__ __forceinline__ void wave_min_pair(uint64_t &a, uint64_t &b)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t x = __shfl_xor((unsigned long long)a, o), y = __shfl_xor((unsigned long long)b, o);
        const bool take = x < a || (x == a && y < b);
        a = take ? x : a;
        b = take ? y : b;
    }
}

__global__ void __launch_bounds__(64, 6) tile_kernel(DevProfile P, PriceArgs A, uint8_t *tiling)
{
    extern __shared__ __align__(16) unsigned char smem[];      // one wavefront per workgroup
    const int lane = threadIdx.x;
    const int L = P.L, R = L + 1, N = P.n_types, K = P.n_tp, E = P.n_ep, F = K * E;
    // rows of Fp = F rounded up to odd 8-byte entries: lanes reading their own
    // stage's row touch distinct LDS banks
    const int Fp = F | 1;
    uint64_t *cT = (uint64_t *)smem;                           // [s_cap][Fp] time (kNoLayout: none)
    uint64_t *cG = cT + (size_t)A.s_cap * Fp;                  // [s_cap][Fp] synchronisation
    int64_t *cM = (int64_t *)(cG + (size_t)A.s_cap * Fp);      // [s_cap][Fp] memory
    uint8_t *cC = (uint8_t *)(cM + (size_t)A.s_cap * Fp);      // [s_cap][Fp] layout index of a kept entry
    uint8_t *cN = cC + (size_t)A.s_cap * Fp;                   // [s_cap] kept layouts of a stage
    const size_t sk_off = ((size_t)A.s_cap * Fp * 25 + A.s_cap + 15) & ~size_t(15);
    StageK *SK = (StageK *)(smem + sk_off);                    // [s_cap]
    uint8_t *tS = (uint8_t *)(SK + A.s_cap);                   // [s_cap * Fp] stage of a threshold entry
    uint8_t *tJ = tS + (size_t)A.s_cap * Fp;                   // [s_cap * Fp] its index among the stage's kept
    const int64_t total = A.n * A.n_m;
    // slot q -> stage q / F as a high product with ceil(2^32 / F), exact for
    // q * F < 2^32 (here q < s_cap * F <= 255 * 256); F = 1 maps q to itself
    const uint32_t invF = F > 1 ? (uint32_t)(0xFFFFFFFFu / (uint32_t)F) + 1u : 0u;

    for (int64_t o = blockIdx.x; o < total; o += gridDim.x) {
        const int64_t t = A.n_m == 1 ? o : total <= 0xFFFFFFFFll ? (int64_t)((uint32_t)o / (uint32_t)A.n_m) : o / A.n_m;
        const int k = (int)(o - t * A.n_m);
        const int st_in = A.status[o];
        const bool has_split = (st_in == HEDDLE_S_OK || st_in == HEDDLE_S_OOM) && A.layers[o * A.s_max] > 0;
        if (!has_split) {                                      // no split: nothing to tile
            if (lane < A.s_max) tiling[o * A.s_max + lane] = 0;
            continue;
        }
        // a split implies a valid template; buffers that do not describe one
        // (inconsistent with the templates) are left alone rather than read out
        // of range
        const int S = A.n_stages[t];
        const bool act = lane < S && lane < A.s_cap;
        const uint32_t rec = act ? A.stages[t * A.s_max + lane] : 0u;
        const int nl = act ? A.layers[o * A.s_max + lane] : 0;
        int i0 = nl;                                           // inclusive scan, then exclusive
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int u = __shfl_up(i0, d);
            i0 += lane >= d ? u : 0;
        }
        const int total_layers = __shfl(i0, 63);
        i0 -= nl;
        const int j0 = i0 + nl;
        const int g = rec & 0xFF, l2tp = (rec >> 8) & 15, l2ep = (rec >> 12) & 15;
        const int ki = nibble(P.tp_index, l2tp);
        const int tp = 1 << l2tp;
        const int D = (int)(__builtin_amdgcn_readfirstlane(rec) >> 16);
        const bool bad = S < 1 || S > A.s_cap || total_layers != L || D < 1 ||
                         __ballot(act && (g >= N || nl < 1 || !((P.tp_present >> l2tp) & 1))) != 0;
        if (bad) {
            if (lane < A.s_max) tiling[o * A.s_max + lane] = 0;
            continue;
        }
        const int32_t m = A.m[k];
        const int64_t Mp = (int64_t)(((uint32_t)m + (uint32_t)D - 1) / (uint32_t)D);
        const int64_t inflight = (int64_t)(S - lane) < Mp ? (int64_t)(S - lane) : Mp;
        const int g_next = __builtin_amdgcn_update_dpp(g, g, kDppWaveShl1, 0xF, 0xF, false);
        const int64_t p2p = lane + 1 < S ? P.p2p_ns[g * N + g_next] : 0;
        const int node = P.node_size[g];
        const int64_t cap = P.mem_cap[g];
        const int64_t W = (int64_t)tp * D;
        const int64_t bw = W <= node ? P.intra_bw[g] : P.link_bw[g * N + g];
        const uint64_t *base = P.rows64[0] + ((size_t)(g * K + ki) * 3 + kA2ANone) * R;
        const uint64_t T0 = base[j0] - base[i0] + (uint64_t)p2p;
        const int64_t n_moe = P.pre_moe[j0] - P.pre_moe[i0];
        const int64_t dstate = P.pre_dstate[ki * R + j0] - P.pre_dstate[ki * R + i0];
        const int64_t act_b = P.pre_act[ki * R + j0] - P.pre_act[ki * R + i0];
        const int64_t gd = P.pre_grad[ki * R + j0] - P.pre_grad[ki * R + i0];
        const int64_t g_dense = allreduce_ns(gd, D, bw);

        // ---- lanes = (stage, layout) slots q = s * F + c: price every layout
        wave_sync();                                           // the previous plan's table reads are done
        if (act) {
            StageK &sk = SK[lane];
            sk.W = W; sk.cap = cap; sk.bw = bw; sk.T0 = (int64_t)T0; sk.n_moe = n_moe; sk.dstate = dstate;
            sk.act_b = act_b; sk.inflight = inflight; sk.g_dense = g_dense;
            sk.g = g; sk.ki = ki; sk.node = node; sk.i0 = i0; sk.j0 = j0;
        }
        wave_sync();
        const int n_cand = S * F;
        for (int q0 = 0; q0 < n_cand; q0 += 64) {
            const int q = q0 + lane;
            if (q < n_cand) {
                const int s = F > 1 ? (int)__umulhi((uint32_t)q, invF) : q, c = q - s * F;
                const StageK &sk = SK[s];
                const int sg = sk.g, ski = sk.ki, snode = sk.node, si0 = sk.i0, sj0 = sk.j0;
                const int ei = c / K, ti = c - ei * K;
                const int l2e = nibble(P.ep_log2, ei), l2t = nibble(P.tp_log2, ti);
                const int et = 1 << l2t;
                const int64_t gmask = ((int64_t)1 << (l2e + l2t)) - 1;    // EP x ETP, a power of two
                const bool allowed = P.profiled[sg * K + ti] && et <= snode && (sk.W & gmask) == 0;
                const int64_t *xd = P.xdelta + ((size_t)(sg * K + ski) * K + ti) * R;
                const uint64_t T = (uint64_t)sk.T0 + (uint64_t)(xd[sj0] - xd[si0]) +
                                   (uint64_t)(sk.n_moe * P.a2a_ns[sg * 3 + a2a_variant(1 << l2e, et, snode)]);
                const int64_t *xs = P.pre_xstate + (size_t)(ti * E + ei) * R;
                const int64_t mem = sk.dstate + (xs[sj0] - xs[si0]) + sk.inflight * sk.act_b;
                const int64_t *xg = P.pre_xgrad + (size_t)(ti * E + ei) * R;
                const int64_t edp = allowed ? sk.W >> (l2e + l2t) : 1;
                const int64_t gs = sk.g_dense + allreduce_ns(xg[sj0] - xg[si0], edp, sk.bw);
                const int qs = s * Fp + c;
                cT[qs] = allowed && mem <= sk.cap ? T : kNoLayout;
                cG[qs] = (uint64_t)gs;
                cM[qs] = mem;
            }
        }
        wave_sync();

        // ---- lanes = (stage, layout) slots again: a layout is kept when no other
        // layout of its stage beats it in both time and synchronisation (an earlier
        // one also by being equal in both); only these can be a stage's fastest
        // layout under a bound on the synchronisation, and only their
        // synchronisation values need to be tried as bounds. The kept layouts move
        // to the front of their stage's row in layout order (a slot's new place is
        // at or before its old one, so no row entry is overwritten before it is read).
        uint8_t *kf = tS;                                      // [n_cand] kept flags, by slot
        for (int q0 = 0; q0 < n_cand; q0 += 64) {
            const int q = q0 + lane;
            const bool in = q < n_cand;
            const int s = !in ? 0 : F > 1 ? (int)__umulhi((uint32_t)q, invF) : q, c = in ? q - s * F : 0;
            const int rb = s * Fp;
            const uint64_t x = in ? cT[rb + c] : kNoLayout, y = in ? cG[rb + c] : 0;
            bool keep = x != kNoLayout;
            for (int c2 = 0; c2 < F; c2++) {
                const uint64_t x2 = cT[rb + c2], y2 = cG[rb + c2];
                keep = keep && !(c2 != c && x2 <= x && y2 <= y && (c2 < c || x2 < x || y2 < y));
            }
            if (in) kf[q] = (uint8_t)keep;
        }
        wave_sync();
        for (int q0 = 0; q0 < n_cand; q0 += 64) {
            const int q = q0 + lane;
            const bool in = q < n_cand;
            const int s = !in ? 0 : F > 1 ? (int)__umulhi((uint32_t)q, invF) : q, c = in ? q - s * F : 0;
            const int rb = s * Fp;
            const bool keep = in && kf[q];
            int rank = 0, tot = 0;
            for (int c2 = 0; c2 < F; c2++) {
                const int f = kf[s * F + c2];
                rank += c2 < c ? f : 0;
                tot += f;
            }
            const uint64_t x = cT[rb + c], y = cG[rb + c];
            const int64_t mx = cM[rb + c];
            wave_sync();
            if (keep) {
                cT[rb + rank] = x;
                cG[rb + rank] = y;
                cM[rb + rank] = mx;
                cC[rb + rank] = (uint8_t)c;
            }
            if (in && c == 0) cN[s] = (uint8_t)tot;
            wave_sync();
        }
        // threshold list: every kept layout of every stage, (stage, index) per entry
        int n_thr = 0;
        {
            const int nfl = act ? cN[lane] : 0;
            int off = nfl;                                     // exclusive scan of the kept counts
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int u = __shfl_up(off, d);
                off += lane >= d ? u : 0;
            }
            n_thr = __shfl(off, 63);
            off -= nfl;
            for (int j = 0; j < nfl; j++) {
                tS[off + j] = (uint8_t)lane;
                tJ[off + j] = (uint8_t)j;
            }
        }
        wave_sync();

        // ---- lanes = frontier layouts as thresholds G: the plan's iteration time
        // with every stage at its fastest kept layout of synchronisation <= G
        uint64_t best_it = kNoLayout, best_G = kNoLayout;
        for (int q0 = 0; q0 < n_thr; q0 += 64) {
            const int q = q0 + lane;
            uint64_t it = kNoLayout, G = kNoLayout;
            if (q < n_thr) {
                G = cG[tS[q] * Fp + tJ[q]];
                uint64_t maxT = 0, sumT = 0, maxg = 0;
                bool ok = true;
                for (int s2 = 0; s2 < S && ok; s2++) {
                    uint64_t bT = kNoLayout, bG = 0;
                    const int n2 = cN[s2];
                    for (int j2 = 0; j2 < n2; j2++) {
                        const uint64_t x = cT[s2 * Fp + j2], y = cG[s2 * Fp + j2];
                        const bool take = y <= G && x < bT;        // kept layouts have distinct times
                        bT = take ? x : bT;
                        bG = take ? y : bG;
                    }
                    ok = bT != kNoLayout;
                    maxT = bT > maxT ? bT : maxT;
                    sumT += bT;
                    maxg = bG > maxg ? bG : maxg;
                }
                if (ok) it = (uint64_t)(Mp - 1) * maxT + sumT + maxg;
            }
            wave_min_pair(it, G);
            if (it < best_it || (it == best_it && G < best_G)) {
                best_it = it;
                best_G = G;
            }
        }

        // ---- lanes = stages: write the chosen layouts
        if (best_it == kNoLayout) {                            // some stage has no fitting layout: unchanged
            if (lane < A.s_max) tiling[o * A.s_max + lane] = act ? (uint8_t)(l2ep | l2tp << 4) : 0;
            continue;
        }
        uint64_t bT = 0;
        int64_t bM = 0;
        int bc = 0;
        if (act) {
            bT = kNoLayout;
            const int rb = lane * Fp, nf = cN[lane];
            for (int j = 0; j < nf; j++) {
                const uint64_t x = cT[rb + j], y = cG[rb + j];
                const bool take = y <= best_G && x < bT;
                bT = take ? x : bT;
                bM = take ? cM[rb + j] : bM;
                bc = take ? cC[rb + j] : bc;
            }
        }
        const uint64_t B = wave_max(bT);
        const int64_t peak = wave_max(bM);
        if (lane == 0) {
            A.status[o] = HEDDLE_S_OK;
            ((int64_t *)A.iter)[o] = (int64_t)best_it;
            ((int64_t *)A.bottleneck)[o] = (int64_t)B;
            A.peak_mem[o] = peak;
        }
        const int bei = bc / K, bti = bc - bei * K;
        if (lane < A.s_max)
            tiling[o * A.s_max + lane] = act ? (uint8_t)(nibble(P.ep_log2, bei) | nibble(P.tp_log2, bti) << 4) : 0;
    }
}

int launch_tile(const heddle_profile *p, const PriceArgs &a, uint8_t *tiling, hipStream_t stream)
{
    const int64_t total = a.n * a.n_m;
    if (total == 0) return HEDDLE_OK;
    const size_t F = (size_t)p->dev.n_tp * p->dev.n_ep;
    // layout tables (time, synchronisation, memory: 8 bytes each; layout index),
    // kept counts, per-stage constants, threshold list (stage, index)
    const size_t lds = (((size_t)a.s_cap * (F | 1) * 25 + a.s_cap + 15) & ~size_t(15)) + (size_t)a.s_cap * sizeof(StageK) +
                       (size_t)a.s_cap * (F | 1) * 2;
    int max_lds = 0;
    HEDDLE_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, p->device));
    if (lds > (size_t)max_lds) return fail(HEDDLE_E_RANGE, "layout table of this (s_max, n_tp, n_ep) does not fit in LDS");
    if (lds > 65536)
        HEDDLE_HIP(hipFuncSetAttribute((const void *)tile_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
    const int blocks = (int)(total < 65536 ? total : 65536);
    hipLaunchKernelGGL(tile_kernel, dim3(blocks), dim3(64), lds, stream, p->dev, a, tiling);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

}  // namespace heddle

using namespace heddle;

extern "C" int heddle_tile_plans(const heddle_profile *p, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                                 const uint32_t *d_stages, const int32_t *h_m, int32_t n_m, uint32_t flags,
                                 void *d_iter, void *d_bottleneck, int64_t *d_peak_mem, const uint8_t *d_layers,
                                 uint8_t *d_status, uint8_t *d_tiling, hipStream_t stream)
{
    int rc = validate_price_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    if (rc) return rc;
    if (flags & HEDDLE_F_FP32) return fail(HEDDLE_E_INVAL, "expert tiling is defined for int64 costs (no HEDDLE_F_FP32)");
    if (n > 0 && (!d_iter || !d_bottleneck || !d_peak_mem || !d_layers || !d_status || !d_tiling))
        return fail(HEDDLE_E_INVAL, "device pointer is NULL");
    int64_t m_max = 0;
    for (int k = 0; k < n_m; k++) m_max = h_m[k] > m_max ? h_m[k] : m_max;
    const int64_t s_cap = s_max < p->dev.L ? s_max : p->dev.L;
    const __int128 bound = (__int128)(m_max - 1 + s_cap) * p->max_tiled_ns + p->max_ar_tiled_ns;
    if (bound >= kLimit62) return fail(HEDDLE_E_RANGE, "tiled iteration time could exceed 2^62 for these m");
    PriceArgs a;
    std::memset(&a, 0, sizeof(a));
    a.n = n;
    a.s_max = s_max;
    a.s_cap = (int32_t)s_cap;
    a.n_m = n_m;
    a.flags = (int32_t)flags;
    for (int k = 0; k < n_m; k++) a.m[k] = h_m[k];
    a.n_stages = d_n_stages;
    a.stages = d_stages;
    a.iter = d_iter;
    a.bottleneck = d_bottleneck;
    a.peak_mem = d_peak_mem;
    a.layers = const_cast<uint8_t *>(d_layers);
    a.status = d_status;
    return launch_tile(p, a, d_tiling, stream);
}
