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
// Mapping: one wavefront per plan (grid-stride). Lanes are stages while the
// stage constants are formed (an LDS record per stage). Lanes are then (stage,
// layout) slots that only test which layouts are allowed, and the allowed
// ones are compacted, in (stage, layout) order, into a list by ballot and
// prefix count; lanes over that list price the layouts (time,
// synchronisation, memory) and compact the ones that fit memory into a second
// list, with each stage's segment of it. Lanes over the fitting list keep the
// layouts that no other layout of their stage beats in both time and
// synchronisation (only those can be chosen under a bound, and only their
// synchronisation values need to be tried as bounds), compacted in place.
// Lanes are then the kept layouts as thresholds G, each pricing the plan under
// its G from the kept list (broadcast reads); a wavefront minimum of
// (iteration time, G) decides, and lanes as stages write the layouts back.
// Times and synchronisation values are held in 32 bits when the profile's
// bounds on them allow it.
#include <cstring>

#include "exact_math.h"
#include "heddle_internal.h"
#include "device_common.h"

namespace heddle {

// per-stage constants of the layout pricing, one LDS record per stage
struct StageK {
    int64_t cap, bw, T0, dstate, act_b, g_dense;
    int32_t W, n_moe, inflight, etp, g, ki, node, i0, j0, pad;
};

// set lanes of a wavefront mask below this lane
__device__ __forceinline__ int lanes_below(uint64_t m)
{
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// time and synchronisation of a list entry, read together
template <class TT> struct alignas(2 * sizeof(TT)) TGPair {
    TT x, y;
};

// table entry i of a profile table, addressed by a 32-bit byte offset (every
// profile table is far below 4 GB)
template <class T> __device__ __forceinline__ T ld_at(const T *base, uint32_t i)
{
    return *(const T *)((const char *)base + i * (uint32_t)sizeof(T));
}

// LDS of one wavefront: the stage records, then per list entry (at most
// s_cap * F) memory, time and synchronisation, the allowed-layout list, layout
// index, stage and kept flag, then the per-stage segment bounds
template <class TT> __host__ __device__ inline size_t tile_lds_bytes(int s_cap, int F)
{
    const size_t n = (size_t)s_cap * F;
    // (the time-synchronisation list has F + 1 entries of padding: the Pareto
    // pass reads up to that far past a segment start)
    return (size_t)s_cap * sizeof(StageK) + n * (8 + sizeof(TGPair<TT>) + 4 + 3) + (size_t)(F + 1) * sizeof(TGPair<TT>) +
           3 + (size_t)s_cap * 4;
}

// TT: uint32_t when every stage time and synchronisation value is below
// 2^32 - 1 (the profile's bounds), else uint64_t; all ones marks no layout
// COUNT: no outputs; the work of the batch is added to A.work[0..2] (layouts
// priced, dominance tests, bound tests).
template <class TT, bool COUNT>
__global__ void __launch_bounds__(64, 6) tile_kernel(DevProfile P, PriceArgs A, uint8_t *tiling)
{
    constexpr TT kNone = (TT)~(TT)0;
    extern __shared__ __align__(16) unsigned char smem[];      // one wavefront per workgroup
    const int lane = threadIdx.x;
    const int L = P.L, R = L + 1, N = P.n_types, K = P.n_tp, E = P.n_ep, F = K * E;
    const int nmax = A.s_cap * F;
    StageK *SK = (StageK *)smem;                               // [s_cap]
    int64_t *cM = (int64_t *)(SK + A.s_cap);                   // [nmax] memory of a list entry
    TGPair<TT> *cTG = (TGPair<TT> *)(cM + nmax);               // [nmax] time, synchronisation
    uint32_t *AL = (uint32_t *)(cTG + nmax + F + 1);           // [nmax] allowed: s | c << 8 | ei << 16 | ti << 24
    uint8_t *cC = (uint8_t *)(AL + nmax);                      // [nmax] layout index c = ei * K + ti
    uint8_t *cS = cC + nmax;                                   // [nmax] stage
    uint8_t *kf = cS + nmax;                                   // [nmax] kept flag
    uint16_t *seg_lo = (uint16_t *)(kf + nmax + ((4 - (3 * nmax) % 4) % 4));   // [s_cap] first entry of a stage
    uint16_t *seg_hi = seg_lo + A.s_cap;                       // [s_cap] one past its last
    const int64_t total = A.n * A.n_m;
    // slot q -> stage q / F and layout c -> EP index c / K as high products with
    // ceil(2^32 / F) and ceil(2^32 / K), exact for q * F, c * K < 2^32 (here
    // q < 64 * 256); a divisor of 1 maps to itself
    const uint32_t invF = F > 1 ? (uint32_t)(0xFFFFFFFFu / (uint32_t)F) + 1u : 0u;
    const uint32_t invK = K > 1 ? (uint32_t)(0xFFFFFFFFu / (uint32_t)K) + 1u : 0u;

    // the segments of a list whose entries are in stage order: lanes over the
    // entries mark where each stage's run starts and ends (stages with no
    // entry keep 0 .. 0); returns, in lane s, first | end << 16 of stage s
    auto segments = [&](int n, bool act) -> uint32_t {
        if (act) {
            seg_lo[lane] = 0;
            seg_hi[lane] = 0;
        }
        wave_sync();
        for (int q0 = 0; q0 < n; q0 += 64) {
            const int q = q0 + lane;
            if (q < n) {
                const int s = cS[q];
                if (q == 0 || cS[q - 1] != s) seg_lo[s] = (uint16_t)q;
                if (q == n - 1 || cS[q + 1] != s) seg_hi[s] = (uint16_t)(q + 1);
            }
        }
        wave_sync();
        return act ? (uint32_t)seg_lo[lane] | (uint32_t)seg_hi[lane] << 16 : 0u;
    };

    auto template_of = [&](int64_t oo) -> int64_t {
        return A.n_m == 1 ? oo : total <= 0xFFFFFFFFll ? (int64_t)((uint32_t)oo / (uint32_t)A.n_m) : oo / A.n_m;
    };
    // a plan's status, layer counts, stage count and records, loaded one
    // iteration ahead (plans are this wavefront's alone, so the status read
    // ahead is not one it writes)
    int st_n = 0, S_n = 0, nl_n = 0;
    uint32_t rec_n = 0;
    auto fetch = [&](int64_t oo) {
        const int64_t tt = template_of(oo);
        st_n = A.status[oo];
        S_n = A.n_stages[tt];
        nl_n = lane < A.s_max ? A.layers[oo * A.s_max + lane] : 0;
        rec_n = lane < A.s_max ? A.stages[tt * A.s_max + lane] : 0u;
    };
    if ((int64_t)blockIdx.x < total) fetch(blockIdx.x);
    unsigned long long w_priced = 0, w_dom = 0, w_bound = 0;  // COUNT: this wavefront's work

    for (int64_t o = blockIdx.x; o < total; o += gridDim.x) {
        const int st_in = st_n, S = S_n, nl_all = nl_n;
        const uint32_t rec_all = rec_n;
        if (o + gridDim.x < total) fetch(o + gridDim.x);
        const int64_t t = template_of(o);
        const int k = (int)(o - t * A.n_m);
        const bool has_split = (st_in == HEDDLE_S_OK || st_in == HEDDLE_S_OOM) && rl32(nl_all, 0) > 0;
        if (!has_split) {                                      // no split: nothing to tile
            if (!COUNT && lane < A.s_max) tiling[o * A.s_max + lane] = 0;
            continue;
        }
        // a split implies a valid template; buffers that do not describe one
        // (inconsistent with the templates) are left alone rather than read out
        // of range
        const bool act = lane < S && lane < A.s_cap;
        const uint32_t rec = act ? rec_all : 0u;
        const int nl = act ? nl_all : 0;
        int i0 = wave_inclusive_sum(nl);                       // inclusive scan, then exclusive
        const int total_layers = rl32(i0, 63);
        i0 -= nl;
        const int j0 = i0 + nl;
        const int g = rec & 0xFF, l2tp = (rec >> 8) & 15, l2ep = (rec >> 12) & 15;
        const int ki = nibble(P.tp_index, l2tp);
        const int tp = 1 << l2tp;
        const int D = (int)(__builtin_amdgcn_readfirstlane(rec) >> 16);
        const bool bad = S < 1 || S > A.s_cap || total_layers != L || D < 1 ||
                         __ballot(act && (g >= N || nl < 1 || !((P.tp_present >> l2tp) & 1))) != 0;
        if (bad) {
            if (!COUNT && lane < A.s_max) tiling[o * A.s_max + lane] = 0;
            continue;
        }
        const int32_t m = A.m[k];
        const int64_t Mp = (int64_t)(((uint32_t)m + (uint32_t)D - 1) / (uint32_t)D);

        // ---- lanes = stages: the stage constants
        wave_sync();                                           // the previous plan's reads are done
        if (act) {
            const int64_t inflight = (int64_t)(S - lane) < Mp ? (int64_t)(S - lane) : Mp;
            const int g_next = __builtin_amdgcn_update_dpp(g, g, kDppWaveShl1, 0xF, 0xF, false);
            const uint32_t ug = (uint32_t)g, uj = (uint32_t)j0, ui = (uint32_t)i0, ur = (uint32_t)(ki * R);
            const int64_t p2p = lane + 1 < S ? ld_at(P.p2p_ns, ug * N + (uint32_t)g_next) : 0;
            const int node = ld_at(P.node_size, ug);
            const int64_t W = (int64_t)tp * D;
            const int64_t bw = W <= node ? ld_at(P.intra_bw, ug) : ld_at(P.link_bw, ug * (N + 1));
            const uint32_t trow = ((ug * K + (uint32_t)ki) * 3 + kA2ANone) * R;
            const int64_t gd = ld_at(P.pre_grad, ur + uj) - ld_at(P.pre_grad, ur + ui);
            StageK &sk = SK[lane];
            sk.W = (int32_t)W;
            sk.etp = (int32_t)ld_at(P.etp_mask, ug);
            sk.cap = ld_at(P.mem_cap, ug);
            sk.bw = bw;
            sk.T0 = (int64_t)(ld_at(P.rows64[0], trow + uj) - ld_at(P.rows64[0], trow + ui) + (uint64_t)p2p);
            sk.n_moe = ld_at(P.pre_moe, uj) - ld_at(P.pre_moe, ui);
            sk.dstate = ld_at(P.pre_dstate, ur + uj) - ld_at(P.pre_dstate, ur + ui);
            sk.act_b = ld_at(P.pre_act, ur + uj) - ld_at(P.pre_act, ur + ui);
            sk.inflight = (int32_t)inflight;
            sk.g_dense = allreduce_ns(gd, D, bw);
            sk.g = g; sk.ki = ki; sk.node = node; sk.i0 = i0; sk.j0 = j0;
        }
        wave_sync();

        // ---- lanes = (stage, layout) slots q = s * F + c: which layouts are
        // allowed (a profiled ETP within the node, EP x ETP dividing the
        // stage's GPUs), compacted in slot order
        const int n_cand = S * F;
        int n_al = 0;
        for (int q0 = 0; q0 < n_cand; q0 += 64) {
            const int q = q0 + lane;
            bool allowed = false;
            uint32_t ent = 0;
            if (q < n_cand) {
                const int s = F > 1 ? (int)__umulhi((uint32_t)q, invF) : q, c = q - s * F;
                const int ei = K > 1 ? (int)__umulhi((uint32_t)c, invK) : c, ti = c - ei * K;
                const StageK &sk = SK[s];
                const int l2e = nibble(P.ep_log2, ei), l2t = nibble(P.tp_log2, ti);
                const int32_t gmask = (int32_t)((1u << (l2e + l2t)) - 1);    // EP x ETP, a power of two
                allowed = ((sk.etp >> ti) & 1) && (sk.W & gmask) == 0;
                ent = (uint32_t)s | (uint32_t)c << 8 | (uint32_t)ei << 16 | (uint32_t)ti << 24;
            }
            const uint64_t mk = ballot(allowed);
            if (allowed) AL[n_al + lanes_below(mk)] = ent;
            n_al += __popcll(mk);
        }
        wave_sync();
        w_priced += (unsigned long long)n_al;

        // ---- lanes = allowed layouts: price them; the ones that fit memory
        // go, in the same order, to the fitting list
        int n_fit = 0;
        for (int q0 = 0; q0 < n_al; q0 += 64) {
            const int q = q0 + lane;
            bool fits = false;
            uint64_t T = 0;
            int64_t mem = 0, gs = 0;
            uint32_t ent = 0;
            if (q < n_al) {
                ent = AL[q];
                const int s = ent & 255, ei = (ent >> 16) & 255, ti = ent >> 24;
                const StageK &sk = SK[s];
                const int sg = sk.g, ski = sk.ki, snode = sk.node, si0 = sk.i0, sj0 = sk.j0;
                const int l2e = nibble(P.ep_log2, ei), l2t = nibble(P.tp_log2, ti);
                const uint32_t xd = ((uint32_t)(sg * K + ski) * K + (uint32_t)ti) * R;
                const uint32_t xe = (uint32_t)(ti * E + ei) * R;
                const uint32_t uj = (uint32_t)sj0, ui = (uint32_t)si0;
                T = (uint64_t)sk.T0 + (uint64_t)(ld_at(P.xdelta, xd + uj) - ld_at(P.xdelta, xd + ui)) +
                    (uint64_t)((int64_t)sk.n_moe * ld_at(P.a2a_ns, (uint32_t)(sg * 3 + a2a_variant(1 << l2e, 1 << l2t, snode))));
                mem = sk.dstate + (ld_at(P.pre_xstate, xe + uj) - ld_at(P.pre_xstate, xe + ui)) +
                      (int64_t)sk.inflight * sk.act_b;
                gs = sk.g_dense + allreduce_ns(ld_at(P.pre_xgrad, xe + uj) - ld_at(P.pre_xgrad, xe + ui),
                                               (int64_t)(sk.W >> (l2e + l2t)), sk.bw);
                fits = mem <= sk.cap;
            }
            const uint64_t mk = ballot(fits);
            if (fits) {
                const int pos = n_fit + lanes_below(mk);
                cTG[pos] = TGPair<TT>{(TT)T, (TT)gs};
                cM[pos] = mem;
                cC[pos] = (uint8_t)(ent >> 8);
                cS[pos] = (uint8_t)ent;
            }
            n_fit += __popcll(mk);
        }
        wave_sync();
        uint32_t sgv = segments(n_fit, act);
        if (ballot(act && (sgv >> 16) == (sgv & 0xFFFF))) {    // a stage with no fitting layout: unchanged
            if (!COUNT && lane < A.s_max) tiling[o * A.s_max + lane] = act ? (uint8_t)(l2ep | l2tp << 4) : 0;
            continue;
        }

        // ---- lanes = fitting layouts: a layout is kept when no other layout of
        // its stage beats it in both time and synchronisation (an earlier one
        // also by being equal in both). Every lane walks the longest segment's
        // length (a wave-uniform loop, so the tests stay lane masks); the steps
        // past its own segment are masked (their reads stay inside the list's
        // padded LDS region).
        const int seg_len = act ? (int)(sgv >> 16) - (int)(sgv & 0xFFFF) : 0;
        const int max_seg = uni(wave_max(seg_len));
        if (COUNT) w_dom += wave_sum((uint32_t)(seg_len * seg_len));   // every pair of a stage's fitting layouts
        for (int q0 = 0; q0 < n_fit; q0 += 64) {
            const int q = q0 + lane;
            const bool in = q < n_fit;
            const int qc = in ? q : n_fit - 1;
            const int s = cS[qc];
            const TGPair<TT> e = cTG[qc];
            const int lo = seg_lo[s], len = seg_hi[s] - lo, qo = qc - lo;
            const TGPair<TT> *row = cTG + lo;
            auto beats = [&](int d, TGPair<TT> f) {
                if constexpr (sizeof(TT) == 4) {
                    // the pair compared as one 64-bit word: at most e in both and a
                    // different pair, or the same pair earlier
                    uint64_t fw, ew;
                    __builtin_memcpy(&fw, &f, 8);
                    __builtin_memcpy(&ew, &e, 8);
                    return (d < len) & (((f.x <= e.x) & (f.y <= e.y) & (fw != ew)) | ((fw == ew) & (d < qo)));
                } else {
                    return (d < len) & (d != qo) & (f.x <= e.x) & (f.y <= e.y) & ((d < qo) | (f.x < e.x) | (f.y < e.y));
                }
            };
            bool keep = true;
            for (int d = 0; d < max_seg; d += 2) {             // two entries per step
                const TGPair<TT> f0 = row[d], f1 = row[d + 1];
                keep &= !beats(d, f0);
                keep &= !beats(d + 1, f1);
            }
            if (in) kf[q] = (uint8_t)keep;
        }
        wave_sync();
        // compacted in place: an entry's new place is at or before its old one
        // and after every place an earlier pass wrote
        int n_k = 0;
        for (int q0 = 0; q0 < n_fit; q0 += 64) {
            const int q = q0 + lane;
            const bool keep = q < n_fit && kf[q];
            TGPair<TT> e = {};
            int64_t mx = 0;
            uint8_t c = 0, s = 0;
            if (keep) {
                e = cTG[q];
                mx = cM[q];
                c = cC[q];
                s = cS[q];
            }
            const uint64_t mk = ballot(keep);
            wave_sync();
            if (keep) {
                const int pos = n_k + lanes_below(mk);
                cTG[pos] = e;
                cM[pos] = mx;
                cC[pos] = c;
                cS[pos] = s;
            }
            n_k += __popcll(mk);
        }
        wave_sync();
        sgv = segments(n_k, act);
        if (COUNT) {                                           // every bound against every kept layout and stage
            w_bound += (unsigned long long)n_k * (unsigned long long)(n_k + S);
            continue;
        }

        // ---- lanes = kept layouts as thresholds G: the plan's iteration time
        // with every stage at its fastest kept layout of synchronisation <= G
        uint64_t best_it = ~0ull, best_G = ~0ull, best_B = 0;
        for (int q0 = 0; q0 < n_k; q0 += 64) {
            const int q = q0 + lane;
            const TT G = q < n_k ? cTG[q].y : (TT)0;
            TT maxT = 0, maxg = 0;
            uint64_t sumT = 0;
            bool ok = true;
            for (int s2 = 0; s2 < S; s2++) {
                const uint32_t b = uni64(sgv, s2);
                TT bT = kNone, bG = 0;
                auto consider = [&](TT x, TT y) {
                    const bool take = y <= G && x < bT;        // kept layouts have distinct times
                    bT = take ? x : bT;
                    bG = take ? y : bG;
                };
                const int hi = (int)(b >> 16);
                int j = (int)(b & 0xFFFF);
                for (; j + 1 < hi; j += 2) {                   // two entries per step
                    const TT x0 = cTG[j].x, y0 = cTG[j].y, x1 = cTG[j + 1].x, y1 = cTG[j + 1].y;
                    consider(x0, y0);
                    consider(x1, y1);
                }
                if (j < hi) consider(cTG[j].x, cTG[j].y);
                ok = ok && bT != kNone;
                maxT = bT > maxT ? bT : maxT;
                sumT += (uint64_t)bT;
                maxg = bG > maxg ? bG : maxg;
            }
            const bool valid = q < n_k && ok;
            const uint64_t it = valid ? (uint64_t)(Mp - 1) * (uint64_t)maxT + sumT + (uint64_t)maxg : ~0ull;
            // the smallest iteration time, then the smallest bound among the lanes
            // that reach it; the bottleneck is the slowest chosen stage of such a lane
            const uint64_t it_min = group_min<uint64_t>(it, 64);
            const TT g_min = group_min<TT>(valid && it == it_min ? G : kNone, 64);
            const uint64_t win = ballot(valid && it == it_min && G == g_min);
            if (win && (it_min < best_it || (it_min == best_it && (uint64_t)g_min < best_G))) {
                best_it = it_min;
                best_G = (uint64_t)g_min;
                best_B = (uint64_t)(TT)rl64((int64_t)(uint64_t)maxT, __ffsll((unsigned long long)win) - 1);
            }
        }

        // ---- lanes = stages: write the chosen layouts
        if (best_it == ~0ull) {                                // no bound serves every stage: unchanged
            if (!COUNT && lane < A.s_max) tiling[o * A.s_max + lane] = act ? (uint8_t)(l2ep | l2tp << 4) : 0;
            continue;
        }
        int64_t bM = 0;
        int bc = 0;
        if (act) {
            uint64_t bT = ~0ull;
            for (int j = (int)(sgv & 0xFFFF); j < (int)(sgv >> 16); j++) {
                const uint64_t x = cTG[j].x, y = cTG[j].y;
                const bool take = y <= best_G && x < bT;
                bT = take ? x : bT;
                bM = take ? cM[j] : bM;
                bc = take ? cC[j] : bc;
            }
        }
        const uint64_t B = best_B;
        const int64_t peak = wave_max(bM);
        if (lane == 0) {
            A.status[o] = HEDDLE_S_OK;
            ((int64_t *)A.iter)[o] = (int64_t)best_it;
            ((int64_t *)A.bottleneck)[o] = (int64_t)B;
            A.peak_mem[o] = peak;
        }
        const int bei = K > 1 ? (int)__umulhi((uint32_t)bc, invK) : bc, bti = bc - bei * K;
        if (lane < A.s_max)
            tiling[o * A.s_max + lane] = act ? (uint8_t)(nibble(P.ep_log2, bei) | nibble(P.tp_log2, bti) << 4) : 0;
    }
    if (COUNT && lane == 0) {
        if (w_priced) atomicAdd(&A.work[0], w_priced);
        if (w_dom) atomicAdd(&A.work[1], w_dom);
        if (w_bound) atomicAdd(&A.work[2], w_bound);
    }
}

template <class TT, bool COUNT>
static int launch_tile_t(const heddle_profile *p, const PriceArgs &a, uint8_t *tiling, hipStream_t stream)
{
    const int64_t total = a.n * a.n_m;
    const size_t lds = tile_lds_bytes<TT>(a.s_cap, p->dev.n_tp * p->dev.n_ep);
    int max_lds = 0;
    HEDDLE_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, p->device));
    if (lds > (size_t)max_lds) return fail(HEDDLE_E_RANGE, "layout table of this (s_max, n_tp, n_ep) does not fit in LDS");
    if (lds > 65536)
        HEDDLE_HIP(hipFuncSetAttribute((const void *)tile_kernel<TT, COUNT>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
    const int blocks = (int)(total < 65536 ? total : 65536);
    hipLaunchKernelGGL((tile_kernel<TT, COUNT>), dim3(blocks), dim3(64), lds, stream, p->dev, a, tiling);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

bool tile_narrow(const heddle_profile *p)
{
    return p->max_tiled_ns < (int64_t)0xFFFFFFFFll && p->max_ar_tiled_ns < (int64_t)0xFFFFFFFFll;
}

int launch_tile(const heddle_profile *p, const PriceArgs &a, uint8_t *tiling, hipStream_t stream)
{
    if (a.n * a.n_m == 0) return HEDDLE_OK;
    if (a.work)
        return tile_narrow(p) ? launch_tile_t<uint32_t, true>(p, a, tiling, stream) : launch_tile_t<uint64_t, true>(p, a, tiling, stream);
    return tile_narrow(p) ? launch_tile_t<uint32_t, false>(p, a, tiling, stream) : launch_tile_t<uint64_t, false>(p, a, tiling, stream);
}

}  // namespace heddle

using namespace heddle;

// host checks and arguments of a tiling launch over priced plans
static int tile_args(const heddle_profile *p, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                     const uint32_t *d_stages, const int32_t *h_m, int32_t n_m, uint32_t flags, PriceArgs &a)
{
    int rc = validate_price_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    if (rc) return rc;
    if (flags & HEDDLE_F_FP32) return fail(HEDDLE_E_INVAL, "expert tiling is defined for int64 costs (no HEDDLE_F_FP32)");
    int64_t m_max = 0;
    for (int k = 0; k < n_m; k++) m_max = h_m[k] > m_max ? h_m[k] : m_max;
    const int64_t s_cap = s_max < p->dev.L ? s_max : p->dev.L;
    const __int128 bound = (__int128)(m_max - 1 + s_cap) * p->max_tiled_ns + p->max_ar_tiled_ns;
    if (bound >= kLimit62) return fail(HEDDLE_E_RANGE, "tiled iteration time could exceed 2^62 for these m");
    std::memset(&a, 0, sizeof(a));
    a.n = n;
    a.s_max = s_max;
    a.s_cap = (int32_t)s_cap;
    a.n_m = n_m;
    a.flags = (int32_t)flags;
    for (int k = 0; k < n_m; k++) a.m[k] = h_m[k];
    a.n_stages = d_n_stages;
    a.stages = d_stages;
    return HEDDLE_OK;
}

extern "C" int heddle_tile_plans(const heddle_profile *p, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                                 const uint32_t *d_stages, const int32_t *h_m, int32_t n_m, uint32_t flags,
                                 void *d_iter, void *d_bottleneck, int64_t *d_peak_mem, const uint8_t *d_layers,
                                 uint8_t *d_status, uint8_t *d_tiling, hipStream_t stream)
{
    PriceArgs a;
    int rc = tile_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags, a);
    if (rc) return rc;
    if (n > 0 && (!d_iter || !d_bottleneck || !d_peak_mem || !d_layers || !d_status || !d_tiling))
        return fail(HEDDLE_E_INVAL, "device pointer is NULL");
    a.iter = d_iter;
    a.bottleneck = d_bottleneck;
    a.peak_mem = d_peak_mem;
    a.layers = const_cast<uint8_t *>(d_layers);
    a.status = d_status;
    return launch_tile(p, a, d_tiling, stream);
}

extern "C" int heddle_count_tile_work(const heddle_profile *p, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                                      const uint32_t *d_stages, const int32_t *h_m, int32_t n_m, uint32_t flags,
                                      const uint8_t *d_layers, const uint8_t *d_status, int64_t *h_counts,
                                      hipStream_t stream)
{
    PriceArgs a;
    int rc = tile_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags, a);
    if (rc) return rc;
    if (!h_counts) return fail(HEDDLE_E_INVAL, "h_counts is NULL");
    if (n > 0 && (!d_layers || !d_status)) return fail(HEDDLE_E_INVAL, "device pointer is NULL");
    a.layers = const_cast<uint8_t *>(d_layers);
    a.status = const_cast<uint8_t *>(d_status);
    unsigned long long *d_work = nullptr;
    hipError_t e = scratch_alloc((void **)&d_work, 3 * sizeof(unsigned long long), stream);
    if (e != hipSuccess) return fail(HEDDLE_E_NOMEM, "device scratch for the work counters could not be allocated");
    e = hipMemsetAsync(d_work, 0, 3 * sizeof(unsigned long long), stream);
    a.work = d_work;
    rc = e == hipSuccess ? launch_tile(p, a, nullptr, stream) : hip_fail(e, "hipMemsetAsync");
    unsigned long long h[3] = {0, 0, 0};
    if (rc == HEDDLE_OK) e = hipMemcpyAsync(h, d_work, sizeof(h), hipMemcpyDeviceToHost, stream);
    (void)hipFreeAsync(d_work, stream);                        // stream-ordered after the copy
    if (rc == HEDDLE_OK && e == hipSuccess) e = hipStreamSynchronize(stream);
    if (rc == HEDDLE_OK && e != hipSuccess) rc = hip_fail(e, "reading the work counters back");
    if (rc == HEDDLE_OK)
        for (int i = 0; i < 3; i++) h_counts[i] = (int64_t)h[i];
    return rc;
}
