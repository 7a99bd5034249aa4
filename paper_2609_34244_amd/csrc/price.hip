// Batched plan pricing on gfx950, split kernel: template decode and
// validation, PartitionLayers (exact min-max layer split) and its canonical
// reconstruction. Evaluate runs in evaluate.hip on the split found here.
//
// Method: Heddle (arXiv 2609.34244). The layer split is the PartitionLayers
// step of the planners' nested-loop backbone (section 3.1), aware of per-stage
// GPU speed (the straggler criticism of speed-blind splits in the same
// section) and of memory (section 5.2, memory validation).
//
// Recurrence (suffix form): G[s][i] is the smallest achievable bottleneck
// when stages s..S-1 hold layers [i, L):
//   G[S-1][i] = T(S-1, i, L)                                    if it fits
//   G[s][i]   = min over i < j <= jl_s(i) of max(T(s,i,j), G[s+1][j])
// with jl_s(i) the last admissible end of row i: the memory limit (a profile
// table indexed by GPU type, TP, EP and in-flight count) capped so that every
// later stage keeps one layer. B* = G[0][0]. T(s,i,j) = P_s[j] - P_s[i] + p2p_s
// with P_s the stage's time prefix (layer costs + MoE all-to-all), also a
// profile table.
//
// Mapping. One wavefront splits one template at a time (grid-stride over
// templates). Lanes are stages for decode and validation, and split rows i
// during the DP: a row takes one lane and walks its ends four at a time; the
// rows of a stage's ragged last slot take several lanes each, which stride
// over the ends and combine with cross-lane minima. Per wavefront, LDS holds
// the pairs W[j] = {P_s[j], G[s+1][j]} of the stage being relaxed, so one
// 64-bit LDS read feeds one relaxation (sub, max, min), and, for every stage,
// the DP row G[s][.] and the end limits J[s][.] that the reconstruction
// needs. The profile rows of stage s-1 are fetched into registers while
// stage s relaxes.
#include <cstring>

#include "device_common.h"

namespace heddle {

// Per-lane (lane = stage s) decoded record and stage constants.
struct StageInfo {
    int status;              // uniform: HEDDLE_S_* of the template (0 if valid)
    int S, D;                // uniform
    int prow;                // offset of the stage's time-prefix row
    int lrow;                // offset of the stage's memory-limit rows (in-flight count 1)
    int64_t p2p;             // outbound p2p (ns, or fixed point for fp32)
};

// Template decode and validation (feasibility masks of section 5.1, exact
// profile match of section 5.2). All per-lane table reads are issued at once
// on clamped indices; the checks then run in status order over all stages.
template <bool F32>
__device__ StageInfo decode(const DevProfile &P, const PriceArgs &A, int64_t t, int lane)
{
    StageInfo x;
    const int L = P.L, R = L + 1, N = P.n_types;
    x.S = A.n_stages[t];
    x.status = 0;
    x.D = 1;
    x.prow = x.lrow = 0;
    x.p2p = 0;
    const bool act = lane < x.S && lane < A.s_max;
    const uint32_t rec = act ? A.stages[t * A.s_max + lane] : 0u;
    const int g = rec & 0xFF;
    const int l2tp = (rec >> 8) & 15, l2ep = (rec >> 12) & 15;
    const int dpv = (int)(rec >> 16);
    const int tp = 1 << l2tp, ep = 1 << l2ep;
    const int ki = nibble(P.tp_index, l2tp), ei = nibble(P.ep_index, l2ep);
    const int gc = g < N ? g : N - 1;                          // clamped for speculative reads
    const int gn = __shfl(gc, lane + 1 < 64 ? lane + 1 : 63);
    const int node = P.node_size[gc];
    const int prof = P.profiled[gc * P.n_tp + ki];
    const int ngpu = P.n_gpus[gc];
    const int64_t p2p = F32 ? P.p2p_fx[gc * N + gn] : P.p2p_ns[gc * N + gn];

    if (x.S < 1 || x.S > A.s_max || x.S > L) { x.status = HEDDLE_S_BAD_SHAPE; return x; }
    if (__ballot(act && g >= N)) { x.status = HEDDLE_S_BAD_TYPE; return x; }
    if (__ballot(act && (!((P.tp_present >> l2tp) & 1) || tp > node))) { x.status = HEDDLE_S_BAD_TP; return x; }
    if (__ballot(act && !prof)) { x.status = HEDDLE_S_UNPROFILED; return x; }
    x.D = rl32(dpv, 0);
    if (__ballot(act && (dpv < 1 || dpv != x.D))) { x.status = HEDDLE_S_BAD_DP; return x; }
    if (__ballot(act && (!((P.ep_present >> l2ep) & 1) || ((uint32_t)x.D % (uint32_t)ep) != 0))) {
        x.status = HEDDLE_S_BAD_EP;
        return x;
    }
    int used = 0;                                              // this lane's type: sum of TP over its stages
    for (int s2 = 0; s2 < x.S; s2++)
        if (rl32(g, s2) == g) used += rl32(tp, s2);
    if (__ballot(act && (int64_t)used * x.D > ngpu)) { x.status = HEDDLE_S_OVERSUBSCRIBED; return x; }

    if (act) {
        x.prow = ((g * P.n_tp + ki) * 3 + a2a_variant(ep, tp, node)) * R;
        x.lrow = ((g * P.n_tp + ki) * P.n_ep + ei) * P.n_f * R;
        x.p2p = lane < x.S - 1 ? p2p : 0;
    }
    return x;
}

// Profile rows of one stage, fetched into registers ahead of use: the time
// prefix and the memory limit of every row (slots of 64 entries).
constexpr int kRowSlots = 4;                       // (L + 1) <= 256 entries
template <class V> struct RowRegs {
    V p[kRowSlots];
    uint32_t l[kRowSlots];
};

template <class V>
__device__ __forceinline__ void fetch_rows(RowRegs<V> &r, const V *prow, const uint8_t *lrow, int L, int nslots,
                                           int lane, bool need_mem)
{
#pragma unroll
    for (int q = 0; q < kRowSlots; q++) {
        if (q < nslots) {                                          // uniform
            const int j = min(lane + 64 * q, L);                   // clamped: no divergent loads
            r.p[q] = prow[j];
            r.l[q] = need_mem ? (uint32_t)lrow[j] : (uint32_t)L;
        }
    }
}

template <class V> __device__ __forceinline__ const V *stage_rows(const DevProfile &P, bool f32);
template <> __device__ __forceinline__ const uint32_t *stage_rows<uint32_t>(const DevProfile &P, bool f32)
{
    return P.rows32[f32 ? 1 : 0];
}
template <> __device__ __forceinline__ const uint64_t *stage_rows<uint64_t>(const DevProfile &P, bool f32)
{
    return P.rows64[f32 ? 1 : 0];
}

// relaxation of one end: max(T(s,i,j), G[s+1][j]) with T = P_s[j] - pi
template <class V, class V2> __device__ __forceinline__ V relax(const V2 &a, V pi)
{
    const V t = a.x - pi;
    return t > a.y ? t : a.y;
}

template <class T> __device__ __forceinline__ T vmin(T a, T b) { return a < b ? a : b; }

// ------------------------------------------------------------ split kernel

template <class V, bool F32, bool COUNT>
__global__ void __launch_bounds__(256, sizeof(V) == 4 ? 5 : 4) split_kernel(DevProfile P, PriceArgs A)
{
    typedef typename Vec2<V>::type V2;
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63, wib = threadIdx.x >> 6, wpb = blockDim.x >> 6;
    const int L = P.L, R = L + 1, gs = A.g_stride;
    const int nslots = (L + 64) / 64;                          // 64-entry slots covering [0, L]
    const bool compute_only = (A.flags & HEDDLE_F_COMPUTE_ONLY) != 0;
    const V INF = DPInf<V>::value;
    unsigned char *wave_lds = smem + (size_t)wib * A.lds_per_wave;
    // two pair rows {P_s, G_{s+1}}: stage s reads one and writes G_s into the
    // other, which the commit of stage s-1 completes with P_{s-1}
    V2 *Wbuf = (V2 *)wave_lds;                                 // [2][gs]
    V *G = (V *)(wave_lds + A.off_g);                          // [s_cap][gs] DP rows, for the reconstruction
    uint8_t *J = wave_lds + A.off_j;                           // [s_cap][gs] last admissible ends
    const V *rows = stage_rows<V>(P, F32);

    int my_m = 1;                                              // lane k: the k-th micro-batch count
    for (int k = 0; k < A.n_m; k++) my_m = lane == k ? A.m[k] : my_m;
    unsigned long long work = 0;

    for (int64_t t = (int64_t)blockIdx.x * wpb + wib; t < A.n; t += (int64_t)gridDim.x * wpb) {
        const StageInfo x = decode<F32>(P, A, t, lane);
        const int S = uni(x.S);
        const size_t obase = (size_t)t * A.n_m;
        bool r_split = false;                                  // lane k: a split was found for m index k
        V r_b = INF;

        if (x.status == 0) {
            const int D = x.D;
            // micro-batches per replica M_p = ceil(m / D); min(M_p, S) fixes the split
            const int Mp_k = (int)(((uint32_t)my_m + (uint32_t)D - 1) / (uint32_t)D);
            const int key_k = compute_only ? 0 : (Mp_k < S ? Mp_k : S);
            uint64_t todo = __ballot(lane < A.n_m);

            while (todo) {
                const int key = uni((int)group_min<uint32_t>(((todo >> lane) & 1) ? (uint32_t)key_k : 0x7FFFFFFFu, 64));
                const uint64_t cls = __ballot(lane < A.n_m && key_k == key) & todo;
                todo &= ~cls;
                auto lim_row = [&](int s) {                    // memory limits of stage s in this class
                    int f = (S - s) < key ? (S - s) : key;
                    f = f < 1 ? 1 : f;                         // compute-only: not read
                    return P.mem_lim + uni(rl32(x.lrow, s) + (f - 1) * R);
                };

                // ---------------- PartitionLayers: suffix min-max DP, stages S-1 .. 0
                RowRegs<V> rr;
                fetch_rows<V>(rr, rows + uni(rl32(x.prow, S - 1)), lim_row(S - 1), L, nslots, lane, !compute_only);
                V Bv = INF;
                for (int s = S - 1; s >= 0; s--) {
                    const V p2p = (V)rl64(x.p2p, s);
                    const int jhi = L - (S - 1 - s);               // leaves one layer per later stage
                    const int ihi = (s == 0) ? 0 : L - (S - s);
                    V2 *Xs = Wbuf + (size_t)(s & 1) * gs;          // {P_s, G_{s+1}}
                    V2 *Xo = Wbuf + (size_t)((s & 1) ^ 1) * gs;    // receives G_s
                    V *Gs = G + (size_t)s * gs;
                    uint8_t *Js = J + (size_t)s * gs;
#pragma unroll
                    for (int q = 0; q < kRowSlots; q++) {
                        if (q < nslots) {
                            const int j = min(lane + 64 * q, gs - 1);   // clamped into the padding
                            ((V *)&Xs[j])[0] = rr.p[q];
                            Js[j] = (uint8_t)min(rr.l[q], (uint32_t)jhi);
                        }
                    }
                    if (s > 0) fetch_rows<V>(rr, rows + uni(rl32(x.prow, s - 1)), lim_row(s - 1), L, nslots, lane, !compute_only);
                    wave_sync();
                    if (s == S - 1) {
                        // last stage: its rows must end at L
                        for (int i = s + lane; i <= ihi; i += 64) {
                            const bool fit = Js[i] == L;
                            if (COUNT) {
                                work += fit ? 1 : 0;
                            } else {
                                const V gv = fit ? (V)(Xs[L].x - Xs[i].x) : INF;
                                if (s > 0) {
                                    ((V *)&Xo[i])[1] = gv;
                                    Gs[i] = gv;
                                } else {
                                    Bv = gv;                    // S = 1: row 0, lane 0
                                }
                            }
                        }
                        if (S == 1) Bv = (V)rl64((int64_t)Bv, 0);
                    } else {
                        // rows [s, ihi] (stage 0: row 0 only): whole slots of 64 rows take
                        // one lane per row, the ragged last slot several lanes per row
                        int base = s;
                        for (; base + 63 <= ihi; base += 64) {
                            const int i = base + lane;
                            const int jl = Js[i];
                            if (COUNT) {
                                work += (unsigned long long)(jl - i);
                                continue;
                            }
                            const V pi = Xs[i].x - p2p;                  // T(s,i,j) = P_s[j] - pi
                            V acc = INF;
                            int j = i + 1;
                            for (; j + 3 <= jl; j += 4) {
                                const V2 a = Xs[j], b = Xs[j + 1], c = Xs[j + 2], d = Xs[j + 3];
                                acc = vmin(acc, vmin(vmin(relax<V>(a, pi), relax<V>(b, pi)),
                                                     vmin(relax<V>(c, pi), relax<V>(d, pi))));
                            }
                            if (j <= jl) {                               // 1 to 3 ends left (padded by 4)
                                const int rem = jl - j;
                                const V2 a = Xs[j], b = Xs[j + 1], c = Xs[j + 2];
                                const V cb = rem >= 1 ? relax<V>(b, pi) : INF;
                                const V cc = rem >= 2 ? relax<V>(c, pi) : INF;
                                acc = vmin(acc, vmin(relax<V>(a, pi), vmin(cb, cc)));
                            }
                            ((V *)&Xo[i])[1] = acc;
                            Gs[i] = acc;
                        }
                        if (base <= ihi) {
                            // r < 64 rows left: k lanes per row, k = 64 >> ceil(log2 r), each
                            // lane striding over the row's ends by k
                            const int r = ihi - base + 1;
                            const int k = 64 >> (r > 1 ? 32 - __clz(r - 1) : 0);
                            const int lk = 31 - __clz(k);
                            const int part = lane & (k - 1);
                            const int i = base + (lane >> lk);
                            const bool row_ok = i <= ihi;
                            const int ic = row_ok ? i : ihi;
                            const int jl = row_ok ? Js[ic] : 0;
                            if (COUNT) {
                                if (row_ok && part == 0) work += (unsigned long long)(jl - i);
                            } else {
                                const V pi = Xs[ic].x - p2p;
                                V acc = INF;
                                for (int j = i + 1 + part; j <= jl; j += k) acc = vmin(acc, relax<V>(Xs[j], pi));
                                acc = group_min<V>(acc, k);
                                if (s == 0) {
                                    Bv = (V)rl64((int64_t)acc, 0);       // one row: the whole wave's minimum
                                } else if (row_ok && part == 0) {
                                    ((V *)&Xo[i])[1] = acc;
                                    Gs[i] = acc;
                                }
                            }
                        }
                    }
                    wave_sync();
                }
                if (COUNT) continue;
                if (Bv == INF) continue;                       // no split fits memory
                const uint64_t B = (uint64_t)Bv;
                const uint64_t B24 = F32 ? rne24(B) : B;       // fp32 bottleneck, as an exact integer

                // ---------------- canonical reconstruction: smallest admissible end per stage
                // (time prefixes from the profile's stage rows, DP rows and limits from LDS)
                int cs = 0, my_start = 0, my_end = 0;
                for (int s = 0; s < S; s++) {
                    const V *prow = rows + uni(rl32(x.prow, s));
                    const V *Gn = G + (size_t)(s + 1) * gs;
                    const uint8_t *Js = J + (size_t)s * gs;
                    const V p2p = (V)rl64(x.p2p, s);
                    int found = -1;
                    for (int base = cs + 1; found < 0; base += 64) {
                        const int j = base + lane;
                        const int jc = j <= L ? j : L;
                        const V pj = prow[jc];                   // issued together with the reads below
                        const V pc = prow[cs] - p2p;
                        const int jl = Js[cs];
                        const V gj = s < S - 1 ? Gn[jc] : INF;
                        bool ok = false;
                        if (j <= jl) {
                            const uint64_t T = (uint64_t)(V)(pj - pc);
                            bool rest_ok;                      // the later stages complete within B*
                            if (s == S - 1) rest_ok = j == L;
                            else rest_ok = gj != INF && (F32 ? rne24((uint64_t)gj) <= B24 : (uint64_t)gj <= B);
                            ok = rest_ok && (F32 ? rne24(T) <= B24 : T <= B);
                        }
                        const uint64_t bal = __ballot(ok);
                        if (bal) found = base + __ffsll((unsigned long long)bal) - 1;
                        else if (base + 63 >= jl) found = jl;      // unreachable: G[s][cs] <= B* has a witness;
                                                                   // the fallback only keeps indexing in bounds
                    }
                    if (lane == s) {
                        my_start = cs;
                        my_end = found;
                    }
                    cs = found;
                }
                for (uint64_t c = cls; c; c &= c - 1) {
                    const int k = __ffsll((unsigned long long)c) - 1;
                    for (int q = lane; q < A.s_max; q += 64)
                        A.layers[(obase + k) * A.s_max + q] = q < S ? (uint8_t)(my_end - my_start) : 0;
                }
                if ((cls >> lane) & 1) {
                    r_split = true;
                    r_b = Bv;
                }
            }
        }
        if (COUNT) continue;
        if (lane < A.n_m) {
            const size_t o = obase + lane;
            A.status[o] = (uint8_t)(x.status != 0 ? x.status : (r_split ? HEDDLE_S_OK : HEDDLE_S_OOM));
            if (F32) ((float *)A.bottleneck)[o] = r_split ? exact_float(rne24((uint64_t)r_b), P.fx_exp) : __builtin_inff();
            else ((int64_t *)A.bottleneck)[o] = r_split ? (int64_t)r_b : INT64_MAX;
        }
        // zero layer counts of the plans without a split (invalid template, or no split fits)
        const uint64_t with_split = __ballot(r_split);
        if (with_split != __ballot(lane < A.n_m))
            for (int q = lane; q < A.n_m * A.s_max; q += 64)
                if (!((with_split >> (q / A.s_max)) & 1)) A.layers[obase * A.s_max + q] = 0;
    }
    if (COUNT) {
        work += __shfl_xor(work, 32);
        work += __shfl_xor(work, 16);
        work += __shfl_xor(work, 8);
        work += __shfl_xor(work, 4);
        work += __shfl_xor(work, 2);
        work += __shfl_xor(work, 1);
        if (lane == 0 && work) atomicAdd(A.work, work);
    }
}

// ------------------------------------------------------------------- host

int validate_price_args(const heddle_profile *p, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                        const uint32_t *d_stages, const int32_t *h_m, int32_t n_m, uint32_t flags)
{
    if (!p) return fail(HEDDLE_E_INVAL, "profile is NULL");
    if (n < 0) return fail(HEDDLE_E_INVAL, "n < 0");
    if (s_max < 1 || s_max > HEDDLE_MAX_STAGES) return fail(HEDDLE_E_INVAL, "s_max out of range 1..64");
    if (n_m < 1 || n_m > HEDDLE_MAX_MLIST) return fail(HEDDLE_E_INVAL, "n_m out of range 1..64");
    if (!h_m) return fail(HEDDLE_E_INVAL, "h_m is NULL");
    if (flags & ~(HEDDLE_F_FP32 | HEDDLE_F_COMPUTE_ONLY)) return fail(HEDDLE_E_INVAL, "unknown flag bits");
    int64_t m_max = 0;
    for (int k = 0; k < n_m; k++) {
        if (h_m[k] < 1 || h_m[k] > HEDDLE_MAX_M) return fail(HEDDLE_E_INVAL, "m out of range 1..2^24");
        m_max = h_m[k] > m_max ? h_m[k] : m_max;
    }
    if (n > 0 && (!d_n_stages || !d_stages)) return fail(HEDDLE_E_INVAL, "template pointer is NULL");
    int dev = -1;
    HEDDLE_HIP(hipGetDevice(&dev));
    if (dev != p->device) return fail(HEDDLE_E_INVAL, "profile was loaded on another device");
    const bool f32 = flags & HEDDLE_F_FP32;
    const int64_t max_stage = f32 ? p->max_stage_fx : p->max_stage_ns;
    const int64_t max_ar = f32 ? p->max_ar_fx : p->max_ar_ns;
    if (max_stage < 0) return fail(HEDDLE_E_RANGE, "fp32 costs span too wide a range to be summed exactly");
    const int64_t s_cap = s_max < p->dev.L ? s_max : p->dev.L;
    const __int128 bound = (__int128)(m_max - 1 + s_cap) * max_stage + max_ar;
    if (bound >= kLimit62) return fail(HEDDLE_E_RANGE, "iteration time could exceed 2^62 for these m");
    return HEDDLE_OK;
}

template <class V, bool F32, bool COUNT>
static int launch_split(const heddle_profile *p, PriceArgs &a, hipStream_t stream)
{
    const int L = p->dev.L;
    a.s_cap = a.s_max < L ? a.s_max : L;
    a.g_stride = L + 5;                                       // L + 1 ends and 4 of padding
    // per wavefront: two rows of pairs {P_s, G_{s+1}}, then the DP rows and the
    // end limits of every stage
    const size_t g_off = (size_t)2 * a.g_stride * 2 * sizeof(V);
    const size_t j_off = g_off + (size_t)a.s_cap * a.g_stride * sizeof(V);
    a.off_g = (int32_t)g_off;
    a.off_j = (int32_t)j_off;
    a.lds_per_wave = (int32_t)((j_off + (size_t)a.s_cap * a.g_stride + 15) & ~size_t(15));
    int max_lds = 0;
    HEDDLE_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, p->device));
    int wpb = max_lds / a.lds_per_wave;
    wpb = wpb > 4 ? 4 : (wpb < 1 ? 1 : wpb);
    const size_t lds = (size_t)wpb * a.lds_per_wave;
    if (lds > (size_t)max_lds) return fail(HEDDLE_E_RANGE, "DP table of this (L, s_max) does not fit in LDS");
    if (lds > 65536)
        HEDDLE_HIP(hipFuncSetAttribute((const void *)split_kernel<V, F32, COUNT>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
    const int64_t want = (a.n + wpb - 1) / wpb;
    const int blocks = (int)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL((split_kernel<V, F32, COUNT>), dim3(blocks), dim3(64 * wpb), lds, stream, p->dev, a);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

int launch_price(const heddle_profile *p, PriceArgs &a, hipStream_t stream, bool count_only)
{
    if (a.n == 0) return HEDDLE_OK;
    const bool f32 = a.flags & HEDDLE_F_FP32;
    const bool narrow = f32 ? p->narrow_f32 : p->narrow_i64;
    int rc;
    if (count_only) return launch_split<uint64_t, false, true>(p, a, stream);
    if (f32) rc = narrow ? launch_split<uint32_t, true, false>(p, a, stream) : launch_split<uint64_t, true, false>(p, a, stream);
    else rc = narrow ? launch_split<uint32_t, false, false>(p, a, stream) : launch_split<uint64_t, false, false>(p, a, stream);
    if (rc != HEDDLE_OK) return rc;
    return launch_evaluate(p, a, stream);
}

static PriceArgs make_args(int64_t n, int32_t s_max, const uint8_t *d_n_stages, const uint32_t *d_stages,
                           const int32_t *h_m, int32_t n_m, uint32_t flags)
{
    PriceArgs a;
    std::memset(&a, 0, sizeof(a));
    a.n = n;
    a.s_max = s_max;
    a.n_m = n_m;
    a.flags = (int32_t)flags;
    for (int k = 0; k < n_m; k++) a.m[k] = h_m[k];
    a.n_stages = d_n_stages;
    a.stages = d_stages;
    return a;
}

}  // namespace heddle

using namespace heddle;

extern "C" int heddle_price_plans(const heddle_profile *p, int64_t n, int32_t s_max,
                                  const uint8_t *d_n_stages, const uint32_t *d_stages,
                                  const int32_t *h_m, int32_t n_m, uint32_t flags,
                                  void *d_iter, void *d_bottleneck, int64_t *d_peak_mem,
                                  uint8_t *d_layers, uint8_t *d_status, hipStream_t stream)
{
    int rc = validate_price_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    if (rc) return rc;
    if (n > 0 && (!d_iter || !d_bottleneck || !d_peak_mem || !d_layers || !d_status))
        return fail(HEDDLE_E_INVAL, "output pointer is NULL");
    PriceArgs a = make_args(n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    a.iter = d_iter;
    a.bottleneck = d_bottleneck;
    a.peak_mem = d_peak_mem;
    a.layers = d_layers;
    a.status = d_status;
    return launch_price(p, a, stream, false);
}

extern "C" int heddle_count_work(const heddle_profile *p, int64_t n, int32_t s_max,
                                 const uint8_t *d_n_stages, const uint32_t *d_stages,
                                 const int32_t *h_m, int32_t n_m, uint32_t flags,
                                 int64_t *h_relaxations, hipStream_t stream)
{
    int rc = validate_price_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    if (rc) return rc;
    if (!h_relaxations) return fail(HEDDLE_E_INVAL, "h_relaxations is NULL");
    PriceArgs a = make_args(n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    unsigned long long *d_work = nullptr;
    hipError_t e = hipMallocAsync((void **)&d_work, sizeof(unsigned long long), stream);
    if (e != hipSuccess) return fail(HEDDLE_E_NOMEM, "hipMallocAsync of the work counter failed");
    HEDDLE_HIP(hipMemsetAsync(d_work, 0, sizeof(unsigned long long), stream));
    a.work = d_work;
    rc = launch_price(p, a, stream, true);
    unsigned long long h = 0;
    if (rc == HEDDLE_OK) {
        HEDDLE_HIP(hipMemcpyAsync(&h, d_work, sizeof(h), hipMemcpyDeviceToHost, stream));
        HEDDLE_HIP(hipStreamSynchronize(stream));
        *h_relaxations = (int64_t)h;
    }
    (void)hipFreeAsync(d_work, stream);
    return rc;
}
