// Batched plan pricing on gfx950: template decode and validation,
// PartitionLayers (exact min-max layer split), canonical reconstruction and
// Evaluate (1F1B iteration time and per-GPU peak memory).
//
// Method: Heddle (arXiv 2609.34244). The layer split is the PartitionLayers
// step of the planners' nested-loop backbone (section 3.1), made aware of
// per-stage GPU speed (the straggler criticism of speed-blind splits in the
// same section) and of memory (section 5.2, memory validation). Evaluate is
// the profile-based cost model of section 5.2 and the 1F1B formula
// (M-1) max_s t_s + sum_s t_s + max_s g_s of section 5.3.
//
// Mapping: one wavefront prices one template at a time (grid-stride over
// templates). Lanes are pipeline stages during decode, validation and
// Evaluate, and split rows during the DP. The DP table of the template
// (stage rows of L+1 entries) and the time-prefix row of the stage being
// relaxed live in LDS; profile tables are read from global memory, where
// they stay cache resident (a few KB to a few hundred KB per profile).
//
// Recurrence (suffix form): G[s][i] is the smallest achievable bottleneck
// when stages s..S-1 hold layers [i, L):
//   G[S-1][i] = T(S-1, i, L)                        if it fits, else inf
//   G[s][i]   = min over i < j <= L-(S-1-s), Fits(s,i,j) of max(T(s,i,j), G[s+1][j])
// and B* = G[0][0]. Memory use of a stage grows with j for fixed i, so the
// feasible ends of row i form a prefix (i, jlim(i)] found by binary search;
// the relaxation loop then carries no memory test.
#include <cstring>

#include "heddle_internal.h"

namespace heddle {

// ----------------------------------------------------------------- helpers

__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int rl32(int v, int lane) { return __builtin_amdgcn_readlane(v, lane); }

__device__ __forceinline__ int64_t rl64(int64_t v, int lane)
{
    uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), lane);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

template <class T> __device__ __forceinline__ T wave_min(T v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        T u = __shfl_xor(v, o);
        v = u < v ? u : v;
    }
    return v;
}

template <class T> __device__ __forceinline__ T wave_max(T v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        T u = __shfl_xor(v, o);
        v = u > v ? u : v;
    }
    return v;
}

template <class T> __device__ __forceinline__ T wave_sum(T v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// Nearest value with at most 24 significant bits (ties to even) of a
// non-negative integer: the fp32 rounding of x, kept as an exact integer.
__device__ __forceinline__ uint64_t rne24(uint64_t x)
{
    if (x < (1ull << 24)) return x;
    const int sh = 40 - __clzll(x);            // bits dropped: top bit lands at position 23
    const uint64_t q = x >> sh, r = x & ((1ull << sh) - 1), half = 1ull << (sh - 1);
    const uint64_t qr = q + ((r > half || (r == half && (q & 1))) ? 1 : 0);
    return qr << sh;
}

// float of an integer with at most 24 significant bits, times 2^e
__device__ __forceinline__ float exact_float(uint64_t x, int e)
{
    if (x == 0) return 0.0f;
    const int sh = x < (1ull << 24) ? 0 : 40 - __clzll(x);
    return ldexpf((float)(uint32_t)(x >> sh), sh + e);
}

// ceil(2 (n-1) b * 1000 / (n bw)): ring all-reduce of b bytes over n ranks
__device__ __forceinline__ int64_t allreduce_ns(int64_t b, int64_t n, int64_t bw)
{
    if (n <= 1 || b == 0) return 0;
    const unsigned __int128 num = (unsigned __int128)(uint64_t)(2 * (n - 1)) * (uint64_t)b * 1000u;
    const unsigned __int128 den = (unsigned __int128)(uint64_t)n * (uint64_t)bw;
    return (int64_t)((num + den - 1) / den);
}

__device__ __forceinline__ int nibble(uint64_t w, int l) { return (int)((w >> (4 * l)) & 15); }

// Per-lane (lane = stage s) decoded record and stage constants.
struct StageInfo {
    int status;          // uniform: HEDDLE_S_* of the template (0 if valid)
    int S, D;            // uniform
    int g, tp, ep, ki, ei;
    int64_t a2a, p2p;    // all-to-all per MoE layer, outbound p2p (ns, or fixed-point for fp32)
    int64_t a2a_ns, p2p_ns;
    int64_t cap, bw_dp;
    int trow, srow, arow; // offsets of the stage's rows in the prefix tables
};

// Template decode and validation (feasibility masks of section 5.1; exact
// profile match of section 5.2). Checks run in status order over all stages.
template <bool F32>
__device__ StageInfo decode(const DevProfile &P, const PriceArgs &A, int64_t t, int lane)
{
    StageInfo x;
    const int L = P.L, R = L + 1;
    x.S = A.n_stages[t];
    x.status = 0;
    x.D = 1;
    const bool act = lane < x.S && lane < A.s_max;
    const uint32_t rec = act ? A.stages[t * A.s_max + lane] : 0u;
    x.g = rec & 0xFF;
    const int l2tp = (rec >> 8) & 15, l2ep = (rec >> 12) & 15;
    const int dpv = (int)(rec >> 16);
    x.tp = 1 << l2tp;
    x.ep = 1 << l2ep;
    x.ki = nibble(P.tp_index, l2tp);
    x.ei = nibble(P.ep_index, l2ep);
    x.a2a = x.p2p = x.a2a_ns = x.p2p_ns = x.cap = x.bw_dp = 0;
    x.trow = x.srow = x.arow = 0;
    if (x.S < 1 || x.S > A.s_max || x.S > L) { x.status = HEDDLE_S_BAD_SHAPE; return x; }
    if (__ballot(act && x.g >= P.n_types)) { x.status = HEDDLE_S_BAD_TYPE; return x; }
    const int node = act ? P.node_size[x.g] : 0;
    if (__ballot(act && (!((P.tp_present >> l2tp) & 1) || x.tp > node))) { x.status = HEDDLE_S_BAD_TP; return x; }
    if (__ballot(act && !P.profiled[x.g * P.n_tp + x.ki])) { x.status = HEDDLE_S_UNPROFILED; return x; }
    x.D = rl32(dpv, 0);
    if (__ballot(act && (dpv < 1 || dpv != x.D))) { x.status = HEDDLE_S_BAD_DP; return x; }
    if (__ballot(act && (!((P.ep_present >> l2ep) & 1) || (x.D % x.ep) != 0))) { x.status = HEDDLE_S_BAD_EP; return x; }
    int64_t used = 0;
    for (int s2 = 0; s2 < x.S; s2++)
        if (rl32(x.g, s2) == x.g) used += rl32(x.tp, s2);
    if (__ballot(act && used * x.D > P.n_gpus[x.g])) { x.status = HEDDLE_S_OVERSUBSCRIBED; return x; }

    // stage constants
    const int N = P.n_types;
    const int gn = __shfl(x.g, lane + 1 < 64 ? lane + 1 : 63);
    if (act) {
        const int var = x.ep == 1 ? 0 : (x.ep * x.tp <= node ? 1 : 2);
        x.a2a_ns = P.a2a_ns[x.g * 3 + var];
        x.p2p_ns = lane < x.S - 1 ? P.p2p_ns[x.g * N + gn] : 0;
        x.a2a = F32 ? P.a2a_fx[x.g * 3 + var] : x.a2a_ns;
        x.p2p = lane < x.S - 1 ? (F32 ? P.p2p_fx[x.g * N + gn] : x.p2p_ns) : 0;
        x.cap = P.mem_cap[x.g];
        x.bw_dp = (int64_t)x.tp * x.D <= node ? P.intra_bw[x.g] : P.link_bw[x.g * N + x.g];
        x.trow = (x.g * P.n_tp + x.ki) * R;
        x.srow = (x.ki * P.n_ep + x.ei) * R;
        x.arow = x.ki * R;
    }
    return x;
}

// Largest end j in [i, jhi] such that stage layers [i, j) fit the cap with
// `f` micro-batches of activations in flight (j = i always "fits").
__device__ __forceinline__ int mem_limit(const int64_t *w, const int64_t *a, int64_t f, int64_t cap, int i, int jhi)
{
    const int64_t wi = w[i], ai = a[i];
    int lo = i, hi = jhi;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((w[mid] - wi) + f * (a[mid] - ai) <= cap) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

template <class V> struct DPInf { static constexpr V value = ~V(0); };

// ------------------------------------------------------------ price kernel

template <class V, bool F32, bool COUNT>
__global__ void __launch_bounds__(256) price_kernel(DevProfile P, PriceArgs A)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63, wib = threadIdx.x >> 6, wpb = blockDim.x >> 6;
    const int L = P.L, gs = A.g_stride;
    const bool compute_only = (A.flags & HEDDLE_F_COMPUTE_ONLY) != 0;
    const V INF = DPInf<V>::value;
    V *G = (V *)(smem + (size_t)wib * A.lds_per_wave);
    const int64_t *time_tab = F32 ? P.pre_time_fx : P.pre_time;

    int my_m = 1;                        // lane k holds the k-th micro-batch count
    for (int k = 0; k < A.n_m; k++) my_m = lane == k ? A.m[k] : my_m;
    unsigned long long work = 0;

    for (int64_t t = (int64_t)blockIdx.x * wpb + wib; t < A.n; t += (int64_t)gridDim.x * wpb) {
        const StageInfo x = decode<F32>(P, A, t, lane);
        const int S = x.S;
        const size_t obase = (size_t)t * A.n_m;
        if (x.status != 0) {
            if (!COUNT) {
                for (int k = lane; k < A.n_m; k += 64) {
                    A.status[obase + k] = (uint8_t)x.status;
                    if (F32) {
                        ((float *)A.iter)[obase + k] = __builtin_inff();
                        ((float *)A.bottleneck)[obase + k] = __builtin_inff();
                    } else {
                        ((int64_t *)A.iter)[obase + k] = INT64_MAX;
                        ((int64_t *)A.bottleneck)[obase + k] = INT64_MAX;
                    }
                    A.peak_mem[obase + k] = INT64_MAX;
                }
                for (int q = lane; q < A.n_m * A.s_max; q += 64) A.layers[obase * A.s_max + q] = 0;
            }
            continue;
        }
        const int D = x.D;
        // in-flight key of each micro-batch count: min(M_p, S) decides the split
        const int64_t Mp_k = ((int64_t)my_m + D - 1) / D;
        const int key_k = compute_only ? 0 : (int)(Mp_k < S ? Mp_k : S);
        uint64_t todo = __ballot(lane < A.n_m);

        while (todo) {
            const int key = wave_min(((todo >> lane) & 1) ? key_k : 0x7FFFFFFF);
            const uint64_t cls = __ballot(lane < A.n_m && key_k == key) & todo;
            todo &= ~cls;

            // ---------------- PartitionLayers: suffix min-max DP
            for (int s = S - 1; s >= 0; s--) {
                const int64_t *trow = time_tab + rl32(x.trow, s);
                const int64_t a2a = rl64(x.a2a, s), cap = rl64(x.cap, s);
                const V p2p = (V)rl64(x.p2p, s);
                const int64_t *wrow = P.pre_state + rl32(x.srow, s);
                const int64_t *arow = P.pre_act + rl32(x.arow, s);
                const int64_t f = (S - s) < key ? (S - s) : key;
                const int jhi = L - (S - 1 - s);
                const int ihi = (s == 0) ? 0 : L - (S - s);
                V *prow = G + (size_t)S * gs;           // time prefix of stage s
                V *Gs = G + (size_t)s * gs, *Gn = G + (size_t)(s + 1) * gs;
                for (int j = lane; j <= L; j += 64) prow[j] = (V)(trow[j] + a2a * P.pre_moe[j]);
                wave_sync();
                if (s == S - 1) {
                    for (int i = s + lane; i <= ihi; i += 64) {
                        const bool fit = compute_only || (wrow[L] - wrow[i]) + f * (arow[L] - arow[i]) <= cap;
                        if (COUNT) work += fit ? 1 : 0;
                        else Gs[i] = fit ? (V)(prow[L] - prow[i]) : INF;
                    }
                } else if (s > 0) {
                    for (int i = s + lane; i <= ihi; i += 64) {
                        const int jl = compute_only ? jhi : mem_limit(wrow, arow, f, cap, i, jhi);
                        if (COUNT) { work += (unsigned long long)(jl - i); continue; }
                        const V pi = prow[i];
                        V acc = INF;
                        for (int j = i + 1; j <= jl; j++) {
                            const V tt = prow[j] - pi + p2p;
                            const V gn = Gn[j];
                            const V c = tt > gn ? tt : gn;
                            acc = c < acc ? c : acc;
                        }
                        Gs[i] = acc;
                    }
                } else {                                   // stage 0: row 0 only, lanes split the ends
                    const int jl = compute_only ? jhi : mem_limit(wrow, arow, f, cap, 0, jhi);
                    if (COUNT) {
                        if (lane == 0) work += (unsigned long long)jl;
                    } else {
                        V acc = INF;
                        for (int j = 1 + lane; j <= jl; j += 64) {
                            const V tt = prow[j] - prow[0] + p2p;
                            const V gn = Gn[j];
                            const V c = tt > gn ? tt : gn;
                            acc = c < acc ? c : acc;
                        }
                        acc = wave_min(acc);
                        if (lane == 0) Gs[0] = acc;
                    }
                }
                wave_sync();
            }
            if (COUNT) continue;

            const V Bv = G[0];
            if (Bv == INF) {                               // no split fits memory
                for (uint64_t c = cls; c; c &= c - 1) {
                    const int k = __ffsll((unsigned long long)c) - 1;
                    if (lane == 0) {
                        A.status[obase + k] = HEDDLE_S_OOM;
                        if (F32) {
                            ((float *)A.iter)[obase + k] = __builtin_inff();
                            ((float *)A.bottleneck)[obase + k] = __builtin_inff();
                        } else {
                            ((int64_t *)A.iter)[obase + k] = INT64_MAX;
                            ((int64_t *)A.bottleneck)[obase + k] = INT64_MAX;
                        }
                        A.peak_mem[obase + k] = INT64_MAX;
                    }
                    for (int q = lane; q < A.s_max; q += 64) A.layers[(obase + k) * A.s_max + q] = 0;
                }
                continue;
            }
            const uint64_t B = (uint64_t)Bv;
            const uint64_t B24 = F32 ? rne24(B) : B;      // fp32 bottleneck, as an exact integer

            // ---------------- canonical reconstruction: smallest feasible end per stage
            int cs = 0, my_start = 0, my_end = 0;
            for (int s = 0; s < S; s++) {
                const int64_t *trow = time_tab + rl32(x.trow, s);
                const int64_t a2a = rl64(x.a2a, s), p2p = rl64(x.p2p, s), cap = rl64(x.cap, s);
                const int64_t *wrow = P.pre_state + rl32(x.srow, s);
                const int64_t *arow = P.pre_act + rl32(x.arow, s);
                const int64_t f = (S - s) < key ? (S - s) : key;
                const int jhi = L - (S - 1 - s);
                const V *Gn = G + (size_t)(s + 1) * gs;
                const int64_t wi = wrow[cs], ai = arow[cs], ti = trow[cs] + a2a * P.pre_moe[cs];
                int found = -1;
                for (int base = cs + 1; base <= jhi && found < 0; base += 64) {
                    const int j = base + lane;
                    bool ok = false;
                    if (j <= jhi) {
                        const uint64_t T = (uint64_t)(trow[j] + a2a * P.pre_moe[j] - ti + p2p);
                        bool rest_ok;                      // the later stages complete within B*
                        if (s == S - 1) {
                            rest_ok = j == L;
                        } else {
                            const V gv = Gn[j];
                            rest_ok = gv != INF && (F32 ? rne24((uint64_t)gv) <= B24 : (uint64_t)gv <= B);
                        }
                        const bool fit = compute_only || (wrow[j] - wi) + f * (arow[j] - ai) <= cap;
                        ok = fit && rest_ok && (F32 ? rne24(T) <= B24 : T <= B);
                    }
                    const uint64_t bal = __ballot(ok);
                    if (bal) found = base + __ffsll((unsigned long long)bal) - 1;
                }
                // an end always exists: the DP value G[s][cs] <= B* has a witness.
                // The clamp only keeps indexing in bounds should that ever fail.
                if (found < 0) found = jhi;
                if (lane == s) { my_start = cs; my_end = found; }
                cs = found;
            }

            // ---------------- Evaluate (lane = stage), once per micro-batch count of this class
            const bool act = lane < S;
            int64_t Tst = 0, gsync = 0, wdiff = 0, adiff = 0;
            if (act) {
                const int i = my_start, j = my_end;
                const int64_t *trow = time_tab + x.trow;
                Tst = trow[j] - trow[i] + x.a2a * (P.pre_moe[j] - P.pre_moe[i]) + x.p2p;
                wdiff = P.pre_state[x.srow + j] - P.pre_state[x.srow + i];
                adiff = P.pre_act[x.arow + j] - P.pre_act[x.arow + i];
                const int64_t gd = P.pre_grad[x.arow + j] - P.pre_grad[x.arow + i];
                const int64_t gx = P.pre_xgrad[x.srow + j] - P.pre_xgrad[x.srow + i];
                gsync = allreduce_ns(gd, D, x.bw_dp) + allreduce_ns(gx, D / x.ep, x.bw_dp);
            }
            const int64_t sumT = wave_sum(act ? (int64_t)(F32 ? rne24((uint64_t)Tst) : (uint64_t)Tst) : int64_t(0));
            const int64_t maxg = wave_max(gsync);
            const int64_t maxg_v = F32 ? (int64_t)(rne24((uint64_t)maxg) << (-P.fx_exp)) : maxg;
            for (uint64_t c = cls; c; c &= c - 1) {
                const int k = __ffsll((unsigned long long)c) - 1;
                const int64_t m = rl32(my_m, k);
                const int64_t Mp = (m + D - 1) / D;
                const int64_t fl = (int64_t)(S - lane) < Mp ? (int64_t)(S - lane) : Mp;
                const int64_t mem = act ? wdiff + fl * adiff : 0;
                const bool oom = act && mem > x.cap;
                const int64_t peak = wave_max(mem);
                const bool any_oom = __ballot(oom) != 0;
                const int64_t iter = (Mp - 1) * (int64_t)B24 + sumT + maxg_v;
                if (lane == 0) {
                    A.status[obase + k] = any_oom ? HEDDLE_S_OOM : HEDDLE_S_OK;
                    if (F32) {
                        ((float *)A.iter)[obase + k] = exact_float(rne24((uint64_t)iter), P.fx_exp);
                        ((float *)A.bottleneck)[obase + k] = exact_float(B24, P.fx_exp);
                    } else {
                        ((int64_t *)A.iter)[obase + k] = iter;
                        ((int64_t *)A.bottleneck)[obase + k] = (int64_t)B;
                    }
                    A.peak_mem[obase + k] = peak;
                }
                for (int q = lane; q < A.s_max; q += 64)
                    A.layers[(obase + k) * A.s_max + q] = q < S ? (uint8_t)(my_end - my_start) : 0;
            }
        }
    }
    if (COUNT) {
        work = wave_sum(work);
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
static int launch_t(const heddle_profile *p, PriceArgs &a, hipStream_t stream)
{
    const int L = p->dev.L;
    const int s_cap = a.s_max < L ? a.s_max : L;
    a.g_stride = L + 1;
    // DP rows for stages 0..S-1, row S holds the stage's time prefix
    a.lds_per_wave = (int32_t)(((size_t)(s_cap + 1) * a.g_stride * sizeof(V) + 15) & ~size_t(15));
    int max_lds = 0;
    HEDDLE_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, p->device));
    int wpb = max_lds / a.lds_per_wave;
    wpb = wpb > 4 ? 4 : (wpb < 1 ? 1 : wpb);
    const size_t lds = (size_t)wpb * a.lds_per_wave;
    if (lds > (size_t)max_lds) return fail(HEDDLE_E_RANGE, "DP table of this (L, s_max) does not fit in LDS");
    if (lds > 65536)
        HEDDLE_HIP(hipFuncSetAttribute((const void *)price_kernel<V, F32, COUNT>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
    const int64_t want = (a.n + wpb - 1) / wpb;
    const int blocks = (int)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL((price_kernel<V, F32, COUNT>), dim3(blocks), dim3(64 * wpb), lds, stream, p->dev, a);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

int launch_price(const heddle_profile *p, PriceArgs &a, hipStream_t stream, bool count_only)
{
    if (a.n == 0) return HEDDLE_OK;
    const bool f32 = a.flags & HEDDLE_F_FP32;
    const bool narrow = f32 ? p->narrow_f32 : p->narrow_i64;
    if (count_only) return launch_t<uint64_t, false, true>(p, a, stream);
    if (f32) return narrow ? launch_t<uint32_t, true, false>(p, a, stream) : launch_t<uint64_t, true, false>(p, a, stream);
    return narrow ? launch_t<uint32_t, false, false>(p, a, stream) : launch_t<uint64_t, false, false>(p, a, stream);
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
