// Batched plan pricing on gfx950: template decode and validation,
// PartitionLayers (exact min-max layer split), canonical reconstruction and
// Evaluate (1F1B iteration time and per-GPU peak memory).
//
// Method: Heddle (arXiv 2609.34244). The layer split is the PartitionLayers
// step of the planners' nested-loop backbone (section 3.1), aware of per-stage
// GPU speed (the straggler criticism of speed-blind splits in the same
// section) and of memory (section 5.2, memory validation). Evaluate is the
// profile-based cost model of section 5.2 with the 1F1B iteration time
// (M-1) max_s t_s + sum_s t_s + max_s g_s of section 5.3.
//
// Recurrence (suffix form): G[s][i] is the smallest achievable bottleneck
// when stages s..S-1 hold layers [i, L):
//   G[S-1][i] = T(S-1, i, L)                                    if it fits
//   G[s][i]   = min over i < j <= jlim_s(i) of max(T(s,i,j), G[s+1][j])
// with jlim_s(i) the largest end that fits memory (and leaves one layer per
// later stage); B* = G[0][0]. Memory grows with j for fixed i, so the
// feasible ends of a row form the prefix (i, jlim_s(i)].
//
// Mapping. One wavefront prices one template at a time (grid-stride over
// templates). Lanes are pipeline stages for decode, validation and Evaluate,
// and split rows i of one stage during the DP, each lane walking its own ends
// j. Per wavefront LDS holds, for every stage s, the pairs
//   X[s][j] = { P_s[j], G[s+1][j] }
// where P_s is the stage's time prefix (layer costs + MoE all-to-all), so one
// 64-bit LDS read feeds one relaxation (sub, max, min); the stage's memory
// prefix U; and the memory limits jlim_s(i) as bytes, which the
// reconstruction reuses. The profile rows of the next stage are fetched from
// global memory into registers while the current stage relaxes.
#include <cstring>

#include "exact_math.h"
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
// non-negative integer below 2^63: its fp32 rounding, kept as an exact integer.
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

__device__ __forceinline__ int nibble(uint64_t w, int l) { return (int)((w >> (4 * l)) & 15); }

template <class V> struct Vec2;
template <> struct Vec2<uint32_t> { typedef uint32_t type __attribute__((ext_vector_type(2))); };
template <> struct Vec2<uint64_t> { typedef uint64_t type __attribute__((ext_vector_type(2))); };
template <class V> struct DPInf { static constexpr V value = ~V(0); };

// Per-lane (lane = stage s) decoded record and stage constants.
struct StageInfo {
    int status;              // uniform: HEDDLE_S_* of the template (0 if valid)
    int S, D;                // uniform
    int tp, ep;
    int64_t a2a, p2p;        // all-to-all per MoE layer, outbound p2p (ns, or fixed point for fp32)
    int64_t cap, bw_dp;
    int trow, srow, arow;    // offsets of the stage's rows in the prefix tables
    int lrow;                // offset of the stage's memory-limit rows (in-flight count 1)
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
    const bool act = lane < x.S && lane < A.s_max;
    const uint32_t rec = act ? A.stages[t * A.s_max + lane] : 0u;
    const int g = rec & 0xFF;
    const int l2tp = (rec >> 8) & 15, l2ep = (rec >> 12) & 15;
    const int dpv = (int)(rec >> 16);
    x.tp = 1 << l2tp;
    x.ep = 1 << l2ep;
    const int ki = nibble(P.tp_index, l2tp), ei = nibble(P.ep_index, l2ep);
    const int gc = g < N ? g : N - 1;                          // clamped for speculative reads
    const int gn = __shfl(gc, lane + 1 < 64 ? lane + 1 : 63);
    const int node = P.node_size[gc];
    const int prof = P.profiled[gc * P.n_tp + ki];
    const int ngpu = P.n_gpus[gc];
    const int var = x.ep == 1 ? kA2ANone : (x.ep * x.tp <= node ? kA2AIntra : kA2AInter);
    const int64_t a2a = F32 ? P.a2a_fx[gc * 3 + var] : P.a2a_ns[gc * 3 + var];
    const int64_t p2p = F32 ? P.p2p_fx[gc * N + gn] : P.p2p_ns[gc * N + gn];
    const int64_t cap = P.mem_cap[gc], intra = P.intra_bw[gc], self = P.link_bw[gc * N + gc];

    x.a2a = x.p2p = x.cap = x.bw_dp = 0;
    x.trow = x.srow = x.arow = x.lrow = 0;
    if (x.S < 1 || x.S > A.s_max || x.S > L) { x.status = HEDDLE_S_BAD_SHAPE; return x; }
    if (__ballot(act && g >= N)) { x.status = HEDDLE_S_BAD_TYPE; return x; }
    if (__ballot(act && (!((P.tp_present >> l2tp) & 1) || x.tp > node))) { x.status = HEDDLE_S_BAD_TP; return x; }
    if (__ballot(act && !prof)) { x.status = HEDDLE_S_UNPROFILED; return x; }
    x.D = rl32(dpv, 0);
    if (__ballot(act && (dpv < 1 || dpv != x.D))) { x.status = HEDDLE_S_BAD_DP; return x; }
    if (__ballot(act && (!((P.ep_present >> l2ep) & 1) || ((uint32_t)x.D % (uint32_t)x.ep) != 0))) {
        x.status = HEDDLE_S_BAD_EP;
        return x;
    }
    int used = 0;                                              // this lane's type: sum of TP over its stages
    for (int s2 = 0; s2 < x.S; s2++)
        if (rl32(g, s2) == g) used += rl32(x.tp, s2);
    if (__ballot(act && (int64_t)used * x.D > ngpu)) { x.status = HEDDLE_S_OVERSUBSCRIBED; return x; }

    if (act) {
        x.a2a = a2a;
        x.p2p = lane < x.S - 1 ? p2p : 0;
        x.cap = cap;
        x.bw_dp = (int64_t)x.tp * x.D <= node ? intra : self;
        x.trow = (g * P.n_tp + ki) * R;
        x.srow = (ki * P.n_ep + ei) * R;
        x.arow = ki * R;
        x.lrow = ((g * P.n_tp + ki) * P.n_ep + ei) * P.n_f * R;
    }
    return x;
}

// Profile rows of one stage, fetched into registers ahead of use: the time
// prefix, the MoE prefix count and the memory limits of every row.
constexpr int kRowSlots = 4;                       // (L + 1) <= 256 entries, 64 per slot
struct RowRegs {
    int64_t t[kRowSlots];
    int32_t m[kRowSlots];
    int32_t l[kRowSlots];
};

__device__ __forceinline__ void fetch_rows(RowRegs &r, const int64_t *trow, const int32_t *moe,
                                           const uint8_t *lrow, int L, int lane, bool need_mem)
{
#pragma unroll
    for (int q = 0; q < kRowSlots; q++) {
        const int j = lane + 64 * q;
        if (j <= L) {
            r.t[q] = trow[j];
            r.m[q] = moe[j];
            r.l[q] = need_mem ? lrow[j] : L;
        }
    }
}

// ------------------------------------------------------------ price kernel

template <class V, bool F32, bool COUNT>
__global__ void __launch_bounds__(256) price_kernel(DevProfile P, PriceArgs A)
{
    typedef typename Vec2<V>::type V2;
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63, wib = threadIdx.x >> 6, wpb = blockDim.x >> 6;
    const int L = P.L, gs = A.g_stride;
    const bool compute_only = (A.flags & HEDDLE_F_COMPUTE_ONLY) != 0;
    const V INF = DPInf<V>::value;
    unsigned char *wave_lds = smem + (size_t)wib * A.lds_per_wave;
    V2 *X = (V2 *)wave_lds;                                   // [s_cap][gs] pairs {P_s, G_{s+1}}
    uint8_t *J = wave_lds + A.off_j;                          // [s_cap][gs] memory limits
    const int64_t *time_tab = F32 ? P.pre_time_fx : P.pre_time;

    int my_m = 1;                                             // lane k: the k-th micro-batch count
    for (int k = 0; k < A.n_m; k++) my_m = lane == k ? A.m[k] : my_m;
    unsigned long long work = 0;

    for (int64_t t = (int64_t)blockIdx.x * wpb + wib; t < A.n; t += (int64_t)gridDim.x * wpb) {
        const StageInfo x = decode<F32>(P, A, t, lane);
        const int S = x.S;
        const size_t obase = (size_t)t * A.n_m;
        // results of m index k live in lane k until the end of the template
        bool r_priced = false, r_oom = false;
        int64_t r_iter = INT64_MAX, r_bn = INT64_MAX, r_peak = INT64_MAX;
        float r_iter_f = __builtin_inff(), r_bn_f = __builtin_inff();

        if (x.status == 0) {
            const int D = x.D;
            // micro-batches per replica M_p = ceil(m / D); min(M_p, S) fixes the split
            const int Mp_k = (int)(((uint32_t)my_m + (uint32_t)D - 1) / (uint32_t)D);
            const int key_k = compute_only ? 0 : (Mp_k < S ? Mp_k : S);
            uint64_t todo = __ballot(lane < A.n_m);

            while (todo) {
                const int key = wave_min(((todo >> lane) & 1) ? key_k : 0x7FFFFFFF);
                const uint64_t cls = __ballot(lane < A.n_m && key_k == key) & todo;
                todo &= ~cls;

                // ---------------- PartitionLayers: suffix min-max DP, stages S-1 .. 0
                const int R = L + 1;
                auto lim_row = [&](int s) {                 // memory limits of stage s at this class
                    const int f = (S - s) < key ? (S - s) : key;
                    return P.mem_lim + rl32(x.lrow, s) + (size_t)(f - 1) * R;
                };
                RowRegs rr;
                fetch_rows(rr, time_tab + rl32(x.trow, S - 1), P.pre_moe, lim_row(S - 1), L, lane, !compute_only);
                V Bv = INF;
                for (int s = S - 1; s >= 0; s--) {
                    const int64_t a2a = rl64(x.a2a, s);
                    const V p2p = (V)rl64(x.p2p, s);
                    const int jhi = L - (S - 1 - s);
                    const int ihi = (s == 0) ? 0 : L - (S - s);
                    V2 *Xs = X + (size_t)s * gs;
                    // commit the fetched rows of stage s to LDS: the time prefix, and
                    // the last admissible end of every row (memory limit, and room
                    // for one layer per later stage)
                    uint8_t *Js = J + (size_t)s * gs;
#pragma unroll
                    for (int q = 0; q < kRowSlots; q++) {
                        const int j = lane + 64 * q;
                        if (j <= L) {
                            ((V *)&Xs[j])[0] = (V)(rr.t[q] + a2a * rr.m[q]);
                            Js[j] = (uint8_t)(rr.l[q] < jhi ? rr.l[q] : jhi);
                        }
                    }
                    if (s > 0) fetch_rows(rr, time_tab + rl32(x.trow, s - 1), P.pre_moe, lim_row(s - 1), L, lane, !compute_only);
                    wave_sync();
                    if (s == S - 1) {
                        // last stage: its rows must end at L
                        for (int i = s + lane; i <= ihi; i += 64) {
                            const bool fit = Js[i] == L;
                            if (COUNT) {
                                work += fit ? 1 : 0;
                            } else {
                                const V gv = fit ? (V)(((V *)&Xs[L])[0] - ((V *)&Xs[i])[0]) : INF;
                                if (s > 0) ((V *)&X[(size_t)(s - 1) * gs + i])[1] = gv;
                                else Bv = gv;                   // S = 1: row 0, lane 0
                            }
                        }
                    } else if (s > 0) {
                        // rows of a middle stage: lane = row i relaxes its admissible ends
                        // (i, jl], four per step (X is padded by four entries)
                        V2 *Xp = X + (size_t)(s - 1) * gs;
                        for (int i = s + lane; i <= ihi; i += 64) {
                            const int jl = Js[i];
                            if (COUNT) {
                                work += (unsigned long long)(jl - i);
                                continue;
                            }
                            const V pi = ((V *)&Xs[i])[0] - p2p;        // T(s,i,j) = P_s[j] - pi
                            V acc = INF;
                            for (int j = i + 1; j <= jl; j += 4) {
                                const int rem = jl - j;                  // ends beyond j still admissible
                                const V2 a = Xs[j], b = Xs[j + 1], c = Xs[j + 2], d = Xs[j + 3];
                                const V ta = a.x - pi, tb = b.x - pi, tc = c.x - pi, td = d.x - pi;
                                const V ca = ta > a.y ? ta : a.y;
                                const V cb = rem >= 1 ? (tb > b.y ? tb : b.y) : INF;
                                const V cc = rem >= 2 ? (tc > c.y ? tc : c.y) : INF;
                                const V cd = rem >= 3 ? (td > d.y ? td : d.y) : INF;
                                const V m1 = ca < cb ? ca : cb, m2 = cc < cd ? cc : cd;
                                const V m3 = m1 < m2 ? m1 : m2;
                                acc = m3 < acc ? m3 : acc;
                            }
                            ((V *)&Xp[i])[1] = acc;
                        }
                    } else {
                        // stage 0 (S > 1): row 0 only; the lanes split its ends
                        const int jl = Js[0];
                        if (COUNT) {
                            if (lane == 0) work += (unsigned long long)jl;
                        } else {
                            const V pi = ((V *)&Xs[0])[0] - p2p;
                            V acc = INF;
                            for (int j = 1 + lane; j <= jl; j += 64) {
                                const V2 a = Xs[j];
                                const V ta = a.x - pi;
                                const V ca = ta > a.y ? ta : a.y;
                                acc = ca < acc ? ca : acc;
                            }
                            Bv = wave_min(acc);
                        }
                    }
                    wave_sync();
                }
                if (COUNT) continue;
                if (S == 1) Bv = (V)rl64((int64_t)Bv, 0);      // computed by lane 0 only
                if (Bv == INF) {                              // no split fits memory
                    if ((cls >> lane) & 1) r_oom = true;
                    continue;
                }
                const uint64_t B = (uint64_t)Bv;
                const uint64_t B24 = F32 ? rne24(B) : B;      // fp32 bottleneck, as an exact integer

                // ---------------- canonical reconstruction: smallest admissible end per stage
                int cs = 0, my_start = 0, my_end = 0;
                for (int s = 0; s < S; s++) {
                    const V2 *Xs = X + (size_t)s * gs;
                    const V pc = ((const V *)&Xs[cs])[0] - (V)rl64(x.p2p, s);
                    const int jl = J[(size_t)s * gs + cs];
                    int found = -1;
                    for (int base = cs + 1; base <= jl && found < 0; base += 64) {
                        const int j = base + lane;
                        bool ok = false;
                        if (j <= jl) {
                            const V2 a = Xs[j];
                            const uint64_t T = (uint64_t)(V)(a.x - pc);
                            bool rest_ok;                     // the later stages complete within B*
                            if (s == S - 1) rest_ok = j == L;
                            else rest_ok = a.y != INF && (F32 ? rne24((uint64_t)a.y) <= B24 : (uint64_t)a.y <= B);
                            ok = rest_ok && (F32 ? rne24(T) <= B24 : T <= B);
                        }
                        const uint64_t bal = __ballot(ok);
                        if (bal) found = base + __ffsll((unsigned long long)bal) - 1;
                    }
                    // an end always exists (G[s][cs] <= B* has a witness); the clamp
                    // only keeps indexing in bounds should that ever fail
                    if (found < 0) found = jl;
                    if (lane == s) {
                        my_start = cs;
                        my_end = found;
                    }
                    cs = found;
                }

                // ---------------- Evaluate (lane = stage) for the m values of this class
                const bool act = lane < S;
                uint64_t Tst = 0;
                int64_t gsync = 0, wdiff = 0, adiff = 0;
                if (act) {
                    const int i = my_start, j = my_end;
                    const V2 *Xs = X + (size_t)lane * gs;
                    Tst = (uint64_t)(V)(((const V *)&Xs[j])[0] - ((const V *)&Xs[i])[0] + (V)x.p2p);
                    wdiff = P.pre_state[x.srow + j] - P.pre_state[x.srow + i];
                    adiff = P.pre_act[x.arow + j] - P.pre_act[x.arow + i];
                    const int64_t gd = P.pre_grad[x.arow + j] - P.pre_grad[x.arow + i];
                    const int64_t gx = P.pre_xgrad[x.srow + j] - P.pre_xgrad[x.srow + i];
                    gsync = allreduce_ns(gd, D, x.bw_dp) + allreduce_ns(gx, (int64_t)((uint32_t)D / (uint32_t)x.ep), x.bw_dp);
                }
                const int64_t sumT = wave_sum(act ? (int64_t)(F32 ? rne24(Tst) : Tst) : int64_t(0));
                const int64_t maxg = wave_max(gsync);
                const int64_t maxg_v = F32 ? (int64_t)(rne24((uint64_t)maxg) << (-P.fx_exp)) : maxg;
                for (uint64_t c = cls; c; c &= c - 1) {
                    const int k = __ffsll((unsigned long long)c) - 1;
                    const int64_t Mp = rl32(Mp_k, k);
                    const int64_t fl = (int64_t)(S - lane) < Mp ? (int64_t)(S - lane) : Mp;
                    const int64_t mem = act ? wdiff + fl * adiff : 0;
                    const int64_t peak = wave_max(mem);
                    const bool any_oom = __ballot(act && mem > x.cap) != 0;
                    const int64_t iter = (Mp - 1) * (int64_t)B24 + sumT + maxg_v;
                    if (lane == k) {
                        r_priced = true;
                        r_oom = any_oom;
                        r_peak = peak;
                        if (F32) {
                            r_iter_f = exact_float(rne24((uint64_t)iter), P.fx_exp);
                            r_bn_f = exact_float(B24, P.fx_exp);
                        } else {
                            r_iter = iter;
                            r_bn = (int64_t)B;
                        }
                    }
                    for (int q = lane; q < A.s_max; q += 64)
                        A.layers[(obase + k) * A.s_max + q] = q < S ? (uint8_t)(my_end - my_start) : 0;
                }
            }
        }
        if (COUNT) continue;
        if (lane < A.n_m) {
            const size_t o = obase + lane;
            A.status[o] = (uint8_t)(x.status != 0 ? x.status : (r_oom ? HEDDLE_S_OOM : HEDDLE_S_OK));
            if (F32) {
                ((float *)A.iter)[o] = r_iter_f;
                ((float *)A.bottleneck)[o] = r_bn_f;
            } else {
                ((int64_t *)A.iter)[o] = r_iter;
                ((int64_t *)A.bottleneck)[o] = r_bn;
            }
            A.peak_mem[o] = r_peak;
        }
        // zero layer counts of the plans without a split (invalid template, or no split fits)
        const uint64_t priced = __ballot(r_priced);
        if (priced != __ballot(lane < A.n_m))
            for (int q = lane; q < A.n_m * A.s_max; q += 64)
                if (!((priced >> (q / A.s_max)) & 1)) A.layers[obase * A.s_max + q] = 0;
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
    a.s_cap = a.s_max < L ? a.s_max : L;
    a.g_stride = L + 5;                                       // L + 1 ends and 4 of padding
    // per wavefront: pairs {P_s, G_{s+1}} and the end limits of every stage
    const size_t j_off = (size_t)a.s_cap * a.g_stride * 2 * sizeof(V);
    a.off_j = (int32_t)j_off;
    a.lds_per_wave = (int32_t)((j_off + (size_t)a.s_cap * a.g_stride + 15) & ~size_t(15));
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
