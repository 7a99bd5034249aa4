// Distribute on gfx950: Heddle's own layer split (arXiv 2609.34244, section
// 5.3, layer split and DP degree) as a second partition mode of
// heddle_price_plans, with its Evaluate.
//
// Every stage gets layers in proportion to its profiled speed. The speed of
// stage s is the inverse of the time of all L layers on its GPU type and TP
// degree (int64 layer costs with the stage's all-to-all terms, p2p
// excluded); the cut after stage s is the nearest integer (halves up) to
// L * (speed of stages 0..s) / (speed of all stages), computed in IEEE double
// in that order, then raised to leave stage s a layer and lowered to leave
// every later stage one. When that split does not fit memory, a fixed list of
// alternatives is priced: for each boundary in order, its cut moved by -1,
// then by +1 (kept only if every stage still holds a layer); the fitting one
// with the smallest iteration time is kept, the first on ties, and none
// fitting leaves the plan OOM without a split. With HEDDLE_F_COMPUTE_ONLY the
// proportional split is kept and only flagged.
//
// Mapping: one wavefront per template (grid-stride), lane s = stage s. The
// proportional cuts are computed once per template; each m value prices the
// split with lanes = stages and wave reductions. If it does not fit, lane q
// prices alternative q: only the two stages around the moved cut change, so
// it costs two stage evaluations plus maxima over the untouched stages
// (prefix and suffix maxima across lanes), and a wave minimum picks the
// fastest fitting one.
#include <cstring>

#include "decode.h"
#include "stage_cost.h"

namespace heddle {

template <class T> __device__ __forceinline__ T wave_sum(T v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ __forceinline__ double rl_double(double v, int lane)
{
    return __longlong_as_double(rl64(__double_as_longlong(v), lane));
}

// max over lanes below (above) this one; lanes past the last stage hold 0
template <class T> __device__ __forceinline__ T max_below(T v, int lane)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const T u = __shfl_up(v, o);
        v = lane >= o && u > v ? u : v;
    }
    const T w = __shfl_up(v, 1);
    return lane >= 1 ? w : T(0);
}
template <class T> __device__ __forceinline__ T max_above(T v, int lane)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const T u = __shfl_down(v, o);
        v = lane + o < 64 && u > v ? u : v;
    }
    const T w = __shfl_down(v, 1);
    return lane + 1 < 64 ? w : T(0);
}

// COUNT: only count the stage-cost evaluations into A.work (S for the
// proportional split, 2 per alternative priced)
template <bool F32, bool COUNT>
__global__ void __launch_bounds__(64) distribute_kernel(DevProfile P, PriceArgs A)
{
    extern __shared__ __align__(16) unsigned char smem[];      // one wavefront per workgroup
    uint32_t *cnt = (uint32_t *)smem;                          // [n_types] GPU counters of decode
    const int lane = threadIdx.x;
    const int L = P.L;
    const bool compute_only = (A.flags & HEDDLE_F_COMPUTE_ONLY) != 0;
    unsigned long long work = 0;

    for (int64_t t = blockIdx.x; t < A.n; t += gridDim.x) {
        const int S_in = A.n_stages[t];
        const uint32_t rec_in = lane < A.s_max ? A.stages[t * A.s_max + lane] : 0u;
        const StageInfo<uint64_t> x = decode<uint64_t, F32>(P, A, S_in, rec_in, lane, cnt);
        const size_t obase = (size_t)t * A.n_m;
        if (x.status != 0) {
            if (COUNT) continue;
            if (lane < A.n_m) {
                A.status[obase + lane] = (uint8_t)x.status;
                if (F32) {
                    ((float *)A.iter)[obase + lane] = __builtin_inff();
                    ((float *)A.bottleneck)[obase + lane] = __builtin_inff();
                } else {
                    ((int64_t *)A.iter)[obase + lane] = INT64_MAX;
                    ((int64_t *)A.bottleneck)[obase + lane] = INT64_MAX;
                }
                A.peak_mem[obase + lane] = INT64_MAX;
            }
            for (int k = 0; k < A.n_m; k++)
                if (lane < A.s_max) A.layers[(obase + k) * A.s_max + lane] = 0;
            continue;
        }
        const int S = uni(x.S), D = x.D;
        const uint32_t rec = lane < S ? rec_in : 0u;
        const int g_next = __builtin_amdgcn_update_dpp((int)(rec & 0xFF), (int)(rec & 0xFF), kDppWaveShl1, 0xF, 0xF,
                                                       false);

        // ---- proportional cuts: lane s holds stage s's layers [lo, hi)
        double speed = 0.0;
        if (lane < S) speed = 1.0 / (double)P.rows64[0][x.prow + L];
        double total = 0.0, below = 0.0;                       // lane s: speed of stages < s
        for (int s = 0; s < S; s++) {
            below = lane == s ? total : below;
            total += rl_double(speed, s);
        }
        const int c_raw = (int)floor((double)L * below / total + 0.5);
        int lo = 0, hi = L, prev = 0;
        for (int s = 1; s < S; s++) {
            int c = uni(rl32(c_raw, s));
            c = c < prev + 1 ? prev + 1 : c;
            c = c > L - (S - s) ? L - (S - s) : c;
            lo = put_lane(lo, c, s);
            hi = put_lane(hi, c, s - 1);
            prev = c;
        }

        for (int k = 0; k < A.n_m; k++) {
            const int32_t m = A.m[k];
            const int64_t Mp = (int64_t)(((uint32_t)m + (uint32_t)D - 1) / (uint32_t)D);
            // the proportional split, lanes = stages
            uint64_t T = 0;
            int64_t mem = 0, g = 0;
            bool nf = false;
            if (lane < S) {
                const StageCost c = stage_cost<F32>(P, rec, g_next, lane, S, lo, hi, D, Mp);
                T = F32 ? rne24(c.T) : c.T;
                mem = c.mem;
                g = c.g;
                nf = !c.fits;
            }
            const uint64_t sumT = wave_sum(T);
            const uint64_t nf_mask = __ballot(nf);
            work += S;
            uint64_t B = wave_max(T), iter = 0;
            int64_t peak = wave_max(mem);
            iter = iteration_time<F32>(P, Mp, B, sumT, wave_max(g));
            iter = F32 ? rne24(iter) : iter;
            bool fits = nf_mask == 0, has_split = fits || compute_only;
            int out_lo = lo, out_hi = hi;
            if (!has_split) {
                // the fixed list of alternatives: lane q prices "cut after stage q/2
                // moved by -1 (q even) or +1 (q odd)"; only stages b and b+1 change, the
                // rest comes from maxima over the stages below b and above b+1
                const uint64_t T_lo = max_below(T, lane), T_hi = max_above(T, lane);
                const int64_t M_lo = max_below(mem, lane), M_hi = max_above(mem, lane);
                const int64_t G_lo = max_below(g, lane), G_hi = max_above(g, lane);
                const int n_alt = 2 * (S - 1);
                uint64_t best_key = ~0ull;
                int best_q = -1;
                for (int q0 = 0; q0 < n_alt; q0 += 64) {
                    const int q = q0 + lane;
                    const int b = min(q >> 1, S - 2);
                    const int lo_b = __shfl(lo, b), cut = __shfl(hi, b), hi_b1 = __shfl(hi, b + 1);
                    const int c = cut + ((q & 1) ? 1 : -1);
                    const bool valid = q < n_alt && c > lo_b && c < hi_b1;
                    const int cc = min(max(c, lo_b), hi_b1);        // in range for the table reads
                    const uint32_t rb = __shfl(rec, b), rb1 = __shfl(rec, b + 1);
                    const int g2 = __shfl(g_next, b + 1);
                    const StageCost c0 = stage_cost<F32>(P, rb, (int)(rb1 & 0xFF), b, S, lo_b, cc, D, Mp);
                    const StageCost c1 = stage_cost<F32>(P, rb1, g2, b + 1, S, cc, hi_b1, D, Mp);
                    const uint64_t t0 = F32 ? rne24(c0.T) : c0.T, t1 = F32 ? rne24(c1.T) : c1.T;
                    uint64_t B2 = max(max(__shfl(T_lo, b), __shfl(T_hi, b + 1)), max(t0, t1));
                    const uint64_t sum2 = sumT - __shfl(T, b) - __shfl(T, b + 1) + t0 + t1;
                    const int64_t g2max = max(max(__shfl(G_lo, b), __shfl(G_hi, b + 1)), max(c0.g, c1.g));
                    uint64_t it2 = iteration_time<F32>(P, Mp, B2, sum2, g2max);
                    it2 = F32 ? rne24(it2) : it2;
                    const bool others_fit = (nf_mask & ~(3ull << b)) == 0;
                    const bool ok = valid && others_fit && c0.fits && c1.fits;
                    const uint64_t key = ok ? it2 : ~0ull;
                    const uint64_t kmin = wave_min(key);
                    if (kmin < best_key) {                              // strictly faster: earlier slots win ties
                        const int win = __ffsll((unsigned long long)__ballot(key == kmin)) - 1;
                        best_key = kmin;
                        best_q = q0 + win;
                        B = (uint64_t)rl64((int64_t)B2, win);
                        iter = (uint64_t)rl64((int64_t)it2, win);
                        const int64_t pk = max(max(__shfl(M_lo, b), __shfl(M_hi, b + 1)), max(c0.mem, c1.mem));
                        peak = rl64(pk, win);
                    }
                    if (COUNT) work += 2 * (uint64_t)__popcll(__ballot(valid));
                }
                if (best_q >= 0) {
                    const int b = best_q >> 1;
                    const int c = uni(rl32(hi, b)) + ((best_q & 1) ? 1 : -1);
                    out_lo = put_lane(lo, c, b + 1);
                    out_hi = put_lane(hi, c, b);
                    fits = has_split = true;
                }
            }
            if (COUNT) continue;
            const size_t o = obase + k;
            if (lane == 0) {
                A.status[o] = (uint8_t)(fits ? HEDDLE_S_OK : HEDDLE_S_OOM);
                if (F32) {
                    ((float *)A.iter)[o] = has_split ? exact_float(iter, P.fx_exp) : __builtin_inff();
                    ((float *)A.bottleneck)[o] = has_split ? exact_float(B, P.fx_exp) : __builtin_inff();
                } else {
                    ((int64_t *)A.iter)[o] = has_split ? (int64_t)iter : INT64_MAX;
                    ((int64_t *)A.bottleneck)[o] = has_split ? (int64_t)B : INT64_MAX;
                }
                A.peak_mem[o] = has_split ? peak : INT64_MAX;
            }
            if (lane < A.s_max) A.layers[o * A.s_max + lane] = (has_split && lane < S) ? (uint8_t)(out_hi - out_lo) : 0;
        }
    }
    if (COUNT && lane == 0 && work) atomicAdd(A.work, work);
}

int launch_distribute(const heddle_profile *p, PriceArgs &a, hipStream_t stream, bool count_only)
{
    if (a.n == 0) return HEDDLE_OK;
    const size_t lds = ((size_t)p->dev.n_types * 4 + 15) & ~size_t(15);
    const int blocks = (int)(a.n < 65536 ? a.n : 65536);
    const bool f32 = a.flags & HEDDLE_F_FP32;
    if (count_only) {
        if (f32) hipLaunchKernelGGL((distribute_kernel<true, true>), dim3(blocks), dim3(64), lds, stream, p->dev, a);
        else hipLaunchKernelGGL((distribute_kernel<false, true>), dim3(blocks), dim3(64), lds, stream, p->dev, a);
    } else if (f32) {
        hipLaunchKernelGGL((distribute_kernel<true, false>), dim3(blocks), dim3(64), lds, stream, p->dev, a);
    } else {
        hipLaunchKernelGGL((distribute_kernel<false, false>), dim3(blocks), dim3(64), lds, stream, p->dev, a);
    }
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

}  // namespace heddle
