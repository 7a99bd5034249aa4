// Distribute on gfx950: Heddle's own layer split (arXiv 2609.34244, section
// 5.3, layer split and DP degree) as a second partition mode of
// heddle_price_plans, with its Evaluate.
//
// Each stage's share of the layers follows its profiled speed. The speed of
// stage s is the inverse of the time of all L layers on its GPU type and TP
// degree (int64 layer costs with the stage's all-to-all terms, p2p
// excluded); the cut after stage s is the nearest integer (halves up) to
// L * (speed of stages 0..s) / (speed of all stages), computed in IEEE double
// in that order, then raised to leave stage s a layer and lowered to leave
// every later stage one. When that split does not fit memory, these
// alternatives are priced: for each boundary in order, its cut moved by -1,
// then by +1 (kept only if every stage still holds a layer); the fitting one
// with the smallest iteration time is kept, the first on ties, and none
// fitting leaves the plan OOM without a split. With HEDDLE_F_COMPUTE_ONLY the
// proportional split is kept and only flagged.
//
// Mapping: one lane per template, 256 templates per workgroup (128 or 64
// for small batches or large tables; grid-stride over such tiles). The
// tile's templates are ranked by stage count (a counting sort in LDS, most
// stages first) so that each wavefront takes 64 templates of nearly the same
// length; each lane then validates its template, computes the cuts and walks
// its stages on its own. Per lane, LDS holds the stage starts c_0..c_S
// (bytes) and one GPU counter per type for the oversubscription check; both
// are laid out [index][lane], so every LDS access of a wavefront hits 64
// distinct banks. For the fallback list, the first pass keeps the three
// largest stage times, memories and synchronisation terms with their stages:
// an alternative that moves the cut after stage b changes stages b and b+1
// only, and the largest value over the other stages is the first of those
// three not at b or b+1.
#include <cstring>

#include "stage_cost.h"
#include "validate.h"

namespace heddle {

// the three largest values pushed (value, stage), zeros at stage -1 to start
template <class T> struct Top3 {
    T v0 = 0, v1 = 0, v2 = 0;
    int i0 = -1, i1 = -1, i2 = -1;
    __device__ __forceinline__ void push(T v, int s)
    {
        if (v > v0) {
            v2 = v1; i2 = i1; v1 = v0; i1 = i0; v0 = v; i0 = s;
        } else if (v > v1) {
            v2 = v1; i2 = i1; v1 = v; i1 = s;
        } else if (v > v2) {
            v2 = v; i2 = s;
        }
    }
    // the largest value over the stages other than b and b + 1
    __device__ __forceinline__ T without(int b) const
    {
        return (i0 != b && i0 != b + 1) ? v0 : (i1 != b && i1 != b + 1) ? v1 : (i2 != b && i2 != b + 1) ? v2 : T(0);
    }
};

template <bool F32> __device__ __forceinline__ uint64_t rounded(uint64_t T) { return F32 ? rne24(T) : T; }

__device__ __forceinline__ int stage_prow(const DevProfile &P, uint32_t r)
{
    const int g = r & 0xFF, l2tp = (r >> 8) & 15, l2ep = (r >> 12) & 15;
    const int ki = nibble(P.tp_index, l2tp);
    return ((g * P.n_tp + ki) * 3 + a2a_variant(1 << l2ep, 1 << l2tp, P.node_size[g])) * (P.L + 1);
}

// COUNT: only count the stage-cost evaluations into A.work (S for the
// proportional split, 2 per alternative priced)
constexpr int kDistTpl = 256;                                  // most templates (and lanes) per workgroup

template <bool F32, bool COUNT>
__global__ void __launch_bounds__(kDistTpl, 3) distribute_kernel(DevProfile P, PriceArgs A)
{
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ uint32_t bins[64];                              // templates per stage-count bin, then bin offsets
    __shared__ uint16_t order[kDistTpl];                       // local template indices, most stages first
    const int tid = threadIdx.x;
    const int nw = blockDim.x;                                 // templates per workgroup: 64, 128 or 256
    uint32_t *cnt = (uint32_t *)smem + tid;                    // [n_types][nw]: this lane's column
    uint8_t *cut = smem + (size_t)P.n_types * nw * 4 + tid;    // [s_cap + 1][nw]: stage starts c_0..c_S
    auto C = [&](int s) -> int { return cut[s * nw]; };
    const int L = P.L;
    const bool compute_only = (A.flags & HEDDLE_F_COMPUTE_ONLY) != 0;
    const bool word_layers = (A.s_max & 3) == 0 && ((uintptr_t)A.layers & 3) == 0;
    unsigned long long work = 0;
    for (int g = 0; g < P.n_types; g++) cnt[g * nw] = 0;

    for (int64_t t0 = (int64_t)blockIdx.x * nw; t0 < A.n; t0 += (int64_t)gridDim.x * nw) {
        // ---- rank the tile's templates by stage count (bin 63 - min(S, 63))
        const int nt = A.n - t0 < nw ? (int)(A.n - t0) : nw;
        __syncthreads();                                       // earlier reads of order are done
        if (tid < 64) bins[tid] = 0;
        const int S_own = tid < nt ? (int)A.n_stages[t0 + tid] : 0;
        __syncthreads();
        const int bin = 63 - (S_own < 63 ? S_own : 63);
        const uint32_t rank = tid < nt ? atomicAdd(&bins[bin], 1u) : 0u;
        __syncthreads();
        if (tid < 64) {
            const int c = (int)bins[tid];
            bins[tid] = (uint32_t)(wave_inclusive_sum(c) - c);
        }
        __syncthreads();
        if (tid < nt) order[bins[bin] + rank] = (uint16_t)tid;
        __syncthreads();
        if (tid >= nt) continue;
        const int64_t t = t0 + order[tid];                     // the template this lane takes
        const int S = A.n_stages[t];
        const uint32_t *rec = A.stages + t * A.s_max;
        const size_t obase = (size_t)t * A.n_m;
        const int status = validate_lane(P, A, S, rec, cnt, nw);
        if (status != HEDDLE_S_OK) {
            if (COUNT) continue;
            for (int k = 0; k < A.n_m; k++) {
                const size_t o = obase + k;
                A.status[o] = (uint8_t)status;
                if (F32) {
                    ((float *)A.iter)[o] = __builtin_inff();
                    ((float *)A.bottleneck)[o] = __builtin_inff();
                } else {
                    ((int64_t *)A.iter)[o] = INT64_MAX;
                    ((int64_t *)A.bottleneck)[o] = INT64_MAX;
                }
                A.peak_mem[o] = INT64_MAX;
                if (word_layers) {
                    for (int w = 0; w < A.s_max; w += 4) *(uint32_t *)&A.layers[o * A.s_max + w] = 0u;
                } else {
                    for (int w = 0; w < A.s_max; w++) A.layers[o * A.s_max + w] = 0;
                }
            }
            continue;
        }
        const int D = (int)(rec[0] >> 16);

        // ---- proportional cuts: c_s = nearest integer to L * (speed of stages < s) / (speed of all)
        double total = 0.0;
        for (int s = 0; s < S; s++) total += 1.0 / (double)P.rows64[0][stage_prow(P, rec[s]) + L];
        {
            double below = 0.0;
            int prev = 0;
            cut[0] = 0;
            for (int s = 1; s < S; s++) {
                below += 1.0 / (double)P.rows64[0][stage_prow(P, rec[s - 1]) + L];
                int c = (int)floor((double)L * below / total + 0.5);
                c = c < prev + 1 ? prev + 1 : c;
                c = c > L - (S - s) ? L - (S - s) : c;
                cut[s * nw] = (uint8_t)c;
                prev = c;
            }
            cut[S * nw] = (uint8_t)L;
        }

        for (int k = 0; k < A.n_m; k++) {
            const int32_t m = A.m[k];
            const int64_t Mp = (int64_t)(((uint32_t)m + (uint32_t)D - 1) / (uint32_t)D);
            // ---- the proportional split
            uint64_t sumT = 0, nf = 0;
            Top3<uint64_t> tT;
            Top3<int64_t> tM, tG;
#pragma unroll 1
            for (int s = 0; s < S; s++) {
                const int g_next = s + 1 < S ? (int)(rec[s + 1] & 0xFF) : 0;
                const StageCost c = stage_cost<F32>(P, rec[s], g_next, s, S, C(s), C(s + 1), D, Mp);
                const uint64_t T = rounded<F32>(c.T);
                sumT += T;
                tT.push(T, s);
                tM.push(c.mem, s);
                tG.push(c.g, s);
                nf |= (uint64_t)(!c.fits) << s;
            }
            if (COUNT) work += S;
            uint64_t B = tT.v0;
            uint64_t iter = rounded<F32>(iteration_time<F32>(P, Mp, B, sumT, tG.v0));
            int64_t peak = tM.v0;
            bool fits = nf == 0, has_split = fits || compute_only;
            int best_b = -1, best_c = 0;
            if (!has_split) {
                // the predefined alternatives, in order: for each boundary b, the cut
                // after stage b moved by -1, then by +1; the fastest fitting one is kept
                // (the first on ties)
                uint64_t best_key = ~0ull;
#pragma unroll 1
                for (int b = 0; b + 1 < S; b++) {
                    const uint32_t rb = rec[b], rb1 = rec[b + 1];
                    const int g2 = b + 2 < S ? (int)(rec[b + 2] & 0xFF) : 0;
                    const int lo = C(b), cb = C(b + 1), hi = C(b + 2);
                    const uint64_t Tb = rounded<F32>(stage_cost<F32>(P, rb, (int)(rb1 & 0xFF), b, S, lo, cb, D, Mp).T);
                    const uint64_t Tb1 = rounded<F32>(stage_cost<F32>(P, rb1, g2, b + 1, S, cb, hi, D, Mp).T);
                    const uint64_t T_rest = tT.without(b);
                    const int64_t M_rest = tM.without(b), G_rest = tG.without(b);
                    const bool others_fit = (nf & ~(3ull << b)) == 0;
#pragma unroll 1
                    for (int d = -1; d <= 1; d += 2) {
                        const int c = cb + d;
                        if (c <= lo || c >= hi) continue;           // every stage keeps a layer
                        if (COUNT) {
                            work += 2;
                            continue;
                        }
                        const StageCost c0 = stage_cost<F32>(P, rb, (int)(rb1 & 0xFF), b, S, lo, c, D, Mp);
                        const StageCost c1 = stage_cost<F32>(P, rb1, g2, b + 1, S, c, hi, D, Mp);
                        const uint64_t t0 = rounded<F32>(c0.T), t1 = rounded<F32>(c1.T);
                        const uint64_t B2 = max(T_rest, max(t0, t1));
                        const uint64_t sum2 = sumT - Tb - Tb1 + t0 + t1;
                        const int64_t g2max = max(G_rest, max(c0.g, c1.g));
                        const uint64_t it2 = rounded<F32>(iteration_time<F32>(P, Mp, B2, sum2, g2max));
                        if (others_fit && c0.fits && c1.fits && it2 < best_key) {
                            best_key = it2;
                            best_b = b;
                            best_c = c;
                            B = B2;
                            iter = it2;
                            peak = max(M_rest, max(c0.mem, c1.mem));
                        }
                    }
                }
                if (best_b >= 0) fits = has_split = true;
            }
            if (COUNT) continue;
            const size_t o = obase + k;
            A.status[o] = (uint8_t)(fits ? HEDDLE_S_OK : HEDDLE_S_OOM);
            if (F32) {
                ((float *)A.iter)[o] = has_split ? exact_float(iter, P.fx_exp) : __builtin_inff();
                ((float *)A.bottleneck)[o] = has_split ? exact_float(B, P.fx_exp) : __builtin_inff();
            } else {
                ((int64_t *)A.iter)[o] = has_split ? (int64_t)iter : INT64_MAX;
                ((int64_t *)A.bottleneck)[o] = has_split ? (int64_t)B : INT64_MAX;
            }
            A.peak_mem[o] = has_split ? peak : INT64_MAX;
            // layer counts; the winning alternative moves the start of stage best_b + 1
            auto layers_of = [&](int s) -> uint32_t {
                if (!has_split || s >= S) return 0u;
                const int a = s == best_b + 1 ? best_c : C(s);
                const int e = s == best_b ? best_c : C(s + 1);
                return (uint32_t)(e - a);
            };
            if (word_layers) {
                for (int w = 0; w < A.s_max; w += 4)
                    *(uint32_t *)&A.layers[o * A.s_max + w] =
                        layers_of(w) | layers_of(w + 1) << 8 | layers_of(w + 2) << 16 | layers_of(w + 3) << 24;
            } else {
                for (int w = 0; w < A.s_max; w++) A.layers[o * A.s_max + w] = (uint8_t)layers_of(w);
            }
        }
    }
    if (COUNT) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) work += __shfl_xor(work, off);
        if ((tid & 63) == 0 && work) atomicAdd(A.work, work);
    }
}

int launch_distribute(const heddle_profile *p, PriceArgs &a, hipStream_t stream, bool count_only)
{
    if (a.n == 0) return HEDDLE_OK;
    const int s_cap = a.s_max < p->dev.L ? a.s_max : p->dev.L;
    // templates per workgroup: the most (256, 128 or 64) whose per-lane tables
    // fit 63 KB of LDS beside the ranking's own 768 bytes and that still give
    // every CU four workgroups of the batch
    int max_lds = 0, cus = 0;
    HEDDLE_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, p->device));
    HEDDLE_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device));
    const size_t per_lane = (size_t)p->dev.n_types * 4 + (size_t)(s_cap + 1);
    int nw = kDistTpl;
    while (nw > 64 && (per_lane * nw > 63 * 1024 || a.n < (int64_t)nw * 4 * (cus > 0 ? cus : 1))) nw >>= 1;
    const size_t lds = per_lane * nw;
    if (lds > (size_t)max_lds) return fail(HEDDLE_E_RANGE, "per-lane tables of this profile do not fit in LDS");
    const int64_t want = (a.n + nw - 1) / nw;
    const int blocks = (int)(want < 65536 ? want : 65536);
    const bool f32 = a.flags & HEDDLE_F_FP32;
    const void *fn = count_only ? (f32 ? (const void *)distribute_kernel<true, true> : (const void *)distribute_kernel<false, true>)
                                : (f32 ? (const void *)distribute_kernel<true, false> : (const void *)distribute_kernel<false, false>);
    if (lds > 65536) HEDDLE_HIP(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
    if (count_only) {
        if (f32) hipLaunchKernelGGL((distribute_kernel<true, true>), dim3(blocks), dim3(nw), lds, stream, p->dev, a);
        else hipLaunchKernelGGL((distribute_kernel<false, true>), dim3(blocks), dim3(nw), lds, stream, p->dev, a);
    } else if (f32) {
        hipLaunchKernelGGL((distribute_kernel<true, false>), dim3(blocks), dim3(nw), lds, stream, p->dev, a);
    } else {
        hipLaunchKernelGGL((distribute_kernel<false, false>), dim3(blocks), dim3(nw), lds, stream, p->dev, a);
    }
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

}  // namespace heddle
