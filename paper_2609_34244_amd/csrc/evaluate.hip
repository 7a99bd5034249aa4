// Evaluate on gfx950: iteration time and per-GPU peak memory of every plan
// whose split the split kernel found (Heddle, arXiv 2609.34244: the
// profile-based cost model of section 5.2 and the 1F1B iteration time
// (M-1) max_s t_s + sum_s t_s + max_s g_s of section 5.3).
//
// One lane prices one (template, m) plan, walking its stages: t_s is the
// stage's time over its layers plus its outbound p2p, g_s the ring
// all-reduce of its dense gradients over the D replicas plus that of its
// expert gradients over D / EP replicas, and the memory of stage s holds
// min(S - s, M_p) micro-batches of activations. Plans without a split keep
// their status and get INT64_MAX (fp32: +inf) values.
#include <cstring>

#include "stage_cost.h"

namespace heddle {

// Iteration time and peak memory of plan o, which has a split.
template <bool F32>
__device__ __forceinline__ void evaluate_plan(const DevProfile &P, const PriceArgs &A, int64_t o, int64_t total)
{
    // plan o = t * n_m + k; a 32-bit division when the batch allows it
    const int64_t t = A.n_m == 1 ? o : total <= 0xFFFFFFFFll ? (int64_t)((uint32_t)o / (uint32_t)A.n_m) : o / A.n_m;
    const int k = (int)(o - t * A.n_m);
    int32_t m = A.m[0];
    for (int q = 1; q < A.n_m; q++) m = q == k ? A.m[q] : m;
    const int S = A.n_stages[t];
    const uint32_t *rec = A.stages + t * A.s_max;
    const uint8_t *lay = A.layers + o * A.s_max;
    const int D = (int)(rec[0] >> 16);
    const int64_t Mp = (int64_t)(((uint32_t)m + (uint32_t)D - 1) / (uint32_t)D);
    const uint64_t B = F32 ? fixed_of_float(((const float *)A.bottleneck)[o], P.fx_exp)
                           : (uint64_t)((const int64_t *)A.bottleneck)[o];
    uint64_t sumT = 0;
    int64_t maxg = 0, peak = 0;
    bool oom = false;
    int i = 0;
    uint32_t r_next = rec[0];
    int l_next = lay[0];                                      // layer counts, like the records, one stage ahead
    for (int s = 0; s < S; s++) {
        const uint32_t r = r_next;
        const int j = i + l_next;
        if (s + 1 < S) {
            r_next = rec[s + 1];
            l_next = lay[s + 1];
        }
        const StageCost c = stage_cost<F32>(P, r, (int)(r_next & 0xFF), s, S, i, j, D, Mp);
        sumT += F32 ? rne24(c.T) : c.T;
        peak = c.mem > peak ? c.mem : peak;
        oom = oom || !c.fits;
        maxg = c.g > maxg ? c.g : maxg;
        i = j;
    }
    const uint64_t iter = iteration_time<F32>(P, Mp, B, sumT, maxg);
    if (F32) ((float *)A.iter)[o] = exact_float(rne24(iter), P.fx_exp);
    else ((int64_t *)A.iter)[o] = (int64_t)iter;
    A.peak_mem[o] = peak;
    if (oom) A.status[o] = HEDDLE_S_OOM;                      // compute-only splits that do not fit
}

// A workgroup takes 256 consecutive plans. Plans without a split get their
// INT64_MAX / +inf values at once; the others are ranked by stage count
// (a counting sort in LDS, most stages first) so that each wavefront walks
// plans of nearly the same length and a wavefront left without plans ends
// at once, instead of every lane waiting on the longest plan of its 64.
template <bool F32>
__global__ void __launch_bounds__(256) evaluate_kernel(DevProfile P, PriceArgs A)
{
    __shared__ uint32_t bins[64];                             // plans per stage count S (bin 64 - S), then bin offsets
    __shared__ uint16_t order[256];                           // tile positions, most stages first
    __shared__ uint32_t n_split;
    const int tid = threadIdx.x;
    const int64_t total = A.n * A.n_m;
    for (int64_t base = (int64_t)blockIdx.x * 256; base < total; base += (int64_t)gridDim.x * 256) {
        if (tid < 64) bins[tid] = 0;
        __syncthreads();
        const int64_t o = base + tid;
        int bin = -1;
        uint32_t rank = 0;
        if (o < total) {
            if (A.status[o] != HEDDLE_S_OK) {                 // no split: invalid template or nothing fits
                if (F32) ((float *)A.iter)[o] = __builtin_inff();
                else ((int64_t *)A.iter)[o] = INT64_MAX;
                A.peak_mem[o] = INT64_MAX;
            } else {
                const int64_t t = A.n_m == 1 ? o : total <= 0xFFFFFFFFll ? (int64_t)((uint32_t)o / (uint32_t)A.n_m) : o / A.n_m;
                bin = 64 - (int)A.n_stages[t];                // 1 <= S <= 64
                rank = atomicAdd(&bins[bin], 1u);
            }
        }
        __syncthreads();
        if (tid < 64) {                                       // exclusive offsets of the bins
            const int c = (int)bins[tid];
            const int incl = wave_inclusive_sum(c);
            bins[tid] = (uint32_t)(incl - c);
            if (tid == 63) n_split = (uint32_t)incl;
        }
        __syncthreads();
        if (bin >= 0) order[bins[bin] + rank] = (uint16_t)tid;
        __syncthreads();
        if ((uint32_t)tid < n_split) evaluate_plan<F32>(P, A, base + order[tid], total);
        __syncthreads();                                      // bins and order are rewritten by the next tile
    }
}

int launch_evaluate(const heddle_profile *p, const PriceArgs &a, hipStream_t stream)
{
    const int64_t total = a.n * a.n_m;
    if (total == 0) return HEDDLE_OK;
    const int64_t want = (total + 255) / 256;
    const int blocks = (int)(want < 65536 ? want : 65536);
    if (a.flags & HEDDLE_F_FP32)
        hipLaunchKernelGGL(evaluate_kernel<true>, dim3(blocks), dim3(256), 0, stream, p->dev, a);
    else
        hipLaunchKernelGGL(evaluate_kernel<false>, dim3(blocks), dim3(256), 0, stream, p->dev, a);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

}  // namespace heddle
