// Validation and row windows of every plan, one lane per template (gfx950),
// ahead of the split kernel.
//
// Validation follows the status order of the feasibility masks (section 5.1)
// and the exact profile match (section 5.2). For a valid template and a
// micro-batch count m, the memory limits of its stages depend on the number
// of micro-batches in flight, min(S - s, ceil(m / D)), so plans with the same
// value of min(ceil(m / D), S) share their windows. The windows are those the
// split kernel relaxes over: with lim(s, i) the largest admissible end of row
// i at stage s (memory limit capped so that every later stage keeps a layer),
// the forward reach R_0 = 0, R_{s+1} = lim(s, R_s) and the backward bound
// Bk_S = L, Bk_s = the smallest start >= s whose limit reaches Bk_{s+1} (an
// inverse-limit table lookup); W_s = [Bk_s, min(R_s, L - (S - s))] (row 0 only
// for s = 0). A plan with an empty window has no split that fits memory.
//
// Mapping: one lane per template, 256 templates per workgroup (128 or 64
// when the staged records of 256 would not fit the workgroup's LDS). The
// workgroup's template records are staged in LDS with coalesced loads (row
// stride s_max + 1 words, so that the lanes' column reads do not share
// banks) and its templates are ranked by stage count (a counting sort in LDS,
// most stages first), so that each wavefront takes 64 templates of nearly the
// same length and its per-stage loops do not run for the longest template of
// an unsorted 64. Each lane validates its template (per-type GPU counters in
// an LDS column of its own), then chases its own limit rows in global memory
// (the forward and backward chases are independent and taken in one loop),
// keeping R_s and Bk_s in the two upper bytes of its staged record s (the DP
// degree they held is read before), and writes its windows four at a time.
#include "validate.h"

namespace heddle {

constexpr int kWinTpl = 256;                                   // most templates (and lanes) per workgroup

__global__ void __launch_bounds__(kWinTpl) window_kernel(DevProfile P, PriceArgs A)
{
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ uint32_t bins[64];                              // templates per stage-count bin, then bin offsets
    __shared__ uint16_t order[kWinTpl];                        // local template indices, most stages first
    const int tid = threadIdx.x;
    const int nw = blockDim.x;                                 // templates per workgroup: 64, 128 or 256
    const int rs = A.s_max + 1;                                // staged record stride, words
    uint32_t *cnt = (uint32_t *)smem + tid;                    // [n_types][nw] GPU counters of validation
    uint32_t *recs = (uint32_t *)smem + (size_t)P.n_types * nw;   // [nw][rs] the workgroup's records
    const int L = P.L, ls = P.lim_stride;
    const int ws = win_stride(A.s_max);
    const bool mem_aware = (A.flags & HEDDLE_F_COMPUTE_ONLY) == 0;
    for (int g = 0; g < P.n_types; g++) cnt[g * nw] = 0;

    for (int64_t t0 = (int64_t)blockIdx.x * nw; t0 < A.n; t0 += (int64_t)gridDim.x * nw) {
        // ---------------- the records of templates t0 .. t0 + nw - 1 into LDS, and
        // their ranking by stage count (bin 63 - min(S, 63))
        const int nt = A.n - t0 < nw ? (int)(A.n - t0) : nw;
        const uint32_t *src = A.stages + t0 * A.s_max;
        __syncthreads();                                       // earlier reads of recs and order are done
        if (tid < 64) bins[tid] = 0;
        for (int i = tid; i < nt * A.s_max; i += nw) {
            const int j = i / A.s_max;
            recs[j * rs + (i - j * A.s_max)] = src[i];
        }
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
        const int me = order[tid];                             // the template this lane takes
        const int64_t t = t0 + me;
        const int S = A.n_stages[t];
        const uint32_t *rec = recs + me * rs;
        uint8_t *rk = (uint8_t *)(recs + me * rs);             // byte 4s + 2: R_s, byte 4s + 3: Bk_s
        const size_t obase = (size_t)t * A.n_m;
        // the final outputs of a template none of whose plans has windows (it
        // failed validation, or no split fits memory): status, no bottleneck and
        // no layers; the split kernel skips such templates. Not written when the
        // call only counts work (no outputs are given then).
        auto close_template = [&](uint32_t code) {
            if (!A.status) return;
            const bool f32 = (A.flags & HEDDLE_F_FP32) != 0;
            const bool words = (A.s_max & 3) == 0 && ((uintptr_t)A.layers & 3) == 0;
            for (int k = 0; k < A.n_m; k++) {
                const size_t o = obase + k;
                A.status[o] = (uint8_t)code;
                if (f32) ((float *)A.bottleneck)[o] = __builtin_inff();
                else ((int64_t *)A.bottleneck)[o] = INT64_MAX;
                if (words) {
                    for (int w = 0; w < A.s_max; w += 4) *(uint32_t *)&A.layers[o * A.s_max + w] = 0u;
                } else {
                    for (int w = 0; w < A.s_max; w++) A.layers[o * A.s_max + w] = 0;
                }
            }
        };
        const int status = validate_lane(P, A, S, rec, cnt, nw);
        if (status != HEDDLE_S_OK) {
            for (int k = 0; k < A.n_m; k++) A.wst[obase + k] = (uint32_t)status;
            close_template((uint32_t)status);
            continue;
        }
        const uint32_t D = rec[0] >> 16;
        auto key_of = [&](int k) -> int {                      // in-flight class of the k-th m
            const int Mp = (int)(((uint32_t)A.m[k] + D - 1) / D);
            return mem_aware ? (Mp < S ? Mp : S) : 0;
        };
        bool any_ok = false;                                   // a plan of the template has windows
        for (int k = 0; k < A.n_m; k++) {
            const size_t o = obase + k;
            uint2 *wout = (uint2 *)(A.wwin + o * ws);
            const int key = key_of(k);
            int k0 = -1;                                       // an earlier plan of the same class
            for (int k2 = 0; k2 < k && k0 < 0; k2++) k0 = key_of(k2) == key ? k2 : -1;
            if (k0 >= 0) {
                const size_t o0 = obase + k0;
                const uint2 *win0 = (const uint2 *)(A.wwin + o0 * ws);
                A.wst[o] = A.wst[o0];
                for (int s = 0; s < S; s += 4) wout[s >> 2] = win0[s >> 2];
                continue;                                      // any_ok already holds plan k0's outcome
            }
            if (mem_aware) {
                int c = 0, nxt = L;                            // R_s, Bk_{u+1}
                for (int s = 0; s < S; s++) {
                    const int u = S - 1 - s;
                    rk[4 * s + 2] = (uint8_t)c;
                    const uint32_t rf = rec[s], rb = rec[u];
                    auto rows_of = [&](uint32_t r, int st) -> const uint8_t * {
                        const int ki = nibble(P.tp_index, (r >> 8) & 15), ei = nibble(P.ep_index, (r >> 12) & 15);
                        int f = S - st < key ? S - st : key;
                        f = f < 1 ? 1 : f;
                        return P.mem_lim + ((size_t)((((r & 0xFF) * P.n_tp + ki) * P.n_ep + ei) * P.n_f) + f - 1) * 2 * ls;
                    };
                    const int cf = rows_of(rf, s)[c];         // lim row of stage s, at R_s
                    const int kb = rows_of(rb, u)[ls + nxt];  // inverse row of stage u, at Bk_{u+1}
                    const int jhi = L - (S - 1 - s);
                    c = cf < jhi ? cf : jhi;                   // R_{s+1}
                    nxt = kb > u ? kb : u;                     // Bk_u
                    rk[4 * u + 3] = (uint8_t)nxt;
                }
            }
            bool fits = true;
            uint32_t rows = 0;                                 // rows of W_1 .. W_{S-1}
            for (int s0 = 0; s0 < S; s0 += 4) {
                uint32_t w[4];
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const int s = s0 + q < S ? s0 + q : S - 1;    // entries beyond S repeat the last one
                    const int ihi = s == 0 ? 0 : L - (S - s);
                    const int a = mem_aware ? (int)rk[4 * s + 3] : s;
                    int b = mem_aware ? (int)rk[4 * s + 2] : ihi;
                    b = b < ihi ? b : ihi;
                    fits = fits && a <= b;
                    rows += s0 + q < S && s > 0 ? (uint32_t)(b - a + 1) : 0u;
                    w[q] = (uint32_t)(a | b << 8);
                }
                wout[s0 >> 2] = make_uint2(w[0] | w[1] << 16, w[2] | w[3] << 16);
            }
            A.wst[o] = fits ? (uint32_t)HEDDLE_S_OK | (uint32_t)key << 8 | rows << 16 : (uint32_t)HEDDLE_S_OOM;
            any_ok = any_ok || fits;
        }
        if (!any_ok) close_template((uint32_t)HEDDLE_S_OOM);
    }
}

// templates per workgroup: the most (256, 128 or 64) whose staged records and
// counters fit 63 KB of LDS beside the ranking's own 768 bytes and that still
// give every CU four workgroups of the batch (a small batch in large
// workgroups leaves CUs idle)
static int window_tile(const heddle_profile *p, const PriceArgs &a)
{
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device) != hipSuccess || cus < 1) cus = 1;
    int nw = kWinTpl;
    while (nw > 64 && ((size_t)nw * (p->dev.n_types + a.s_max + 1) * 4 > 63 * 1024 || a.n < (int64_t)nw * 4 * cus))
        nw >>= 1;
    return nw;
}

int prepare_windows(const heddle_profile *p, const PriceArgs &a, int max_lds, size_t *lds)
{
    *lds = (size_t)window_tile(p, a) * (p->dev.n_types + a.s_max + 1) * 4;
    if (*lds > (size_t)max_lds) return fail(HEDDLE_E_RANGE, "per-lane tables of this profile do not fit in LDS");
    if (*lds > 65536)
        HEDDLE_HIP(hipFuncSetAttribute((const void *)window_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)*lds));
    return HEDDLE_OK;
}

int launch_windows(const heddle_profile *p, const PriceArgs &a, size_t lds, hipStream_t stream)
{
    if (a.n == 0) return HEDDLE_OK;
    const int wg = window_tile(p, a);
    const int64_t want = (a.n + wg - 1) / wg;
    const int blocks = (int)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(window_kernel, dim3(blocks), dim3(wg), lds, stream, p->dev, a);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

}  // namespace heddle
