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
// Mapping: one lane per template, 64 templates per wavefront. The
// wavefront's template records are staged in LDS with coalesced loads
// (row stride s_max + 1 words, so that the lanes' column reads do not share
// banks); each lane validates its template (per-type GPU counters in an LDS
// column of its own), then chases its own limit rows in global memory (the
// forward and backward chases are independent and taken in one loop),
// keeping R_s and Bk_s in the two upper bytes of its staged record s (the DP
// degree they held is read before), and writes its windows four at a time.
#include "validate.h"

namespace heddle {

__global__ void __launch_bounds__(64, 8) window_kernel(DevProfile P, PriceArgs A)
{
    extern __shared__ __align__(16) unsigned char smem[];      // one wavefront per workgroup
    const int lane = threadIdx.x;
    const int rs = A.s_max + 1;                                // staged record stride, words
    uint32_t *cnt = (uint32_t *)smem + lane;                   // [n_types][64] GPU counters of validation
    uint32_t *recs = (uint32_t *)smem + (size_t)P.n_types * 64;   // [64][rs] the wavefront's records
    const int L = P.L, ls = P.lim_stride;
    const int ws = win_stride(A.s_max);
    const bool mem_aware = (A.flags & HEDDLE_F_COMPUTE_ONLY) == 0;
    for (int g = 0; g < P.n_types; g++) cnt[g * 64] = 0;

    for (int64_t t0 = (int64_t)blockIdx.x * 64; t0 < A.n; t0 += (int64_t)gridDim.x * 64) {
        // ---------------- the records of templates t0 .. t0 + 63 into LDS
        const int nt = A.n - t0 < 64 ? (int)(A.n - t0) : 64;
        const uint32_t *src = A.stages + t0 * A.s_max;
        wave_sync();                                           // earlier reads of recs are done
        for (int i = lane; i < nt * A.s_max; i += 64) {
            const int j = i / A.s_max;
            recs[j * rs + (i - j * A.s_max)] = src[i];
        }
        wave_sync();
        if (lane >= nt) continue;
        const int64_t t = t0 + lane;
        const int S = A.n_stages[t];
        const uint32_t *rec = recs + lane * rs;
        uint8_t *rk = (uint8_t *)(recs + lane * rs);           // byte 4s + 2: R_s, byte 4s + 3: Bk_s
        const size_t obase = (size_t)t * A.n_m;
        const int status = validate_lane(P, A, S, rec, cnt);
        if (status != HEDDLE_S_OK) {
            for (int k = 0; k < A.n_m; k++) A.wst[obase + k] = (uint32_t)status;
            continue;
        }
        const uint32_t D = rec[0] >> 16;
        auto key_of = [&](int k) -> int {                      // in-flight class of the k-th m
            const int Mp = (int)(((uint32_t)A.m[k] + D - 1) / D);
            return mem_aware ? (Mp < S ? Mp : S) : 0;
        };
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
                continue;
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
        }
    }
}

int prepare_windows(const heddle_profile *p, const PriceArgs &a, int max_lds, size_t *lds)
{
    *lds = (size_t)p->dev.n_types * 256 + (size_t)64 * (a.s_max + 1) * 4;
    if (*lds > (size_t)max_lds) return fail(HEDDLE_E_RANGE, "per-lane tables of this profile do not fit in LDS");
    if (*lds > 65536)
        HEDDLE_HIP(hipFuncSetAttribute((const void *)window_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)*lds));
    return HEDDLE_OK;
}

int launch_windows(const heddle_profile *p, const PriceArgs &a, size_t lds, hipStream_t stream)
{
    if (a.n == 0) return HEDDLE_OK;
    const int64_t want = (a.n + 63) / 64;
    const int blocks = (int)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(window_kernel, dim3(blocks), dim3(64), lds, stream, p->dev, a);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

}  // namespace heddle
