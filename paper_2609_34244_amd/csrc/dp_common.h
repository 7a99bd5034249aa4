// Pieces of the min-max recurrence shared by the split kernels (gfx950).
#pragma once

#include "device_common.h"

namespace heddle {

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
template <class T> __device__ __forceinline__ T vmax(T a, T b) { return a > b ? a : b; }

// min over the ends [j, je] of one row, in steps of four ends; the ends of
// the last step past je are read (they lie inside the pair row) and masked
template <class V, class V2> __device__ __forceinline__ V relax_range(const V2 *X, int j, int je, V pi, V acc)
{
    const V INF = DPInf<V>::value;
    for (; j <= je; j += 4) {
        const V2 a = X[j], b = X[j + 1], c = X[j + 2], d = X[j + 3];
        const int rem = je - j;
        const V rb = rem >= 1 ? relax<V>(b, pi) : INF;
        const V rc = rem >= 2 ? relax<V>(c, pi) : INF;
        const V rd = rem >= 3 ? relax<V>(d, pi) : INF;
        acc = vmin(vmin(acc, relax<V>(a, pi)), vmin(rb, vmin(rc, rd)));
    }
    return acc;
}

}  // namespace heddle
