// Argmin over priced plans: the feasible plan of highest throughput m / iter
// (Heddle, arXiv 2609.34244, section 5 overview: candidates are ordered by
// the throughput the cost model predicts; section 5.3: the fastest fitting
// choice is kept).
//
// Key: iter / m, compared exactly by cross-multiplication (128-bit for int64
// iteration times; fp32 times scaled by m <= 2^24 are exact in fp64). Ties
// go to the lowest flat index t * n_m + k, i.e. the lowest template, then
// the lowest m index. The comparison is a total order, so the two-pass
// reduction (wave shuffles -> LDS -> one block over the partials) returns
// the same answer for any grid shape; no atomics are involved.
#include <cstring>

#include "heddle_internal.h"

namespace heddle {

constexpr int kArgBlock = 256;
constexpr int kArgMaxBlocks = 2048;

struct Cand {
    uint64_t iter;   // int64 value, or the bit pattern of a non-negative float
    int64_t idx;     // flat index; -1 = none
    int32_t m;
};

__device__ __forceinline__ bool better(const Cand &a, const Cand &b, bool f32)
{
    if (a.idx < 0) return false;
    if (b.idx < 0) return true;
    bool lt, eq;
    if (a.m == b.m) {
        // one micro-batch count: iter / m orders as iter (non-negative floats
        // order as their bit patterns)
        lt = a.iter < b.iter;
        eq = a.iter == b.iter;
    } else if (f32) {
        const double x = (double)__uint_as_float((uint32_t)a.iter) * (double)b.m;
        const double y = (double)__uint_as_float((uint32_t)b.iter) * (double)a.m;
        lt = x < y;
        eq = x == y;
    } else {
        const unsigned __int128 x = (unsigned __int128)a.iter * (uint32_t)b.m;
        const unsigned __int128 y = (unsigned __int128)b.iter * (uint32_t)a.m;
        lt = x < y;
        eq = x == y;
    }
    return lt || (eq && a.idx < b.idx);
}

// A candidate from another lane: DPP within rows of 16 lanes, ds_swizzle
// across the two rows of a 32-lane half, one value per word.
template <int CTRL> __device__ __forceinline__ uint32_t dpp_word(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}
template <int PAT> __device__ __forceinline__ uint32_t swz_word(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, PAT);
}
template <class F> __device__ __forceinline__ Cand move_cand(const Cand &c, F mv)
{
    Cand r;
    r.iter = ((uint64_t)mv((uint32_t)(c.iter >> 32)) << 32) | mv((uint32_t)c.iter);
    r.idx = (int64_t)(((uint64_t)mv((uint32_t)((uint64_t)c.idx >> 32)) << 32) | mv((uint32_t)(uint64_t)c.idx));
    r.m = (int32_t)mv((uint32_t)c.m);
    return r;
}
__device__ __forceinline__ Cand from_lane(const Cand &c, int lane)
{
    return move_cand(c, [lane](uint32_t v) { return (uint32_t)__builtin_amdgcn_readlane((int)v, lane); });
}

// best candidate of the wavefront, valid in lane 0: pairs of lanes, quads
// (quad permutations), groups of 8 and 16 (row half-mirror and mirror: after
// the earlier steps every lane of a group holds the group's best, so any
// pairing of two groups combines them), the two rows of 16 of each half
// (swizzle, bit mode: and 0x1F, xor 0x10), then the halves (lane 32 read into
// lane 0). The order is total, so the result does not depend on the pairing.
__device__ __forceinline__ Cand wave_best(Cand c, bool f32)
{
    Cand u;
    u = move_cand(c, dpp_word<0xB1>);            // quad_perm [1, 0, 3, 2]
    if (better(u, c, f32)) c = u;
    u = move_cand(c, dpp_word<0x4E>);            // quad_perm [2, 3, 0, 1]
    if (better(u, c, f32)) c = u;
    u = move_cand(c, dpp_word<0x141>);           // row_half_mirror
    if (better(u, c, f32)) c = u;
    u = move_cand(c, dpp_word<0x140>);           // row_mirror
    if (better(u, c, f32)) c = u;
    u = move_cand(c, swz_word<(0x10 << 10) | 0x1F>);
    if (better(u, c, f32)) c = u;
    u = from_lane(c, 32);
    const Cand l0 = from_lane(c, 0);
    return better(u, l0, f32) ? u : l0;
}

__device__ Cand block_best(Cand c, bool f32)
{
    __shared__ Cand part[kArgBlock / 64];
    c = wave_best(c, f32);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (lane == 0) part[w] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int i = 1; i < (int)(blockDim.x >> 6); i++)
            if (better(part[i], c, f32)) c = part[i];
    }
    return c;
}

struct ArgArgs {
    int64_t total;          // n * n_m
    int32_t n_m, f32;
    int32_t m[kMaxMList];
    const void *iter;
    const uint8_t *status;
    Cand *partial;
};

__global__ void __launch_bounds__(kArgBlock) argmin_pass1(ArgArgs A)
{
    __shared__ int32_t sm[kMaxMList];
    for (int k = 0; k < A.n_m; k++)
        if ((int)threadIdx.x == k) sm[k] = A.m[k];
    __syncthreads();
    Cand best;
    best.idx = -1;
    best.iter = 0;
    best.m = 1;
    const bool f32 = A.f32 != 0;
    const int64_t o0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (int64_t)gridDim.x * blockDim.x;
    // m index of plan o = t * n_m + k, advanced with o (no division per plan)
    int k = (int)(o0 % A.n_m);
    const int dk = (int)(stride % A.n_m);
    for (int64_t o = o0; o < A.total; o += stride) {
        if (A.status[o] == HEDDLE_S_OK) {
            Cand c;
            c.idx = o;
            c.m = sm[k];
            c.iter = f32 ? (uint64_t)__float_as_uint(((const float *)A.iter)[o]) : (uint64_t)((const int64_t *)A.iter)[o];
            if (better(c, best, f32)) best = c;
        }
        k += dk;
        k -= k >= A.n_m ? A.n_m : 0;
    }
    best = block_best(best, f32);
    if (threadIdx.x == 0) A.partial[blockIdx.x] = best;
}

__global__ void __launch_bounds__(kArgBlock) argmin_pass2(const Cand *partial, int n_part, int f32, Cand *out)
{
    Cand best;
    best.idx = -1;
    best.iter = 0;
    best.m = 1;
    for (int i = threadIdx.x; i < n_part; i += blockDim.x)
        if (better(partial[i], best, f32 != 0)) best = partial[i];
    best = block_best(best, f32 != 0);
    if (threadIdx.x == 0) *out = best;
}

// Pass 2 writes its result straight into pinned, coherent host memory: one
// slot per host thread (the call waits for its stream before reading it, so
// calls of one thread never overlap), allocated on first use and kept.
static thread_local Cand *t_result = nullptr;

static Cand *result_slot()
{
    if (!t_result && hipHostMalloc((void **)&t_result, sizeof(Cand), hipHostMallocPortable | hipHostMallocCoherent) != hipSuccess)
        t_result = nullptr;
    return t_result;
}

int launch_argmin(int64_t n, const int32_t *h_m, int32_t n_m, uint32_t flags, const void *d_iter,
                  const uint8_t *d_status, int64_t *h_best_template, int32_t *h_best_m_index,
                  void *h_best_iter, hipStream_t stream)
{
    const int64_t total = n * n_m;
    if (total == 0) return fail(HEDDLE_E_NOFEASIBLE, "no plans");
    ArgArgs a;
    std::memset(&a, 0, sizeof(a));
    a.total = total;
    a.n_m = n_m;
    a.f32 = (flags & HEDDLE_F_FP32) ? 1 : 0;
    for (int k = 0; k < n_m; k++) a.m[k] = h_m[k];
    a.iter = d_iter;
    a.status = d_status;
    const int64_t want = (total + kArgBlock * 8 - 1) / (kArgBlock * 8);
    const int blocks = (int)(want < kArgMaxBlocks ? (want > 0 ? want : 1) : kArgMaxBlocks);
    Cand *scratch = nullptr;
    hipError_t e = scratch_alloc((void **)&scratch, sizeof(Cand) * blocks, stream);
    if (e != hipSuccess) return fail(HEDDLE_E_NOMEM, "device scratch for argmin partials could not be allocated");
    a.partial = scratch;
    hipLaunchKernelGGL(argmin_pass1, dim3(blocks), dim3(kArgBlock), 0, stream, a);
    Cand *res = result_slot();
    if (!res) {
        (void)hipFreeAsync(scratch, stream);
        return fail(HEDDLE_E_NOMEM, "pinned host memory for the argmin result could not be allocated");
    }
    hipLaunchKernelGGL(argmin_pass2, dim3(1), dim3(kArgBlock), 0, stream, (const Cand *)scratch, blocks, a.f32, res);
    e = hipGetLastError();
    (void)hipFreeAsync(scratch, stream);                       // stream-ordered after pass 2
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e, "argmin");
    Cand h;
    std::memcpy(&h, (const void *)res, sizeof(h));
    if (h.idx < 0) return fail(HEDDLE_E_NOFEASIBLE, "no plan has status OK");
    *h_best_template = h.idx / n_m;
    *h_best_m_index = (int32_t)(h.idx % n_m);
    if (h_best_iter) {
        if (a.f32) {
            const uint32_t bits = (uint32_t)h.iter;
            std::memcpy(h_best_iter, &bits, 4);
        } else {
            const int64_t v = (int64_t)h.iter;
            std::memcpy(h_best_iter, &v, 8);
        }
    }
    return HEDDLE_OK;
}

}  // namespace heddle

using namespace heddle;

extern "C" int heddle_argmin_plans(int64_t n, const int32_t *h_m, int32_t n_m, uint32_t flags,
                                   const void *d_iter, const uint8_t *d_status,
                                   int64_t *h_best_template, int32_t *h_best_m_index, void *h_best_iter,
                                   hipStream_t stream)
{
    if (n < 0 || n_m < 1 || n_m > HEDDLE_MAX_MLIST || !h_m) return fail(HEDDLE_E_INVAL, "bad n / n_m / h_m");
    if (flags & ~(HEDDLE_F_FP32 | HEDDLE_F_COMPUTE_ONLY | HEDDLE_F_DISTRIBUTE)) return fail(HEDDLE_E_INVAL, "unknown flag bits");
    for (int k = 0; k < n_m; k++)
        if (h_m[k] < 1 || h_m[k] > HEDDLE_MAX_M) return fail(HEDDLE_E_INVAL, "m out of range 1..2^24");
    if (!h_best_template || !h_best_m_index) return fail(HEDDLE_E_INVAL, "result pointer is NULL");
    if (n > 0 && (!d_iter || !d_status)) return fail(HEDDLE_E_INVAL, "device pointer is NULL");
    return launch_argmin(n, h_m, n_m, flags, d_iter, d_status, h_best_template, h_best_m_index, h_best_iter,
                         stream);
}

extern "C" int heddle_best_plan(const heddle_profile *p, int64_t n, int32_t s_max,
                                const uint8_t *d_n_stages, const uint32_t *d_stages,
                                const int32_t *h_m, int32_t n_m, uint32_t flags,
                                int64_t *h_best_template, int32_t *h_best_m_index, void *h_best_iter,
                                hipStream_t stream)
{
    int rc = validate_price_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    if (rc) return rc;
    if (!h_best_template || !h_best_m_index) return fail(HEDDLE_E_INVAL, "result pointer is NULL");
    if (n == 0) return fail(HEDDLE_E_NOFEASIBLE, "no plans");
    const size_t total = (size_t)n * n_m;
    // iter | bottleneck | peak_mem | status | layers, one stream-ordered allocation
    const size_t o_iter = 0, o_bn = o_iter + total * 8, o_pk = o_bn + total * 8, o_st = o_pk + total * 8,
                 o_ly = (o_st + total + 255) & ~size_t(255), bytes = o_ly + total * (size_t)s_max;
    unsigned char *buf = nullptr;
    hipError_t e = scratch_alloc((void **)&buf, bytes, stream);
    if (e != hipSuccess) return fail(HEDDLE_E_NOMEM, "device scratch for pricing outputs could not be allocated");
    PriceArgs a;
    std::memset(&a, 0, sizeof(a));
    a.n = n;
    a.s_max = s_max;
    a.n_m = n_m;
    a.flags = (int32_t)flags;
    for (int k = 0; k < n_m; k++) a.m[k] = h_m[k];
    a.n_stages = d_n_stages;
    a.stages = d_stages;
    a.iter = buf + o_iter;
    a.bottleneck = buf + o_bn;
    a.peak_mem = (int64_t *)(buf + o_pk);
    a.status = buf + o_st;
    a.layers = buf + o_ly;
    rc = launch_price(p, a, stream, 0);
    if (rc == HEDDLE_OK)
        rc = launch_argmin(n, h_m, n_m, flags, a.iter, a.status, h_best_template, h_best_m_index, h_best_iter,
                           stream);
    (void)hipFreeAsync(buf, stream);
    if (rc == HEDDLE_OK) {
        e = hipStreamSynchronize(stream);
        if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    }
    return rc;
}
