// BestFill on gfx950 (Heddle, arXiv 2609.34244, section 5.3, arithmetic
// auto-fill): the DP degree of each template from the GPU composition's node
// lists, then the micro-batch size among the profiled sizes (powers of two).
//
// DP degree: the TP group of every stage is packed into the nodes of the
// stage's GPU type (section 5.1: a group goes to a node whose free GPUs equal
// its size, otherwise on a node with more free GPUs), one replica after
// another with the stages in order. Nodes with the same number of free GPUs
// are interchangeable, so a type's nodes are kept as counts per number of
// free GPUs (0..64); a group of t GPUs takes a node from count[t] if there is
// one, else from the smallest c > t with count[c] > 0, which becomes a node
// with c - t free. Types pack independently; D is the smallest number of
// whole replicas over the types used, capped, and rounded down to a multiple
// of the template's largest EP degree so that the template stays valid.
//
// Mapping: one lane per template (64 templates per wavefront). Each lane keeps
// its type's counts in an LDS column of its own ([free GPUs][lane]), so every
// LDS access of a wavefront hits 64 distinct banks; the 64 templates' records
// are read once, coalesced, into LDS columns by stage ([stage][lane]).
//
// Micro-batch size: each size has its own profile (profile entries are keyed
// by GPU type, TP degree and micro-batch size, section 5.2); every template is
// priced once per size at the micro-batch count that covers the global batch,
// and a per-template pass keeps, among the sizes whose plan fits, the one of
// smallest iteration time (the smaller size on ties).
#include <cstring>
#include <vector>

#include "heddle_internal.h"
#include "device_common.h"

struct heddle_cluster {
    int device;
    int n_types, max_gpus;           // max_gpus: largest node, 1..64
    int32_t *counts;                 // device [n_types][65]: nodes with b GPUs
};

namespace heddle {

constexpr int kMaxMbs = 16;

__global__ void __launch_bounds__(64) fill_dp_kernel(const int32_t *counts, int n_types, int max_gpus, int64_t n,
                                                     int s_max, const uint8_t *n_stages, uint32_t *stages,
                                                     int dp_cap, int32_t *dp_out)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x;
    uint32_t *cnt = (uint32_t *)smem + lane;                   // [max_gpus + 1][64]: this lane's column
    uint32_t *rc = (uint32_t *)smem + (max_gpus + 1) * 64;     // [s_max][64]: the block's records, by stage
    auto C = [&](int b) -> uint32_t & { return cnt[b * 64]; };
    uint8_t *lst = (uint8_t *)(rc + s_max * 64) + lane;        // [s_max][64]: one type's TP degrees
    auto R = [&](int s) -> uint32_t { return rc[s * 64 + lane]; };
    for (int64_t t0 = (int64_t)blockIdx.x * 64; t0 < n; t0 += (int64_t)gridDim.x * 64) {
        // the records of the block's 64 templates, read coalesced and stored by stage
        const int nt = n - t0 < 64 ? (int)(n - t0) : 64;
        const uint32_t *src = stages + t0 * s_max;
        __syncthreads();
        for (int d = lane; d < nt * s_max; d += 64) {
            const int q = d / s_max;
            rc[(d - q * s_max) * 64 + q] = src[d];
        }
        __syncthreads();
        const int64_t t = t0 + lane;
        if (t >= n) continue;
        const int S = n_stages[t];
        int D = 0;
        bool ok = S >= 1 && S <= s_max;
        int max_ep = 1;
        for (int s = 0; s < S && ok; s++) {
            const uint32_t r = R(s);
            ok = (int)(r & 0xFF) < n_types && ((r >> 8) & 15) <= 6;
            max_ep = max(max_ep, 1 << ((r >> 12) & 15));
        }
        if (ok) {
            D = dp_cap;
            uint64_t done = 0;                                 // stages whose type is packed
            for (int s = 0; s < S && D > 0; s++) {
                if ((done >> s) & 1) continue;                 // each type once, at its first stage
                const int g = R(s) & 0xFF;
                // the TP degrees (log2) of this type's stages, in stage order
                int k = 0;
                for (int s2 = s; s2 < S; s2++) {
                    const uint32_t r2 = R(s2);
                    if ((int)(r2 & 0xFF) != g) continue;
                    lst[k++ * 64] = (uint8_t)((r2 >> 8) & 15);
                    done |= 1ull << s2;
                }
                // counts per number of free GPUs, and a bit (b - 1) for every b >= 1 with
                // nodes of b free GPUs: the node a group of tp takes is the lowest set bit
                // at or above tp - 1
                uint64_t avail = 0;
                for (int b = 0; b <= max_gpus; b++) {
                    const uint32_t cb = (uint32_t)counts[g * 65 + b];
                    C(b) = cb;
                    if (b > 0 && cb) avail |= 1ull << (b - 1);
                }
                int r = 0;
                while (r < D) {
                    bool placed = true;
                    for (int q = 0; q < k && placed; q++) {
                        const int tp = 1 << lst[q * 64];
                        const uint64_t up = avail >> (tp - 1);
                        placed = up != 0;
                        if (placed) {
                            const int b = tp + __ffsll((unsigned long long)up) - 1;
                            if (--C(b) == 0) avail &= ~(1ull << (b - 1));
                            if (b > tp) {
                                C(b - tp) += 1;
                                avail |= 1ull << (b - tp - 1);
                            }
                        }
                    }
                    if (!placed) break;
                    r++;
                }
                D = r < D ? r : D;
            }
            D = D / max_ep * max_ep;
            uint32_t *rec = stages + t * s_max;
            for (int s = 0; s < S; s++) rec[s] = (R(s) & 0xFFFFu) | ((uint32_t)D << 16);
        }
        dp_out[t] = D;
    }
}

struct SelectArgs {
    int64_t n;
    int32_t s_max, n_mbs;
    bool f32;
    const void *iter[kMaxMbs];
    const void *bottleneck[kMaxMbs];
    const int64_t *peak_mem[kMaxMbs];
    const uint8_t *layers[kMaxMbs];
    const uint8_t *status[kMaxMbs];
    void *o_iter, *o_bottleneck;
    int64_t *o_peak_mem;
    uint8_t *o_layers, *o_status, *o_mbs;
};

__global__ void __launch_bounds__(256) select_mbs_kernel(SelectArgs A)
{
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < A.n; t += (int64_t)gridDim.x * blockDim.x) {
        int best = -1;
        int64_t bi = 0;
        float bf = 0.f;
        for (int b = 0; b < A.n_mbs; b++) {
            if (A.status[b][t] != HEDDLE_S_OK) continue;
            const int64_t xi = A.f32 ? 0 : ((const int64_t *)A.iter[b])[t];
            const float xf = A.f32 ? ((const float *)A.iter[b])[t] : 0.f;
            const bool take = best < 0 || (A.f32 ? xf < bf : xi < bi);
            best = take ? b : best;
            bi = take ? xi : bi;
            bf = take ? xf : bf;
        }
        const int b = best < 0 ? 0 : best;
        if (A.f32) {
            ((float *)A.o_iter)[t] = ((const float *)A.iter[b])[t];
            ((float *)A.o_bottleneck)[t] = ((const float *)A.bottleneck[b])[t];
        } else {
            ((int64_t *)A.o_iter)[t] = ((const int64_t *)A.iter[b])[t];
            ((int64_t *)A.o_bottleneck)[t] = ((const int64_t *)A.bottleneck[b])[t];
        }
        A.o_peak_mem[t] = A.peak_mem[b][t];
        A.o_status[t] = A.status[b][t];
        A.o_mbs[t] = (uint8_t)b;
        for (int s = 0; s < A.s_max; s++) A.o_layers[t * A.s_max + s] = A.layers[b][t * A.s_max + s];
    }
}

static int launch_fill_dp(const heddle_cluster *c, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                          uint32_t *d_stages, int32_t dp_cap, int32_t *d_dp, hipStream_t stream)
{
    if (n == 0) return HEDDLE_OK;
    const size_t lds = ((size_t)(c->max_gpus + 1) + (size_t)s_max) * 64 * 4 + (size_t)s_max * 64;
    const int64_t want = (n + 63) / 64;
    const int blocks = (int)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(fill_dp_kernel, dim3(blocks), dim3(64), lds, stream, (const int32_t *)c->counts, c->n_types,
                       c->max_gpus, n, s_max, d_n_stages, d_stages, dp_cap, d_dp);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

}  // namespace heddle

using namespace heddle;

extern "C" int heddle_load_cluster(const heddle_cluster_desc *d, heddle_cluster **out)
{
    if (!out) return fail(HEDDLE_E_INVAL, "out is NULL");
    *out = nullptr;
    if (!d || !d->n_nodes) return fail(HEDDLE_E_INVAL, "descriptor or n_nodes is NULL");
    if (d->n_types < 1 || d->n_types > HEDDLE_MAX_TYPES) return fail(HEDDLE_E_INVAL, "n_types out of range 1..255");
    std::vector<int32_t> counts((size_t)d->n_types * 65, 0);
    int64_t k = 0;
    int max_gpus = 1;
    for (int g = 0; g < d->n_types; g++) {
        if (d->n_nodes[g] < 0) return fail(HEDDLE_E_INVAL, "n_nodes must be >= 0");
        if (d->n_nodes[g] > 0 && !d->node_gpus) return fail(HEDDLE_E_INVAL, "node_gpus is NULL");
        for (int i = 0; i < d->n_nodes[g]; i++, k++) {
            const int x = d->node_gpus[k];
            if (x < 1 || x > 64) return fail(HEDDLE_E_INVAL, "node sizes must be 1..64 GPUs");
            if (counts[(size_t)g * 65 + x] == INT32_MAX) return fail(HEDDLE_E_RANGE, "too many nodes");
            counts[(size_t)g * 65 + x]++;
            max_gpus = x > max_gpus ? x : max_gpus;
        }
    }
    heddle_cluster *c = new (std::nothrow) heddle_cluster;
    if (!c) return fail(HEDDLE_E_NOMEM, "host allocation failed");
    c->n_types = d->n_types;
    c->max_gpus = max_gpus;
    hipError_t e = hipGetDevice(&c->device);
    if (e == hipSuccess) e = hipMalloc((void **)&c->counts, counts.size() * sizeof(int32_t));
    if (e != hipSuccess) {
        delete c;
        return e == hipErrorOutOfMemory ? fail(HEDDLE_E_NOMEM, "hipMalloc of node counts failed") : hip_fail(e, "cluster");
    }
    e = hipMemcpy(c->counts, counts.data(), counts.size() * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(c->counts);
        delete c;
        return hip_fail(e, "hipMemcpy");
    }
    *out = c;
    return HEDDLE_OK;
}

extern "C" void heddle_free_cluster(heddle_cluster *c)
{
    if (!c) return;
    (void)hipFree(c->counts);
    delete c;
}

static int check_fill_args(const heddle_cluster *c, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                           const uint32_t *d_stages, int32_t dp_cap, const int32_t *d_dp)
{
    if (!c) return fail(HEDDLE_E_INVAL, "cluster is NULL");
    if (n < 0) return fail(HEDDLE_E_INVAL, "n < 0");
    if (s_max < 1 || s_max > HEDDLE_MAX_STAGES) return fail(HEDDLE_E_INVAL, "s_max out of range 1..64");
    if (dp_cap < 1 || dp_cap > 0xFFFF) return fail(HEDDLE_E_INVAL, "dp_cap out of range 1..65535");
    if (n > 0 && (!d_n_stages || !d_stages || !d_dp)) return fail(HEDDLE_E_INVAL, "device pointer is NULL");
    int dev = -1;
    HEDDLE_HIP(hipGetDevice(&dev));
    if (dev != c->device) return fail(HEDDLE_E_INVAL, "cluster was loaded on another device");
    return HEDDLE_OK;
}

extern "C" int heddle_fill_dp(const heddle_cluster *c, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                              uint32_t *d_stages, int32_t dp_cap, int32_t *d_dp, hipStream_t stream)
{
    int rc = check_fill_args(c, n, s_max, d_n_stages, d_stages, dp_cap, d_dp);
    if (rc) return rc;
    return launch_fill_dp(c, n, s_max, d_n_stages, d_stages, dp_cap, d_dp, stream);
}

extern "C" int heddle_fill_plans(const heddle_profile *const *profiles, const int32_t *h_mbs, int32_t n_mbs,
                                 const heddle_cluster *c, int64_t global_batch, int32_t dp_cap, int64_t n,
                                 int32_t s_max, const uint8_t *d_n_stages, uint32_t *d_stages, uint32_t flags,
                                 void *d_iter, void *d_bottleneck, int64_t *d_peak_mem, uint8_t *d_layers,
                                 uint8_t *d_status, int32_t *d_dp, uint8_t *d_mbs_index, hipStream_t stream)
{
    if (!profiles || !h_mbs || n_mbs < 1 || n_mbs > kMaxMbs) return fail(HEDDLE_E_INVAL, "1..16 micro-batch sizes");
    if (global_batch < 1) return fail(HEDDLE_E_INVAL, "global_batch < 1");
    int rc = check_fill_args(c, n, s_max, d_n_stages, d_stages, dp_cap, d_dp);
    if (rc) return rc;
    if (n > 0 && (!d_iter || !d_bottleneck || !d_peak_mem || !d_layers || !d_status || !d_mbs_index))
        return fail(HEDDLE_E_INVAL, "output pointer is NULL");
    int32_t m_of[kMaxMbs];
    for (int b = 0; b < n_mbs; b++) {
        if (!profiles[b]) return fail(HEDDLE_E_INVAL, "profile is NULL");
        if (h_mbs[b] < 1 || (b > 0 && h_mbs[b] <= h_mbs[b - 1])) return fail(HEDDLE_E_INVAL, "sizes must be ascending and >= 1");
        if (profiles[b]->dev.L != profiles[0]->dev.L) return fail(HEDDLE_E_INVAL, "profiles of different L");
        const int64_t m = (global_batch + h_mbs[b] - 1) / h_mbs[b];
        if (m > HEDDLE_MAX_M) return fail(HEDDLE_E_INVAL, "micro-batch count above 2^24");
        m_of[b] = (int32_t)m;
        // placeholders stand for the template pointers, checked above
        rc = validate_price_args(profiles[b], n, s_max, (const uint8_t *)1, (const uint32_t *)1, &m_of[b], 1, flags);
        if (rc) return rc;
    }
    if (n == 0) return HEDDLE_OK;
    rc = launch_fill_dp(c, n, s_max, d_n_stages, d_stages, dp_cap, d_dp, stream);
    if (rc) return rc;
    // per size: iter | bottleneck | peak_mem | status | layers
    const size_t un = (size_t)n, o_it = 0, o_bn = un * 8, o_pk = o_bn + un * 8, o_st = o_pk + un * 8,
                 o_ly = (o_st + un + 255) & ~size_t(255), per = (o_ly + un * s_max + 255) & ~size_t(255);
    unsigned char *buf = nullptr;
    hipError_t e = scratch_alloc((void **)&buf, per * n_mbs, stream);
    if (e != hipSuccess) return fail(HEDDLE_E_NOMEM, "device scratch for per-size outputs could not be allocated");
    SelectArgs sa;
    std::memset(&sa, 0, sizeof(sa));
    sa.n = n;
    sa.s_max = s_max;
    sa.n_mbs = n_mbs;
    sa.f32 = (flags & HEDDLE_F_FP32) != 0;
    for (int b = 0; b < n_mbs && rc == HEDDLE_OK; b++) {
        unsigned char *base = buf + per * b;
        PriceArgs a;
        std::memset(&a, 0, sizeof(a));
        a.n = n;
        a.s_max = s_max;
        a.n_m = 1;
        a.flags = (int32_t)flags;
        a.m[0] = m_of[b];
        a.n_stages = d_n_stages;
        a.stages = d_stages;
        a.iter = base + o_it;
        a.bottleneck = base + o_bn;
        a.peak_mem = (int64_t *)(base + o_pk);
        a.status = base + o_st;
        a.layers = base + o_ly;
        rc = launch_price(profiles[b], a, stream, 0);
        sa.iter[b] = a.iter;
        sa.bottleneck[b] = a.bottleneck;
        sa.peak_mem[b] = a.peak_mem;
        sa.layers[b] = a.layers;
        sa.status[b] = a.status;
    }
    if (rc == HEDDLE_OK) {
        sa.o_iter = d_iter;
        sa.o_bottleneck = d_bottleneck;
        sa.o_peak_mem = d_peak_mem;
        sa.o_layers = d_layers;
        sa.o_status = d_status;
        sa.o_mbs = d_mbs_index;
        const int64_t want = (n + 255) / 256;
        const int blocks = (int)(want < 65536 ? want : 65536);
        hipLaunchKernelGGL(select_mbs_kernel, dim3(blocks), dim3(256), 0, stream, sa);
        e = hipGetLastError();
        if (e != hipSuccess) rc = hip_fail(e, "select_mbs_kernel");
    }
    (void)hipFreeAsync(buf, stream);
    if (rc == HEDDLE_OK) {
        e = hipStreamSynchronize(stream);
        if (e != hipSuccess) rc = hip_fail(e, "hipStreamSynchronize");
    }
    return rc;
}
