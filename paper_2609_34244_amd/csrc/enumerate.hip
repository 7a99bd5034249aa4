// Exhaustive structural enumeration on gfx950: the search backbone that the
// planners Heddle analyses share (arXiv 2609.34244, section 3.1: loops over
// the stage count, the GPU type of every stage, the TP degree of every stage
// and the DP degree, with a layer split and an Evaluate per configuration),
// run as one data-parallel workload. Section 2 counts (N * K)^D structures
// for N GPU types, K TP degrees and D stages.
//
// Order of the space, outermost first: the stage count S = 1 .. d_max; the
// type vector (g_0 .. g_{S-1}), each entry running over the spec's type list
// in list order with g_0 slowest; the TP vector, likewise; the DP degree
// over the spec's DP list. Index u of this order is decoded independently by
// each thread (mixed radix, least significant digit first), so any range of
// the space can be generated on the device without a host list. The micro-
// batch count m is the innermost loop, as the m axis of heddle_price_plans.
//
// heddle_best_enumerated walks the whole space in chunks: generate, price
// (the split and evaluate kernels of heddle_price_plans), argmin, and keeps
// the best plan over the chunks (strictly better replaces, so ties keep the
// lowest index, as the argmin does inside a chunk).
#include <cstring>

#include "heddle_internal.h"

namespace heddle {

constexpr int kEnumMaxDp = 64;

struct EnumArgs {
    int64_t first, n;
    int32_t d_max, n_g, n_k, n_dp;
    uint32_t ep_bits;                      // log2 EP, already shifted into place
    uint8_t types[256];
    uint8_t log2_tp[16];
    int32_t dp[kEnumMaxDp];
    int64_t start[kMaxStages + 1];         // start[S - 1]: index of the first template with S stages
    uint8_t *n_stages;
    uint32_t *stages;
};

// x /= d, returns x % d (32-bit division when x fits)
__device__ __forceinline__ uint32_t divmod(uint64_t &x, uint32_t d)
{
    if ((x >> 32) == 0) {
        const uint32_t x32 = (uint32_t)x, q = x32 / d;
        x = q;
        return x32 - q * d;
    }
    const uint64_t q = x / d;
    const uint32_t r = (uint32_t)(x - q * d);
    x = q;
    return r;
}

__global__ void __launch_bounds__(256) enum_kernel(EnumArgs E)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < E.n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t u = E.first + i;
        int S = 1;
        while (u >= E.start[S]) S++;                       // start[d_max] = the size of the space
        uint64_t r = (uint64_t)(u - E.start[S - 1]);
        const uint32_t di = divmod(r, (uint32_t)E.n_dp);
        // r = type-vector index * n_k^S + TP-vector index
        uint64_t kpow = 1;
        for (int s = 0; s < S; s++) kpow *= (uint64_t)E.n_k;
        uint64_t g_idx = r / kpow;
        uint64_t t_idx = r - g_idx * kpow;
        const uint32_t common = E.ep_bits | ((uint32_t)E.dp[di] << 16);
        uint32_t *rec = E.stages + i * E.d_max;
        for (int s = S - 1; s >= 0; s--) {
            const uint32_t k = divmod(t_idx, (uint32_t)E.n_k);
            const uint32_t g = divmod(g_idx, (uint32_t)E.n_g);
            rec[s] = common | ((uint32_t)E.log2_tp[k] << 8) | E.types[g];
        }
        for (int s = S; s < E.d_max; s++) rec[s] = 0u;
        E.n_stages[i] = (uint8_t)S;
    }
}

// spec checks and the start index of every stage count; returns the size of
// the space in *total
static int setup_enum(const heddle_enum_spec *sp, EnumArgs &E, int64_t *total)
{
    if (!sp) return fail(HEDDLE_E_INVAL, "spec is NULL");
    if (sp->d_max < 1 || sp->d_max > HEDDLE_MAX_STAGES) return fail(HEDDLE_E_INVAL, "d_max out of range 1..64");
    if (sp->n_types < 1 || sp->n_types > 255 || !sp->types) return fail(HEDDLE_E_INVAL, "type list empty or too long");
    if (sp->n_tp < 1 || sp->n_tp > 16 || !sp->log2_tp) return fail(HEDDLE_E_INVAL, "TP list empty or too long");
    if (sp->n_dp < 1 || sp->n_dp > kEnumMaxDp || !sp->dp) return fail(HEDDLE_E_INVAL, "DP list empty or too long");
    if (sp->log2_ep < 0 || sp->log2_ep > 15) return fail(HEDDLE_E_INVAL, "log2_ep out of range 0..15");
    std::memset(&E, 0, sizeof(E));
    bool seen[256] = {false};
    for (int i = 0; i < sp->n_types; i++) {
        if (seen[sp->types[i]]) return fail(HEDDLE_E_INVAL, "duplicate GPU type in the type list");
        seen[sp->types[i]] = true;
        E.types[i] = sp->types[i];
    }
    uint32_t tp_seen = 0;
    for (int i = 0; i < sp->n_tp; i++) {
        const uint8_t l = sp->log2_tp[i];
        if (l > 15) return fail(HEDDLE_E_INVAL, "log2 TP out of range 0..15");
        if ((tp_seen >> l) & 1) return fail(HEDDLE_E_INVAL, "duplicate TP degree in the TP list");
        tp_seen |= 1u << l;
        E.log2_tp[i] = l;
    }
    for (int i = 0; i < sp->n_dp; i++) {
        if (sp->dp[i] < 1 || sp->dp[i] > 0xFFFF) return fail(HEDDLE_E_INVAL, "DP degree out of range 1..65535");
        for (int j = 0; j < i; j++)
            if (sp->dp[j] == sp->dp[i]) return fail(HEDDLE_E_INVAL, "duplicate DP degree in the DP list");
        E.dp[i] = sp->dp[i];
    }
    E.d_max = sp->d_max;
    E.n_g = sp->n_types;
    E.n_k = sp->n_tp;
    E.n_dp = sp->n_dp;
    E.ep_bits = (uint32_t)sp->log2_ep << 12;
    // start[S] = sum over d <= S of (n_g * n_k)^d * n_dp, all below 2^62
    const unsigned __int128 base = (unsigned __int128)sp->n_types * (unsigned)sp->n_tp;
    unsigned __int128 block = (unsigned)sp->n_dp, acc = 0;
    E.start[0] = 0;
    for (int d = 1; d <= sp->d_max; d++) {
        block *= base;
        acc += block;
        if (acc >= (unsigned __int128)kLimit62) return fail(HEDDLE_E_RANGE, "the space has 2^62 or more templates");
        E.start[d] = (int64_t)acc;
    }
    for (int d = sp->d_max + 1; d <= kMaxStages; d++) E.start[d] = E.start[sp->d_max];
    *total = E.start[sp->d_max];
    return HEDDLE_OK;
}

static int launch_enum(EnumArgs &E, hipStream_t stream)
{
    if (E.n == 0) return HEDDLE_OK;
    const int64_t want = (E.n + 255) / 256;
    const int blocks = (int)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(enum_kernel, dim3(blocks), dim3(256), 0, stream, E);
    HEDDLE_HIP(hipGetLastError());
    return HEDDLE_OK;
}

__global__ void __launch_bounds__(256) count_ok_kernel(const uint8_t *status, int64_t total, unsigned long long *out)
{
    unsigned long long c = 0;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total; o += (int64_t)gridDim.x * blockDim.x)
        c += status[o] == HEDDLE_S_OK;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
    if ((threadIdx.x & 63) == 0 && c) atomicAdd(out, c);
}

// iter_a / m_a < iter_b / m_b, exactly (the argmin's key)
static bool key_less(bool f32, int64_t ia, float fa, int32_t ma, int64_t ib, float fb, int32_t mb)
{
    if (f32) return (double)fa * (double)mb < (double)fb * (double)ma;
    return (unsigned __int128)ia * (uint32_t)mb < (unsigned __int128)ib * (uint32_t)ma;
}

}  // namespace heddle

using namespace heddle;

extern "C" int heddle_enum_count(const heddle_enum_spec *sp, int64_t *h_count)
{
    if (!h_count) return fail(HEDDLE_E_INVAL, "h_count is NULL");
    EnumArgs E;
    return setup_enum(sp, E, h_count);
}

extern "C" int heddle_enum_templates(const heddle_enum_spec *sp, int64_t first, int64_t n, uint8_t *d_n_stages,
                                     uint32_t *d_stages, hipStream_t stream)
{
    EnumArgs E;
    int64_t total = 0;
    int rc = setup_enum(sp, E, &total);
    if (rc) return rc;
    if (first < 0 || n < 0 || first > total || n > total - first) return fail(HEDDLE_E_INVAL, "range outside the space");
    if (n > 0 && (!d_n_stages || !d_stages)) return fail(HEDDLE_E_INVAL, "output pointer is NULL");
    E.first = first;
    E.n = n;
    E.n_stages = d_n_stages;
    E.stages = d_stages;
    return launch_enum(E, stream);
}

extern "C" int heddle_best_enumerated(const heddle_profile *p, const heddle_enum_spec *sp, const int32_t *h_m,
                                      int32_t n_m, uint32_t flags, int64_t chunk, int64_t *h_best_index,
                                      int32_t *h_best_m_index, void *h_best_iter, int64_t *h_n_ok,
                                      hipStream_t stream)
{
    EnumArgs E;
    int64_t total = 0;
    int rc = setup_enum(sp, E, &total);
    if (rc) return rc;
    if (!h_best_index || !h_best_m_index) return fail(HEDDLE_E_INVAL, "result pointer is NULL");
    if (chunk < 0) return fail(HEDDLE_E_INVAL, "chunk < 0");
    if (chunk == 0) chunk = int64_t(1) << 22;
    if (chunk > total) chunk = total;
    // the price arguments are checked once, as for a chunk (non-null placeholders)
    rc = validate_price_args(p, chunk, sp->d_max, (const uint8_t *)1, (const uint32_t *)1, h_m, n_m, flags);
    if (rc) return rc;
    const int s_max = sp->d_max;
    const size_t c = (size_t)chunk, cm = c * (size_t)n_m;
    // templates | iter | bottleneck | peak_mem | status | layers | OK counter
    const size_t o_ns = 0, o_st = (o_ns + c + 255) & ~size_t(255), o_it = (o_st + c * 4 * s_max + 255) & ~size_t(255),
                 o_bn = o_it + cm * 8, o_pk = o_bn + cm * 8, o_ss = o_pk + cm * 8,
                 o_ly = (o_ss + cm + 255) & ~size_t(255), o_ok = (o_ly + cm * s_max + 255) & ~size_t(255),
                 bytes = o_ok + 8;
    unsigned char *buf = nullptr;
    hipError_t e = scratch_alloc((void **)&buf, bytes, stream);
    if (e != hipSuccess) return fail(HEDDLE_E_NOMEM, "device scratch for the enumeration buffers could not be allocated");
    unsigned long long *d_ok = (unsigned long long *)(buf + o_ok);
    e = hipMemsetAsync(d_ok, 0, 8, stream);
    if (e != hipSuccess) {
        (void)hipFreeAsync(buf, stream);
        return hip_fail(e, "hipMemsetAsync");
    }
    const bool f32 = flags & HEDDLE_F_FP32;
    bool found = false;
    int64_t best_idx = -1, best_i = 0;
    int32_t best_k = -1;
    float best_f = 0.f;
    for (int64_t first = 0; first < total && rc == HEDDLE_OK; first += chunk) {
        const int64_t n = total - first < chunk ? total - first : chunk;
        E.first = first;
        E.n = n;
        E.n_stages = buf + o_ns;
        E.stages = (uint32_t *)(buf + o_st);
        rc = launch_enum(E, stream);
        if (rc) break;
        PriceArgs a;
        std::memset(&a, 0, sizeof(a));
        a.n = n;
        a.s_max = s_max;
        a.n_m = n_m;
        a.flags = (int32_t)flags;
        for (int k = 0; k < n_m; k++) a.m[k] = h_m[k];
        a.n_stages = E.n_stages;
        a.stages = E.stages;
        a.iter = buf + o_it;
        a.bottleneck = buf + o_bn;
        a.peak_mem = (int64_t *)(buf + o_pk);
        a.status = buf + o_ss;
        a.layers = buf + o_ly;
        rc = launch_price(p, a, stream, 0);
        if (rc) break;
        if (h_n_ok) {
            const int64_t want = ((int64_t)n * n_m + 255) / 256;
            const int blocks = (int)(want < 4096 ? want : 4096);
            hipLaunchKernelGGL(count_ok_kernel, dim3(blocks), dim3(256), 0, stream, (const uint8_t *)a.status,
                               (int64_t)n * n_m, d_ok);
            e = hipGetLastError();
            if (e != hipSuccess) {
                rc = hip_fail(e, "count_ok_kernel");
                break;
            }
        }
        int64_t t = -1, it_i = 0;
        int32_t k = -1;
        float it_f = 0.f;
        rc = launch_argmin(n, h_m, n_m, flags, a.iter, a.status, &t, &k, f32 ? (void *)&it_f : (void *)&it_i,
                           stream);
        if (rc == HEDDLE_E_NOFEASIBLE) {
            rc = HEDDLE_OK;
            continue;
        }
        if (rc) break;
        if (!found || key_less(f32, it_i, it_f, h_m[k], best_i, best_f, h_m[best_k])) {
            found = true;
            best_idx = first + t;
            best_k = k;
            best_i = it_i;
            best_f = it_f;
        }
    }
    unsigned long long n_ok = 0;
    if (rc == HEDDLE_OK && h_n_ok) {
        e = hipMemcpyAsync(&n_ok, d_ok, 8, hipMemcpyDeviceToHost, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) rc = hip_fail(e, "reading the OK count");
    }
    (void)hipFreeAsync(buf, stream);
    if (rc == HEDDLE_OK) {
        e = hipStreamSynchronize(stream);
        if (e != hipSuccess) rc = hip_fail(e, "hipStreamSynchronize");
    }
    if (rc) return rc;
    if (h_n_ok) *h_n_ok = (int64_t)n_ok;
    if (!found) return fail(HEDDLE_E_NOFEASIBLE, "no plan of the space has status OK");
    *h_best_index = best_idx;
    *h_best_m_index = best_k;
    if (h_best_iter) {
        if (f32) *(float *)h_best_iter = best_f;
        else *(int64_t *)h_best_iter = best_i;
    }
    return HEDDLE_OK;
}
