// Profile loading: validation of the descriptor, derived prefix tables and
// transfer-time terms, range proofs, and upload to the device.
//
// Derived tables follow the profile-based cost model (Heddle, section 5.2):
// per-(type, TP) layer costs are summed into prefix rows so that a stage's
// time over layers [i, j) is one subtraction; memory and gradient bytes per
// TP degree likewise. Transfer times of the MoE all-to-all (section 5.3,
// expert tiling) and the inter-stage p2p are precomputed per type and per
// type pair.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <vector>

#include "heddle_internal.h"

namespace heddle {

static thread_local std::string g_last_error;

void set_error(const std::string &msg) { g_last_error = msg; }

int fail(int code, const std::string &msg)
{
    g_last_error = msg;
    return code;
}

int hip_fail(hipError_t e, const char *what)
{
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return HEDDLE_E_DEVICE;
}

// Stream-ordered scratch of every entry point comes from one memory pool per
// device that the library owns. Its release threshold keeps freed blocks
// mapped between calls (a pool that hands them back at every synchronisation
// pays a fresh mapping on the next call); they go back when the process ends.
static std::mutex g_pool_mu;
static hipMemPool_t g_pool[kMaxDevices];

hipError_t scratch_alloc(void **ptr, size_t bytes, hipStream_t stream)
{
    int dev = 0;
    hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    hipMemPool_t pool = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_pool_mu);
        if (!g_pool[dev]) {
            hipMemPoolProps props;
            std::memset(&props, 0, sizeof(props));
            props.allocType = hipMemAllocationTypePinned;
            props.location.type = hipMemLocationTypeDevice;
            props.location.id = dev;
            hipMemPool_t created = nullptr;
            e = hipMemPoolCreate(&created, &props);
            if (e != hipSuccess) return e;
            uint64_t keep = UINT64_MAX;
            e = hipMemPoolSetAttribute(created, hipMemPoolAttrReleaseThreshold, &keep);
            if (e != hipSuccess) {
                (void)hipMemPoolDestroy(created);
                return e;
            }
            g_pool[dev] = created;
        }
        pool = g_pool[dev];
    }
    return hipMallocFromPoolAsync(ptr, bytes, pool, stream);
}

int profile_scratch(const heddle_profile *p, hipStream_t stream, size_t bytes, void **ptr, bool *owned)
{
    *ptr = nullptr;
    *owned = false;
    if (stream == hipStreamPerThread) {
        if (scratch_alloc(ptr, bytes, stream) != hipSuccess) return fail(HEDDLE_E_NOMEM, "device scratch could not be allocated");
        *owned = true;
        return HEDDLE_OK;
    }
    heddle_profile::Scratch *slot = nullptr;
    for (auto &sl : p->scratch)
        if (sl.stream == stream) slot = &sl;
    if (!slot) {
        hipEvent_t ev = nullptr;
        HEDDLE_HIP(hipEventCreateWithFlags(&ev, hipEventDisableTiming));
        try {
            p->scratch.push_back({stream, nullptr, 0, ev});
        } catch (...) {
            (void)hipEventDestroy(ev);
            return fail(HEDDLE_E_NOMEM, "host allocation failed");
        }
        slot = &p->scratch.back();
    } else {
        // the last use was on this handle; should the stream have been
        // destroyed and the handle reused, the wait orders this call after it
        HEDDLE_HIP(hipStreamWaitEvent(stream, slot->done, 0));
    }
    if (slot->bytes < bytes) {
        if (slot->ptr) HEDDLE_HIP(hipFreeAsync(slot->ptr, stream));
        slot->ptr = nullptr;
        slot->bytes = 0;
        const size_t want = (bytes + (size_t(1) << 21) - 1) & ~((size_t(1) << 21) - 1);   // 2 MiB steps
        if (scratch_alloc(&slot->ptr, want, stream) != hipSuccess) {
            slot->ptr = nullptr;
            return fail(HEDDLE_E_NOMEM, "device scratch could not be allocated");
        }
        slot->bytes = want;
    }
    *ptr = slot->ptr;
    return HEDDLE_OK;
}

int profile_scratch_done(const heddle_profile *p, hipStream_t stream, void *ptr, bool owned)
{
    if (owned) {
        HEDDLE_HIP(hipFreeAsync(ptr, stream));
        return HEDDLE_OK;
    }
    for (auto &sl : p->scratch)
        if (sl.stream == stream) HEDDLE_HIP(hipEventRecord(sl.done, stream));
    return HEDDLE_OK;
}

typedef __int128 i128;

// ceil(b * 1000 / MBps) ns: b bytes at MBps megabytes per second
static i128 transfer_ns(int64_t bytes, int64_t MBps) { return ((i128)bytes * 1000 + MBps - 1) / MBps; }

static int log2_exact(int32_t v)
{
    if (v < 1 || (v & (v - 1))) return -1;
    int l = 0;
    while ((1 << l) < v) l++;
    return l;
}

// exponent of the lowest set bit of a positive finite float (v = odd * 2^e)
static int low_bit_exp(float v)
{
    int e;
    double fr = std::frexp((double)v, &e);
    int64_t mant = (int64_t)std::ldexp(fr, 24);   // exact 24-bit integer
    int tz = 0;
    while (!(mant & 1)) { mant >>= 1; tz++; }
    return e - 24 + tz;
}

struct Builder {
    std::vector<unsigned char> bytes;
    size_t add(const void *src, size_t n)
    {
        size_t off = (bytes.size() + 255) & ~size_t(255);
        bytes.resize(off + n);
        std::memcpy(bytes.data() + off, src, n);
        return off;
    }
    template <class T> size_t add(const std::vector<T> &v) { return add(v.data(), v.size() * sizeof(T)); }
};

}  // namespace heddle

using namespace heddle;

extern "C" const char *heddle_last_error(void) { return g_last_error.c_str(); }

extern "C" int heddle_load_profile(const heddle_profile_desc *d, heddle_profile **out)
{
    if (!out) return fail(HEDDLE_E_INVAL, "out is NULL");
    *out = nullptr;
    if (!d) return fail(HEDDLE_E_INVAL, "descriptor is NULL");
    const int L = d->L, N = d->n_types, K = d->n_tp, E = d->n_ep;
    if (L < 1 || L > HEDDLE_MAX_LAYERS) return fail(HEDDLE_E_INVAL, "L out of range 1..255");
    if (N < 1 || N > HEDDLE_MAX_TYPES) return fail(HEDDLE_E_INVAL, "n_types out of range 1..255");
    if (K < 1 || K > 16 || E < 1 || E > 16) return fail(HEDDLE_E_INVAL, "n_tp / n_ep out of range 1..16");
    if (!d->tp_degrees || !d->ep_degrees || !d->layer_ns || !d->profiled || !d->is_moe || !d->state_bytes ||
        !d->xstate_bytes || !d->act_bytes || !d->grad_bytes || !d->xgrad_bytes || !d->mem_cap_bytes ||
        !d->node_size || !d->n_gpus || !d->intra_bw_MBps || !d->link_bw_MBps)
        return fail(HEDDLE_E_INVAL, "a required table pointer is NULL");

    DevProfile dp;
    std::memset(&dp, 0, sizeof(dp));
    dp.L = L; dp.n_types = N; dp.n_tp = K; dp.n_ep = E;
    for (int k = 0; k < K; k++) {
        int l = log2_exact(d->tp_degrees[k]);
        if (l < 0 || l > 15 || ((dp.tp_present >> l) & 1)) return fail(HEDDLE_E_INVAL, "tp_degrees must be distinct powers of two <= 32768");
        dp.tp_present |= 1u << l;
        dp.tp_index |= (uint64_t)k << (4 * l);
        dp.tp_log2 |= (uint64_t)l << (4 * k);
    }
    for (int e = 0; e < E; e++) {
        int l = log2_exact(d->ep_degrees[e]);
        if (l < 0 || l > 15 || ((dp.ep_present >> l) & 1)) return fail(HEDDLE_E_INVAL, "ep_degrees must be distinct powers of two <= 32768");
        dp.ep_present |= 1u << l;
        dp.ep_index |= (uint64_t)e << (4 * l);
        dp.ep_log2 |= (uint64_t)l << (4 * e);
    }
    for (int g = 0; g < N; g++) {
        if (d->node_size[g] < 1) return fail(HEDDLE_E_INVAL, "node_size must be >= 1");
        if (d->n_gpus[g] < 0 || d->mem_cap_bytes[g] < 0) return fail(HEDDLE_E_INVAL, "negative GPU count or memory");
        if (d->intra_bw_MBps[g] < 1 || d->intra_bw_MBps[g] > kMaxBandwidth)
            return fail(HEDDLE_E_INVAL, "bandwidths must be in 1 .. 2^34-1 MB/s");
        for (int h = 0; h < N; h++)
            if (d->link_bw_MBps[g * N + h] < 1 || d->link_bw_MBps[g * N + h] > kMaxBandwidth)
                return fail(HEDDLE_E_INVAL, "bandwidths must be in 1 .. 2^34-1 MB/s");
    }
    if (d->boundary_bytes < 0 || d->a2a_bytes < 0 || d->boundary_bytes > kLimit62 / 2000 ||
        d->a2a_bytes > kLimit62 / 1000)
        return fail(HEDDLE_E_RANGE, "boundary_bytes / a2a_bytes out of range");

    const size_t R = (size_t)L + 1;
    int n_moe = 0;
    std::vector<int32_t> pre_moe(R, 0);
    for (int l = 0; l < L; l++) {
        n_moe += d->is_moe[l] ? 1 : 0;
        pre_moe[l + 1] = n_moe;
    }

    // ---- int64 time prefix rows and transfer terms
    std::vector<int64_t> pre_time((size_t)N * K * R);
    for (int g = 0; g < N; g++)
        for (int k = 0; k < K; k++) {
            i128 acc = 0;
            int64_t *row = &pre_time[((size_t)g * K + k) * R];
            row[0] = 0;
            for (int l = 0; l < L; l++) {
                int64_t c = d->layer_ns[((size_t)g * K + k) * L + l];
                if (c < 1) return fail(HEDDLE_E_INVAL, "layer_ns entries must be >= 1 ns");
                acc += c;
                if (acc >= kLimit62) return fail(HEDDLE_E_RANGE, "layer_ns row total exceeds 2^62");
                row[l + 1] = (int64_t)acc;
            }
        }
    std::vector<int64_t> a2a_ns((size_t)N * 3), p2p_ns((size_t)N * N);
    for (int g = 0; g < N; g++) {
        a2a_ns[g * 3 + kA2ANone] = 0;
        a2a_ns[g * 3 + kA2AIntra] = (int64_t)transfer_ns(d->a2a_bytes, d->intra_bw_MBps[g]);
        a2a_ns[g * 3 + kA2AInter] = (int64_t)transfer_ns(d->a2a_bytes, d->link_bw_MBps[g * N + g]);
        for (int h = 0; h < N; h++) p2p_ns[g * N + h] = (int64_t)transfer_ns(2 * d->boundary_bytes, d->link_bw_MBps[g * N + h]);
    }
    // bound on any stage time: full row + all-to-all on every MoE layer + the largest p2p
    i128 max_stage = 0;
    for (int g = 0; g < N; g++)
        for (int k = 0; k < K; k++) {
            int64_t a2a_max = a2a_ns[g * 3 + 1] > a2a_ns[g * 3 + 2] ? a2a_ns[g * 3 + 1] : a2a_ns[g * 3 + 2];
            int64_t p2p_max = 0;
            for (int h = 0; h < N; h++) p2p_max = p2p_ns[g * N + h] > p2p_max ? p2p_ns[g * N + h] : p2p_max;
            i128 b = (i128)pre_time[((size_t)g * K + k) * R + L] + (i128)n_moe * a2a_max + p2p_max;
            if (b > max_stage) max_stage = b;
        }
    if (max_stage >= kLimit62) return fail(HEDDLE_E_RANGE, "stage times could exceed 2^62 ns");

    // ---- memory and gradient prefix rows
    std::vector<int64_t> pre_state((size_t)K * E * R), pre_act((size_t)K * R), pre_grad((size_t)K * R),
        pre_xgrad((size_t)K * E * R);
    i128 max_grad = 0;
    for (int k = 0; k < K; k++) {
        i128 a = 0, gsum = 0;
        pre_act[k * R] = pre_grad[k * R] = 0;
        for (int l = 0; l < L; l++) {
            int64_t av = d->act_bytes[(size_t)k * L + l], gv = d->grad_bytes[(size_t)k * L + l];
            if (av < 0 || gv < 0) return fail(HEDDLE_E_INVAL, "byte counts must be >= 0");
            a += av;
            gsum += gv;
            if (a >= kLimit62 / 64 || gsum >= kLimit62 / 4096) return fail(HEDDLE_E_RANGE, "byte totals too large");
            pre_act[k * R + l + 1] = (int64_t)a;
            pre_grad[k * R + l + 1] = (int64_t)gsum;
        }
        for (int e = 0; e < E; e++) {
            const int64_t ep = d->ep_degrees[e];
            i128 w = 0, xg = 0;
            pre_state[(k * E + e) * R] = pre_xgrad[(k * E + e) * R] = 0;
            for (int l = 0; l < L; l++) {
                int64_t sv = d->state_bytes[(size_t)k * L + l], xv = d->xstate_bytes[(size_t)k * L + l];
                int64_t xgv = d->xgrad_bytes[(size_t)k * L + l];
                if (sv < 0 || xv < 0 || xgv < 0) return fail(HEDDLE_E_INVAL, "byte counts must be >= 0");
                w += (i128)sv + (xv + ep - 1) / ep;
                xg += (xgv + ep - 1) / ep;
                if (w >= kLimit62 / 2 || xg >= kLimit62 / 4096) return fail(HEDDLE_E_RANGE, "byte totals too large");
                pre_state[(k * E + e) * R + l + 1] = (int64_t)w;
                pre_xgrad[(k * E + e) * R + l + 1] = (int64_t)xg;
            }
            if (gsum + xg > max_grad) max_grad = gsum + xg;
        }
    }
    std::vector<int64_t> pair_sx(pre_state.size() * 2), pair_ag(pre_act.size() * 2);
    for (size_t x = 0; x < pre_state.size(); x++) {
        pair_sx[2 * x] = pre_state[x];
        pair_sx[2 * x + 1] = pre_xgrad[x];
    }
    for (size_t x = 0; x < pre_act.size(); x++) {
        pair_ag[2 * x] = pre_act[x];
        pair_ag[2 * x + 1] = pre_grad[x];
    }
    // Memory limits of a stage (section 5.2 memory validation): for GPU type g,
    // TP index k, EP index e and f micro-batches of activations in flight,
    // lim[i] is the largest end j >= i such that layers [i, j) fit one GPU's
    // memory. Ends that fit form a prefix because every term is non-negative,
    // so one two-pointer sweep per (g, k, e, f) builds a row; lim is
    // non-decreasing in i. Each limit row is followed by its inverse,
    // inv[x] = the smallest i with lim[i] >= x (lim[L] = L, so x <= L always
    // has one). Half-rows are padded to a multiple of 16 bytes so kernels copy
    // them as dwords.
    const int F = std::min(L, HEDDLE_MAX_STAGES);
    const int RL = (R + 15) & ~15;
    const size_t lim_entries = (size_t)N * K * E * F * 2 * RL;
    if (lim_entries > kMaxLimitTable) return fail(HEDDLE_E_RANGE, "memory-limit table would exceed 256 MB");
    std::vector<uint8_t> lim_tab(lim_entries, 0);
    for (int g = 0; g < N; g++)
        for (int k = 0; k < K; k++)
            for (int e = 0; e < E; e++)
                for (int f = 1; f <= F; f++) {
                    const int64_t *w = &pre_state[(k * E + e) * R], *a = &pre_act[k * R];
                    uint8_t *row = &lim_tab[((((size_t)g * K + k) * E + e) * F + (f - 1)) * 2 * RL];
                    uint8_t *inv = row + RL;
                    int j = 0;
                    for (int i = 0; i <= L; i++) {
                        if (j < i) j = i;
                        while (j < L && (w[j + 1] - w[i]) + (i128)f * (a[j + 1] - a[i]) <= d->mem_cap_bytes[g]) j++;
                        row[i] = (uint8_t)j;
                    }
                    int i = 0;
                    for (int x = 0; x <= L; x++) {
                        while (row[i] < x) i++;
                        inv[x] = (uint8_t)i;
                    }
                }
    // gradient synchronisation is below 2 * bytes * 1000 / min bandwidth (+1 per ceiling)
    int64_t min_bw = INT64_MAX;
    for (int g = 0; g < N; g++) {
        min_bw = d->intra_bw_MBps[g] < min_bw ? d->intra_bw_MBps[g] : min_bw;
        for (int h = 0; h < N; h++) min_bw = d->link_bw_MBps[g * N + h] < min_bw ? d->link_bw_MBps[g * N + h] : min_bw;
    }
    i128 max_ar = (2 * max_grad * 1000) / min_bw + 2;
    if (max_ar >= kLimit62) return fail(HEDDLE_E_RANGE, "gradient synchronisation time could exceed 2^62 ns");

    // ---- expert tiling (section 5.3): the experts' part x of an MoE layer's
    // time at ETP t, scaled to a stage of TP k, is ceil(x_t * t / k); the
    // layer's time there is layer_ns_k - x_k + ceil(x_t * t / k), never
    // negative since x_k <= layer_ns_k. Memory splits into dense state at TP k
    // and expert state at ETP t / EP e.
    std::vector<int64_t> pre_dstate((size_t)K * R), pre_xstate((size_t)K * E * R),
        xdelta((size_t)N * K * K * R, 0);
    for (int k = 0; k < K; k++) {
        i128 w = 0;
        pre_dstate[k * R] = 0;
        for (int l = 0; l < L; l++) {
            w += d->state_bytes[(size_t)k * L + l];
            pre_dstate[k * R + l + 1] = (int64_t)w;
        }
        for (int e = 0; e < E; e++) {
            const int64_t ep = d->ep_degrees[e];
            i128 x = 0;
            pre_xstate[(k * E + e) * R] = 0;
            for (int l = 0; l < L; l++) {
                x += (d->xstate_bytes[(size_t)k * L + l] + ep - 1) / ep;
                pre_xstate[(k * E + e) * R + l + 1] = (int64_t)x;
            }
        }
    }
    i128 max_tiled = 0;
    for (int g = 0; g < N; g++)
        for (int k = 0; k < K; k++) {
            int64_t a2a_max = std::max(a2a_ns[g * 3 + 1], a2a_ns[g * 3 + 2]), p2p_max = 0;
            for (int h = 0; h < N; h++) p2p_max = std::max(p2p_max, p2p_ns[g * N + h]);
            for (int t = 0; t < K; t++) {
                i128 acc = 0;
                int64_t *row = &xdelta[(((size_t)g * K + k) * K + t) * R];
                for (int l = 0; l < L; l++) {
                    if (d->is_moe[l] && d->xlayer_ns) {
                        const int64_t xk = d->xlayer_ns[((size_t)g * K + k) * L + l];
                        const int64_t xt = d->xlayer_ns[((size_t)g * K + t) * L + l];
                        if (xk < 0 || xt < 0 || xk > d->layer_ns[((size_t)g * K + k) * L + l])
                            return fail(HEDDLE_E_INVAL, "xlayer_ns entries must lie in 0 .. layer_ns");
                        const i128 num = (i128)xt * d->tp_degrees[t], den = d->tp_degrees[k];
                        acc += (num + den - 1) / den - xk;
                        if (acc >= kLimit62 || acc <= -kLimit62) return fail(HEDDLE_E_RANGE, "tiled layer times exceed 2^62");
                    }
                    row[l + 1] = (int64_t)acc;
                }
                i128 b = (i128)pre_time[((size_t)g * K + k) * R + L] + acc + (i128)n_moe * a2a_max + p2p_max;
                if (b > max_tiled) max_tiled = b;
            }
        }
    if (max_tiled >= kLimit62) return fail(HEDDLE_E_RANGE, "tiled stage times could exceed 2^62 ns");
    i128 max_xg = 0;
    for (int k = 0; k < K; k++)
        for (int e = 0; e < E; e++) max_xg = std::max(max_xg, (i128)pre_xgrad[(k * E + e) * R + L]);
    i128 max_dg = 0;
    for (int k = 0; k < K; k++) max_dg = std::max(max_dg, (i128)pre_grad[k * R + L]);
    const i128 max_ar_tiled = (2 * (max_dg + max_xg) * 1000) / min_bw + 2;
    if (max_ar_tiled >= kLimit62) return fail(HEDDLE_E_RANGE, "gradient synchronisation time could exceed 2^62 ns");

    // ---- fp32 variant: exact fixed-point image of the fp32 costs
    std::vector<float> cost32((size_t)N * K * L);
    for (size_t i = 0; i < cost32.size(); i++) {
        float v = d->layer_ns_f32 ? d->layer_ns_f32[i] : (float)d->layer_ns[i];
        if (!(v > 0.0f) || !std::isfinite(v)) return fail(HEDDLE_E_INVAL, "layer_ns_f32 entries must be finite and > 0");
        cost32[i] = v;
    }
    std::vector<float> a2a32((size_t)N * 3), p2p32((size_t)N * N);
    for (size_t i = 0; i < a2a32.size(); i++) a2a32[i] = (float)a2a_ns[i];
    for (size_t i = 0; i < p2p32.size(); i++) p2p32[i] = (float)p2p_ns[i];
    int e0 = 0;
    for (float v : cost32) e0 = std::min(e0, low_bit_exp(v));
    for (float v : a2a32) if (v > 0) e0 = std::min(e0, low_bit_exp(v));
    for (float v : p2p32) if (v > 0) e0 = std::min(e0, low_bit_exp(v));
    bool fx_ok = e0 > -80;
    auto to_fx = [&](float v, bool &ok) -> int64_t {
        if (v == 0.0f) return 0;
        long double x = std::ldexp((long double)v, -e0);      // exact: v is a multiple of 2^e0
        if (x >= (long double)kLimit62) { ok = false; return 0; }
        return (int64_t)x;
    };
    std::vector<int64_t> pre_time_fx((size_t)N * K * R, 0), a2a_fx((size_t)N * 3, 0), p2p_fx((size_t)N * N, 0);
    i128 max_stage_fx = 0;
    if (fx_ok) {
        for (size_t i = 0; i < a2a32.size() && fx_ok; i++) a2a_fx[i] = to_fx(a2a32[i], fx_ok);
        for (size_t i = 0; i < p2p32.size() && fx_ok; i++) p2p_fx[i] = to_fx(p2p32[i], fx_ok);
        for (int g = 0; g < N && fx_ok; g++)
            for (int k = 0; k < K && fx_ok; k++) {
                i128 acc = 0;
                int64_t *row = &pre_time_fx[((size_t)g * K + k) * R];
                for (int l = 0; l < L && fx_ok; l++) {
                    acc += to_fx(cost32[((size_t)g * K + k) * L + l], fx_ok);
                    if (acc >= kLimit62) fx_ok = false;
                    row[l + 1] = (int64_t)acc;
                }
                int64_t a2a_max = std::max(a2a_fx[g * 3 + 1], a2a_fx[g * 3 + 2]), p2p_max = 0;
                for (int h = 0; h < N; h++) p2p_max = std::max(p2p_max, p2p_fx[g * N + h]);
                i128 b = (i128)row[L] + (i128)n_moe * a2a_max + p2p_max;
                if (b >= kLimit62) fx_ok = false;
                if (b > max_stage_fx) max_stage_fx = b;
            }
    }

    // ---- stage rows: time prefix of a stage per (type, TP, all-to-all variant),
    // P[j] = pre_time[j] + a2a * (MoE layers before j), exact in 64 bits and, when
    // the range proof allows, narrowed to 32 bits; the same for the fp32 image
    const bool narrow_i64 = max_stage < (i128)kNarrowLimit;
    const bool narrow_f32 = fx_ok && max_stage_fx < (i128)kNarrowLimit;
    std::vector<uint64_t> rows64[2];
    std::vector<uint32_t> rows32[2];
    for (int v = 0; v < 2; v++) {
        const std::vector<int64_t> &pt = v ? pre_time_fx : pre_time;
        const std::vector<int64_t> &aa = v ? a2a_fx : a2a_ns;
        rows64[v].assign((size_t)N * K * 3 * R, 0);
        if (v == 1 && !fx_ok) continue;
        for (int g = 0; g < N; g++)
            for (int k = 0; k < K; k++)
                for (int var = 0; var < 3; var++)
                    for (int j = 0; j <= L; j++)
                        rows64[v][(((size_t)g * K + k) * 3 + var) * R + j] =
                            (uint64_t)(pt[((size_t)g * K + k) * R + j] + aa[g * 3 + var] * pre_moe[j]);
        if (v ? narrow_f32 : narrow_i64) {
            rows32[v].resize(rows64[v].size());
            for (size_t i = 0; i < rows64[v].size(); i++) rows32[v][i] = (uint32_t)rows64[v][i];
        } else {
            rows32[v].assign(1, 0);
        }
    }

    // ---- per stage record: time-row and limit-row offsets
    std::vector<uint32_t> stage_tab((size_t)65536 * 2, 0);
    for (int g = 0; g < N; g++)
        for (int l2tp = 0; l2tp < 16; l2tp++) {
            if (!((dp.tp_present >> l2tp) & 1)) continue;
            const int k = (int)((dp.tp_index >> (4 * l2tp)) & 15);
            for (int l2ep = 0; l2ep < 16; l2ep++) {
                if (!((dp.ep_present >> l2ep) & 1)) continue;
                const int e = (int)((dp.ep_index >> (4 * l2ep)) & 15);
                const size_t idx = (size_t)(g | l2tp << 8 | l2ep << 12);
                const int var = a2a_variant(1 << l2ep, 1 << l2tp, d->node_size[g]);
                stage_tab[2 * idx] = (uint32_t)((((size_t)g * K + k) * 3 + var) * R);
                stage_tab[2 * idx + 1] = (uint32_t)((((size_t)g * K + k) * E + e) * F * 2 * RL);
            }
        }

    // ---- upload
    Builder B;
    const size_t o_r64a = B.add(rows64[0]), o_r64b = B.add(rows64[1]), o_r32a = B.add(rows32[0]),
                 o_r32b = B.add(rows32[1]);
    size_t o_time = B.add(pre_time), o_time_fx = B.add(pre_time_fx), o_moe = B.add(pre_moe),
           o_state = B.add(pre_state), o_act = B.add(pre_act), o_grad = B.add(pre_grad),
           o_xgrad = B.add(pre_xgrad), o_psx = B.add(pair_sx), o_pag = B.add(pair_ag), o_stab = B.add(stage_tab), o_prof = B.add(d->profiled, (size_t)N * K),
           o_a2a = B.add(a2a_ns), o_a2a_fx = B.add(a2a_fx), o_p2p = B.add(p2p_ns), o_p2p_fx = B.add(p2p_fx),
           o_cap = B.add(d->mem_cap_bytes, (size_t)N * 8), o_node = B.add(d->node_size, (size_t)N * 4),
           o_ngpu = B.add(d->n_gpus, (size_t)N * 4), o_intra = B.add(d->intra_bw_MBps, (size_t)N * 8),
           o_link = B.add(d->link_bw_MBps, (size_t)N * N * 8), o_epd = B.add(d->ep_degrees, (size_t)E * 4),
           o_lim = B.add(lim_tab), o_dstate = B.add(pre_dstate), o_xstate = B.add(pre_xstate),
           o_xdelta = B.add(xdelta);
    // expert tiling: per GPU type the TP indices usable as ETP (profiled, at
    // most the type's node size), one bit each
    std::vector<uint32_t> etp_mask(N, 0);
    for (int g = 0; g < N; g++)
        for (int k = 0; k < K; k++)
            if (d->profiled[(size_t)g * K + k] && d->tp_degrees[k] <= d->node_size[g]) etp_mask[g] |= 1u << k;
    const size_t o_etp = B.add(etp_mask);

    heddle_profile *p = new (std::nothrow) heddle_profile;
    if (!p) return fail(HEDDLE_E_NOMEM, "host allocation failed");
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) { delete p; return hip_fail(e, "hipGetDevice"); }
    e = hipMalloc(&p->dev_block, B.bytes.size());
    if (e != hipSuccess) { delete p; return e == hipErrorOutOfMemory ? fail(HEDDLE_E_NOMEM, "hipMalloc of profile tables failed") : hip_fail(e, "hipMalloc"); }
    e = hipMemcpy(p->dev_block, B.bytes.data(), B.bytes.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) { (void)hipFree(p->dev_block); delete p; return hip_fail(e, "hipMemcpy"); }
    unsigned char *base = (unsigned char *)p->dev_block;
    dp.fx_exp = e0;
    dp.pre_time = (const int64_t *)(base + o_time);
    dp.pre_time_fx = (const int64_t *)(base + o_time_fx);
    dp.pre_moe = (const int32_t *)(base + o_moe);
    dp.pre_state = (const int64_t *)(base + o_state);
    dp.pre_act = (const int64_t *)(base + o_act);
    dp.pre_grad = (const int64_t *)(base + o_grad);
    dp.pre_xgrad = (const int64_t *)(base + o_xgrad);
    dp.pair_sx = (const longlong2 *)(base + o_psx);
    dp.pair_ag = (const longlong2 *)(base + o_pag);
    dp.stage_tab = (const uint2 *)(base + o_stab);
    dp.profiled = (const uint8_t *)(base + o_prof);
    dp.a2a_ns = (const int64_t *)(base + o_a2a);
    dp.a2a_fx = (const int64_t *)(base + o_a2a_fx);
    dp.p2p_ns = (const int64_t *)(base + o_p2p);
    dp.p2p_fx = (const int64_t *)(base + o_p2p_fx);
    dp.mem_cap = (const int64_t *)(base + o_cap);
    dp.node_size = (const int32_t *)(base + o_node);
    dp.n_gpus = (const int32_t *)(base + o_ngpu);
    dp.intra_bw = (const int64_t *)(base + o_intra);
    dp.link_bw = (const int64_t *)(base + o_link);
    dp.ep_degrees = (const int32_t *)(base + o_epd);
    dp.mem_lim = (const uint8_t *)(base + o_lim);
    dp.pre_dstate = (const int64_t *)(base + o_dstate);
    dp.pre_xstate = (const int64_t *)(base + o_xstate);
    dp.xdelta = (const int64_t *)(base + o_xdelta);
    dp.etp_mask = (const uint32_t *)(base + o_etp);
    dp.rows64[0] = (const uint64_t *)(base + o_r64a);
    dp.rows64[1] = (const uint64_t *)(base + o_r64b);
    dp.rows32[0] = (const uint32_t *)(base + o_r32a);
    dp.rows32[1] = (const uint32_t *)(base + o_r32b);
    dp.n_f = F;
    dp.lim_stride = RL;
    p->dev = dp;
    p->max_stage_ns = (int64_t)max_stage;
    p->max_ar_ns = (int64_t)max_ar;
    p->max_tiled_ns = (int64_t)max_tiled;
    p->max_ar_tiled_ns = (int64_t)max_ar_tiled;
    p->narrow_i64 = narrow_i64;
    p->max_stage_fx = fx_ok ? (int64_t)max_stage_fx : -1;
    // fp32-rounded all-reduce terms are within a factor (1 + 2^-24) of the int64 ones
    {
        long double b = std::ldexp((long double)max_ar * (1.0L + std::ldexp(1.0L, -20)) + 1.0L, -e0);
        p->max_ar_fx = !fx_ok ? -1 : (b >= (long double)kLimit62 ? kLimit62 : (int64_t)b);
    }
    p->narrow_f32 = narrow_f32;
    *out = p;
    return HEDDLE_OK;
}

extern "C" void heddle_free_profile(heddle_profile *p)
{
    if (!p) return;
    // device work of earlier calls may still read the tables or the scratch
    // buffers: wait for the profile's device before releasing them
    int prev = -1;
    const bool switched = hipGetDevice(&prev) == hipSuccess && prev != p->device && hipSetDevice(p->device) == hipSuccess;
    hipError_t e = hipDeviceSynchronize();
    // the per-stream buffers came from the library's memory pool: they go
    // back to it stream-ordered (on the device's null stream, since the
    // streams they were used on may no longer exist), so later calls reuse them
    for (auto &sl : p->scratch) {
        if (sl.ptr) {
            const hipError_t f = hipFreeAsync(sl.ptr, nullptr);
            e = e == hipSuccess ? f : e;
        }
        (void)hipEventDestroy(sl.done);
    }
    const hipError_t q = hipStreamSynchronize(nullptr);
    e = e == hipSuccess ? q : e;
    const hipError_t b = hipFree(p->dev_block);
    e = e == hipSuccess ? b : e;
    if (e != hipSuccess) (void)hip_fail(e, "heddle_free_profile: releasing the profile's device memory");
    if (switched) (void)hipSetDevice(prev);
    delete p;
}

extern "C" int heddle_profile_info_get(const heddle_profile *p, heddle_profile_info *info)
{
    if (!p || !info) return fail(HEDDLE_E_INVAL, "NULL argument");
    info->narrow[0] = p->narrow_i64;
    info->narrow[1] = p->narrow_f32;
    info->fx_exp = p->dev.fx_exp;
    info->L = p->dev.L;
    info->n_types = p->dev.n_types;
    info->n_tp = p->dev.n_tp;
    info->n_ep = p->dev.n_ep;
    info->max_stage_ns = p->max_stage_ns;
    std::lock_guard<std::mutex> lock(p->scratch_mu);
    int64_t bytes = 0;
    for (const auto &sl : p->scratch) bytes += (int64_t)sl.bytes;
    info->scratch_bytes = bytes;
    info->narrow_tile = tile_narrow(p) ? 1 : 0;
    return HEDDLE_OK;
}
