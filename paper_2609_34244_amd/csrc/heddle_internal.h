// Internal declarations of the gfx950 plan-pricing library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/heddle.h"

namespace heddle {

constexpr int kWave = 64;
constexpr int kMaxStages = HEDDLE_MAX_STAGES;
constexpr int kMaxMList = HEDDLE_MAX_MLIST;
constexpr int64_t kLimit62 = int64_t(1) << 62;
constexpr size_t kMaxLimitTable = size_t(256) << 20;       // bytes of the memory-limit table
constexpr int64_t kMaxBandwidth = (int64_t(1) << 34) - 1;   // MB/s; keeps n * bw below 2^50
constexpr uint32_t kNarrowLimit = 0x7FFFFFFFu;   // exact 32-bit DP when every stage time is below this

// a2a variant of a stage: no all-to-all (EP = 1), EP x TP group inside one
// node (intra-node bandwidth), or spanning nodes (same-type inter-node link)
enum A2AVariant { kA2ANone = 0, kA2AIntra = 1, kA2AInter = 2 };
__host__ __device__ inline int a2a_variant(int ep, int tp, int node)
{
    return ep == 1 ? kA2ANone : (ep * tp <= node ? kA2AIntra : kA2AInter);
}

// Device-resident derived tables of one profile. Passed by value to kernels.
// Prefix rows have L + 1 entries: row[j] = sum over layers l < j.
struct DevProfile {
    int32_t L, n_types, n_tp, n_ep;
    int32_t fx_exp;                  // fixed-point unit of the fp32 variant is 2^fx_exp
    uint32_t tp_present, ep_present; // bit l set: 2^l is a profiled TP / an allowed EP degree
    uint64_t tp_index, ep_index;     // nibble l: index of 2^l in tp_degrees / ep_degrees
    uint64_t tp_log2, ep_log2;       // nibble k: log2 of tp_degrees[k] / ep_degrees[k]
    const int64_t *pre_time;         // [n_types][n_tp][L+1] prefix of layer_ns
    const int64_t *pre_time_fx;      // [n_types][n_tp][L+1] prefix of fp32 costs in 2^fx_exp units
    const int32_t *pre_moe;          // [L+1] prefix count of MoE layers
    const int64_t *pre_state;        // [n_tp][n_ep][L+1] prefix of state + ceil(xstate / e)
    const int64_t *pre_act;          // [n_tp][L+1] prefix of act
    const int64_t *pre_grad;         // [n_tp][L+1] prefix of grad
    const int64_t *pre_xgrad;        // [n_tp][n_ep][L+1] prefix of ceil(xgrad / e)
    // the same prefixes interleaved by the index they share, so that one
    // 16-byte read serves a stage boundary: {pre_state, pre_xgrad} and
    // {pre_act, pre_grad}
    const longlong2 *pair_sx;        // [n_tp][n_ep][L+1]
    const longlong2 *pair_ag;        // [n_tp][L+1]
    // by the low 16 bits of a valid stage record (type | log2 TP << 8 | log2 EP
    // << 12): {offset of its time-prefix row in rows32 / rows64, byte offset of
    // its memory-limit rows (in-flight count 1)}; 0 for invalid combinations
    const uint2 *stage_tab;          // [65536]
    const uint8_t *profiled;         // [n_types][n_tp]
    const int64_t *a2a_ns;           // [n_types][3] all-to-all time per MoE layer by variant
    const int64_t *a2a_fx;           // [n_types][3] fp32-rounded, in fixed-point units
    const int64_t *p2p_ns;           // [n_types][n_types] p2p time, sender type x receiver type
    const int64_t *p2p_fx;           // [n_types][n_types] fp32-rounded, fixed-point units
    const int64_t *mem_cap;          // [n_types]
    const int32_t *node_size;        // [n_types]
    const int32_t *n_gpus;           // [n_types]
    const int64_t *intra_bw;         // [n_types] MB/s
    const int64_t *link_bw;          // [n_types][n_types] MB/s
    const int32_t *ep_degrees;       // [n_ep]
    // expert tiling: dense state prefix per TP, expert state prefix per
    // (ETP, EP) with a per-layer ceiling, and per (type, TP, ETP) the prefix
    // of the change of MoE layer time when the experts run at ETP instead of TP
    const int64_t *pre_dstate;       // [n_tp][L+1]
    const int64_t *pre_xstate;       // [n_tp][n_ep][L+1]
    const int64_t *xdelta;           // [n_types][n_tp][n_tp][L+1]
    const uint32_t *etp_mask;        // [n_types] bit k: tp_degrees[k] is profiled and fits a node
    // [n_types][n_tp][n_ep][n_f][2][lim_stride]: per row, the largest end that
    // fits from row i, then its inverse (smallest row whose limit reaches x)
    const uint8_t *mem_lim;
    int32_t n_f;                     // in-flight counts covered by mem_lim: 1 .. min(L, 64)
    int32_t lim_stride;              // bytes per half-row: L + 1 rounded up to a multiple of 16
    // [n_types][n_tp][3][L+1] stage time prefix (layer costs + all-to-all of the
    // variant); index 0: int64 ns, 1: fp32 image in fixed point; the 32-bit
    // copies exist only when the range proof allows narrowing
    const uint64_t *rows64[2];
    const uint32_t *rows32[2];
};

}  // namespace heddle

struct heddle_profile {
    heddle::DevProfile dev;
    void *dev_block;                 // one device allocation holding every table
    int device;
    int narrow_i64, narrow_f32;      // 32-bit DP proven exact
    int64_t max_stage_ns;            // bound on any int64 stage time
    int64_t max_stage_fx;            // bound on any fp32 stage time, fixed-point units
    int64_t max_ar_ns;               // bound on any stage's gradient synchronisation time
    int64_t max_ar_fx;               // the same, fp32-rounded, fixed-point units
    int64_t max_tiled_ns;            // bound on any stage time under any expert layout
    int64_t max_ar_tiled_ns;         // bound on any stage's synchronisation under any expert layout
    // Scratch of the pricing path, one buffer per stream, grown on demand and
    // kept until the profile is freed (a fresh stream-ordered block per call
    // costs tens of microseconds of host time before the first launch).
    // scratch_mu is held from taking a buffer until the call's last launch
    // is enqueued and `done` recorded after it, so a buffer is reused only in
    // stream order.
    struct Scratch {
        hipStream_t stream;
        void *ptr;
        size_t bytes;
        hipEvent_t done;
    };
    mutable std::mutex scratch_mu;
    mutable std::vector<Scratch> scratch;
};

namespace heddle {

// thread-local last error
void set_error(const std::string &msg);
int fail(int code, const std::string &msg);
int hip_fail(hipError_t e, const char *what);

// stream-ordered device scratch from the library's pool of the stream's
// device; release with hipFreeAsync on the same stream
constexpr int kMaxDevices = 64;
hipError_t scratch_alloc(void **ptr, size_t bytes, hipStream_t stream);

// The profile's scratch buffer of `stream`, at least `bytes` long; the caller
// holds p->scratch_mu until profile_scratch_done. With hipStreamPerThread (one
// handle for many streams) the block is a fresh one that *owned marks, which
// profile_scratch_done releases on the stream.
int profile_scratch(const heddle_profile *p, hipStream_t stream, size_t bytes, void **ptr, bool *owned);
int profile_scratch_done(const heddle_profile *p, hipStream_t stream, void *ptr, bool owned);

#define HEDDLE_HIP(call)                                         \
    do {                                                         \
        hipError_t _e = (call);                                  \
        if (_e != hipSuccess) return ::heddle::hip_fail(_e, #call); \
    } while (0)

// Arguments of one pricing launch (host-validated).
struct PriceArgs {
    int64_t n;
    int32_t s_max, n_m, flags;
    int32_t m[kMaxMList];
    const uint8_t *n_stages;
    const uint32_t *stages;
    void *iter, *bottleneck;
    int64_t *peak_mem;
    uint8_t *layers, *status;
    unsigned long long *work;        // count-only launches: accumulated relaxations
    int32_t g_stride;                // LDS entries per pair row (L + 1 and padding)
    int32_t s_cap;                   // stage rows: min(s_max, L)
    int32_t lds_per_wave;            // bytes of one wavefront's LDS region
    int32_t off_j, off_x;            // byte offsets of the per-stage limit rows and of the next-row
                                     // tables (shared with the G arena)
    int32_t arena_cap;               // entries of the G arena
    uint32_t *wst;                   // [n][n_m] status after validation and windows (0: windows found)
                                     // | in-flight class min(ceil(m / D), S) << 8 (0: memory ignored)
                                     // | rows of the windows W_1 .. W_{S-1} << 16 (status 0 only)
    uint16_t *wwin;                  // [n][n_m][win_stride(s_max)] window of stage s: first row | last row << 8
    bool scratch_owned;              // host side: wst lives in a block of its own (hipStreamPerThread)
    unsigned char *ext_scratch;      // host side: a fixed device buffer for wst and wwin (no
    size_t ext_bytes;                // allocation, no profile buffer); NULL: the profile's buffer
};

int validate_price_args(const heddle_profile *p, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                        const uint32_t *d_stages, const int32_t *h_m, int32_t n_m, uint32_t flags);
// count: 0 prices; 1 counts the relaxations over the windows; 2 counts those the
// split kernel evaluates (it runs the DP); 1 and 2 write no plan outputs
int launch_price(const heddle_profile *p, PriceArgs &a, hipStream_t stream, int count);
int launch_evaluate(const heddle_profile *p, const PriceArgs &a, hipStream_t stream);
// window pass outputs: row stride of a plan's windows, in entries (a
// multiple of 4, so that rows are stored 8 bytes at a time)
__host__ __device__ inline int win_stride(int s_max) { return (s_max + 3) & ~3; }
// window pass: LDS check and attribute set-up (nothing enqueued), then the launch
int prepare_windows(const heddle_profile *p, const PriceArgs &a, int max_lds, size_t *lds);
int launch_windows(const heddle_profile *p, const PriceArgs &a, size_t lds, hipStream_t stream);
int launch_distribute(const heddle_profile *p, PriceArgs &a, hipStream_t stream, bool count_only);
int launch_tile(const heddle_profile *p, const PriceArgs &a, uint8_t *tiling, hipStream_t stream);
// expert tiling holds stage times and synchronisation values in 32 bits
bool tile_narrow(const heddle_profile *p);
int launch_argmin(int64_t n, const int32_t *h_m, int32_t n_m, uint32_t flags, const void *d_iter,
                  const uint8_t *d_status, int64_t *h_best_template, int32_t *h_best_m_index,
                  void *h_best_iter, hipStream_t stream);

}  // namespace heddle
