/*
 * heddle.h -- C ABI of the MI355X (gfx950) batched plan-pricing library.
 *
 * The library prices a batch of candidate parallelism plans of one model on
 * one heterogeneous GPU cluster, following the profile-based cost model of
 * Heddle (arXiv 2609.34244):
 *
 *   - a plan is a structural template (section 5.1: pipeline depth, and per
 *     stage a GPU type and a TP degree; here also the DP degree and the EP
 *     degree of each stage) together with a global micro-batch count m;
 *   - PartitionLayers (the layer-split step of the nested-loop backbone in
 *     section 3.1) splits the model's L layers over the S stages so that the
 *     slowest stage is as fast as possible, every stage holding at least one
 *     layer and fitting its GPUs' memory (memory validation, section 5.2);
 *   - Evaluate (section 3.1 backbone; section 5.2 cost model) returns the
 *     1F1B iteration time (M-1) max_s t_s + sum_s t_s + max_s g_s (section
 *     5.3, expert tiling paragraph) and the peak memory of each GPU;
 *   - the best plan is the one of highest throughput m / iter among the
 *     feasible ones (section 5 overview: candidate plans are ordered by the
 *     throughput the cost model predicts for them).
 *
 * All time quantities are int64 nanoseconds and all sizes int64 bytes; with
 * HEDDLE_F_FP32 the time quantities are fp32 (see heddle_price_plans).
 *
 * Threading: every entry point may be called from any host thread. A loaded
 * profile is immutable, so concurrent pricing calls on different streams
 * may share it. heddle_last_error() is per host thread.
 *
 * Scratch: device memory that an entry point needs beyond its caller's
 * buffers is allocated stream-ordered on the call's stream, from a memory
 * pool per device that the library creates on first use, and freed on that
 * stream before the call returns; the pool keeps freed memory for later
 * calls until the process ends. The exception is the pricing path's per-plan
 * scratch (heddle_price_plans and the entry points built on it): a profile
 * keeps one buffer per stream it was used on, grown on demand, until
 * heddle_free_profile. Pricing calls
 * that share a profile take its lock while they enqueue their launches (their
 * device work still overlaps across streams). With hipStreamPerThread the
 * buffer is a fresh stream-ordered block per call. heddle_price_plans_noalloc
 * allocates nothing: it uses a fixed buffer per GPU instead. The argmin entry points
 * return their result through a small pinned host buffer per host thread,
 * allocated on the thread's first call and kept until the process ends.
 */
#ifndef HEDDLE_H
#define HEDDLE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes of the entry points (call-level errors are negative) ---- */
#define HEDDLE_OK            0
#define HEDDLE_E_INVAL      -1  /* bad argument: null pointer, size or flag out of range    */
#define HEDDLE_E_NOMEM      -2  /* host or device allocation failed                         */
#define HEDDLE_E_DEVICE     -3  /* a HIP call failed (message from hipGetErrorString)       */
#define HEDDLE_E_RANGE      -4  /* table values could overflow the exact integer arithmetic */
#define HEDDLE_E_NOFEASIBLE -5  /* best-plan queries only: no plan has status OK            */

/* ---- flags ---- */
#define HEDDLE_F_FP32         1u  /* fp32 time quantities (iter, bottleneck outputs are float) */
#define HEDDLE_F_COMPUTE_ONLY 2u  /* split ignores memory; the fit is checked afterwards       */
#define HEDDLE_F_DISTRIBUTE   4u  /* speed-proportional split with a fallback list (section 5.3) */
#define HEDDLE_F_COUNT_EVALUATED 8u  /* heddle_count_work only: count what the kernel evaluates */

/* ---- per-plan status codes (data, not errors); the first failing check wins ---- */
#define HEDDLE_S_OK             0  /* priced and fits                                         */
#define HEDDLE_S_BAD_SHAPE      1  /* S < 1, S > s_max or S > L                               */
#define HEDDLE_S_BAD_TYPE       2  /* a stage's GPU type >= n_types                           */
#define HEDDLE_S_BAD_TP         3  /* TP not a profiled degree, or TP > node size (5.1 mask)  */
#define HEDDLE_S_UNPROFILED     4  /* no profile entry for (type, TP): profiles match exactly (5.2) */
#define HEDDLE_S_BAD_DP         5  /* DP < 1, or stages disagree on DP                        */
#define HEDDLE_S_BAD_EP         6  /* EP not an allowed degree, or EP does not divide DP      */
#define HEDDLE_S_OVERSUBSCRIBED 7  /* sum over a type's stages of TP * DP > its GPU count     */
#define HEDDLE_S_OOM            8  /* no split fits memory (or, compute-only, the split OOMs) */

/* ---- limits ---- */
#define HEDDLE_MAX_LAYERS  255     /* L (layer counts are returned as uint8)   */
#define HEDDLE_MAX_STAGES  64      /* s_max                                     */
#define HEDDLE_MAX_TYPES   255     /* n_types                                   */
#define HEDDLE_MAX_MLIST   64      /* n_m                                       */
#define HEDDLE_MAX_M       (1 << 24) /* each m                                  */

/*
 * Stage record of a template: one uint32 per stage,
 *   bits  0..7   GPU type index g          (0 .. n_types-1)
 *   bits  8..11  log2 of the TP degree
 *   bits 12..15  log2 of the EP degree     (0 for a dense model)
 *   bits 16..31  DP degree D (pipeline replica count; equal on all stages)
 * The expert layout of a stage is EP = e, ETP = TP, EDP = D / e, so that
 * EP * ETP * EDP equals the stage's TP * D GPUs (section 3.2).
 */
#define HEDDLE_STAGE(g, log2_tp, log2_ep, dp) \
    ((uint32_t)(g) | ((uint32_t)(log2_tp) << 8) | ((uint32_t)(log2_ep) << 12) | ((uint32_t)(dp) << 16))

/*
 * Profile of one model on one cluster (the offline profiles of section 5.2,
 * keyed by GPU type and TP degree at one fixed micro-batch size).
 * All pointers are HOST memory and are only read during heddle_load_profile.
 * Index k runs over tp_degrees, e over ep_degrees, l over layers.
 */
typedef struct heddle_profile_desc {
    int32_t L;                    /* layers, 1..255                                        */
    int32_t n_types;              /* GPU types, 1..255                                     */
    int32_t n_tp, n_ep;           /* entries of tp_degrees / ep_degrees (each 1..16)       */
    const int32_t *tp_degrees;    /* [n_tp] distinct powers of two, 1..32768               */
    const int32_t *ep_degrees;    /* [n_ep] distinct powers of two; {1} for a dense model  */
    const int64_t *layer_ns;      /* [n_types][n_tp][L] fwd+bwd ns per micro-batch
                                     (computation + TP communication), each >= 1          */
    const uint8_t *profiled;      /* [n_types][n_tp] 0: no profile entry                   */
    const float   *layer_ns_f32;  /* [n_types][n_tp][L] fp32 costs for HEDDLE_F_FP32, each
                                     finite and > 0; NULL: the int64 table rounded to fp32 */
    const uint8_t *is_moe;        /* [L] 1 for a mixture-of-experts layer                  */
    const int64_t *state_bytes;   /* [n_tp][L] per-GPU params+grads+optimizer, dense part  */
    const int64_t *xstate_bytes;  /* [n_tp][L] the same for the experts at EP = 1          */
    const int64_t *act_bytes;     /* [n_tp][L] per-GPU activations of one micro-batch      */
    const int64_t *grad_bytes;    /* [n_tp][L] per-GPU gradient bytes, dense part          */
    const int64_t *xgrad_bytes;   /* [n_tp][L] per-GPU gradient bytes of experts at EP = 1 */
    int64_t boundary_bytes;       /* activation tensor crossing a stage boundary, one way  */
    int64_t a2a_bytes;            /* all-to-all bytes of one MoE layer per micro-batch     */
    const int64_t *mem_cap_bytes; /* [n_types] physical memory per GPU                     */
    const int32_t *node_size;     /* [n_types] GPUs in the largest node of the type        */
    const int32_t *n_gpus;        /* [n_types] GPUs of the type in the cluster             */
    const int64_t *intra_bw_MBps; /* [n_types] intra-node bandwidth, MB/s, >= 1            */
    const int64_t *link_bw_MBps;  /* [n_types][n_types] inter-node bandwidth, MB/s, >= 1   */
    const int64_t *xlayer_ns;     /* [n_types][n_tp][L] the experts' part of layer_ns of
                                     each MoE layer (ETP = TP, EP = 1), 0 <= x <= layer_ns;
                                     entries of dense layers are ignored. Used only by
                                     heddle_tile_plans; NULL: 0                            */
} heddle_profile_desc;

typedef struct heddle_profile heddle_profile;   /* opaque, device-resident tables */

/*
 * heddle_load_profile -- validate a profile, build its derived tables
 * (exclusive prefix sums of per-layer time, memory and gradient bytes; the
 * transfer-time terms of every type and type pair) and upload them to the
 * current HIP device.
 *   d    host descriptor; only read during the call.
 *   out  receives a handle owned by the caller, released with
 *        heddle_free_profile. The handle may be used on the device that was
 *        current at load time only.
 * Returns HEDDLE_OK, HEDDLE_E_INVAL (null pointer, size out of range, a
 * non-power-of-two degree, a cost < 1, a negative byte count, a bandwidth
 * < 1), HEDDLE_E_RANGE (prefix totals or transfer times would exceed 2^62),
 * HEDDLE_E_NOMEM or HEDDLE_E_DEVICE. On error *out is set to NULL.
 * Cost: O(n_types * n_tp * L) host work and one host-to-device copy.
 */
int heddle_load_profile(const heddle_profile_desc *d, heddle_profile **out);

/* Release a profile and its per-stream scratch buffers. Waits for the work
 * on the profile's device first, so device work of earlier calls may still
 * be in flight; no host thread may be inside a call that uses the profile.
 * The scratch buffers go back to the library's memory pool (reused by later
 * calls), the tables to the device. There is no return code: if the device
 * reports an error while releasing, heddle_last_error() of the calling
 * thread names it. NULL is ignored. */
void heddle_free_profile(heddle_profile *p);

/*
 * heddle_price_plans -- price n templates at each of n_m micro-batch counts
 * (the "plans" are the n * n_m pairs). Asynchronous: enqueued on `stream`;
 * outputs are valid once the stream has completed the work.
 *   p            profile from heddle_load_profile.
 *   n            templates (>= 0; n = 0 enqueues nothing).
 *   s_max        stage slots per template record, 1..64.
 *   d_n_stages   DEVICE [n] uint8, stage count S of each template.
 *   d_stages     DEVICE [n][s_max] uint32 stage records (HEDDLE_STAGE);
 *                slots s >= S are ignored.
 *   h_m          HOST [n_m] micro-batch counts, each 1..HEDDLE_MAX_M; read
 *                during the call. Micro-batches per replica: M_p = ceil(m/D).
 *   n_m          1..HEDDLE_MAX_MLIST.
 *   flags        any of HEDDLE_F_FP32, HEDDLE_F_COMPUTE_ONLY, HEDDLE_F_DISTRIBUTE.
 * Outputs (DEVICE, caller-allocated, index o = t * n_m + k):
 *   d_iter        [n][n_m] iteration time: int64 ns, or float with FP32.
 *   d_bottleneck  [n][n_m] slowest stage time B* (same type as d_iter).
 *   d_peak_mem    [n][n_m] int64 max over stages of per-GPU peak bytes.
 *   d_layers      [n][n_m][s_max] uint8 layers of each stage (0 beyond S).
 *   d_status      [n][n_m] uint8 HEDDLE_S_*.
 * Split: lexicographically smallest (n_0..n_{S-1}) among the splits of
 * minimum bottleneck, where a stage's time is its layers' profiled cost
 * plus, for MoE layers with EP > 1, one all-to-all, plus its outbound p2p of
 * 2 * boundary_bytes; a stage holds min(S - s, M_p) micro-batches of
 * activations (1F1B). Without COMPUTE_ONLY only splits that fit memory
 * qualify. Plans with status 1..7, and OOM plans without COMPUTE_ONLY, get
 * iter = bottleneck = peak_mem = INT64_MAX (float: +inf) and zero layers;
 * COMPUTE_ONLY OOM plans carry their computed values.
 * FP32: every time quantity is the fp32 nearest (ties to even) to its exact
 * value computed from fp32 per-layer costs and fp32-rounded transfer terms
 * (one rounding per stage time and one for the iteration time).
 * DISTRIBUTE (Heddle's own split, section 5.3, layer split and DP degree):
 * instead of the min-max split, stage s's share of the layers is set by its
 * speed 1 / (int64 time of all L layers on its type and TP, all-to-all
 * included, p2p excluded): the cut after stage s is floor(x + 0.5) with
 * x = L * (speeds of stages 0..s) / (speeds of all stages) in IEEE double
 * (speeds summed in stage order), raised to leave stage s a layer and
 * lowered to leave each later stage one. If it does not fit memory, the
 * alternatives "cut after stage b moved by -1, then by +1" for b = 0..S-2
 * (each stage keeping a layer) are priced and the fitting one with the
 * smallest iteration time is kept (the first on ties); none fitting gives
 * OOM without a split. With COMPUTE_ONLY the proportional split is kept and
 * flagged OOM if it does not fit. The bottleneck output is then the split's
 * slowest stage time.
 * Scratch: without DISTRIBUTE, about n * n_m * (4 + 2 * s_max) bytes (s_max
 * rounded up to a multiple of 4) for the per-plan validation and row
 * windows, in the profile's buffer of `stream`.
 * Returns HEDDLE_OK, HEDDLE_E_INVAL, HEDDLE_E_RANGE (the iteration time could
 * exceed 2^62 for these m, or the fp32 costs span too wide a range to sum
 * exactly), HEDDLE_E_NOMEM (the scratch) or HEDDLE_E_DEVICE. With
 * HEDDLE_E_INVAL or HEDDLE_E_RANGE nothing is enqueued; with HEDDLE_E_NOMEM or
 * HEDDLE_E_DEVICE part of the call's work (scratch set-up, the window pass)
 * may already be on the stream and the outputs are undefined.
 */
int heddle_price_plans(const heddle_profile *p, int64_t n, int32_t s_max,
                       const uint8_t *d_n_stages, const uint32_t *d_stages,
                       const int32_t *h_m, int32_t n_m, uint32_t flags,
                       void *d_iter, void *d_bottleneck, int64_t *d_peak_mem,
                       uint8_t *d_layers, uint8_t *d_status, hipStream_t stream);

/* Device memory the allocation-free pricing entry point holds, per GPU. */
#define HEDDLE_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * heddle_price_plans_noalloc -- heddle_price_plans for callers that cannot
 * allocate device memory: code under HIP graph capture, serving loops that
 * forbid hipMalloc, harnesses that count allocations. Same arguments,
 * outputs, kernels and results as heddle_price_plans; it calls no hipMalloc,
 * hipFree or allocating library routine and does not touch the profile's
 * per-stream buffers.
 * Scratch: the per-plan validation and row windows go to a buffer of
 * HEDDLE_NOALLOC_SCRATCH_BYTES that the library holds in each GPU's memory
 * from the first call on that GPU until the process ends. Without DISTRIBUTE
 * a call needs R(4 * n * n_m, 256) + 2 * n * n_m * R(s_max, 4) bytes of it
 * (R(x, k): x rounded up to a multiple of k) -- 36 MB for a million
 * templates of 16 stage slots at one m; with DISTRIBUTE none. Every cell
 * the kernels read is written earlier in the same call, so what an earlier
 * call left there does not matter.
 * Every call on one GPU shares that GPU's buffer: calls whose device work
 * overlaps (calls on different streams without an ordering between them)
 * race on it and give undefined outputs; calls on one stream are ordered.
 * Returns what heddle_price_plans returns, except HEDDLE_E_NOMEM, plus
 * HEDDLE_E_RANGE (nothing enqueued) when the call needs more than
 * HEDDLE_NOALLOC_SCRATCH_BYTES of the buffer.
 */
int heddle_price_plans_noalloc(const heddle_profile *p, int64_t n, int32_t s_max,
                               const uint8_t *d_n_stages, const uint32_t *d_stages,
                               const int32_t *h_m, int32_t n_m, uint32_t flags,
                               void *d_iter, void *d_bottleneck, int64_t *d_peak_mem,
                               uint8_t *d_layers, uint8_t *d_status, hipStream_t stream);

/*
 * heddle_argmin_plans -- best plan among priced outputs: the plan of status
 * OK with the smallest iter / m (highest throughput m / iter), compared
 * exactly as iter_a * m_b < iter_b * m_a; ties go to the lowest template
 * index, then the lowest m index (section 5.3: the fastest candidate is kept).
 * Synchronous: waits for `stream`.
 *   d_iter, d_status  DEVICE outputs of heddle_price_plans with the same
 *                     n, n_m, h_m and the same FP32 flag.
 *   h_best_template, h_best_m_index  HOST results.
 *   h_best_iter       HOST int64 (or float with FP32) iteration time; may be NULL.
 * Returns HEDDLE_OK, HEDDLE_E_NOFEASIBLE (nothing written), HEDDLE_E_INVAL,
 * HEDDLE_E_NOMEM or HEDDLE_E_DEVICE.
 */
int heddle_argmin_plans(int64_t n, const int32_t *h_m, int32_t n_m, uint32_t flags,
                        const void *d_iter, const uint8_t *d_status,
                        int64_t *h_best_template, int32_t *h_best_m_index, void *h_best_iter,
                        hipStream_t stream);

/*
 * heddle_best_plan -- the whole planning step of one batch: every plan
 * priced (heddle_price_plans, into library-allocated device buffers) and the
 * fitting plan with the largest m / iter, the throughput the cost model
 * gives it, returned (heddle_argmin_plans). This is the selection the
 * planner makes over its priced candidates (section 5 overview: candidates
 * are ordered by the cost model's throughput estimate; section 5.3: of a
 * template's fill choices the quickest one that fits is retained).
 * Synchronous. Arguments as in those two
 * calls; the library allocates and frees its own buffers as scratch on
 * `stream`.
 */
int heddle_best_plan(const heddle_profile *p, int64_t n, int32_t s_max,
                     const uint8_t *d_n_stages, const uint32_t *d_stages,
                     const int32_t *h_m, int32_t n_m, uint32_t flags,
                     int64_t *h_best_template, int32_t *h_best_m_index, void *h_best_iter,
                     hipStream_t stream);

/*
 * heddle_count_work -- algorithmic work of pricing this batch: the number of
 * (row i, end j) pairs the min-max recurrence relaxes, summed over the
 * distinct splits the batch needs (a template's m values that imply the
 * same in-flight activation counts share one split). Only rows that can lie
 * on a complete split are relaxed: with lim(s, i) the last admissible end of
 * row i at stage s (memory limit, capped so that each later stage keeps a
 * layer), stage s takes the rows from Bk_s (the smallest start from which
 * lim reaches Bk_{s+1}, Bk_S = L) to min(R_s, L - (S - s)) (R_0 = 0,
 * R_{s+1} = lim(s, R_s): the furthest reachable start; stage 0: row 0), each
 * against the ends max(i + 1, Bk_{s+1}) .. lim(s, i); a last-stage row
 * counts one. A template with an empty range at some stage has no split
 * that fits memory and counts zero. Synchronous.
 *   h_relaxations  HOST result.
 * With HEDDLE_F_COUNT_EVALUATED the count is of the pairs the split kernel
 * actually relaxes, which is at most the count above: it runs the recurrence
 * and a row's ends are taken in chunks of four by 64 >> ceil(log2 r) lanes
 * for r window rows (one lane when r >= 64), lane p taking chunks p, p + k,
 * ... from the first end; a lane stops after a chunk whose last end has a
 * stage time at or above the lane's running minimum (later ends cannot
 * lower it). Each chunk counts the ends it adds (a last chunk moved back to
 * end at the row's last end counts those from its own start); a last-stage
 * row counts one. The values follow the flags' arithmetic (HEDDLE_F_FP32:
 * the fp32 image), so the count is exact, not a model. For a template with
 * several in-flight classes (int64 pricing), the classes run from the
 * largest key down, and a row's running minimum starts at the previous
 * class's B* + 1, so lanes also stop once a stage time passes that bound.
 * With HEDDLE_F_DISTRIBUTE the unit is one stage-cost evaluation (time,
 * memory and gradient synchronisation of one stage): S for the proportional
 * split and, when it does not fit, 2 per alternative priced (only the two
 * stages around the moved cut change); HEDDLE_F_COUNT_EVALUATED changes
 * nothing there.
 * Returns HEDDLE_OK, HEDDLE_E_INVAL, HEDDLE_E_NOMEM or HEDDLE_E_DEVICE.
 */
int heddle_count_work(const heddle_profile *p, int64_t n, int32_t s_max,
                      const uint8_t *d_n_stages, const uint32_t *d_stages,
                      const int32_t *h_m, int32_t n_m, uint32_t flags,
                      int64_t *h_relaxations, hipStream_t stream);

/*
 * heddle_tile_plans -- expert tiling (section 5.3, expert tiling paragraph)
 * of priced plans, in place. A stage of TP k and DP D spans W = k * D GPUs;
 * its expert layout is EP e x ETP t x EDP W / (e t), with e from ep_degrees,
 * t a profiled TP degree of the stage's type no larger than its node, and
 * e * t dividing W. Under a layout an MoE layer costs
 * layer_ns_k - xlayer_ns_k + ceil(xlayer_ns_t * t / k) plus one all-to-all
 * (intra-node bandwidth if e * t fits the node, else the same-type link);
 * the stage holds dense state at TP k, expert state at ETP t divided by e
 * (per layer, rounded up) and its in-flight activations; its
 * synchronisation all-reduces dense gradients over D and expert gradients
 * (ETP t, divided by e) over W / (e t) replicas. The template's own layout
 * (e from its record, t = k) is one of them. The layouts of a plan are
 * chosen together for the smallest 1F1B iteration time among the layouts
 * that fit memory; ties: the smaller largest synchronisation term, then per
 * stage the faster layout, the smaller synchronisation, the first in
 * (ep_degrees, tp_degrees) order.
 * Inputs are the outputs of heddle_price_plans for the same templates, m and
 * flags (any split mode); int64 costs only (HEDDLE_F_FP32 is rejected).
 * A plan has a split when its status is OK or OOM and it has layer counts.
 * Such a plan gets status OK, its new iter, bottleneck and peak_mem, and
 * d_tiling[(t * n_m + k) * s_max + s] = log2 EP | log2 ETP << 4 per stage;
 * if some stage has no layout that fits, the plan keeps its values and gets
 * its template's layouts. Plans without a split are left as they are and
 * get zero tiling bytes (0 beyond S too). Asynchronous on `stream`.
 *   d_iter, d_bottleneck, d_peak_mem, d_status  DEVICE, read and rewritten.
 *   d_layers  DEVICE [n][n_m][s_max], read.
 *   d_tiling  DEVICE [n][n_m][s_max] uint8, written.
 * Returns HEDDLE_OK, HEDDLE_E_INVAL, HEDDLE_E_RANGE (the tiled iteration time
 * could exceed 2^62, or the layout table of s_max x n_tp x n_ep does not fit
 * the device's LDS) or HEDDLE_E_DEVICE.
 */
int heddle_tile_plans(const heddle_profile *p, int64_t n, int32_t s_max,
                      const uint8_t *d_n_stages, const uint32_t *d_stages,
                      const int32_t *h_m, int32_t n_m, uint32_t flags,
                      void *d_iter, void *d_bottleneck, int64_t *d_peak_mem,
                      const uint8_t *d_layers, uint8_t *d_status, uint8_t *d_tiling,
                      hipStream_t stream);

/*
 * heddle_count_tile_work -- algorithmic work of heddle_tile_plans on the same
 * priced plans (section 5.3, expert tiling paragraph), for throughput
 * reports. Synchronous. Over the plans that are tiled (a split and a valid
 * template):
 *   h_counts[0]  layouts priced: the allowed (stage, EP x ETP) layouts, each
 *                priced for time, memory and synchronisation;
 *   h_counts[1]  dominance tests: for every stage, its fitting layouts
 *                squared (each against each, to keep the layouts no other
 *                one beats in both time and synchronisation);
 *   h_counts[2]  bound tests: kept layouts x (kept layouts + stages), every
 *                kept layout's synchronisation tried as the bound against
 *                every kept layout and folded over every stage;
 * plans with a stage that has no fitting layout add only to h_counts[0].
 *   d_layers, d_status  DEVICE outputs of heddle_price_plans (unchanged).
 * Returns HEDDLE_OK, HEDDLE_E_INVAL, HEDDLE_E_RANGE, HEDDLE_E_NOMEM or
 * HEDDLE_E_DEVICE.
 */
int heddle_count_tile_work(const heddle_profile *p, int64_t n, int32_t s_max,
                           const uint8_t *d_n_stages, const uint32_t *d_stages,
                           const int32_t *h_m, int32_t n_m, uint32_t flags,
                           const uint8_t *d_layers, const uint8_t *d_status,
                           int64_t *h_counts, hipStream_t stream);

/*
 * The cluster's machines (section 5.1, support for non-uniform GPU
 * compositions): for every GPU type, the GPU count of each of its nodes;
 * the nodes of a type may differ in size. HOST memory,
 * read during heddle_load_cluster.
 */
typedef struct heddle_cluster_desc {
    int32_t n_types;              /* 1..255, the profile's type indices                    */
    const int32_t *n_nodes;       /* [n_types] nodes of each type, >= 0                    */
    const int32_t *node_gpus;     /* [sum n_nodes] GPUs per node, 1..64, type 0's first    */
} heddle_cluster_desc;

typedef struct heddle_cluster heddle_cluster;   /* opaque, device-resident node counts */

/* Load a node list to the current device (per type, the number of nodes of
 * each size). Returns HEDDLE_OK, HEDDLE_E_INVAL, HEDDLE_E_NOMEM or
 * HEDDLE_E_DEVICE; *out is NULL on error. Release with heddle_free_cluster. */
int heddle_load_cluster(const heddle_cluster_desc *d, heddle_cluster **out);
void heddle_free_cluster(heddle_cluster *c);

/*
 * heddle_fill_dp -- the DP degree of each template from the node lists
 * (section 5.3, layer split and DP degree; section 5.1 packing rule). The TP
 * group of every stage is packed into the nodes of the stage's GPU type, one
 * replica after another (replica 1: stages 0..S-1 in order, then replica 2,
 * ...); a group of TP t goes to a node with exactly t free GPUs if there is
 * one, else takes t GPUs from the node with the fewest free GPUs above t;
 * types pack independently. D is the number of whole replicas packed before
 * the first group that finds no node, capped at dp_cap and rounded down to a
 * multiple of the template's largest EP degree. D is written into the DP
 * field of every stage record (in place) and into d_dp[t]; D = 0 means not
 * even one replica packs (heddle_price_plans then reports BAD_DP). Templates
 * with S < 1, S > s_max, a type outside the cluster or TP above 64 are left
 * unchanged with d_dp = 0. Asynchronous on `stream`.
 *   d_stages  DEVICE [n][s_max] records, DP fields rewritten.
 *   d_dp      DEVICE [n] int32.
 *   dp_cap    1..65535.
 * Returns HEDDLE_OK, HEDDLE_E_INVAL or HEDDLE_E_DEVICE.
 */
int heddle_fill_dp(const heddle_cluster *c, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                   uint32_t *d_stages, int32_t dp_cap, int32_t *d_dp, hipStream_t stream);

/*
 * heddle_fill_plans -- BestFill (section 5.3, arithmetic auto-fill): the DP
 * degree from the node lists (heddle_fill_dp, records rewritten in place),
 * then the micro-batch size among the profiled sizes: profiles[b] is
 * the profile measured at micro-batch size h_mbs[b] (ascending), and a
 * global batch of `global_batch` samples is m_b = ceil(global_batch /
 * h_mbs[b]) micro-batches. Each template is priced at every size (as
 * heddle_price_plans with m = m_b and `flags`); among the sizes whose plan
 * fits (status OK) the one of smallest iteration time wins, the smaller
 * size on ties; with none OK the smallest size's results are kept.
 * Outputs as heddle_price_plans with n_m = 1, plus d_dp [n] int32 and
 * d_mbs_index [n] uint8 (index into h_mbs). The library allocates one set
 * of outputs per size on `stream` and frees it before returning.
 * Synchronous.
 * Returns HEDDLE_OK, HEDDLE_E_INVAL (profiles of different L or s_max, m_b
 * out of range), HEDDLE_E_RANGE, HEDDLE_E_NOMEM or HEDDLE_E_DEVICE.
 */
int heddle_fill_plans(const heddle_profile *const *profiles, const int32_t *h_mbs, int32_t n_mbs,
                      const heddle_cluster *c, int64_t global_batch, int32_t dp_cap,
                      int64_t n, int32_t s_max, const uint8_t *d_n_stages, uint32_t *d_stages,
                      uint32_t flags, void *d_iter, void *d_bottleneck, int64_t *d_peak_mem,
                      uint8_t *d_layers, uint8_t *d_status, int32_t *d_dp, uint8_t *d_mbs_index,
                      hipStream_t stream);

/*
 * Exhaustive enumeration of structures: the search backbone of the planners
 * Heddle analyses (section 3.1), with (N * K)^D structures for N GPU types,
 * K TP degrees and D stages (section 2), run as one data-parallel workload.
 * The space, in order (outermost first): S = 1 .. d_max stages; the type
 * vector (g_0 .. g_{S-1}), each entry over `types` in list order, g_0
 * slowest; the TP vector (over `log2_tp`) likewise; the DP degree (over
 * `dp`). Every stage of a template gets the template's DP degree and EP
 * degree 2^log2_ep. Index u of this order is template u of the space. The
 * micro-batch count is the innermost loop (the m list of the calls below).
 * All pointers are HOST memory, read during the call.
 */
typedef struct heddle_enum_spec {
    int32_t d_max;                /* stage counts 1 .. d_max, d_max in 1..64                */
    int32_t n_types;              /* 1..255                                                 */
    const uint8_t *types;         /* [n_types] distinct GPU type indices, in loop order     */
    int32_t n_tp;                 /* 1..16                                                  */
    const uint8_t *log2_tp;       /* [n_tp] distinct log2 TP degrees 0..15, in loop order   */
    int32_t n_dp;                 /* 1..64                                                  */
    const int32_t *dp;            /* [n_dp] distinct DP degrees 1..65535, in loop order     */
    int32_t log2_ep;              /* EP degree of every stage, log2, 0..15                  */
} heddle_enum_spec;

/*
 * heddle_enum_count -- size of the space: sum over S of
 * (n_types * n_tp)^S * n_dp. Returns HEDDLE_OK, HEDDLE_E_INVAL (bad spec:
 * size out of range, a duplicate list entry) or HEDDLE_E_RANGE (2^62 or
 * more templates).
 */
int heddle_enum_count(const heddle_enum_spec *sp, int64_t *h_count);

/*
 * heddle_enum_templates -- write templates first .. first + n - 1 of the
 * space as template records (the layout of heddle_price_plans with
 * s_max = d_max; slots s >= S are zero). Asynchronous on `stream`.
 *   d_n_stages  DEVICE [n] uint8; d_stages DEVICE [n][d_max] uint32.
 * Returns HEDDLE_OK, HEDDLE_E_INVAL (bad spec, range outside the space, null
 * output), HEDDLE_E_RANGE or HEDDLE_E_DEVICE.
 */
int heddle_enum_templates(const heddle_enum_spec *sp, int64_t first, int64_t n,
                          uint8_t *d_n_stages, uint32_t *d_stages, hipStream_t stream);

/*
 * heddle_best_enumerated -- the best plan of the whole space: every
 * template at every m, priced as heddle_price_plans (s_max = d_max, the
 * same flags) and ranked as heddle_argmin_plans, ties to the lowest template
 * index, then the lowest m index. The space is walked in chunks of `chunk`
 * templates (0: 4,194,304); the library allocates the chunk buffers on
 * `stream` (stream-ordered) and frees them before returning. Synchronous.
 *   h_best_index    HOST template index in the space (heddle_enum_templates
 *                   with n = 1 gives its records).
 *   h_best_m_index  HOST index into h_m.
 *   h_best_iter     HOST int64 (float with FP32) iteration time; may be NULL.
 *   h_n_ok          HOST number of plans of status OK; may be NULL.
 * Returns HEDDLE_OK, HEDDLE_E_NOFEASIBLE (no plan of the space has status
 * OK; *h_n_ok is still written), HEDDLE_E_INVAL, HEDDLE_E_RANGE,
 * HEDDLE_E_NOMEM or HEDDLE_E_DEVICE.
 */
int heddle_best_enumerated(const heddle_profile *p, const heddle_enum_spec *sp,
                           const int32_t *h_m, int32_t n_m, uint32_t flags, int64_t chunk,
                           int64_t *h_best_index, int32_t *h_best_m_index, void *h_best_iter,
                           int64_t *h_n_ok, hipStream_t stream);

/*
 * heddle_profile_info -- facts about a loaded profile for tests and reports.
 *   narrow[0]  1 if the int64 split runs in exact 32-bit arithmetic
 *   narrow[1]  1 if the fp32 split does
 *   fx_exp     exponent of the fixed-point unit of the fp32 variant (<= 0)
 */
typedef struct heddle_profile_info {
    int32_t narrow[2];
    int32_t fx_exp;
    int32_t L, n_types, n_tp, n_ep;
    int64_t max_stage_ns;        /* bound on any stage time, ns            */
    int64_t scratch_bytes;       /* device bytes of the per-stream buffers the
                                    profile holds now (see heddle_price_plans) */
    int32_t narrow_tile;         /* 1 if expert tiling holds times in 32 bits */
} heddle_profile_info;
int heddle_profile_info_get(const heddle_profile *p, heddle_profile_info *info);

/* Message of the last negative return on this host thread ("" if none). */
const char *heddle_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HEDDLE_H */
