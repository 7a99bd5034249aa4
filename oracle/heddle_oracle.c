/*
 * heddle_oracle.c -- plain CPU oracle of batched plan pricing.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this file's library. The GPU library
 * shares no code with it: no headers, helpers, tables or generators.
 *
 * What it computes (Heddle, arXiv 2609.34244): for each structural template
 * (section 5.1: pipeline depth plus per-stage GPU type and TP degree; here
 * also per-stage DP and EP degrees) and each global micro-batch count m,
 *   1. validate the template (feasibility masks of section 5.1, exact-match
 *      profile lookup of section 5.2),
 *   2. PartitionLayers: split the L layers over the S stages so that the
 *      slowest stage is as fast as possible (the min-max layer split of the
 *      nested-loop backbone, section 3.1), honouring per-GPU memory
 *      (memory validation, section 5.2),
 *   3. Evaluate: the 1F1B iteration time (M-1) max_s t_s + sum_s t_s +
 *      max_s g_s (section 5.3, expert tiling paragraph) and the per-GPU peak
 *      memory (section 5.2),
 * and finally the argmin over all feasible plans of iteration time per
 * micro-batch (section 5 overview: candidates are ordered by the cost
 * model's throughput estimate; section 5.3: the quickest fitting choice is
 * retained).
 *
 * Expert tiling (oracle_tile_plans): each stage of a priced plan re-chooses
 * its expert layout EP x ETP x EDP among the factorisations of its GPUs that
 * fit memory, and the layouts are chosen together for the shortest 1F1B
 * iteration (section 5.3, expert tiling; see tile_plan).
 *
 * Second partition mode (OR_F_DISTRIBUTE): Heddle's own layer split of the
 * arithmetic auto-fill (section 5.3, layer split and DP degree): the layer
 * shares follow the stages' profiled speeds; if that split overflows memory,
 * a predefined set of neighbouring splits is evaluated and the quickest one
 * within memory wins (see distribute_cuts and price_distribute).
 *
 * Everything is written the slow, obvious way: every sum is a loop, every
 * product and quotient of a transfer time is done in 128-bit integers, and
 * the DP is the textbook suffix recurrence over all (row, column) pairs.
 *
 * Readings of the paper where it is silent:
 *  - the split minimises the bottleneck stage time (stage compute + its
 *    outbound p2p), every stage holds >= 1 layer, ties are broken to the
 *    lexicographically smallest layer-count vector;
 *  - a stage holds min(S - s, M_p) in-flight micro-batches of activations
 *    (1F1B), M_p = ceil(m / D) micro-batches per pipeline replica;
 *  - transfer time of b bytes at B MB/s is ceil(b * 1000 / B) ns; the ring
 *    all-reduce of b bytes over n ranks is ceil(2 (n-1) b * 1000 / (n B)) ns;
 *  - an MoE layer on a stage with EP degree e > 1 adds one all-to-all of
 *    a2a_bytes, priced at the intra-node bandwidth when the e*TP group fits
 *    one node and at the same-type inter-node bandwidth otherwise (expert
 *    tiling paragraph of section 5.3); expert state is sharded by e and
 *    expert gradients are all-reduced over D / e replicas.
 *
 * fp32 variant: every time quantity is the fp32 value nearest (ties to even)
 * to the exact real-valued quantity computed from the fp32 per-layer costs;
 * see oracle_price_plans_f32 below.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

typedef __int128 i128;

#define OR_INF INT64_MAX

enum {
    OR_OK = 0, OR_BAD_SHAPE = 1, OR_BAD_TYPE = 2, OR_BAD_TP = 3, OR_UNPROFILED = 4,
    OR_BAD_DP = 5, OR_BAD_EP = 6, OR_OVERSUBSCRIBED = 7, OR_OOM = 8
};

#define OR_F_FP32 1u
#define OR_F_COMPUTE_ONLY 2u
#define OR_F_DISTRIBUTE 4u

typedef struct {
    int32_t L, n_types, n_tp, n_ep;
    const int32_t *tp_degrees, *ep_degrees;
    const int64_t *layer_ns;       /* [n_types][n_tp][L] */
    const uint8_t *profiled;       /* [n_types][n_tp] */
    const float *layer_ns_f32;     /* [n_types][n_tp][L] or NULL */
    const uint8_t *is_moe;         /* [L] */
    const int64_t *state_bytes, *xstate_bytes, *act_bytes, *grad_bytes, *xgrad_bytes; /* [n_tp][L] */
    int64_t boundary_bytes, a2a_bytes;
    const int64_t *mem_cap_bytes;  /* [n_types] */
    const int32_t *node_size, *n_gpus; /* [n_types] */
    const int64_t *intra_bw_MBps;  /* [n_types] */
    const int64_t *link_bw_MBps;   /* [n_types][n_types] */
    const int64_t *xlayer_ns;      /* [n_types][n_tp][L] experts' part of layer_ns, or NULL (0) */
} oracle_profile;

/* one decoded stage */
typedef struct { int g, tp, tpi, ep, dp; } ostage;

static i128 ceil_div128(i128 a, i128 b) { return (a + b - 1) / b; }

/* Transfer time in ns of `bytes` at `MBps` megabytes per second. */
static int64_t xfer_ns(int64_t bytes, int64_t MBps)
{
    return (int64_t)ceil_div128((i128)bytes * 1000, (i128)MBps);
}

/* Ring all-reduce of `bytes` over `n` ranks: 2 (n-1)/n * bytes / bw
 * (Patarasuk & Yuan's bandwidth-optimal ring); zero for a single rank. */
static int64_t allreduce_ns(int64_t bytes, int64_t n, int64_t MBps)
{
    if (n == 1) return 0;
    return (int64_t)ceil_div128((i128)2 * (n - 1) * bytes * 1000, (i128)n * MBps);
}

static int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

/* ---------------------------------------------------------------------- */
/* Template decode and validation (feasibility masks, section 5.1; exact-   */
/* match profile lookup, section 5.2). First failing check wins.           */
/* ---------------------------------------------------------------------- */
static int validate(const oracle_profile *p, int S, int s_max, const uint32_t *rec, ostage *st)
{
    if (S < 1 || S > s_max || S > p->L) return OR_BAD_SHAPE;
    for (int s = 0; s < S; s++) {
        st[s].g = (int)(rec[s] & 0xFF);
        st[s].tp = 1 << ((rec[s] >> 8) & 0xF);
        st[s].ep = 1 << ((rec[s] >> 12) & 0xF);
        st[s].dp = (int)(rec[s] >> 16);
        st[s].tpi = -1;
    }
    for (int s = 0; s < S; s++)
        if (st[s].g >= p->n_types) return OR_BAD_TYPE;
    for (int s = 0; s < S; s++) {
        for (int k = 0; k < p->n_tp; k++)
            if (p->tp_degrees[k] == st[s].tp) st[s].tpi = k;
        if (st[s].tpi < 0 || st[s].tp > p->node_size[st[s].g]) return OR_BAD_TP;
    }
    for (int s = 0; s < S; s++)
        if (!p->profiled[st[s].g * p->n_tp + st[s].tpi]) return OR_UNPROFILED;
    for (int s = 0; s < S; s++)
        if (st[s].dp < 1 || st[s].dp != st[0].dp) return OR_BAD_DP;
    for (int s = 0; s < S; s++) {
        int found = 0;
        for (int e = 0; e < p->n_ep; e++)
            if (p->ep_degrees[e] == st[s].ep) found = 1;
        if (!found || st[s].dp % st[s].ep != 0) return OR_BAD_EP;
    }
    for (int g = 0; g < p->n_types; g++) {
        int64_t used = 0;
        for (int s = 0; s < S; s++)
            if (st[s].g == g) used += (int64_t)st[s].tp * st[s].dp;
        if (used > p->n_gpus[g]) return OR_OVERSUBSCRIBED;
    }
    return OR_OK;
}

/* ---------------------------------------------------------------------- */
/* Per-stage cost terms.                                                   */
/* ---------------------------------------------------------------------- */

/* All-to-all time per MoE layer on a stage (expert tiling, section 5.3):
 * zero without EP; intra-node bandwidth when the EP x TP group fits one
 * node, otherwise the same-type inter-node link. */
static int64_t a2a_ns(const oracle_profile *p, const ostage *st)
{
    if (st->ep == 1) return 0;
    int64_t bw = ((int64_t)st->ep * st->tp <= p->node_size[st->g])
                     ? p->intra_bw_MBps[st->g] : p->link_bw_MBps[st->g * p->n_types + st->g];
    return xfer_ns(p->a2a_bytes, bw);
}

/* Inter-stage p2p per micro-batch (forward activation + backward gradient),
 * charged to the sending stage; the last stage sends nothing. */
static int64_t p2p_ns(const oracle_profile *p, const ostage *st, int s, int S)
{
    if (s == S - 1) return 0;
    return xfer_ns(2 * p->boundary_bytes, p->link_bw_MBps[st[s].g * p->n_types + st[s + 1].g]);
}

/* Cost of layer l on stage st: profiled compute + TP comm, plus the
 * all-to-all of an MoE layer. */
static int64_t layer_cost(const oracle_profile *p, const ostage *st, int l)
{
    int64_t c = p->layer_ns[((int64_t)st->g * p->n_tp + st->tpi) * p->L + l];
    if (p->is_moe[l]) c += a2a_ns(p, st);
    return c;
}

/* T(s, i, j): time of stage s holding layers [i, j). */
static int64_t stage_time(const oracle_profile *p, const ostage *st, int s, int S, int i, int j)
{
    int64_t t = p2p_ns(p, st, s, S);
    for (int l = i; l < j; l++) t += layer_cost(p, &st[s], l);
    return t;
}

/* Mem(s, i, j): the peak memory of one GPU of stage s holding layers [i, j) with
 * `inflight` micro-batches of activations resident (memory validation,
 * section 5.2: parameters + optimizer state + gradients + activations). */
static int64_t stage_mem(const oracle_profile *p, const ostage *st, int i, int j, int64_t inflight)
{
    i128 w = 0, a = 0;
    for (int l = i; l < j; l++) {
        w += p->state_bytes[st->tpi * p->L + l] + ceil_div64(p->xstate_bytes[st->tpi * p->L + l], st->ep);
        a += p->act_bytes[st->tpi * p->L + l];
    }
    i128 mem = w + (i128)inflight * a;
    return mem > INT64_MAX ? INT64_MAX : (int64_t)mem;
}

/* Gradient synchronisation g_s of one stage: ring all-reduce of the dense
 * gradients over the D replicas, plus the expert gradients over the D / e
 * expert-data-parallel replicas. Intra-node bandwidth if the TP x D group
 * fits one node, else the same-type inter-node link. */
static int64_t stage_sync(const oracle_profile *p, const ostage *st, int i, int j)
{
    int64_t bw = ((int64_t)st->tp * st->dp <= p->node_size[st->g])
                     ? p->intra_bw_MBps[st->g] : p->link_bw_MBps[st->g * p->n_types + st->g];
    int64_t gd = 0, gx = 0;
    for (int l = i; l < j; l++) {
        gd += p->grad_bytes[st->tpi * p->L + l];
        gx += ceil_div64(p->xgrad_bytes[st->tpi * p->L + l], st->ep);
    }
    return allreduce_ns(gd, st->dp, bw) + allreduce_ns(gx, st->dp / st->ep, bw);
}

/* ---------------------------------------------------------------------- */
/* PartitionLayers: exact min-max split. G[s][i] is the smallest achievable */
/* bottleneck when stages s..S-1 hold layers [i, L); G[S][L] = 0 and        */
/* G[S][j] = inf for j < L closes the recurrence. Stage time is an integer  */
/* here; the fp32 variant passes a rounding hook.                          */
/* ---------------------------------------------------------------------- */
typedef int64_t (*time_fn)(const oracle_profile *, const ostage *, int s, int S, int i, int j);

static int64_t inflight_of(int s, int S, int64_t Mp) { return (S - s) < Mp ? (S - s) : Mp; }

static int fits(const oracle_profile *p, const ostage *st, int s, int S, int i, int j,
                int64_t Mp, int compute_only)
{
    if (compute_only) return 1;
    return stage_mem(p, &st[s], i, j, inflight_of(s, S, Mp)) <= p->mem_cap_bytes[st[s].g];
}

/* Returns B* (OR_INF if no split fits) and fills cut[0..S] (cut[0] = 0,
 * cut[S] = L) with the lexicographically smallest optimal layer counts. */
static int64_t partition(const oracle_profile *p, const ostage *st, int S, int64_t Mp,
                         int compute_only, time_fn T, int *cut)
{
    int L = p->L;
    int64_t *G = (int64_t *)malloc(sizeof(int64_t) * (size_t)(S + 1) * (L + 1));
#define Gat(s, i) G[(size_t)(s) * (L + 1) + (i)]
    for (int i = 0; i <= L; i++) Gat(S, i) = (i == L) ? 0 : OR_INF;
    for (int s = S - 1; s >= 0; s--) {
        for (int i = 0; i <= L; i++) Gat(s, i) = OR_INF;
        /* stage s starts at i with at least one layer left for each later stage */
        for (int i = s; i <= L - (S - s); i++) {
            int64_t best = OR_INF;
            for (int j = i + 1; j <= L - (S - 1 - s); j++) {
                if (!fits(p, st, s, S, i, j, Mp, compute_only)) continue;
                int64_t t = T(p, st, s, S, i, j);
                int64_t cand = t > Gat(s + 1, j) ? t : Gat(s + 1, j);
                if (cand < best) best = cand;
            }
            Gat(s, i) = best;
        }
    }
    int64_t B = Gat(0, 0);
    if (B != OR_INF) {
        /* canonical forward reconstruction: at each stage take the smallest
         * end that keeps an optimal completion */
        cut[0] = 0;
        for (int s = 0; s < S; s++) {
            int found = -1;
            for (int j = cut[s] + 1; j <= L - (S - 1 - s); j++) {
                if (!fits(p, st, s, S, cut[s], j, Mp, compute_only)) continue;
                if (T(p, st, s, S, cut[s], j) <= B && Gat(s + 1, j) <= B) { found = j; break; }
            }
            if (found < 0) { B = OR_INF; break; }   /* unreachable by construction */
            cut[s + 1] = found;
        }
    }
    free(G);
#undef Gat
    return B;
}

/* Largest admissible end of row i at stage s: the largest j in
 * (i, L-(S-1-s)] with Fits(s,i,j), or i itself when no such j fits. */
static int last_end(const oracle_profile *p, const ostage *st, int s, int S, int i, int64_t Mp, int co)
{
    int best = i;
    for (int j = i + 1; j <= p->L - (S - 1 - s); j++)
        if (fits(p, st, s, S, i, j, Mp, co)) best = j;
    return best;
}

/* Work of the suffix DP over the rows that can lie on a complete split.
 * R_s is the furthest start stage s can be reached at from row 0:
 * R_0 = 0, R_{s+1} = last_end(s, R_s). Bk_s is the smallest start i in
 * [s, min(R_s, L-(S-s))] with last_end(s, i) >= Bk_{s+1}, where Bk_S = L; when
 * some stage has no such start, no split fits and there is no work. Stage
 * s < S-1 relaxes each row i in [Bk_s, min(R_s, L-(S-s))] against the ends
 * max(i+1, Bk_{s+1}) .. last_end(s, i); each row of the last stage counts one.
 * This is the algorithmic work unit of the GPU kernel. */
static int64_t count_distribute(const oracle_profile *p, const ostage *st, int S, int64_t m, uint32_t flags);

int64_t oracle_count_relaxations(const oracle_profile *p, int S, const uint32_t *rec, int s_max,
                                 int64_t m, uint32_t flags)
{
    ostage st[256];
    if (validate(p, S, s_max, rec, st) != OR_OK) return 0;
    if (flags & OR_F_DISTRIBUTE) return count_distribute(p, st, S, m, flags);
    int64_t Mp = ceil_div64(m, st[0].dp), count = 0;
    int L = p->L, co = (flags & OR_F_COMPUTE_ONLY) != 0;
    int R[257], Bk[258], top[257];
    R[0] = 0;
    for (int s = 0; s + 1 < S; s++) R[s + 1] = last_end(p, st, s, S, R[s], Mp, co);
    Bk[S] = L;
    for (int s = S - 1; s >= 0; s--) {
        int ihi = (s == 0) ? 0 : L - (S - s);
        top[s] = R[s] < ihi ? R[s] : ihi;
        Bk[s] = -1;
        for (int i = s; i <= top[s]; i++)
            if (last_end(p, st, s, S, i, Mp, co) >= Bk[s + 1]) { Bk[s] = i; break; }
        if (Bk[s] < 0) return 0;
    }
    for (int s = 0; s < S; s++)
        for (int i = Bk[s]; i <= top[s]; i++) {
            if (s == S - 1) { count++; continue; }
            int lo = i + 1 > Bk[s + 1] ? i + 1 : Bk[s + 1];
            int hi = last_end(p, st, s, S, i, Mp, co);
            if (hi >= lo) count += hi - lo + 1;
        }
    return count;
}

/* ---------------------------------------------------------------------- */
/* int64 pricing of one (template, m) plan.                                */
/* ---------------------------------------------------------------------- */
typedef struct {
    int status;
    int64_t iter, bottleneck, peak_mem;
    double iter_f, bottleneck_f;     /* fp32 variant (exactly representable) */
    int cut[257];
} oplan;

static int64_t time_i64(const oracle_profile *p, const ostage *st, int s, int S, int i, int j)
{
    return stage_time(p, st, s, S, i, j);
}

/* Evaluate (section 5.3) the split out->cut: bottleneck max_s t_s,
 * iteration time (M-1) max_s t_s + sum_s t_s + max_s g_s, peak memory, and
 * status OOM when some stage does not fit. */
static void evaluate_i64(const oracle_profile *p, const ostage *st, int S, int64_t Mp, oplan *out)
{
    i128 sum_t = 0;
    int64_t B = 0, max_g = 0, peak = 0;
    int oom = 0;
    for (int s = 0; s < S; s++) {
        int i = out->cut[s], j = out->cut[s + 1];
        int64_t t = stage_time(p, st, s, S, i, j);
        sum_t += t;
        if (t > B) B = t;
        int64_t g = stage_sync(p, &st[s], i, j);
        if (g > max_g) max_g = g;
        int64_t mem = stage_mem(p, &st[s], i, j, inflight_of(s, S, Mp));
        if (mem > peak) peak = mem;
        if (mem > p->mem_cap_bytes[st[s].g]) oom = 1;
    }
    out->status = oom ? OR_OOM : OR_OK;
    out->bottleneck = B;
    out->iter = (int64_t)((i128)(Mp - 1) * B + sum_t + max_g);
    out->peak_mem = peak;
}

static void price_one(const oracle_profile *p, const ostage *st, int S, int64_t m, uint32_t flags,
                      oplan *out)
{
    int co = (flags & OR_F_COMPUTE_ONLY) != 0;
    int64_t D = st[0].dp, Mp = ceil_div64(m, D);
    int64_t B = partition(p, st, S, Mp, co, time_i64, out->cut);
    if (B == OR_INF) { out->status = OR_OOM; return; }
    evaluate_i64(p, st, S, Mp, out);     /* the canonical split's max_s t_s is B */
}

/* ---------------------------------------------------------------------- */
/* fp32 variant. Per-layer costs are the fp32 table (or the int64 table    */
/* rounded to fp32); transfer terms are the int64 ns values rounded to     */
/* fp32. A stage time is the exact real sum of its fp32 terms, rounded     */
/* once to the nearest fp32. The sum is formed exactly in a 128-bit fixed  */
/* point with 2^-FX fractional bits, which holds every fp32 of magnitude   */
/* >= 2^-FX+23 exactly; the loader rejects tables outside that range.      */
/* ---------------------------------------------------------------------- */
#define FX 40

static i128 fx_of_float(float v)
{
    /* v = mant * 2^exp exactly, with |mant| < 2^24 */
    int e;
    double fr = frexp((double)v, &e);             /* v = fr * 2^e, 0.5 <= fr < 1 */
    i128 mant = (i128)ldexp(fr, 24);               /* exact: fr has 24 bits */
    int sh = e - 24 + FX;
    if (sh >= 0) return mant << sh;
    return mant >> (-sh);                          /* caller guarantees no bits lost */
}

/* nearest fp32 (ties to even) of the fixed-point value x >= 0 */
static float float_of_fx(i128 x)
{
    if (x == 0) return 0.0f;
    /* find the top bit */
    int top = 127;
    while (top > 0 && !((x >> top) & 1)) top--;
    /* keep 24 significant bits, round half to even on the rest */
    int drop = top - 23;
    i128 q, r, half;
    if (drop <= 0) return (float)ldexp((double)(int64_t)x, -FX);   /* exact */
    q = x >> drop;
    r = x - (q << drop);
    half = (i128)1 << (drop - 1);
    if (r > half || (r == half && (q & 1))) q += 1;
    return (float)ldexp((double)(int64_t)q, drop - FX);            /* q <= 2^24: exact */
}

static float layer_cost_f32(const oracle_profile *p, const ostage *st, int l)
{
    size_t idx = ((size_t)st->g * p->n_tp + st->tpi) * p->L + l;
    return p->layer_ns_f32 ? p->layer_ns_f32[idx] : (float)p->layer_ns[idx];
}

static i128 stage_time_fx(const oracle_profile *p, const ostage *st, int s, int S, int i, int j)
{
    i128 t = fx_of_float((float)p2p_ns(p, st, s, S));
    float a2a = (float)a2a_ns(p, &st[s]);
    for (int l = i; l < j; l++) {
        t += fx_of_float(layer_cost_f32(p, &st[s], l));
        if (p->is_moe[l]) t += fx_of_float(a2a);
    }
    return t;
}

/* fp32 stage time, carried as the bit pattern of a non-negative float so
 * that integer order equals float order. */
static int64_t time_f32bits(const oracle_profile *p, const ostage *st, int s, int S, int i, int j)
{
    float f = float_of_fx(stage_time_fx(p, st, s, S, i, j));
    uint32_t u;
    memcpy(&u, &f, 4);
    return (int64_t)u;
}

static float bits_to_float(int64_t b)
{
    uint32_t u = (uint32_t)b;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* fp32 Evaluate of the split out->cut: stage times rounded to fp32 once
 * each, the iteration time rounded once from the exact sum of its fp32 terms. */
static void evaluate_f32(const oracle_profile *p, const ostage *st, int S, int64_t Mp, oplan *out)
{
    float B = 0.0f, max_g = 0.0f;
    i128 sum_t = 0;
    int64_t peak = 0;
    int oom = 0;
    for (int s = 0; s < S; s++) {
        int i = out->cut[s], j = out->cut[s + 1];
        float t = float_of_fx(stage_time_fx(p, st, s, S, i, j));
        sum_t += fx_of_float(t);
        if (t > B) B = t;
        float g = (float)stage_sync(p, &st[s], i, j);
        if (g > max_g) max_g = g;
        int64_t mem = stage_mem(p, &st[s], i, j, inflight_of(s, S, Mp));
        if (mem > peak) peak = mem;
        if (mem > p->mem_cap_bytes[st[s].g]) oom = 1;
    }
    i128 total = (i128)(Mp - 1) * fx_of_float(B) + sum_t + fx_of_float(max_g);
    out->status = oom ? OR_OOM : OR_OK;
    out->bottleneck_f = B;
    out->iter_f = float_of_fx(total);
    out->peak_mem = peak;
}

static void price_one_f32(const oracle_profile *p, const ostage *st, int S, int64_t m, uint32_t flags,
                          oplan *out)
{
    int co = (flags & OR_F_COMPUTE_ONLY) != 0;
    int64_t D = st[0].dp, Mp = ceil_div64(m, D);
    int64_t Bbits = partition(p, st, S, Mp, co, time_f32bits, out->cut);
    if (Bbits == OR_INF) { out->status = OR_OOM; return; }
    evaluate_f32(p, st, S, Mp, out);     /* the canonical split's max_s t_s is B */
}

/* ---------------------------------------------------------------------- */
/* Distribute (section 5.3, layer split and DP degree).                    */
/* Readings: the profiled speed of stage s is the inverse of the time of   */
/* all L layers on its GPU type and TP degree (int64 layer costs with the  */
/* stage's all-to-all terms, p2p excluded). The cut after stage s is the   */
/* nearest integer (halves up) to L * (sum_{t<=s} speed_t) / sum_t speed_t, */
/* computed in IEEE double in this order, then moved up to leave stage s   */
/* one layer and down to leave every later stage one layer. When that      */
/* split does not fit memory, the alternatives tried are: for each         */
/* boundary b = 0 .. S-2 in order, the cut after stage b moved by -1, then */
/* by +1 (kept only if every stage still holds a layer); the fitting       */
/* alternative with the smallest iteration time is kept, the first in list */
/* order on ties; none fitting leaves the plan OOM without a split. With   */
/* OR_F_COMPUTE_ONLY the proportional split is kept and only flagged.      */
/* ---------------------------------------------------------------------- */
static void distribute_cuts(const oracle_profile *p, const ostage *st, int S, int *cut)
{
    int L = p->L;
    double speed[256], total = 0.0, below = 0.0;
    for (int s = 0; s < S; s++) {
        int64_t all = 0;
        for (int l = 0; l < L; l++) all += layer_cost(p, &st[s], l);
        speed[s] = 1.0 / (double)all;
    }
    for (int s = 0; s < S; s++) total += speed[s];
    cut[0] = 0;
    for (int s = 1; s < S; s++) {
        below += speed[s - 1];
        int c = (int)floor((double)L * below / total + 0.5);
        if (c < cut[s - 1] + 1) c = cut[s - 1] + 1;
        if (c > L - (S - s)) c = L - (S - s);
        cut[s] = c;
    }
    cut[S] = L;
}

static int faster(const oplan *a, const oplan *b, int f32)
{
    return f32 ? a->iter_f < b->iter_f : a->iter < b->iter;
}

static void price_distribute(const oracle_profile *p, const ostage *st, int S, int64_t m, uint32_t flags,
                             oplan *out)
{
    int co = (flags & OR_F_COMPUTE_ONLY) != 0, f32 = (flags & OR_F_FP32) != 0;
    int64_t Mp = ceil_div64(m, st[0].dp);
    distribute_cuts(p, st, S, out->cut);
    if (f32) evaluate_f32(p, st, S, Mp, out);
    else evaluate_i64(p, st, S, Mp, out);
    if (out->status == OR_OK || co) return;
    oplan best, cand;
    int found = 0;
    for (int b = 0; b + 1 < S; b++) {
        for (int d = -1; d <= 1; d += 2) {
            memcpy(cand.cut, out->cut, sizeof(int) * (size_t)(S + 1));
            cand.cut[b + 1] += d;
            if (cand.cut[b + 1] <= cand.cut[b] || cand.cut[b + 1] >= cand.cut[b + 2]) continue;
            if (f32) evaluate_f32(p, st, S, Mp, &cand);
            else evaluate_i64(p, st, S, Mp, &cand);
            if (cand.status != OR_OK) continue;
            if (!found || faster(&cand, &best, f32)) { best = cand; found = 1; }
        }
    }
    if (found) *out = best;
    else out->status = OR_OOM;
}

/* Work of Distribute, in stage-cost evaluations: S for the proportional
 * split and, when it does not fit (and memory is checked), 2 for every
 * alternative of the list (only the two stages around the moved cut change;
 * the others are already priced). */
static int64_t count_distribute(const oracle_profile *p, const ostage *st, int S, int64_t m, uint32_t flags)
{
    oplan pl;
    int64_t Mp = ceil_div64(m, st[0].dp), n = S;
    distribute_cuts(p, st, S, pl.cut);
    evaluate_i64(p, st, S, Mp, &pl);
    if (pl.status == OR_OK || (flags & OR_F_COMPUTE_ONLY)) return n;
    for (int b = 0; b + 1 < S; b++)
        for (int d = -1; d <= 1; d += 2) {
            int c = pl.cut[b + 1] + d;
            if (c > pl.cut[b] && c < pl.cut[b + 2]) n += 2;
        }
    return n;
}

/* ---------------------------------------------------------------------- */
/* Batch entry points.                                                     */
/* Outputs per (template t, m index k), index t * n_m + k:                 */
/*   iter, bottleneck (int64, or float when OR_F_FP32), peak_mem, status,  */
/*   layers[(t * n_m + k) * s_max + s] (0 beyond S).                       */
/* Non-OK plans whose split is undefined get iter = bottleneck = peak_mem  */
/* = INT64_MAX (float: +inf) and all-zero layer counts.                    */
/* ---------------------------------------------------------------------- */
int oracle_price_plans(const oracle_profile *p, int64_t t0, int64_t t1, int s_max,
                       const uint8_t *n_stages, const uint32_t *stages,
                       const int32_t *m, int n_m, uint32_t flags,
                       void *iter, void *bottleneck, int64_t *peak_mem,
                       uint8_t *layers, uint8_t *status)
{
    ostage st[256];
    oplan pl;
    int f32 = (flags & OR_F_FP32) != 0;
    for (int64_t t = t0; t < t1; t++) {
        int S = n_stages[t];
        const uint32_t *rec = stages + (size_t)t * s_max;
        int v = validate(p, S, s_max, rec, st);
        for (int k = 0; k < n_m; k++) {
            size_t o = (size_t)t * n_m + k;
            pl.status = v;
            if (v == OR_OK) {
                if (flags & OR_F_DISTRIBUTE) price_distribute(p, st, S, m[k], flags, &pl);
                else if (f32) price_one_f32(p, st, S, m[k], flags, &pl);
                else price_one(p, st, S, m[k], flags, &pl);
            }
            int has_split = (pl.status == OR_OK) ||
                            (pl.status == OR_OOM && (flags & OR_F_COMPUTE_ONLY));
            status[o] = (uint8_t)pl.status;
            for (int s = 0; s < s_max; s++)
                layers[o * s_max + s] = (has_split && s < S) ? (uint8_t)(pl.cut[s + 1] - pl.cut[s]) : 0;
            if (f32) {
                ((float *)iter)[o] = has_split ? (float)pl.iter_f : INFINITY;
                ((float *)bottleneck)[o] = has_split ? (float)pl.bottleneck_f : INFINITY;
            } else {
                ((int64_t *)iter)[o] = has_split ? pl.iter : INT64_MAX;
                ((int64_t *)bottleneck)[o] = has_split ? pl.bottleneck : INT64_MAX;
            }
            peak_mem[o] = has_split ? pl.peak_mem : INT64_MAX;
        }
    }
    return 0;
}

/* ---------------------------------------------------------------------- */
/* Expert tiling (section 5.3, expert tiling paragraph). A stage of TP k   */
/* and DP D spans W = k * D GPUs, and its expert layout is EP e x ETP t x  */
/* EDP W / (e t). The layouts priced for a stage: e from the EP list, t    */
/* from the TP list, t profiled for the stage's GPU type and no larger     */
/* than its node (ETP stays within a node like TP; EP may span nodes), e t */
/* dividing                                                                */
/* W. For one layout:                                                      */
/*  - an MoE layer costs its profiled time at TP k with the experts' part  */
/*    at ETP k replaced by the experts' part at ETP t scaled to the        */
/*    stage's tokens per GPU (x_t * t / k, rounded up), plus one all-to-all */
/*    at intra-node bandwidth if the e t GPUs of an EP group fit one node, */
/*    else at the same-type inter-node link;                               */
/*  - memory: dense state at TP k, expert state at ETP t divided by e      */
/*    (rounded up per layer), in-flight activations at TP k;               */
/*  - synchronisation: dense gradients over the D replicas, expert         */
/*    gradients at ETP t divided by e over the W / (e t) EDP replicas.     */
/* With t = k and e the template's EP these are the untiled terms.         */
/* A stage is tiled on its own (its layout reaches no other stage); the    */
/* plan's layouts are then chosen together to minimise the whole 1F1B      */
/* iteration (M-1) max_s t_s + sum_s t_s + max_s g_s over the layouts that */
/* fit memory (see tile_plan).                                             */
/* ---------------------------------------------------------------------- */
typedef struct { int e, ei, t, ti; } otile;

static int64_t xlayer(const oracle_profile *p, int g, int ti, int l)
{
    return p->xlayer_ns ? p->xlayer_ns[((int64_t)g * p->n_tp + ti) * p->L + l] : 0;
}

static int64_t tiled_layer_cost(const oracle_profile *p, const ostage *st, const otile *tl, int l)
{
    int64_t c = p->layer_ns[((int64_t)st->g * p->n_tp + st->tpi) * p->L + l];
    if (p->is_moe[l]) {
        i128 scaled = ceil_div128((i128)xlayer(p, st->g, tl->ti, l) * tl->t, st->tp);
        c += (int64_t)scaled - xlayer(p, st->g, st->tpi, l);
        if (tl->e > 1) {
            int64_t bw = ((int64_t)tl->e * tl->t <= p->node_size[st->g])
                             ? p->intra_bw_MBps[st->g] : p->link_bw_MBps[st->g * p->n_types + st->g];
            c += xfer_ns(p->a2a_bytes, bw);
        }
    }
    return c;
}

static int64_t tiled_time(const oracle_profile *p, const ostage *st, int s, int S, const otile *tl, int i, int j)
{
    int64_t t = p2p_ns(p, st, s, S);
    for (int l = i; l < j; l++) t += tiled_layer_cost(p, &st[s], tl, l);
    return t;
}

static int64_t tiled_mem(const oracle_profile *p, const ostage *st, const otile *tl, int i, int j, int64_t inflight)
{
    i128 w = 0, a = 0;
    for (int l = i; l < j; l++) {
        w += p->state_bytes[st->tpi * p->L + l] + ceil_div64(p->xstate_bytes[tl->ti * p->L + l], tl->e);
        a += p->act_bytes[st->tpi * p->L + l];
    }
    i128 mem = w + (i128)inflight * a;
    return mem > INT64_MAX ? INT64_MAX : (int64_t)mem;
}

static int64_t tiled_sync(const oracle_profile *p, const ostage *st, const otile *tl, int i, int j)
{
    int64_t bw = ((int64_t)st->tp * st->dp <= p->node_size[st->g])
                     ? p->intra_bw_MBps[st->g] : p->link_bw_MBps[st->g * p->n_types + st->g];
    int64_t gd = 0, gx = 0;
    for (int l = i; l < j; l++) {
        gd += p->grad_bytes[st->tpi * p->L + l];
        gx += ceil_div64(p->xgrad_bytes[tl->ti * p->L + l], tl->e);
    }
    int64_t edp = (int64_t)st->tp * st->dp / ((int64_t)tl->e * tl->t);
    return allreduce_ns(gd, st->dp, bw) + allreduce_ns(gx, edp, bw);
}

/* the layouts priced for one stage, EP list order, then TP list order */
static int tiles_of(const oracle_profile *p, const ostage *st, otile *out)
{
    int n = 0;
    for (int ei = 0; ei < p->n_ep; ei++)
        for (int ti = 0; ti < p->n_tp; ti++) {
            int e = p->ep_degrees[ei], t = p->tp_degrees[ti];
            if (!p->profiled[st->g * p->n_tp + ti] || t > p->node_size[st->g]) continue;
            if (((int64_t)st->tp * st->dp) % ((int64_t)e * t) != 0) continue;
            out[n].e = e; out[n].ei = ei; out[n].t = t; out[n].ti = ti;
            n++;
        }
    return n;
}

typedef struct { int64_t T, mem, g; int fits; otile tl; } ocand;

static int cmp_i64(const void *a, const void *b)
{
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return x < y ? -1 : x > y;
}

/* the fastest fitting layout of stage s whose synchronisation is <= G:
 * smallest time, then smallest synchronisation, then the first listed */
static int pick(const ocand *c, int n, int64_t G)
{
    int best = -1;
    for (int q = 0; q < n; q++) {
        if (!c[q].fits || c[q].g > G) continue;
        if (best < 0 || c[q].T < c[best].T || (c[q].T == c[best].T && c[q].g < c[best].g)) best = q;
    }
    return best;
}

/* Tile one plan of split cut[0..S]. With every stage's fastest fitting
 * layout under a bound G on the synchronisation term, both (M-1) max t and
 * sum t are as small as G allows, so the smallest iteration time over all
 * combinations of fitting layouts is the smallest over the thresholds G =
 * the synchronisation of some fitting layout; ties keep the smallest G.
 * Returns 0 (and leaves the outputs) if some stage has no fitting layout. */
static int tile_plan(const oracle_profile *p, const ostage *st, int S, int64_t Mp, const int *cut,
                     otile *choice, int64_t *iter, int64_t *bn, int64_t *pk)
{
    int maxc = p->n_ep * p->n_tp;
    ocand *c = (ocand *)malloc(sizeof(ocand) * (size_t)S * maxc);
    otile *tl = (otile *)malloc(sizeof(otile) * (size_t)maxc);
    int64_t *G = (int64_t *)malloc(sizeof(int64_t) * (size_t)S * maxc);
    int *nc = (int *)malloc(sizeof(int) * (size_t)S);
    int nG = 0, found = 0;
    int64_t best_it = 0, best_G = 0;
    for (int s = 0; s < S; s++) {
        nc[s] = tiles_of(p, &st[s], tl);
        for (int q = 0; q < nc[s]; q++) {
            ocand *x = &c[s * maxc + q];
            x->tl = tl[q];
            x->T = tiled_time(p, st, s, S, &tl[q], cut[s], cut[s + 1]);
            x->mem = tiled_mem(p, &st[s], &tl[q], cut[s], cut[s + 1], inflight_of(s, S, Mp));
            x->g = tiled_sync(p, &st[s], &tl[q], cut[s], cut[s + 1]);
            x->fits = x->mem <= p->mem_cap_bytes[st[s].g];
            if (x->fits) G[nG++] = x->g;
        }
    }
    qsort(G, nG, sizeof(int64_t), cmp_i64);
    for (int a = 0; a < nG; a++) {
        if (a > 0 && G[a] == G[a - 1]) continue;
        i128 sum_t = 0;
        int64_t B = 0, max_g = 0;
        int ok = 1;
        for (int s = 0; s < S && ok; s++) {
            int q = pick(&c[s * maxc], nc[s], G[a]);
            if (q < 0) { ok = 0; break; }
            const ocand *x = &c[s * maxc + q];
            sum_t += x->T;
            if (x->T > B) B = x->T;
            if (x->g > max_g) max_g = x->g;
        }
        if (!ok) continue;
        int64_t it = (int64_t)((i128)(Mp - 1) * B + sum_t + max_g);
        if (!found || it < best_it) { found = 1; best_it = it; best_G = G[a]; }
    }
    if (found) {
        int64_t B = 0, peak = 0;
        for (int s = 0; s < S; s++) {
            const ocand *x = &c[s * maxc + pick(&c[s * maxc], nc[s], best_G)];
            choice[s] = x->tl;
            if (x->T > B) B = x->T;
            if (x->mem > peak) peak = x->mem;
        }
        *iter = best_it;
        *bn = B;
        *pk = peak;
    }
    free(c); free(tl); free(G); free(nc);
    return found;
}

static int log2_of(int v) { int l = 0; while ((1 << l) < v) l++; return l; }

/* Re-tile priced plans in place (the outputs of oracle_price_plans for the
 * same templates and m list, int64 costs only). A plan with a split (status
 * OK, or OOM with layer counts) gets the best layouts: status OK, new iter,
 * bottleneck and peak memory, and tiling[o * s_max + s] = log2 EP | log2 ETP
 * << 4 per stage; if some stage has no fitting layout it keeps its values
 * and gets its starting layouts. Plans without a split are left as they are
 * with zero tiling bytes. Returns -1 for fp32 costs. */
int oracle_tile_plans(const oracle_profile *p, int64_t n, int s_max, const uint8_t *n_stages,
                      const uint32_t *stages, const int32_t *m, int n_m, uint32_t flags,
                      const uint8_t *layers, uint8_t *status, int64_t *iter, int64_t *bottleneck,
                      int64_t *peak_mem, uint8_t *tiling)
{
    ostage st[256];
    otile choice[256];
    int cut[257];
    if (flags & OR_F_FP32) return -1;
    for (int64_t t = 0; t < n; t++) {
        int S = n_stages[t];
        const uint32_t *rec = stages + (size_t)t * s_max;
        int v = validate(p, S, s_max, rec, st);
        for (int k = 0; k < n_m; k++) {
            size_t o = (size_t)t * n_m + k;
            for (int s = 0; s < s_max; s++) tiling[o * s_max + s] = 0;
            if (v != OR_OK || (status[o] != OR_OK && status[o] != OR_OOM) || layers[o * s_max] == 0) continue;
            cut[0] = 0;
            for (int s = 0; s < S; s++) cut[s + 1] = cut[s] + layers[o * s_max + s];
            int64_t Mp = ceil_div64(m[k], st[0].dp), it, bn, pk;
            if (tile_plan(p, st, S, Mp, cut, choice, &it, &bn, &pk)) {
                status[o] = OR_OK;
                iter[o] = it;
                bottleneck[o] = bn;
                peak_mem[o] = pk;
                for (int s = 0; s < S; s++)
                    tiling[o * s_max + s] = (uint8_t)(log2_of(choice[s].e) | log2_of(choice[s].t) << 4);
            } else {
                for (int s = 0; s < S; s++)
                    tiling[o * s_max + s] = (uint8_t)(log2_of(st[s].ep) | log2_of(st[s].tp) << 4);
            }
        }
    }
    return 0;
}

/* ---------------------------------------------------------------------- */
/* DP degree by packing (section 5.3, layer split and DP degree; section   */
/* 5.1, non-uniform GPU composition): the TP group of every stage is       */
/* packed into the nodes of its GPU type, replica after replica (stages in */
/* order within a replica); a group of t GPUs goes to the first node with  */
/* exactly t free GPUs, else to the node with the fewest free GPUs above t */
/* (the first such). Types pack independently; D is the smallest number of */
/* whole replicas over the types used, capped at dp_cap, rounded down to a */
/* multiple of the template's largest EP degree.                           */
/* ---------------------------------------------------------------------- */
static int place_group(const int *free_gpus, int n_nodes, int t)
{
    for (int i = 0; i < n_nodes; i++)
        if (free_gpus[i] == t) return i;
    int pick = -1;
    for (int i = 0; i < n_nodes; i++)
        if (free_gpus[i] > t && (pick < 0 || free_gpus[i] < free_gpus[pick])) pick = i;
    return pick;
}

int oracle_fill_dp(int n_types, const int32_t *n_nodes, const int32_t *node_gpus, int64_t n, int s_max,
                   const uint8_t *n_stages, uint32_t *stages, int dp_cap, int32_t *dp)
{
    int64_t first[256];
    int64_t acc = 0;
    for (int g = 0; g < n_types; g++) { first[g] = acc; acc += n_nodes[g]; }
    int *free_gpus = (int *)malloc(sizeof(int) * (size_t)(acc > 0 ? acc : 1));
    for (int64_t t = 0; t < n; t++) {
        int S = n_stages[t];
        uint32_t *rec = stages + (size_t)t * s_max;
        dp[t] = 0;
        if (S < 1 || S > s_max) continue;
        int ok_types = 1, max_ep = 1;
        for (int s = 0; s < S; s++) {
            int g = (int)(rec[s] & 0xFF), tp = 1 << ((rec[s] >> 8) & 15), ep = 1 << ((rec[s] >> 12) & 15);
            if (g >= n_types || tp > 64) ok_types = 0;
            if (ep > max_ep) max_ep = ep;
        }
        if (!ok_types) continue;
        int D = dp_cap;
        for (int g = 0; g < n_types; g++) {
            int used = 0;
            for (int s = 0; s < S; s++) used |= (int)(rec[s] & 0xFF) == g;
            if (!used) continue;
            for (int i = 0; i < n_nodes[g]; i++) free_gpus[i] = node_gpus[first[g] + i];
            int r = 0;
            while (r < dp_cap) {
                int ok = 1;
                for (int s = 0; s < S && ok; s++) {
                    if ((int)(rec[s] & 0xFF) != g) continue;
                    int tp = 1 << ((rec[s] >> 8) & 15);
                    int i = place_group(free_gpus, n_nodes[g], tp);
                    if (i < 0) ok = 0;
                    else free_gpus[i] -= tp;
                }
                if (!ok) break;
                r++;
            }
            if (r < D) D = r;
        }
        D = D / max_ep * max_ep;
        dp[t] = D;
        for (int s = 0; s < S; s++) rec[s] = (rec[s] & 0xFFFFu) | ((uint32_t)D << 16);
    }
    free(free_gpus);
    return 0;
}

/* Argmin over OK plans of iter / m (maximum throughput m / iter), compared
 * exactly as iter_a * m_b < iter_b * m_a; ties to the lowest template
 * index, then the lowest m index. Returns 0 and fills the answer, or -1
 * if no plan is OK. */
int oracle_best_plan(int64_t n, int n_m, const int32_t *m, uint32_t flags,
                     const void *iter, const uint8_t *status,
                     int64_t *best_t, int32_t *best_k)
{
    int64_t bt = -1;
    int32_t bk = -1;
    int f32 = (flags & OR_F_FP32) != 0;
    for (int64_t t = 0; t < n; t++) {
        for (int k = 0; k < n_m; k++) {
            size_t o = (size_t)t * n_m + k;
            if (status[o] != OR_OK) continue;
            int better;
            if (bt < 0) better = 1;
            else {
                size_t ob = (size_t)bt * n_m + bk;
                if (f32) {
                    /* fp32 values are exact dyadic rationals: compare exactly */
                    i128 a = fx_of_float(((const float *)iter)[o]) * m[bk];
                    i128 b = fx_of_float(((const float *)iter)[ob]) * m[k];
                    better = a < b;
                } else {
                    i128 a = (i128)((const int64_t *)iter)[o] * m[bk];
                    i128 b = (i128)((const int64_t *)iter)[ob] * m[k];
                    better = a < b;
                }
            }
            if (better) { bt = t; bk = k; }
        }
    }
    if (bt < 0) return -1;
    *best_t = bt;
    *best_k = bk;
    return 0;
}

/* Stage-level helpers exposed for closed-form tests of the formulas. */
int64_t oracle_xfer_ns(int64_t bytes, int64_t MBps) { return xfer_ns(bytes, MBps); }
int64_t oracle_allreduce_ns(int64_t bytes, int64_t n, int64_t MBps) { return allreduce_ns(bytes, n, MBps); }
float oracle_round_sum_f32(const float *v, int n)
{
    i128 t = 0;
    for (int i = 0; i < n; i++) t += fx_of_float(v[i]);
    return float_of_fx(t);
}
