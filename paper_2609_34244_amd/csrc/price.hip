// Batched plan pricing on gfx950, split kernel: PartitionLayers (exact
// min-max layer split) and its canonical reconstruction over the row windows
// that the window pass (windows.hip) found for every valid plan. Evaluate
// runs in evaluate.hip on the split found here.
//
// Method: Heddle (arXiv 2609.34244). The layer split is the PartitionLayers
// step of the planners' nested-loop backbone (section 3.1), aware of per-stage
// GPU speed (the straggler criticism of speed-blind splits in the same
// section) and of memory (section 5.2, memory validation).
//
// Recurrence (suffix form): G[s][i] is the smallest achievable bottleneck
// when stages s..S-1 hold layers [i, L):
//   G[S-1][i] = T(S-1, i, L)                                    if it fits
//   G[s][i]   = min over i < j <= jl_s(i) of max(T(s,i,j), G[s+1][j])
// with jl_s(i) the last admissible end of row i: the memory limit (a profile
// table indexed by GPU type, TP, EP and in-flight count) capped so that every
// later stage keeps one layer. B* = G[0][0]. T(s,i,j) = P_s[j] - P_s[i] + p2p_s
// with P_s the stage's time prefix (layer costs + MoE all-to-all), also a
// profile table.
//
// Mapping. One wavefront splits one template at a time (grid-stride over
// templates); templates whose plans all failed validation or have an empty
// window cost one status read. Lanes are stages while the per-stage table
// offsets are formed. A row's last admissible end is read from its stage's
// memory-limit row in the profile (through the caches; one byte per row),
// and the DP relaxes only the rows of each stage's window (rows that can lie
// on a complete split, see the split kernel). Lanes are split rows
// during the DP: r rows of a window take 64 >> ceil(log2 r) lanes each, which
// share the row's ends and combine with a cross-lane minimum. Per wavefront,
// one LDS pair row holds X[j] = {P_s[j], G[s+1][j]}, so one 64-bit read feeds
// one relaxation (sub, max, min); G[s][i] overwrites G[s+1][i] in place. The
// time prefix of stage s-1 is fetched into registers while stage s relaxes.
#include <cstring>

#include "decode.h"
#include "dp_common.h"

namespace heddle {

// Time prefix of one stage over the entries [a, e], fetched into registers
// ahead of use (slots of 64 entries; lanes past e repeat entry e).
// NS slots: 2 when L + 1 <= 128, else 4 ((L + 1) <= 256 entries)
template <class V, int NS> struct RowRegs {
    V p[NS];
};

// (row: the row's offset in the table, in entries; it joins the lanes' index
// rather than the table's base, so the base stays one scalar pair)
template <class V, int NS>
__device__ __forceinline__ void fetch_rows(RowRegs<V, NS> &r, const V *rows, uint32_t row, int a, int e, int lane)
{
#pragma unroll
    for (int q = 0; q < NS; q++)
        if (q == 0 || 64 * q <= e - a) r.p[q] = rows[row + (uint32_t)min(a + lane + 64 * q, e)];   // uniform; e >= a
}

// ------------------------------------------------------------ split kernel
//
// Row windows. With lim(s, i) the largest admissible end of row i at stage s
// (memory limit capped so that every later stage keeps a layer), lim is
// non-decreasing in i. So the starts stage s can be reached at from row 0 lie
// in [s, R_s] with R_0 = 0 and R_{s+1} = lim(s, R_s), and the rows from which
// stages s..S-1 can still complete lie in [Bk_s, L - (S - s)] with Bk_S = L and
// Bk_s the smallest i >= s whose limit reaches Bk_{s+1} (an inverse-limit
// table lookup). Rows outside the window
// W_s = [Bk_s, min(R_s, L - (S - s))] are unreachable or have G = inf, so the
// DP relaxes only rows of W_s and ends in W_{s+1}, which gives the same G on
// every row of every complete split, hence the same B*. An empty window means
// no split fits memory.
//
// Canonical split without stored DP rows. Given B*, let F_s[i] be true when
// stages s..S-1 can cover [i, L) with bottleneck <= B*, i.e. G_s[i] <= B*.
// Because T(s, i, j) grows with j, F_s[i] holds exactly when the smallest j
// >= max(i + 1, Bk_{s+1}) with F_{s+1}[j] (call it nx(i)) is admissible and
// T(s, i, nx(i)) <= B*. A second backward pass evaluates F_s this way for the
// window rows and stores, per row, the next row at or after it with F true;
// the forward reconstruction then takes c_{s+1} = nx(c_s), which is the
// smallest admissible end keeping an optimal completion at every stage, i.e.
// the lexicographically smallest optimal split.

// MA: memory-aware (the flags do not ask to ignore memory); M1: one
// micro-batch count per template. Compile-time choices, so that the hot
// loops carry no test of them.
// COUNT: 0 prices; 1 counts the relaxations over the windows (no DP); 2 runs the DP
// and counts the (row, end) pairs it relaxes under the row loop's exit rule
template <class V, bool F32, int COUNT, int NS, bool MA, bool M1>
__global__ void __launch_bounds__(64, sizeof(V) == 4 ? 8 : 4) split_kernel(DevProfile P, PriceArgs A)
{
    typedef typename Vec2<V>::type V2;
    constexpr int kNone = 255;                                 // no row with F true at or after this one
    extern __shared__ __align__(16) unsigned char smem[];      // one wavefront per workgroup
    const int lane = threadIdx.x;
    const int L = P.L, ls = P.lim_stride;
    constexpr bool mem_aware = MA;
    const int n_m = M1 ? 1 : A.n_m;                            // plans per template
    const V INF = DPInf<V>::value;
    V2 *X = (V2 *)smem;                                        // [gs] pair row {P_s[j], G_{s+1}[j]}
    // [ls] a limit row of 255s (no memory limit); [s_cap][ls] next-row tables
    // of the second backward pass, a region that, with what follows it up to
    // the end of the wavefront's LDS, holds the G arena instead when the
    // template's windows fit it
    uint8_t *JX = smem + A.off_j;
    uint8_t *IX = smem + A.off_x;
    const V *rows = stage_rows<V>(P, F32);
    auto xrow = [&](int s) -> uint8_t * { return IX + s * ls; };

    unsigned long long work = 0;
    // without memory limits every stage reads the limit row of 255s (no limit
    // below the last end of a row), so that a row's last end is always a read
    // of a limit row, capped
    if (!mem_aware) {
        for (int q = lane; 4 * q < ls; q += 64) ((uint32_t *)JX)[q] = ~0u;
        wave_sync();
    }

    // the template records of the next iteration are loaded one iteration ahead
    // Workgroups are handed to the 8 XCDs round robin (workgroup b to XCD
    // x = b mod 8). With a grid that is a multiple of 512, each round of the
    // grid-stride loop gives XCD x the runs of 64 consecutive templates whose
    // run index is x mod 8 (workgroup b, j = b / 8, takes position j mod 64 of
    // run 8 (j / 64) + x), so a run's records, status words and outputs share
    // one XCD's L2 lines while a partial last round still spreads over all XCDs.
    const int64_t stride = gridDim.x;
    int64_t t = blockIdx.x;
    if ((gridDim.x & 511) == 0) {
        const uint32_t x = blockIdx.x & 7, j = blockIdx.x >> 3;
        t = (int64_t)((((j >> 6) << 3) + x) << 6) + (j & 63);
    }
    int S_next = 0;
    uint32_t rec_next = 0;
    if (t < A.n) {
        S_next = A.n_stages[t];
        rec_next = lane < A.s_max ? A.stages[t * A.s_max + lane] : 0u;
    }
    for (; t < A.n; t += stride) {
        const int S_in = S_next;
        const uint32_t rec_in = rec_next;
        if (t + stride < A.n) {
            S_next = A.n_stages[t + stride];
            rec_next = lane < A.s_max ? A.stages[(t + stride) * A.s_max + lane] : 0u;
        }
        const size_t obase = (size_t)t * n_m;
        // lane k: status of plan k after validation and windows (0: windows found),
        // its in-flight class min(M_p, S) (0 when memory is ignored), which fixes
        // the split (M_p = ceil(m / D) micro-batches per replica), and the rows of
        // its windows W_1 .. W_{S-1}
        const uint32_t wv = lane < n_m ? A.wst[obase + lane] : (uint32_t)HEDDLE_S_OOM;
        const int pst = (int)(wv & 255), key_k = (int)((wv >> 8) & 255);
        uint64_t todo = ballot(lane < n_m && pst == HEDDLE_S_OK);
        if (!todo) continue;                                   // the window pass wrote this template's outputs
        bool r_split = false;                                  // lane k: a split was found for m index k
        V r_b = INF;

        if (todo) {
            const int S_t = uni(S_in);
            const StageInfo<V> x = stage_info<V, F32>(P, A, S_t, rec_in, lane);

            // Classes are taken from the largest key down: a larger key holds more
            // micro-batches in flight at every stage, so fewer splits fit memory and
            // its B* bounds those of the classes after it. A row's running minimum
            // starts at U = that bound + 1 instead of INF: every row whose G is at
            // most the bound keeps its exact value, the others end at U or above
            // (above every B* to come), and the row loop's exit rule stops lanes once
            // a stage time exceeds the bound. (Not under fp32 pricing, whose tests of the
            // reconstruction round: a row held at U could round level with B*.)
            V U = INF;
            while (todo) {
                // an opaque copy of the stage count per class: tests on it are formed
                // where they are used, not hoisted out of this loop and kept in scalar
                // registers across the DP
                int S = S_t;
                asm volatile("" : "+s"(S));
                const int key = n_m == 1 ? uni(key_k)
                                           : 255 - uni((int)group_min<uint32_t>(((todo >> lane) & 1) ? 255u - (uint32_t)key_k : 255u, 64));
                const uint64_t cls = M1 ? todo : ballot(lane < n_m && key_k == key) & todo;
                todo &= ~cls;
                auto jhi_of = [&](int s) { return L - (S - 1 - s); };   // last end leaving a layer per later stage

                // lane s: offset of stage s's memory-limit row for this class (in-flight
                // count min(S - s, class key), at least one)
                int f_row = min(S - lane, key);
                f_row = f_row < 1 ? 1 : f_row;
                const int my_row = x.lrow + (f_row - 1) * 2 * ls;

                // ---------------- row windows (from the window pass): lane s holds [a_s, b_s]
                int Al, Bl, g_total;
                {
                    const int k0 = __ffsll((unsigned long long)cls) - 1;   // a plan of this class
                    const uint32_t w = lane < S ? A.wwin[(obase + k0) * win_stride(A.s_max) + lane] : 0u;
                    Al = (int)(w & 255);
                    Bl = (int)(w >> 8);
                    g_total = uni(rl32((int)(wv >> 16), k0));
                }
                // G arena: G_s over the rows of W_s for s = S-1 .. 1, stored in that order,
                // when all of them fit; else the second backward pass rebuilds F
                const bool arena = COUNT == 0 && g_total <= A.arena_cap;

                // ---------------- PartitionLayers: suffix min-max DP over the windows, stages S-1 .. 0
                // Per-stage constants packed into lanes, one readlane per stage each:
                // lane s: a_s | b_s << 8 | e_s << 16 | a_{s+1} << 24, with e_s the last end
                // of a row of stage s (L for the last stage, else b_{s+1}) and a_S = L;
                // lane s: offset of the time row of stage s-1 | a_{s-1} << 24.
                const int An = __builtin_amdgcn_update_dpp(L, Al, kDppWaveShl1, 0xF, 0xF, false);
                const int Bn = __builtin_amdgcn_update_dpp(L, Bl, kDppWaveShl1, 0xF, 0xF, false);
                const bool last = lane >= S - 1;
                const uint32_t pk = (uint32_t)Al | ((uint32_t)Bl << 8) | ((uint32_t)(last ? L : Bn) << 16) |
                                    ((uint32_t)(last ? L : An) << 24);
                const uint32_t prv = (uint32_t)__builtin_amdgcn_update_dpp(
                    0, (int)((uint32_t)x.prow | ((uint32_t)Al << 24)), kDppWaveShr1, 0xF, 0xF, false);
                // lane s: lk_s | jhi_s << 8, with 2^lk_s the lanes per row at stage s
                // (64 >> ceil(log2 r) for r window rows, one when r >= 64) and jhi_s the
                // last end leaving a layer to every later stage
                // and (bits 16..31) the LDS byte address at which G_s[i] would sit for
                // i = 0 (G_s[i] at that address + i * sizeof(V)): the arena holds the
                // windows of stages S-1 .. 1 in that order, so stage s's starts after
                // those of stages s+1 .. S-1. The address is positive (the pair row
                // before the arena is longer than L entries of V) and, while the arena
                // is used, within the wavefront's LDS, which the host keeps under 64 KB
                uint32_t aux;
                {
                    const int r = Bl - Al + 1;
                    const int lk = r >= 64 ? 0 : 6 - (r > 1 ? 32 - __clz(r - 1) : 0);
                    const int before = wave_inclusive_sum(lane >= 1 && lane < S ? r : 0);   // windows of stages 1..s
                    aux = (uint32_t)lk | (uint32_t)(L - (S - 1 - lane)) << 8 |
                          (uint32_t)(A.off_x + (int)sizeof(V) * (g_total - before - Al)) << 16;
                }
                RowRegs<V, NS> rr;
                fetch_rows<V, NS>(rr, rows, (uint32_t)uni(rl32(x.prow, S - 1)), uni(rl32(Al, S - 1)), L, lane);
                V Bv = INF;
                for (int s = S - 1; s >= 0; s--) {
                    const uint32_t ks = uni64(pk, s);
                    const int a = ks & 255, b = (ks >> 8) & 255, e = (ks >> 16) & 255, a_next = ks >> 24;
                    const uint32_t ax = uni64(aux, s);
                    V *Gs = (V *)(smem + (ax >> 16));                   // G_s[i] in the arena at Gs[i]
                    // P_s into the pair row over [a, e]; G_{s+1} stays in place
#pragma unroll
                    for (int q = 0; q < NS; q++)
                        if (q == 0 || 64 * q <= e - a) ((V *)&X[min(a + lane + 64 * q, e)])[0] = rr.p[q];
                    if (s > 0) {
                        const uint32_t kp = uni64(prv, s);
                        fetch_rows<V, NS>(rr, rows, kp & 0xFFFFFFu, (int)(kp >> 24), b, lane);
                    }
                    wave_sync();
                    if (s == S - 1) {
                        // last stage: every window row ends at L
                        if (COUNT != 0 && lane == 0) work += (unsigned long long)(b - a + 1);
                        if (COUNT != 1) {
                            const V pL = X[L].x;
                            for (int i = a + lane; i <= b; i += 64) {
                                const V gv = (V)(pL - X[i].x);
                                if (S > 1) {                           // s = S - 1 > 0
                                    ((V *)&X[i])[1] = gv;
                                    if (arena) Gs[i] = gv;
                                } else {
                                    Bv = gv;                           // S = 1: row 0, lane 0
                                }
                            }
                            if (S == 1) Bv = (V)rl64((int64_t)Bv, 0);
                        }
                    } else {
                        // r rows, k = 64 >> ceil(log2 r) lanes per row (one when r >= 64). The
                        // ends of a row are relaxed four at a time, chunk c of the row by lane
                        // c mod k; a chunk reaching past the row's last end is moved back to end
                        // there (rows of four or more ends), and the ends past the last one of a
                        // shorter row are masked. G_s[i] replaces G_{s+1}[i] in place: rows are
                        // taken in increasing order and every end read lies above its row.
                        const V p2p = (V)uni64(x.p2p, s);
                        const int jhi = (int)((ax >> 8) & 255), lk = (int)(ax & 7);
                        // a row's last admissible end: byte jrow + ic of the limit table (the
                        // row's offset joins the lanes' index, the table's base stays fixed)
                        const uint8_t *Jb = mem_aware ? P.mem_lim : JX;
                        const uint32_t jrow = mem_aware ? (uint32_t)uni(rl32(my_row, s)) : 0u;
                        const int k = 1 << lk;
                        const int part = lane & (k - 1);
                        int base = a;                                      // windows are not empty
                        do {
                            const int i = base + (lane >> lk);
                            const int ic = min(i, b);
                            int lo = max(ic + 1, a_next);
                            // one copy of the row's first end: the compiler otherwise keeps a
                            // second induction variable for the chunk addresses and derives
                            // the first end again from it
                            asm volatile("" : "+v"(lo));
                            const int hi = min((int)Jb[jrow + (uint32_t)ic], jhi);
                            if (COUNT == 1) {
                                if (part == 0 && i <= b && hi >= lo) work += (unsigned long long)(hi - lo + 1);
                                continue;
                            }
                            // lanes past b repeat row b (the same ends, so no longer loop);
                            // only the lanes of rows up to b store
                            // a relaxation past the row's last end is forced to INF by a mask
                            // taken into its max (ends 1..3 of a row with fewer than four ends):
                            // end e of the chunk is missing when hi - lo < e, and bit t of
                            // 0b1, 0b11, 0b111 at t = min(hi - lo, 3), spread over the word,
                            // is all ones (INF) exactly then. A lane with hi < lo has no chunk.
                            // (the builtin's result type is unsigned: taken as int before it is
                            // widened, so that the 64-bit DP gets all ones too)
                            const int t3 = min(hi - lo, 3);
                            const V m1 = (V)(int64_t)(int)__builtin_amdgcn_sbfe(1, t3, 1);
                            const V m2 = (V)(int64_t)(int)__builtin_amdgcn_sbfe(3, t3, 1);
                            const V m3 = (V)(int64_t)(int)__builtin_amdgcn_sbfe(7, t3, 1);
                            const V pi = X[ic].x - p2p;                      // T(s,i,j) = P_s[j] - pi
                            // chunk starts walk by 4k ends and stop at the row's last chunk start
                            const V2 *cm = X + max(hi - 3, lo);
                            const V2 *ce = X + hi;
                            const V2 *cx = X + lo + 4 * part;
                            V acc = M1 || F32 ? INF : U;
                            asm volatile("" : "+v"(acc));                    // one definition, not one per path
                            if (lo <= hi) {
                                // the chunk loop runs while any lane of the group has a chunk
                                // left; a lane past its own chunks relaxes the row's last chunk
                                // again, which leaves its minimum as it is
                                bool more, own = cx <= ce;         // own: the lane's chunk is its own
                                do {
                                    // the ends the chunk adds: four, or those from its start to the
                                    // row's last end when it was moved back (rows past b repeat b)
                                    if (COUNT == 2 && own && i <= b) work += (unsigned long long)min(4, (int)(ce - cx) + 1);
                                    const V2 *c = cx < cm ? cx : cm;
                                    const V2 c0 = c[0], c1 = c[1], c2 = c[2], c3 = c[3];
                                    acc = vmin(vmin(acc, relax<V>(c0, pi)), vmax(relax<V>(c1, pi), m1));
                                    acc = vmin(vmin(acc, vmax(relax<V>(c2, pi), m2)), vmax(relax<V>(c3, pi), m3));
                                    cx += 4 * k;
                                    // the stage time grows with the end: once the chunk's last end
                                    // alone reaches the lane's minimum, no later end can lower it
                                    more = cx <= ce && (V)(c3.x - pi) < acc;
                                    own = more;
                                } while (ballot(more));
                            }
                            // the stage index re-read opaquely: the test is made here, not held
                            // as a lane mask built once per stage
                            int s_here = s;
                            asm volatile("" : "+s"(s_here));
                            if (s_here == 0) {
                                Bv = (V)rl64((int64_t)group_min<V>(acc, 64), 0);   // row 0 only
                            } else {
                                // an opaque copy of k keeps the level tests of the minimum at
                                // their use (one compare and branch each) instead of masks
                                // hoisted out of the row loop for every level
                                int kr = k;
                                asm volatile("" : "+s"(kr));
                                acc = group_min<V>(acc, kr);
                                if (i <= b && part == 0) {             // then ic = i
                                    ((V *)&X[ic])[1] = acc;
                                    if (arena) Gs[ic] = acc;
                                }
                            }
                        } while ((base += 64 >> lk) <= b);
                    }
                    wave_sync();
                }
                if (!M1 && !F32 && Bv != INF) U = Bv + 1;
                if (COUNT) continue;
                if (Bv == INF) continue;                       // no split fits memory
                const uint64_t B = (uint64_t)Bv;
                const uint64_t B24 = F32 ? rne24(B) : B;       // fp32 bottleneck, as an exact integer
                auto within = [&](uint64_t T) { return F32 ? rne24(T) <= B24 : T <= B; };

                int cs = 0, my_end = L;                                // lane s < S-1: c_{s+1}
                if (arena) {
                    // ---------------- canonical reconstruction from the arena: c_{s+1} = the
                    // smallest row j >= max(c_s + 1, a_{s+1}) of W_{s+1} with G_{s+1}[j] within
                    // B*. Such a j is admissible from c_s and T(s, c_s, j) is within B*: some
                    // row with both properties exists (F_s[c_s] holds on the path) and T grows
                    // with j.
                    for (int s = 0; s < S - 1; s++) {
                        const uint32_t k1 = uni64(pk, s + 1);
                        const int a1 = k1 & 255, b1 = (k1 >> 8) & 255;  // W_{s+1}: rows a1 .. b1
                        const V *G1 = (const V *)(smem + (uni64(aux, s + 1) >> 16));   // G_{s+1}[j] at G1[j]
                        const int lo = max(cs + 1, a1);                // lowest admissible row
                        // 64 rows at a time from lo (a later word only when the window runs
                        // more than 64 rows past lo). Bits past the window's last row repeat
                        // that row's bit (the read is clamped to it), and a set bit at or
                        // after lo and at or before the last row always exists: G_s[c_s] is
                        // within B*, so is G_{s+1} at the end minimising it, an admissible row
                        // of W_{s+1} at or after lo (rounding to fp32 is monotone, so this
                        // holds for the fp32 test too). The first set bit is therefore the
                        // row sought, with no test of the window's end.
                        auto word = [&](int r0) -> uint64_t {
                            const V g = G1[min(r0 + lane, b1)];
                            return ballot(F32 ? g != INF && within((uint64_t)g) : (uint64_t)g <= B);
                        };
                        int r0 = lo;
                        uint64_t mk = word(r0);
                        if (!mk) {                                     // more than 64 rows from lo
                            while (r0 + 64 <= b1) {
                                r0 += 64;
                                mk = word(r0);
                                if (mk) break;
                            }
                        }
                        cs = r0 + __builtin_ctzll(mk);                 // mk is not zero (see above)
                        asm volatile("v_writelane_b32 %0, %1, m0" : "+v"(my_end) : "s"(cs), "{m0}"(s));   // lane s := c_{s+1}
                    }
                } else {
                    // ---------------- F_s for stages S-1 .. 1; xrow(s)[i] := the smallest row >= i
                    // of W_s with F_s true (kNone if there is none)
                    for (int s = S - 1; s >= 1; s--) {
                        const int a = uni(rl32(Al, s)), b = uni(rl32(Bl, s));
                        const V *prow = rows + uni(rl32(x.prow, s));
                        const V p2p = (V)uni64(x.p2p, s);
                        const int a_next = s < S - 1 ? uni(rl32(Al, s + 1)) : L;
                        const int jhi = jhi_of(s);
                        const uint8_t *Js = mem_aware ? P.mem_lim + uni(rl32(my_row, s)) : JX;
                        const uint8_t *NXn = xrow(s + 1);
                        uint8_t *NXs = xrow(s);
                        int first_above = kNone;                           // smallest row with F true in higher slots
                        for (int q = (b - a) >> 6; q >= 0; q--) {
                            const int i = a + 64 * q + lane;
                            const int ic = min(i, b);
                            int nx = L;                                    // last stage: the end is L
                            bool ok = i <= b;
                            if (s < S - 1) {
                                // read unconditionally (lo <= L lies inside the row); an entry past
                                // hi, or a stale one when lo > hi, is rejected by the tests below
                                const int lo = max(ic + 1, a_next);
                                const int hi = mem_aware ? min((int)Js[ic], jhi) : jhi;
                                nx = NXn[lo];
                                ok = ok & (lo <= hi) & (nx <= hi);
                            }
                            const uint32_t nxc = min(nx, L);
                            ok = ok & within((uint64_t)(V)(prow[nxc] - prow[(uint32_t)ic] + p2p));
                            const uint64_t mask = ballot(ok);
                            const uint64_t rest = mask >> lane;            // rows >= i of this slot with F true
                            const int nxi = rest ? i + __ffsll((unsigned long long)rest) - 1 : first_above;
                            if (i <= b) NXs[i] = (uint8_t)nxi;
                            if (mask) first_above = a + 64 * q + __ffsll((unsigned long long)mask) - 1;
                        }
                        wave_sync();
                    }

                    // ---------------- canonical reconstruction: c_{s+1} = nx(c_s)
                    for (int s = 0; s < S - 1; s++) {
                        const int a_next = uni(rl32(Al, s + 1));
                        const int lo = cs + 1 > a_next ? cs + 1 : a_next;
                        int nx = uni((int)xrow(s + 1)[lo <= L ? lo : L]);
                        nx = nx <= L ? nx : L;                             // unreachable: F_s[c_s] holds on the path
                        my_end = put_lane(my_end, nx, s);
                        cs = nx;
                    }
                }
                // lane s: c_s (c_0 = 0)
                int my_start = __builtin_amdgcn_update_dpp(0, my_end, kDppWaveShr1, 0xF, 0xF, false);
                // kept a value of its own: folded into the subtraction below as one
                // DPP subtract-reverse, the shift gave negated layer counts on gfx950
                asm volatile("" : "+v"(my_start));
                const uint8_t my_layers = lane < S ? (uint8_t)(my_end - my_start) : 0;
                for (uint64_t c = cls; c; c &= c - 1) {            // s_max <= 64: a lane per stage
                    const int k = __ffsll((unsigned long long)c) - 1;
                    if (lane < A.s_max) A.layers[(obase + k) * A.s_max + lane] = my_layers;
                }
                if ((cls >> lane) & 1) {
                    r_split = true;
                    r_b = Bv;
                }
            }
        }
        if (COUNT) continue;
        if (lane < n_m) {
            const size_t o = obase + lane;
            A.status[o] = (uint8_t)(pst != HEDDLE_S_OK ? pst : (r_split ? HEDDLE_S_OK : HEDDLE_S_OOM));
            if (F32) ((float *)A.bottleneck)[o] = r_split ? exact_float(rne24((uint64_t)r_b), P.fx_exp) : __builtin_inff();
            else ((int64_t *)A.bottleneck)[o] = r_split ? (int64_t)r_b : INT64_MAX;
        }
        // zero layer counts of the plans without a split (invalid template, or no split fits)
        const uint64_t without = ballot(lane < n_m && !r_split);
        for (uint64_t c = without; c; c &= c - 1) {
            const int k = __ffsll((unsigned long long)c) - 1;
            if (lane < A.s_max) A.layers[(obase + k) * A.s_max + lane] = 0;
        }
    }
    if (COUNT) {
        work += __shfl_xor(work, 32);
        work += __shfl_xor(work, 16);
        work += __shfl_xor(work, 8);
        work += __shfl_xor(work, 4);
        work += __shfl_xor(work, 2);
        work += __shfl_xor(work, 1);
        if (lane == 0 && work) atomicAdd(A.work, work);
    }
}

// ------------------------------------------------------------------- host

int validate_price_args(const heddle_profile *p, int64_t n, int32_t s_max, const uint8_t *d_n_stages,
                        const uint32_t *d_stages, const int32_t *h_m, int32_t n_m, uint32_t flags)
{
    if (!p) return fail(HEDDLE_E_INVAL, "profile is NULL");
    if (n < 0) return fail(HEDDLE_E_INVAL, "n < 0");
    if (s_max < 1 || s_max > HEDDLE_MAX_STAGES) return fail(HEDDLE_E_INVAL, "s_max out of range 1..64");
    if (n_m < 1 || n_m > HEDDLE_MAX_MLIST) return fail(HEDDLE_E_INVAL, "n_m out of range 1..64");
    if (!h_m) return fail(HEDDLE_E_INVAL, "h_m is NULL");
    if (flags & ~(HEDDLE_F_FP32 | HEDDLE_F_COMPUTE_ONLY | HEDDLE_F_DISTRIBUTE)) return fail(HEDDLE_E_INVAL, "unknown flag bits");
    int64_t m_max = 0;
    for (int k = 0; k < n_m; k++) {
        if (h_m[k] < 1 || h_m[k] > HEDDLE_MAX_M) return fail(HEDDLE_E_INVAL, "m out of range 1..2^24");
        m_max = h_m[k] > m_max ? h_m[k] : m_max;
    }
    if (n > 0 && (!d_n_stages || !d_stages)) return fail(HEDDLE_E_INVAL, "template pointer is NULL");
    int dev = -1;
    HEDDLE_HIP(hipGetDevice(&dev));
    if (dev != p->device) return fail(HEDDLE_E_INVAL, "profile was loaded on another device");
    const bool f32 = flags & HEDDLE_F_FP32;
    const int64_t max_stage = f32 ? p->max_stage_fx : p->max_stage_ns;
    const int64_t max_ar = f32 ? p->max_ar_fx : p->max_ar_ns;
    if (max_stage < 0) return fail(HEDDLE_E_RANGE, "fp32 costs span too wide a range to be summed exactly");
    const int64_t s_cap = s_max < p->dev.L ? s_max : p->dev.L;
    const __int128 bound = (__int128)(m_max - 1 + s_cap) * max_stage + max_ar;
    if (bound >= kLimit62) return fail(HEDDLE_E_RANGE, "iteration time could exceed 2^62 for these m");
    return HEDDLE_OK;
}

// bytes of the window pass's outputs: the status word of every plan (256-byte
// aligned) and then the row windows of every plan
static size_t window_scratch_bytes(int64_t n, int32_t n_m, int32_t s_max)
{
    const size_t plans = (size_t)n * n_m;
    return ((plans * sizeof(uint32_t) + 255) & ~size_t(255)) + plans * win_stride(s_max) * sizeof(uint16_t);
}

template <class V, bool F32, int COUNT>
static int launch_split(const heddle_profile *p, PriceArgs &a, hipStream_t stream)
{
    const int L = p->dev.L, ls = p->dev.lim_stride;
    a.s_cap = a.s_max < L ? a.s_max : L;
    a.g_stride = L + 5;                                       // L + 1 ends and 4 of padding
    // per wavefront: one pair row {P_s, G_{s+1}}; one limit row of 255s (read
    // in place of the stages' limit rows when memory is ignored; with memory
    // limits a row's last end is read from the profile's limit rows through
    // the caches); per stage its next-row table (second backward pass), a
    // region that the G arena shares and extends up to the wavefront's share
    // of the CU's LDS at the occupancy the registers allow
    const size_t j_off = ((size_t)a.g_stride * 2 * sizeof(V) + 15) & ~size_t(15);
    const size_t rows_lds = (size_t)a.s_cap * ls;            // the next-row tables of every stage
    int max_lds = 0, lds_cu = 0;
    HEDDLE_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, p->device));
    HEDDLE_HIP(hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, p->device));
    const size_t waves_regs = sizeof(V) == 4 ? 32 : 20;       // wavefronts per CU the registers allow
    const size_t x_off = j_off + (size_t)ls;
    size_t x_bytes = rows_lds;
    if (!COUNT && lds_cu > 0) {
        const size_t need = x_off + x_bytes;
        size_t waves = (size_t)lds_cu / need;
        waves = waves < waves_regs ? waves : waves_regs;
        if (waves > 0) {
            size_t share = ((size_t)lds_cu / waves) & ~size_t(511);   // LDS is allocated in 512-byte blocks
            share = share < (size_t)max_lds ? share : ((size_t)max_lds & ~size_t(15));
            if (share > need) x_bytes += (share - need) & ~size_t(15);
        }
    }
    a.off_j = (int32_t)j_off;
    a.off_x = (int32_t)x_off;
    // the split kernel addresses the arena with 16-bit LDS byte offsets
    const size_t x_max = x_off < 65535 ? 65535 - x_off : 0;
    a.arena_cap = (int32_t)((x_bytes < x_max ? x_bytes : x_max) / sizeof(V));
    a.lds_per_wave = (int32_t)(x_off + x_bytes);
    // one wavefront per workgroup: a wavefront's LDS is released as soon as it
    // is done, whatever the other wavefronts on the CU are doing
    const int wpb = 1;
    const size_t lds = (size_t)wpb * a.lds_per_wave;
    if (lds > (size_t)max_lds) return fail(HEDDLE_E_RANGE, "DP table of this (L, s_max) does not fit in LDS");
    // time-prefix slots of 64 entries held in registers: 2 cover L + 1 <= 128
    const bool ma = (a.flags & HEDDLE_F_COMPUTE_ONLY) == 0;
    const void *kern;
    if (a.n_m == 1)
        kern = L + 1 <= 128 ? (ma ? (const void *)split_kernel<V, F32, COUNT, 2, true, true>
                                  : (const void *)split_kernel<V, F32, COUNT, 2, false, true>)
                            : (ma ? (const void *)split_kernel<V, F32, COUNT, 4, true, true>
                                  : (const void *)split_kernel<V, F32, COUNT, 4, false, true>);
    else
        kern = L + 1 <= 128 ? (ma ? (const void *)split_kernel<V, F32, COUNT, 2, true, false>
                                  : (const void *)split_kernel<V, F32, COUNT, 2, false, false>)
                            : (ma ? (const void *)split_kernel<V, F32, COUNT, 4, true, false>
                                  : (const void *)split_kernel<V, F32, COUNT, 4, false, false>);
    if (lds > 65536) HEDDLE_HIP(hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
    size_t w_lds = 0;
    const int rc = prepare_windows(p, a, max_lds, &w_lds);
    if (rc != HEDDLE_OK) return rc;
    // validation and windows of every plan into the profile's scratch of this
    // stream (the caller holds its lock and marks the end of its use)
    const size_t plans = (size_t)a.n * a.n_m;
    const size_t st_bytes = (plans * sizeof(uint32_t) + 255) & ~size_t(255);
    const size_t bytes = window_scratch_bytes(a.n, a.n_m, a.s_max);
    unsigned char *buf = nullptr;
    if (a.ext_scratch) {
        if (bytes > a.ext_bytes) return fail(HEDDLE_E_RANGE, "window scratch exceeds the fixed buffer");
        buf = a.ext_scratch;
    } else {
        const int rs = profile_scratch(p, stream, bytes, (void **)&buf, &a.scratch_owned);
        if (rs != HEDDLE_OK) return rs;
    }
    a.wst = (uint32_t *)buf;
    a.wwin = (uint16_t *)(buf + st_bytes);
    const int rw = launch_windows(p, a, w_lds, stream);
    if (rw != HEDDLE_OK) return rw;
    // at least 65,536 workgroups (one per template for a smaller batch) and at
    // least one per four templates, as a power of two: the hardware hands a
    // finished workgroup's slot to the next one, which evens out the
    // templates' uneven costs better than long grid-stride runs, while a few
    // templates per workgroup keep the next one's records loaded ahead and the
    // set-up shared (c3, 1,000,000 templates: 1.29 ms at 65,536 workgroups,
    // 1.22 ms at 262,144, 1.26 ms at one per template)
    const int64_t per_wg = (a.n + 4 * wpb - 1) / (4 * wpb);
    const int64_t floor_wg = a.n < 65536 ? a.n : 65536;
    const int64_t want = per_wg > floor_wg ? per_wg : floor_wg;
    int blocks = 1;
    while (blocks < want && blocks < (1 << 30)) blocks <<= 1;  // from 512 on, a multiple of 512: XCD-aware runs
    const DevProfile dev = p->dev;
    void *args[] = {(void *)&dev, (void *)&a};
    HEDDLE_HIP(hipLaunchKernel(kern, dim3(blocks), dim3(64 * wpb), args, lds, stream));
    return HEDDLE_OK;
}

int launch_price(const heddle_profile *p, PriceArgs &a, hipStream_t stream, int count)
{
    if (a.n == 0) return HEDDLE_OK;
    const bool f32 = a.flags & HEDDLE_F_FP32;
    const bool narrow = f32 ? p->narrow_f32 : p->narrow_i64;
    if (a.flags & HEDDLE_F_DISTRIBUTE) return launch_distribute(p, a, stream, count != 0);
    // validation and windows of every plan (window_kernel), then the split
    // kernel over the plans with windows, then Evaluate
    // the profile's buffer of the stream is taken under its lock; a fixed
    // buffer of the caller's needs no lock
    std::unique_lock<std::mutex> lock(p->scratch_mu, std::defer_lock);
    if (!a.ext_scratch) lock.lock();
    a.wst = nullptr;
    a.wwin = nullptr;
    a.scratch_owned = false;
    int rc;
    if (count == 1) rc = launch_split<uint64_t, false, 1>(p, a, stream);
    else if (count == 2) rc = f32 ? launch_split<uint64_t, true, 2>(p, a, stream) : launch_split<uint64_t, false, 2>(p, a, stream);
    else if (f32) rc = narrow ? launch_split<uint32_t, true, 0>(p, a, stream) : launch_split<uint64_t, true, 0>(p, a, stream);
    else rc = narrow ? launch_split<uint32_t, false, 0>(p, a, stream) : launch_split<uint64_t, false, 0>(p, a, stream);
    if (rc == HEDDLE_OK && count == 0) rc = launch_evaluate(p, a, stream);
    if (a.wst && !a.ext_scratch) {
        const int rd = profile_scratch_done(p, stream, a.wst, a.scratch_owned);
        if (rc == HEDDLE_OK) rc = rd;
    }
    a.wst = nullptr;
    a.wwin = nullptr;
    return rc;
}

static PriceArgs make_args(int64_t n, int32_t s_max, const uint8_t *d_n_stages, const uint32_t *d_stages,
                           const int32_t *h_m, int32_t n_m, uint32_t flags)
{
    PriceArgs a;
    std::memset(&a, 0, sizeof(a));
    a.n = n;
    a.s_max = s_max;
    a.n_m = n_m;
    a.flags = (int32_t)flags;
    for (int k = 0; k < n_m; k++) a.m[k] = h_m[k];
    a.n_stages = d_n_stages;
    a.stages = d_stages;
    return a;
}

}  // namespace heddle

using namespace heddle;

extern "C" int heddle_price_plans(const heddle_profile *p, int64_t n, int32_t s_max,
                                  const uint8_t *d_n_stages, const uint32_t *d_stages,
                                  const int32_t *h_m, int32_t n_m, uint32_t flags,
                                  void *d_iter, void *d_bottleneck, int64_t *d_peak_mem,
                                  uint8_t *d_layers, uint8_t *d_status, hipStream_t stream)
{
    int rc = validate_price_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    if (rc) return rc;
    if (n > 0 && (!d_iter || !d_bottleneck || !d_peak_mem || !d_layers || !d_status))
        return fail(HEDDLE_E_INVAL, "output pointer is NULL");
    PriceArgs a = make_args(n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    a.iter = d_iter;
    a.bottleneck = d_bottleneck;
    a.peak_mem = d_peak_mem;
    a.layers = d_layers;
    a.status = d_status;
    return launch_price(p, a, stream, 0);
}

extern "C" int heddle_count_work(const heddle_profile *p, int64_t n, int32_t s_max,
                                 const uint8_t *d_n_stages, const uint32_t *d_stages,
                                 const int32_t *h_m, int32_t n_m, uint32_t flags,
                                 int64_t *h_relaxations, hipStream_t stream)
{
    const int mode = (flags & HEDDLE_F_COUNT_EVALUATED) ? 2 : 1;
    flags &= ~HEDDLE_F_COUNT_EVALUATED;
    int rc = validate_price_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    if (rc) return rc;
    if (!h_relaxations) return fail(HEDDLE_E_INVAL, "h_relaxations is NULL");
    PriceArgs a = make_args(n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    unsigned long long *d_work = nullptr;
    hipError_t e = scratch_alloc((void **)&d_work, sizeof(unsigned long long), stream);
    if (e != hipSuccess) return fail(HEDDLE_E_NOMEM, "device scratch for the work counter could not be allocated");
    e = hipMemsetAsync(d_work, 0, sizeof(unsigned long long), stream);
    a.work = d_work;
    rc = e == hipSuccess ? launch_price(p, a, stream, mode) : hip_fail(e, "hipMemsetAsync");
    unsigned long long h = 0;
    if (rc == HEDDLE_OK) e = hipMemcpyAsync(&h, d_work, sizeof(h), hipMemcpyDeviceToHost, stream);
    (void)hipFreeAsync(d_work, stream);                        // stream-ordered after the copy
    if (rc == HEDDLE_OK && e == hipSuccess) e = hipStreamSynchronize(stream);
    if (rc == HEDDLE_OK && e != hipSuccess) rc = hip_fail(e, "reading the work counter back");
    if (rc == HEDDLE_OK) *h_relaxations = (int64_t)h;
    return rc;
}

// ---------------------------------------------------------------------------
// Pricing without allocation. The window pass's outputs go to this fixed
// array, one copy per GPU, held until the process ends. Host code never uses
// the array's name as a device address: the address of each GPU's copy is
// taken once per device with hipGetSymbolAddress (with that device current)
// and kept below.
static __device__ __align__(256) unsigned char scratch[HEDDLE_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char *g_scratch_ptr[kMaxDevices];   // device address of `scratch` on each device, or NULL

// the current device's copy of `scratch` (the caller has checked that the
// current device is the profile's)
int noalloc_scratch(int dev, unsigned char **ptr)
{
    if (dev < 0 || dev >= kMaxDevices) return fail(HEDDLE_E_INVAL, "device index beyond the library's device table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *q = nullptr;
        const hipError_t e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress of the fixed pricing scratch");
        if (!q) return fail(HEDDLE_E_DEVICE, "hipGetSymbolAddress gave no address for the fixed pricing scratch");
        g_scratch_ptr[dev] = (unsigned char *)q;
    }
    *ptr = g_scratch_ptr[dev];
    return HEDDLE_OK;
}
}  // namespace

extern "C" int heddle_price_plans_noalloc(const heddle_profile *p, int64_t n, int32_t s_max,
                                          const uint8_t *d_n_stages, const uint32_t *d_stages,
                                          const int32_t *h_m, int32_t n_m, uint32_t flags,
                                          void *d_iter, void *d_bottleneck, int64_t *d_peak_mem,
                                          uint8_t *d_layers, uint8_t *d_status, hipStream_t stream)
{
    int rc = validate_price_args(p, n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    if (rc) return rc;
    if (n > 0 && (!d_iter || !d_bottleneck || !d_peak_mem || !d_layers || !d_status))
        return fail(HEDDLE_E_INVAL, "output pointer is NULL");
    PriceArgs a = make_args(n, s_max, d_n_stages, d_stages, h_m, n_m, flags);
    a.iter = d_iter;
    a.bottleneck = d_bottleneck;
    a.peak_mem = d_peak_mem;
    a.layers = d_layers;
    a.status = d_status;
    if (n > 0 && !(flags & HEDDLE_F_DISTRIBUTE)) {
        const size_t need = window_scratch_bytes(n, n_m, s_max);
        if (need > (size_t)HEDDLE_NOALLOC_SCRATCH_BYTES)
            return fail(HEDDLE_E_RANGE, "this batch needs more window scratch than the fixed buffer of "
                                        "heddle_price_plans_noalloc holds (HEDDLE_NOALLOC_SCRATCH_BYTES)");
        rc = noalloc_scratch(p->device, &a.ext_scratch);
        if (rc) return rc;
        a.ext_bytes = HEDDLE_NOALLOC_SCRATCH_BYTES;
    }
    return launch_price(p, a, stream, 0);
}
