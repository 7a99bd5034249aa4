"""A model of the split kernel's relaxation schedule, for its work counter.

The GPU library can count the (row, end) pairs its split kernel relaxes
(heddle_count_work with HEDDLE_F_COUNT_EVALUATED). That count belongs to the
kernel's schedule, not to the method, so it is checked against this model of
the schedule rather than against the oracle: the windowed min-max recurrence
(section 5.2, the suffix recurrence over layer splits) over the rows that can
lie on a complete split, with each row's ends taken in chunks of four by k
lanes and a lane stopping after a chunk whose last end has a stage time at
or above the lane's running minimum. Stage times and memory come from
brute.Plan (plain sums of the per-layer terms), here as prefix differences.
template_relaxations() takes a template's several micro-batch counts the
way the kernel does: one recurrence per in-flight class (key min(ceil(m/D),
S), or 0 when memory is ignored), from the largest key down, each later
class's rows starting at the previous class's B* + 1 instead of INF.
"""
from __future__ import annotations

import numpy as np

from brute import Plan, ceil_div, status_of

INF = 1 << 63


def _prefix(xs):
    return np.concatenate([[0], np.cumsum(np.asarray(xs, dtype=object))])


def evaluated_relaxations(p, S, s_max, recs, m, compute_only=False, exit_rule=True, bottleneck=False, start=None):
    """pairs relaxed for one plan (one in-flight class), as the kernel counts them;
    without the exit rule every end of every window row is relaxed. With
    bottleneck=True also returns G_0[0] (None when no split fits). start: the
    value a row's running minimum starts from (INF when None)."""
    acc0 = INF if start is None else start
    stt, st = status_of(p, S, s_max, recs)
    if stt != 0:
        return (0, None) if bottleneck else 0
    Plan(p, st)                                   # fills each stage's per-layer terms
    L = p.L
    Mp = ceil_div(int(m), st[0]["dp"])
    C = [_prefix(x["cost"]) for x in st]
    W = [_prefix(x["w"]) for x in st]
    A = [_prefix(x["a"]) for x in st]
    cap = [int(p.mem_cap_bytes[x["g"]]) for x in st]

    def t(s, i, j):
        return int(C[s][j] - C[s][i]) + st[s]["p2p"]

    def fits(s, i, j):
        if compute_only:
            return True
        return int(W[s][j] - W[s][i]) + min(S - s, Mp) * int(A[s][j] - A[s][i]) <= cap[s]

    def lim(s, i):
        best = i
        for j in range(i + 1, L - (S - 1 - s) + 1):
            if fits(s, i, j):
                best = j
        return best

    # windows: R_s the furthest reachable start, Bk_s the smallest start that reaches Bk_{s+1}
    R = [0] * S
    for s in range(S - 1):
        R[s + 1] = lim(s, R[s])
    Bk = [0] * (S + 1)
    Bk[S] = L
    top = [0] * S
    for s in range(S - 1, -1, -1):
        top[s] = min(R[s], 0 if s == 0 else L - (S - s))
        Bk[s] = next((i for i in range(s, top[s] + 1) if lim(s, i) >= Bk[s + 1]), -1)
        if Bk[s] < 0:
            return (0, None) if bottleneck else 0
    count = top[S - 1] - Bk[S - 1] + 1
    G = {i: t(S - 1, i, L) for i in range(Bk[S - 1], top[S - 1] + 1)}
    for s in range(S - 2, -1, -1):
        a, b = Bk[s], top[s]
        r = b - a + 1
        k = 1 if r >= 64 else 64 >> (0 if r == 1 else (r - 1).bit_length())
        Gs = {}
        for i in range(a, b + 1):
            lo, hi = max(i + 1, Bk[s + 1]), lim(s, i)
            best = acc0
            if lo <= hi:
                cm = max(hi - 3, lo)
                for part in range(k):
                    cx, acc = lo + 4 * part, acc0
                    while cx <= hi:
                        count += min(4, hi - cx + 1)
                        c = min(cx, cm)
                        for j in range(c, min(c + 3, hi) + 1):
                            acc = min(acc, max(t(s, i, j), G[j]))
                        cx += 4 * k
                        if cx > hi or (exit_rule and t(s, i, c + 3) >= acc):
                            break
                    best = min(best, acc)
            Gs[i] = best
        G = Gs
    if bottleneck:
        return count, (G[0] if G[0] < acc0 else None)
    return count


def template_relaxations(p, S, s_max, recs, ms, compute_only=False):
    """pairs relaxed for one template priced at every m of ms, as the kernel
    counts them, and B* per m (None when no split fits)"""
    stt, st = status_of(p, S, s_max, recs)
    if stt != 0:
        return 0, [None] * len(ms)
    D = st[0]["dp"]
    key = [0 if compute_only else min(ceil_div(int(m), D), S) for m in ms]
    total, U, best = 0, None, {}
    for k in sorted(set(key), reverse=True):
        m = ms[key.index(k)]
        c, b = evaluated_relaxations(p, S, s_max, recs, m, compute_only, bottleneck=True,
                                     start=None if U is None else U + 1)
        total += c
        best[k] = b
        if b is not None:
            U = b
    return total, [best[k] for k in key]
