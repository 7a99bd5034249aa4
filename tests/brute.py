"""Brute-force pricing of tiny plans, in pure Python.

Enumerates every composition (n_0, ..., n_{S-1}) of L layers into S
non-empty stages in lexicographic order, keeps the memory-feasible ones,
takes the smallest bottleneck (first in lexicographic order among equals),
then evaluates the 1F1B iteration time. It shares nothing with the C oracle
beyond the input arrays and is only usable for L <= ~16.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

INF = (1 << 63) - 1


def compositions(L, S):
    """All (n_0..n_{S-1}), n_s >= 1, sum L, in lexicographic order."""
    if S == 1:
        yield (L,)
        return
    for first in range(1, L - S + 2):
        for rest in compositions(L - first, S - 1):
            yield (first,) + rest


def ceil_div(a, b):
    return -((-a) // b)


def decode(p, rec):
    return dict(g=int(rec & 0xFF), tp=1 << int((rec >> 8) & 0xF), ep=1 << int((rec >> 12) & 0xF),
                dp=int(rec >> 16))


def status_of(p, S, s_max, recs):
    tp_list = [int(x) for x in p.tp_degrees]
    ep_list = [int(x) for x in p.ep_degrees]
    N = p.layer_ns.shape[0]
    if S < 1 or S > s_max or S > p.L:
        return 1, None
    st = [decode(p, int(recs[s])) for s in range(S)]
    if any(x["g"] >= N for x in st):
        return 2, None
    if any(x["tp"] not in tp_list or x["tp"] > int(p.node_size[x["g"]]) for x in st):
        return 3, None
    for x in st:
        x["k"] = tp_list.index(x["tp"])
    if any(not p.profiled[x["g"], x["k"]] for x in st):
        return 4, None
    if any(x["dp"] < 1 or x["dp"] != st[0]["dp"] for x in st):
        return 5, None
    if any(x["ep"] not in ep_list or x["dp"] % x["ep"] for x in st):
        return 6, None
    for g in range(N):
        if sum(x["tp"] * x["dp"] for x in st if x["g"] == g) > int(p.n_gpus[g]):
            return 7, None
    return 0, st


def xfer(b, bw):
    return ceil_div(int(b) * 1000, int(bw))


def allreduce(b, n, bw):
    return 0 if n == 1 else ceil_div(2 * (n - 1) * int(b) * 1000, n * int(bw))


class Plan:
    """Per-stage cost pieces of one valid template."""

    def __init__(self, p, st):
        self.p, self.st, self.S = p, st, len(st)
        N = p.layer_ns.shape[0]
        for s, x in enumerate(st):
            g, k, e = x["g"], x["k"], x["ep"]
            node = int(p.node_size[g])
            same = int(p.link_bw_MBps[g, g])
            x["a2a"] = 0 if e == 1 else xfer(p.a2a_bytes, int(p.intra_bw_MBps[g]) if e * x["tp"] <= node else same)
            x["p2p"] = 0 if s == self.S - 1 else xfer(2 * p.boundary_bytes, int(p.link_bw_MBps[g, st[s + 1]["g"]]))
            x["bw_dp"] = int(p.intra_bw_MBps[g]) if x["tp"] * x["dp"] <= node else same
            x["cost"] = [int(p.layer_ns[g, k, l]) + (x["a2a"] if p.is_moe[l] else 0) for l in range(p.L)]
            x["w"] = [int(p.state_bytes[k, l]) + ceil_div(int(p.xstate_bytes[k, l]), e) for l in range(p.L)]
            x["a"] = [int(p.act_bytes[k, l]) for l in range(p.L)]
            x["gd"] = [int(p.grad_bytes[k, l]) for l in range(p.L)]
            x["gx"] = [ceil_div(int(p.xgrad_bytes[k, l]), e) for l in range(p.L)]
        del N

    def stage(self, s, i, j, Mp):
        x = self.st[s]
        t = sum(x["cost"][i:j]) + x["p2p"]
        mem = sum(x["w"][i:j]) + min(self.S - s, Mp) * sum(x["a"][i:j])
        g = allreduce(sum(x["gd"][i:j]), x["dp"], x["bw_dp"]) + \
            allreduce(sum(x["gx"][i:j]), x["dp"] // x["ep"], x["bw_dp"])
        return t, mem, g

    def stage_f32(self, s, i, j):
        """exact real stage time from fp32 terms, rounded once to fp32"""
        x, p = self.st[s], self.p
        f32 = p.layer_ns_f32 if p.layer_ns_f32 is not None else p.layer_ns.astype(np.float32)
        a2a = Fraction(float(np.float32(x["a2a"])))
        tot = Fraction(float(np.float32(x["p2p"])))
        for l in range(i, j):
            tot += Fraction(float(f32[x["g"], x["k"], l]))
            if p.is_moe[l]:
                tot += a2a
        return round_f32(tot)


def round_f32(fr):
    """nearest float32 of an exact Fraction (ties to even), via an exact float64"""
    d = float(fr)
    assert Fraction(d) == fr, "test range must keep the sum exact in float64"
    return np.float32(d)


def price(p, S, s_max, recs, m, compute_only=False, fp32=False):
    """Returns dict(status, iter, bottleneck, peak_mem, layers) for one plan."""
    stt, st = status_of(p, S, s_max, recs)
    none = dict(status=stt, iter=None, bottleneck=None, peak_mem=None, layers=[0] * s_max)
    if stt != 0:
        return none
    plan = Plan(p, st)
    D = st[0]["dp"]
    Mp = ceil_div(int(m), D)
    best, best_c = None, None
    for comp in compositions(p.L, S):
        cuts = np.concatenate([[0], np.cumsum(comp)]).astype(int)
        stages = [plan.stage(s, cuts[s], cuts[s + 1], Mp) for s in range(S)]
        if not compute_only and any(mem > int(p.mem_cap_bytes[st[s]["g"]]) for s, (_, mem, _) in enumerate(stages)):
            continue
        if fp32:
            b = max(plan.stage_f32(s, cuts[s], cuts[s + 1]) for s in range(S))
        else:
            b = max(t for t, _, _ in stages)
        if best is None or b < best:
            best, best_c = b, (comp, cuts, stages)
    if best is None:
        return dict(none, status=8)
    comp, cuts, stages = best_c
    peak = max(mem for _, mem, _ in stages)
    oom = any(mem > int(p.mem_cap_bytes[st[s]["g"]]) for s, (_, mem, _) in enumerate(stages))
    if fp32:
        tprime = [plan.stage_f32(s, cuts[s], cuts[s + 1]) for s in range(S)]
        maxg = max(np.float32(g) for _, _, g in stages)
        tot = (Mp - 1) * Fraction(float(best)) + sum(Fraction(float(t)) for t in tprime) + Fraction(float(maxg))
        it = round_f32(tot)
    else:
        it = (Mp - 1) * best + sum(t for t, _, _ in stages) + max(g for _, _, g in stages)
    return dict(status=8 if oom else 0, iter=it, bottleneck=best, peak_mem=peak,
                layers=list(comp) + [0] * (s_max - S))


def best_iter(p, S, s_max, recs, m, fp32=False):
    """smallest iteration time over every memory-feasible composition (its
    own bottleneck per composition), or None if none fits."""
    stt, st = status_of(p, S, s_max, recs)
    if stt != 0:
        return None
    plan = Plan(p, st)
    Mp = ceil_div(int(m), st[0]["dp"])
    best = None
    for comp in compositions(p.L, S):
        cuts = np.concatenate([[0], np.cumsum(comp)]).astype(int)
        stages = [plan.stage(s, cuts[s], cuts[s + 1], Mp) for s in range(S)]
        if any(mem > int(p.mem_cap_bytes[st[s]["g"]]) for s, (_, mem, _) in enumerate(stages)):
            continue
        if fp32:
            tprime = [plan.stage_f32(s, cuts[s], cuts[s + 1]) for s in range(S)]
            maxg = max(np.float32(g) for _, _, g in stages)
            tot = (Mp - 1) * Fraction(float(max(tprime))) + sum(Fraction(float(t)) for t in tprime) + \
                Fraction(float(maxg))
            it = round_f32(tot)
        else:
            it = (Mp - 1) * max(t for t, _, _ in stages) + sum(t for t, _, _ in stages) + \
                max(g for _, _, g in stages)
        best = it if best is None or it < best else best
    return best


def best_plan(m, iters, status):
    """argmin over OK plans of iter / m, ties to lowest (template, m index)."""
    best, arg = None, None
    n, n_m = status.shape
    for t in range(n):
        for k in range(n_m):
            if status[t, k] != 0:
                continue
            key = Fraction(Fraction(float(iters[t, k])) if isinstance(iters[t, k], np.floating) else int(iters[t, k]),
                           int(m[k]))
            if best is None or key < best:
                best, arg = key, (t, k)
    return arg


# ------------------------------------------------------------ expert tiling

def stage_layouts(p, x):
    """(EP, ETP, ETP index) factorisations of a stage's TP * D GPUs: EP from
    the EP list, ETP a profiled TP degree within the node, EP * ETP | TP * D"""
    out = []
    for e in p.ep_degrees:
        for ti, t in enumerate(p.tp_degrees):
            e, t = int(e), int(t)
            if p.profiled[x["g"], ti] and t <= int(p.node_size[x["g"]]) and (x["tp"] * x["dp"]) % (e * t) == 0:
                out.append((e, t, ti))
    return out


def tiled_stage(p, st, s, i, j, Mp, e, t, ti):
    """time, memory, synchronisation of stage s on layers [i, j) with experts
    laid out as EP e x ETP t"""
    x, S = st[s], len(st)
    g, k, tp, dp = x["g"], x["k"], x["tp"], x["dp"]
    node, same = int(p.node_size[g]), int(p.link_bw_MBps[g, g])
    xl = p.xlayer_ns if p.xlayer_ns is not None else np.zeros_like(p.layer_ns)
    a2a = 0 if e == 1 else xfer(p.a2a_bytes, int(p.intra_bw_MBps[g]) if e * t <= node else same)
    p2p = 0 if s == S - 1 else xfer(2 * p.boundary_bytes, int(p.link_bw_MBps[g, st[s + 1]["g"]]))
    T = p2p
    for l in range(i, j):
        T += int(p.layer_ns[g, k, l])
        if p.is_moe[l]:
            T += ceil_div(int(xl[g, ti, l]) * t, tp) - int(xl[g, k, l]) + a2a
    w = sum(int(p.state_bytes[k, l]) + ceil_div(int(p.xstate_bytes[ti, l]), e) for l in range(i, j))
    mem = w + min(S - s, Mp) * sum(int(p.act_bytes[k, l]) for l in range(i, j))
    bw = int(p.intra_bw_MBps[g]) if tp * dp <= node else same
    gs = allreduce(sum(int(p.grad_bytes[k, l]) for l in range(i, j)), dp, bw) + \
        allreduce(sum(ceil_div(int(p.xgrad_bytes[ti, l]), e) for l in range(i, j)), tp * dp // (e * t), bw)
    return T, mem, gs


def tile_brute(p, S, s_max, recs, m, layers):
    """Every combination of memory-fitting layouts over the stages of a split:
    (smallest 1F1B iteration time, {combination: (iter, bottleneck, peak)}
    of the minimisers), or None if some stage has no fitting layout."""
    import itertools
    _, st = status_of(p, S, s_max, recs)
    cuts = np.concatenate([[0], np.cumsum(layers[:S])]).astype(int)
    Mp = ceil_div(int(m), st[0]["dp"])
    opts = []
    for s in range(S):
        o = []
        for e, t, ti in stage_layouts(p, st[s]):
            T, mem, gs = tiled_stage(p, st, s, cuts[s], cuts[s + 1], Mp, e, t, ti)
            if mem <= int(p.mem_cap_bytes[st[s]["g"]]):
                o.append(((e, t), T, mem, gs))
        if not o:
            return None
        opts.append(o)
    best, arg = None, {}
    for combo in itertools.product(*opts):
        B = max(c[1] for c in combo)
        it = (Mp - 1) * B + sum(c[1] for c in combo) + max(c[3] for c in combo)
        key = tuple(c[0] for c in combo)
        if best is None or it < best:
            best, arg = it, {key: (it, B, max(c[2] for c in combo))}
        elif it == best:
            arg[key] = (it, B, max(c[2] for c in combo))
    return best, arg
