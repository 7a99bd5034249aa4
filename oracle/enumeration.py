"""Oracle of the exhaustive structural enumeration.

TEST INFRASTRUCTURE ONLY: imported by the test suite and by the CPU-baseline
leg of the benchmark. The GPU library never imports it, and it shares no code
with the library.

What it computes (Heddle, arXiv 2609.34244): the search backbone that the
planners of section 3.1 share -- for each pipeline depth, for each GPU type
of every stage, for each TP degree of every stage, for each DP degree (and,
innermost, each micro-batch choice): split the layers, then Evaluate -- run
over a whole space, and the best plan of that space. Section 2 counts the
structures of this loop nest: (N * K)^D for N GPU types, K TP degrees and D
stages.

The space is written exactly as that loop nest (``all_templates``), with
itertools.product standing for "for g[1..S] in types" (its first position
varies slowest, as the outermost loop). ``template_at`` is a second,
independent formulation (mixed-radix decoding of an index) used to address
large spaces; the tests pin the two against each other on small spaces.
Every stage of a template carries the template's DP degree and the spec's
EP degree.
"""
from __future__ import annotations

import itertools

import numpy as np

from . import oracle as O


def _record(g, log2_tp, log2_ep, dp):
    # the stage record of the library's ABI: type | log2 TP << 8 | log2 EP << 12 | DP << 16
    return int(g) | int(log2_tp) << 8 | int(log2_ep) << 12 | int(dp) << 16


def space_size(d_max, n_types, n_tp, n_dp):
    """number of templates: sum over S = 1..d_max of (n_types * n_tp)^S * n_dp"""
    return sum((n_types * n_tp) ** S * n_dp for S in range(1, d_max + 1))


def all_templates(d_max, types, log2_tp, dp, log2_ep=0):
    """the backbone's loops, outermost first; yields (S, [records])"""
    for S in range(1, d_max + 1):
        for gv in itertools.product(types, repeat=S):
            for tv in itertools.product(log2_tp, repeat=S):
                for D in dp:
                    yield S, [_record(g, t, log2_ep, D) for g, t in zip(gv, tv)]


def template_at(d_max, types, log2_tp, dp, log2_ep, u):
    """template u of the same order, by mixed-radix decoding"""
    n_g, n_k, n_d = len(types), len(log2_tp), len(dp)
    for S in range(1, d_max + 1):
        block = (n_g * n_k) ** S * n_d
        if u < block:
            break
        u -= block
    else:
        raise IndexError("index outside the space")
    u, di = divmod(u, n_d)
    g_index, t_index = divmod(u, n_k ** S)
    recs = []
    for s in range(S):                   # stage 0 is the most significant digit
        gs = (g_index // n_g ** (S - 1 - s)) % n_g
        ts = (t_index // n_k ** (S - 1 - s)) % n_k
        recs.append(_record(types[gs], log2_tp[ts], log2_ep, dp[di]))
    return S, recs


def as_arrays(templates, d_max):
    """(n_stages uint8 [n], stages uint32 [n][d_max]) of (S, records) pairs"""
    templates = list(templates)
    ns = np.zeros(len(templates), dtype=np.uint8)
    st = np.zeros((len(templates), d_max), dtype=np.uint32)
    for i, (S, recs) in enumerate(templates):
        ns[i] = S
        st[i, :S] = recs
    return ns, st


def best_enumerated(oprof, d_max, types, log2_tp, dp, log2_ep, m, flags=0):
    """(index, m index, iter, number of OK plans) of the best plan of the
    whole space, ranked as the oracle's argmin (iter / m, ties to the lowest
    template index, then the lowest m index); index None if no plan is OK.
    For small spaces: every template is priced."""
    ns, st = as_arrays(all_templates(d_max, types, log2_tp, dp, log2_ep), d_max)
    out = O.price_plans(oprof, ns, st, m, flags)
    n_ok = int((out["status"] == 0).sum())
    best = O.best_plan(m, out["iter"], out["status"], flags)
    if best is None:
        return None, None, None, n_ok
    t, k = best
    return t, k, out["iter"][t, k], n_ok
