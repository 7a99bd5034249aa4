"""The model of the split kernel's relaxation schedule (kernel_schedule.py),
pinned to the oracle: without its exit rule it relaxes exactly the pairs the
oracle counts over the windows, and with or without the rule it reaches the
oracle's bottleneck (the exit rule changes the work, never the minimum).
CPU only."""
import numpy as np
import pytest

import kernel_schedule as KS
from oracle import oracle as O
from workloads.gen import make_workload, random_instance

# lengths 20..55 with costs up to 40, so that rows are long enough for a lane
# to take several chunks and the exit rule to fire
CASES = [(7000 + s, 20 + 5 * (s % 8)) for s in range(16)]
I64_MAX = (1 << 63) - 1


@pytest.mark.parametrize("co", [False, True])
def test_schedule_model_against_oracle(co):
    flags = O.F_COMPUTE_ONLY if co else 0
    fired = checked = 0
    for seed, L in CASES:
        w = random_instance(seed, L=L, s_max=8, n=24, max_cost=40)
        op = O.OracleProfile(w.profile)
        m = int(w.m[0])
        o = O.price_plans(op, w.n_stages, w.stages, [m], flags)
        for t in range(w.n):
            S = int(w.n_stages[t])
            full, b_full = KS.evaluated_relaxations(w.profile, S, w.s_max, w.stages[t], m, co, exit_rule=False,
                                                    bottleneck=True)
            ev, b_ev = KS.evaluated_relaxations(w.profile, S, w.s_max, w.stages[t], m, co, bottleneck=True)
            assert full == O.count_relaxations(op, S, w.stages[t], w.s_max, m, flags), (seed, t)
            assert ev <= full and b_ev == b_full, (seed, t)
            want = int(o["bottleneck"][t, 0])
            assert (b_ev if b_ev is not None else I64_MAX) == want, (seed, t)
            fired += ev < full
            checked += b_ev is not None
    assert fired >= 10 and checked >= 50, (fired, checked)


def test_class_ordered_bound_keeps_every_bottleneck():
    """several micro-batch counts per template: classes from the largest key
    down, later rows starting at the previous B* + 1, still reach the
    oracle's bottleneck at every m, and never relax more pairs than pricing
    each class from INF"""
    checked = classes = fired = 0
    cases = [random_instance(seed, L=L, s_max=8, n=24, max_cost=40) for seed, L in CASES]
    # the stress workload's first templates (128 layers, up to 32 stages, six
    # micro-batch counts), where the bound cuts rows
    c5 = make_workload("c5_stress", n=12)
    for w in cases + [c5]:
        ms = [int(m) for m in w.m]
        op = O.OracleProfile(w.profile)
        o = O.price_plans(op, w.n_stages, w.stages, ms, 0)
        for t in range(w.n):
            S = int(w.n_stages[t])
            total, best = KS.template_relaxations(w.profile, S, w.s_max, w.stages[t], ms)
            for k in range(len(ms)):
                want = int(o["bottleneck"][t, k])
                assert (best[k] if best[k] is not None else I64_MAX) == want, (w.name, t, k)
                checked += best[k] is not None
            D = int(w.stages[t, 0] >> 16) or 1
            keys = {min(-(-m // D), S) for m in ms}
            plain = sum(KS.evaluated_relaxations(w.profile, S, w.s_max, w.stages[t], ms[[min(-(-m // D), S) for m in ms].index(k)])
                        for k in keys)
            assert total <= plain, (w.name, t)
            classes += len(keys)
            fired += total < plain
    assert checked >= 50 and classes > len(CASES) * 24 and fired >= 5, (checked, classes, fired)
