"""GPU parity of the exhaustive enumeration (the planners' search backbone of
section 3.1 over a whole space): the library's device generator against the
oracle's loop nest, record for record, and the best plan of a space against
the oracle pricing every template of it. Needs an MI355X."""
import sys

import numpy as np
import pytest

from gpu_common import CO, F32
from oracle import enumeration as EN
from oracle import oracle as O
from workloads.gen import make_workload, random_instance

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="session")
def H():
    import torch
    assert torch.cuda.is_available(), "no GPU"
    from paper_2609_34244_amd import heddle
    heddle.lib()
    return heddle


def gpu_range(H, spec, first, n):
    ns, st = H.heddle_enum_templates(spec, first, n)
    return ns.cpu().numpy(), st.cpu().numpy().view(np.uint32)


SPECS = [(4, [2, 0, 1], [1, 0], [1, 3], 0), (3, [0], [0, 1, 2, 3], [2], 1), (6, [0, 1], [0, 1], [1], 0),
         (2, [7, 3, 5, 1], [2], [8, 2, 4], 3), (1, [4], [0], [1], 0)]


@pytest.mark.parametrize("spec", SPECS)
def test_enum_templates_whole_space(H, spec):
    d_max, types, tps, dps, ep = spec
    s = H.EnumSpec(d_max, types, tps, dps, ep)
    total = H.heddle_enum_count(s)
    assert total == EN.space_size(d_max, len(types), len(tps), len(dps))
    ns_o, st_o = EN.as_arrays(EN.all_templates(d_max, types, tps, dps, ep), d_max)
    ns, st = gpu_range(H, s, 0, total)
    assert np.array_equal(ns, ns_o) and np.array_equal(st, st_o)
    # ragged ranges across the depth boundaries
    starts = np.cumsum([(len(types) * len(tps)) ** S * len(dps) for S in range(1, d_max + 1)])
    for b in [0, *starts[:-1].tolist()]:
        for first, n in [(max(b - 3, 0), 7), (b, 1)]:
            n = min(n, total - first)
            ns, st = gpu_range(H, s, first, n)
            assert np.array_equal(ns, ns_o[first:first + n]) and np.array_equal(st, st_o[first:first + n])


def test_enum_templates_large_space_sampled(H):
    """N = K = 3, D = 8 (48,427,560 templates): seeded ranges decoded on the
    GPU against the oracle's random access, and the last template"""
    d_max, types, tps, dps, ep = 8, [0, 1, 2], [0, 1, 2], [1], 0
    s = H.EnumSpec(d_max, types, tps, dps, ep)
    total = H.heddle_enum_count(s)
    assert total == 48_427_560
    rng = np.random.default_rng(7)
    firsts = sorted(set(rng.integers(0, total - 64, size=12).tolist()) | {total - 64, 0})
    for first in firsts:
        ns, st = gpu_range(H, s, first, 64)
        want = EN.as_arrays([EN.template_at(d_max, types, tps, dps, ep, u) for u in range(first, first + 64)], d_max)
        assert np.array_equal(ns, want[0]) and np.array_equal(st, want[1]), first


def small_space_instance(seed):
    """a random profile and a spec over all of its GPU types and TP degrees"""
    rng = np.random.default_rng(900 + seed)
    w = random_instance(900 + seed, L=int(rng.integers(3, 12)), n_types=int(rng.integers(1, 4)), n=2)
    p = w.profile
    types = list(rng.permutation(p.layer_ns.shape[0]))
    tps = [int(np.log2(t)) for t in rng.permutation(p.tp_degrees)]
    d_max = int(rng.integers(1, 5)) if len(types) * len(tps) <= 4 else int(rng.integers(1, 4))
    dps = sorted(set(int(x) for x in rng.choice([1, 2, 3, 4], size=int(rng.integers(1, 3)))))
    ep = int(np.log2(rng.choice(p.ep_degrees)))
    m = np.unique(rng.integers(1, 20, size=int(rng.integers(1, 4)))).astype(np.int32)
    return w, (d_max, types, tps, dps, ep), m


@pytest.mark.parametrize("flags", [0, CO, F32, F32 | CO, 4])
def test_best_enumerated_matches_oracle(H, flags):
    n_spaces = 0
    for seed in range(16):
        w, (d_max, types, tps, dps, ep), m = small_space_instance(seed)
        prof = H.heddle_load_profile(w.profile)
        op = O.OracleProfile(w.profile)
        want = EN.best_enumerated(op, d_max, types, tps, dps, ep, m, flags)
        s = H.EnumSpec(d_max, types, tps, dps, ep)
        total = H.heddle_enum_count(s)
        for chunk in (0, 7, max(total // 3, 1)):
            got = H.heddle_best_enumerated(prof, s, m, flags, chunk)
            ctx = f"seed {seed} spec {(d_max, types, tps, dps, ep)} m {m.tolist()} chunk {chunk}"
            assert got[3] == want[3], ctx
            assert got[:2] == want[:2], ctx
            if want[0] is not None:
                assert np.array_equal(np.array(got[2], dtype=want[2].dtype), want[2]), ctx
        n_spaces += 1
    say("spaces checked", n_spaces)


def test_best_enumerated_full_size_sampled(H):
    """the 70B-like profile over N = K = 3, D = 8: the best plan re-priced by
    the oracle, and no plan of a seeded sample ranks above it"""
    from fractions import Fraction
    w = make_workload("c3_70b_dense", n=16)
    prof = H.heddle_load_profile(w.profile)
    d_max, types, tps, dps, ep = 8, [0, 1, 2], [0, 1, 2], [1], 0
    s = H.EnumSpec(d_max, types, tps, dps, ep)
    m = [64]
    t, k, it, n_ok = H.heddle_best_enumerated(prof, s, m, 0)
    say("best", t, k, it, "ok plans", n_ok)
    assert t is not None and 0 < n_ok <= H.heddle_enum_count(s)
    op = O.OracleProfile(w.profile)
    ns, st = EN.as_arrays([EN.template_at(d_max, types, tps, dps, ep, t)], d_max)
    o = O.price_plans(op, ns, st, m, 0)
    assert o["status"][0, k] == 0 and int(o["iter"][0, k]) == it
    rng = np.random.default_rng(11)
    idx = rng.integers(0, H.heddle_enum_count(s), size=400)
    ns, st = EN.as_arrays([EN.template_at(d_max, types, tps, dps, ep, int(u)) for u in idx], d_max)
    o = O.price_plans(op, ns, st, m, 0)
    ok = o["status"][:, 0] == 0
    assert all(Fraction(int(x), m[0]) >= Fraction(it, m[k]) for x in o["iter"][ok, 0])


def test_enumeration_edges(H):
    """a one-template space, chunks of one template, and a space where no
    plan fits (every stage count above the layers)"""
    w = make_workload("c1_tiny_dense", n=8)
    prof = H.heddle_load_profile(w.profile)
    op = O.OracleProfile(w.profile)
    s1 = H.EnumSpec(1, [1], [0], [1], 0)
    assert H.heddle_enum_count(s1) == 1
    got = H.heddle_best_enumerated(prof, s1, [16], 0, 1)
    want = EN.best_enumerated(op, 1, [1], [0], [1], 0, np.array([16], np.int32), 0)
    assert got[:2] == want[:2] and got[3] == want[3]
    s2 = H.EnumSpec(2, [0, 1], [1, 0], [2, 1], 0)
    for chunk in (1, 3):
        got = H.heddle_best_enumerated(prof, s2, [16, 4], 0, chunk)
        want = EN.best_enumerated(op, 2, [0, 1], [1, 0], [2, 1], 0, np.array([16, 4], np.int32), 0)
        assert got[:2] == want[:2] and got[3] == want[3]
        assert want[0] is None or got[2] == int(want[2])
    L = w.profile.L
    big = H.EnumSpec(min(L + 2, 64), [0], [0], [1], 0)            # depths above L are BAD_SHAPE
    got = H.heddle_best_enumerated(prof, big, [16], 0, 0)
    want = EN.best_enumerated(op, min(L + 2, 64), [0], [0], [1], 0, np.array([16], np.int32), 0)
    assert got[:2] == want[:2] and got[3] == want[3]
