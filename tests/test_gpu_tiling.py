"""GPU parity of expert tiling (section 5.3, expert tiling paragraph): the
library's tile kernel, run on the library's own priced plans, against the
oracle's re-tiling of the oracle's priced plans, bit for bit (status, iter,
bottleneck, peak memory, layer counts and the chosen layouts). Needs an
MI355X."""
import sys

import numpy as np
import pytest

from gpu_common import CO, F32, POISON, assert_same, oracle_price, sub_workload
from oracle import oracle as O
from workloads.gen import make_workload, pack_stage, random_instance

pytestmark = pytest.mark.gpu
DIST = 4


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


def gpu_tiled(H, prof, w, flags):
    import torch
    ns, st = H.to_device(w.n_stages, w.stages)
    m = [int(x) for x in w.m]
    out = H.alloc_outputs(w.n, len(m), w.s_max, flags)
    out["tiling"] = torch.full_like(out["layers"], POISON)
    H.heddle_price_plans(prof, ns, st, m, flags, out)
    H.heddle_tile_plans(prof, ns, st, m, flags, out)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def oracle_tiled(w, flags):
    op = O.OracleProfile(w.profile)
    return O.tile_plans(op, w.n_stages, w.stages, w.m, flags, oracle_price(w, flags))


def check(g, o, flags, ctx):
    assert_same(g, o, flags, ctx)
    if not np.array_equal(g["tiling"], o["tiling"]):
        bad = np.argwhere(g["tiling"] != o["tiling"])
        i = tuple(bad[0])
        raise AssertionError(f"{ctx}: tiling differs at {len(bad)} places, first {i}: gpu={g['tiling'][i[:2]].tolist()} "
                             f"oracle={o['tiling'][i[:2]].tolist()}")


@pytest.mark.parametrize("flags", [0, CO, DIST, CO | DIST])
def test_tile_random_instances(H, flags):
    n_plans = 0
    for seed in range(80):
        w = random_instance(2000 + seed, moe=seed % 4 != 0, s_max=int([6, 9, 13][seed % 3]), n=41)
        prof = H.heddle_load_profile(w.profile)
        check(gpu_tiled(H, prof, w, flags), oracle_tiled(w, flags), flags, f"seed {2000 + seed} flags {flags}")
        n_plans += w.n * len(w.m)
    say("tiled random plans", n_plans)


@pytest.mark.parametrize("flags", [0, CO, DIST])
def test_tile_wide_costs(H, flags):
    """layer costs above 2^32 ns: the tile kernel's 64-bit variant"""
    n_plans = 0
    for seed in range(30):
        w = random_instance(2700 + seed, moe=True, s_max=int([6, 9, 13][seed % 3]), n=41)
        p = w.profile
        p.layer_ns = np.ascontiguousarray(p.layer_ns << 30)
        p.xlayer_ns = np.ascontiguousarray(p.xlayer_ns << 30)
        prof = H.heddle_load_profile(p)
        assert not H.heddle_profile_info_get(prof)["narrow_tile"]
        check(gpu_tiled(H, prof, w, flags), oracle_tiled(w, flags), flags, f"wide seed {2700 + seed} flags {flags}")
        n_plans += w.n * len(w.m)
    say("tiled wide-cost plans", n_plans)


def test_tile_variants_of_the_configs(H):
    """the MoE benchmark config tiles in 32 bits, the stress config in 64"""
    got = {name: H.heddle_profile_info_get(H.heddle_load_profile(make_workload(name, n=8).profile))["narrow_tile"]
           for name in ("c2_7b_dense", "c4_moe", "c5_stress")}
    say("32-bit tiling", got)
    assert got["c4_moe"] and not got["c5_stress"]


@pytest.mark.parametrize("name,n", [("c4_moe", 1500), ("c5_stress", 30), ("c2_7b_dense", 500)])
@pytest.mark.parametrize("flags", [0, CO])
def test_tile_config_subsets(H, name, n, flags):
    w = sub_workload(make_workload(name, n=max(n, 2000)), np.arange(n))
    prof = H.heddle_load_profile(w.profile)
    g = gpu_tiled(H, prof, w, flags)
    check(g, oracle_tiled(w, flags), flags, f"{name} flags {flags}")
    say(name, flags, "statuses", np.bincount(g["status"].ravel(), minlength=9).tolist())


def test_tile_full_c4_sampled(H):
    """the full MoE batch (500,000 templates) in the benchmark's launch
    configuration; a seeded sample recomputed by the oracle; tiling never
    slows a plan that fitted with its template's layouts"""
    import torch
    w = make_workload("c4_moe")
    prof = H.heddle_load_profile(w.profile)
    ns, st = H.to_device(w.n_stages, w.stages)
    m = [int(x) for x in w.m]
    out = H.alloc_outputs(w.n, len(m), w.s_max, 0)
    H.heddle_price_plans(prof, ns, st, m, 0, out)
    before = {k: v.cpu().numpy() for k, v in out.items()}
    H.heddle_tile_plans(prof, ns, st, m, 0, out)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    ok = before["status"] == 0
    assert np.all(g["status"][ok] == 0) and np.all(g["iter"][ok] <= before["iter"][ok])
    say("c4 OK plans", int(ok.sum()), "faster after tiling", int((g["iter"][ok] < before["iter"][ok]).sum()),
        "mean ratio", float(np.mean(g["iter"][ok] / before["iter"][ok])))
    idx = np.sort(np.random.default_rng(5).choice(w.n, size=400, replace=False))
    o = oracle_tiled(sub_workload(w, idx), 0)
    check({k: v[idx] for k, v in g.items()}, o, 0, "c4 full sampled")


def test_tile_edges(H):
    """fp32 is rejected; buffers that describe no split (layer counts that do
    not add up to L) are left alone with zero tiling bytes"""
    import torch
    w = random_instance(2500, moe=True, n=8)
    prof = H.heddle_load_profile(w.profile)
    ns, st = H.to_device(w.n_stages, w.stages)
    m = [int(x) for x in w.m]
    out = H.alloc_outputs(w.n, len(m), w.s_max, F32)
    with pytest.raises(H.HeddleError) as e:
        H.heddle_tile_plans(prof, ns, st, m, F32, out)
    assert e.value.code == H.HEDDLE_E_INVAL
    out = H.alloc_outputs(w.n, len(m), w.s_max, 0)
    H.heddle_price_plans(prof, ns, st, m, 0, out)
    out["status"].zero_()
    out["layers"][:, :, 0] = 1                 # stage 0 claims one layer; the rest as priced
    out["layers"][:, :, 1:] = 0
    out["iter"].fill_(7)
    H.heddle_tile_plans(prof, ns, st, m, 0, out)
    torch.cuda.synchronize()
    bad = (w.profile.L != 1)
    if bad:
        assert int(out["tiling"].count_nonzero()) == 0
        assert bool((out["iter"] == 7).all())


def test_tile_max_shapes_and_empty(H):
    """L = 255 layers, s_max = 64 stage slots, four TP and four EP degrees
    (the largest layout table); an empty batch enqueues nothing"""
    import torch
    rng = np.random.default_rng(9)
    w = random_instance(2600, L=255, n_types=2, s_max=64, n=6, moe=True, max_cost=40, cap_scale=100.0)
    p = w.profile
    # four TP and four EP degrees: widen the instance's tables to TP {1, 2, 4, 8}
    K = 4
    tp = np.array([1, 2, 4, 8], np.int32)
    rep = lambda a, ax: np.ascontiguousarray(np.concatenate([a] + [a[:, :1] if ax == 1 else a[:1]] * (K - a.shape[ax]),
                                                            axis=ax)) if a.shape[ax] < K else a
    p.tp_degrees = tp
    p.layer_ns = rep(p.layer_ns, 1)
    p.xlayer_ns = np.ascontiguousarray(p.layer_ns * p.is_moe[None, None, :] // 3, dtype=np.int64)
    p.profiled = np.ones((p.layer_ns.shape[0], K), np.uint8)
    for f in ("state_bytes", "xstate_bytes", "act_bytes", "grad_bytes", "xgrad_bytes"):
        setattr(p, f, rep(getattr(p, f), 0))
    p.ep_degrees = np.array([1, 2, 4, 8], np.int32)
    p.node_size[:] = 8
    p.n_gpus[:] = 1 << 20
    p.check()
    S = np.array([1, 64, 40, 17, 64, 2], np.uint8)
    rec = np.zeros((6, 64), np.uint32)
    for t in range(6):
        rec[t, :S[t]] = pack_stage(rng.integers(0, 2, S[t]), rng.integers(0, 4, S[t]), rng.integers(0, 3, S[t]), 8)
    w.n_stages, w.stages, w.s_max = S, rec, 64
    prof = H.heddle_load_profile(p)
    for flags in (0, CO):
        check(gpu_tiled(H, prof, w, flags), oracle_tiled(w, flags), flags, f"max shapes flags {flags}")
    ns, st = H.to_device(S[:0], rec[:0])
    out = H.alloc_outputs(0, 1, 64, 0)
    H.heddle_price_plans(prof, ns, st, [4], 0, out)
    H.heddle_tile_plans(prof, ns, st, [4], 0, out)
    torch.cuda.synchronize()


def _tiled_plans(w, g):
    """(template, m index) of the plans the tile kernel works on: a split and
    a valid template"""
    has = ((g["status"] == 0) | (g["status"] == 8)) & (g["layers"][:, :, 0] > 0)
    return np.argwhere(has)


def _allowed_layouts(p, rec):
    """allowed (EP, ETP) layouts of one stage record: a profiled ETP within the
    type's node, EP x ETP dividing the stage's TP x DP GPUs (counted here on
    the host from the profile arrays)"""
    g, l2tp, dp = int(rec & 0xFF), int((rec >> 8) & 15), int(rec >> 16)
    W = (1 << l2tp) * dp
    n = 0
    for e in p.ep_degrees:
        for k, t in enumerate(p.tp_degrees):
            n += bool(p.profiled[g, k]) and t <= p.node_size[g] and W % (int(e) * int(t)) == 0
    return n


@pytest.mark.parametrize("flags", [0, CO])
def test_tile_work_counts(H, flags):
    """the counted layouts priced equal a host count of the allowed layouts of
    the tiled plans; the other two counts lie within their definitions'
    bounds; on one-layout profiles every count has its closed form"""
    import torch
    for seed in range(40):
        w = random_instance(2900 + seed, moe=seed % 3 != 0, s_max=int([6, 9, 13][seed % 3]), n=41)
        p = w.profile
        prof = H.heddle_load_profile(p)
        ns, st = H.to_device(w.n_stages, w.stages)
        m = [int(x) for x in w.m]
        out = H.alloc_outputs(w.n, len(m), w.s_max, flags)
        H.heddle_price_plans(prof, ns, st, m, flags, out)
        torch.cuda.synchronize()
        g = {k: v.cpu().numpy() for k, v in out.items()}
        priced, dom, bound = H.heddle_count_tile_work(prof, ns, st, m, flags, out)
        plans = _tiled_plans(w, g)
        allowed = [[_allowed_layouts(p, w.stages[t, s]) for s in range(w.n_stages[t])] for t, _ in plans]
        assert priced == sum(sum(a) for a in allowed), f"seed {2900 + seed}"
        assert dom <= sum(sum(x * x for x in a) for a in allowed)
        F = len(p.tp_degrees) * len(p.ep_degrees)
        if F == 1:
            S = np.array([w.n_stages[t] for t, _ in plans], dtype=np.int64)
            assert priced == S.sum() and dom <= S.sum() and bound <= int((2 * S * S).sum())
            # every stage's one layout fits exactly when the plan keeps its status
            fits = np.array([g["status"][t, k] == 0 for t, k in plans])
            assert dom == int(S[fits].sum()) and bound == int((2 * S[fits] * S[fits]).sum())
    # the MoE config subset: bounds only
    w = sub_workload(make_workload("c4_moe", n=2000), np.arange(1500))
    prof = H.heddle_load_profile(w.profile)
    ns, st = H.to_device(w.n_stages, w.stages)
    m = [int(x) for x in w.m]
    out = H.alloc_outputs(w.n, len(m), w.s_max, flags)
    H.heddle_price_plans(prof, ns, st, m, flags, out)
    priced, dom, bound = H.heddle_count_tile_work(prof, ns, st, m, flags, out)
    g = {k: v.cpu().numpy() for k, v in out.items()}
    plans = _tiled_plans(w, g)
    allowed = [[_allowed_layouts(w.profile, w.stages[t, s]) for s in range(w.n_stages[t])] for t, _ in plans]
    assert priced == sum(sum(a) for a in allowed)
    assert 0 < dom <= sum(sum(x * x for x in a) for a in allowed) and bound > 0
    say("c4 subset tile work", priced, dom, bound, "per tiled plan", priced / len(plans), dom / len(plans),
        bound / len(plans))
