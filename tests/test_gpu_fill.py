"""GPU parity of BestFill (section 5.3, arithmetic auto-fill): the DP degree
from packing TP groups into node lists, and the micro-batch size chosen over
per-size profiles; the library against the oracle on the same seeded
inputs, bit for bit. Needs an MI355X."""
import sys

import numpy as np
import pytest

from gpu_common import CO, F32, assert_same, sub_workload
from oracle import oracle as O
from workloads.gen import cluster_nodes, make_workload, mbs_profile, pack_stage, random_instance

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


def random_cluster(rng, N):
    n_nodes = rng.integers(0, 7, size=N).astype(np.int32)
    node_gpus = rng.choice([1, 2, 3, 4, 6, 8, 12, 16, 64], size=int(n_nodes.sum())).astype(np.int32)
    return n_nodes, node_gpus


def random_templates(rng, n, s_max, N):
    S = rng.integers(0, s_max + 2, size=n)                        # 0 and s_max + 1: bad shapes
    rec = np.zeros((n, s_max), dtype=np.uint32)
    for t in range(n):
        k = min(int(S[t]), s_max)
        rec[t, :k] = pack_stage(rng.integers(0, N + 1, size=k), rng.integers(0, 8, size=k),
                                rng.integers(0, 4, size=k), rng.integers(0, 5, size=k))
    return S.astype(np.uint8), rec


def test_fill_dp_random(H):
    import torch
    rng = np.random.default_rng(31)
    for trial in range(60):
        N = int(rng.integers(1, 5))
        nn, ng = random_cluster(rng, N)
        ns, rec = random_templates(rng, int(rng.integers(1, 200)), int(rng.integers(1, 12)), N)
        dp_cap = int(rng.choice([1, 3, 8, 40, 65535]))
        cl = H.heddle_load_cluster(nn, ng)
        d_ns, d_st = H.to_device(ns, rec)
        dp = H.heddle_fill_dp(cl, d_ns, d_st, dp_cap)
        torch.cuda.synchronize()
        o_dp, o_st = O.fill_dp(nn, ng, ns, rec, dp_cap)
        assert np.array_equal(dp.cpu().numpy(), o_dp), trial
        assert np.array_equal(d_st.cpu().numpy().view(np.uint32), o_st), trial


def test_fill_dp_c3(H):
    import torch
    w0 = make_workload("c3_70b_dense", n=50000)
    nn, ng = cluster_nodes(w0.profile)
    cl = H.heddle_load_cluster(nn, ng)
    for dp_cap, n in ((8, 50000), (1024, 1500)):
        w = sub_workload(w0, np.arange(n))
        d_ns, d_st = H.to_device(w.n_stages, w.stages)
        dp = H.heddle_fill_dp(cl, d_ns, d_st, dp_cap)
        torch.cuda.synchronize()
        o_dp, o_st = O.fill_dp(nn, ng, w.n_stages, w.stages, dp_cap)
        assert np.array_equal(dp.cpu().numpy(), o_dp) and np.array_equal(d_st.cpu().numpy().view(np.uint32), o_st)
        say("dp_cap", dp_cap, "D histogram", np.bincount(o_dp)[:12].tolist())


def fill_both(H, w, mbs, G, dp_cap, flags):
    import torch
    nn, ng = cluster_nodes(w.profile)
    profs = [mbs_profile(w.profile, b) for b in mbs]
    cl = H.heddle_load_cluster(nn, ng)
    hp = [H.heddle_load_profile(p) for p in profs]
    d_ns, d_st = H.to_device(w.n_stages, w.stages)
    out = H.heddle_fill_plans(hp, mbs, cl, G, dp_cap, d_ns, d_st, flags)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    g["stages"] = d_st.cpu().numpy().view(np.uint32)
    o = O.fill_plans([O.OracleProfile(p) for p in profs], mbs, nn, ng, G, dp_cap, w.n_stages, w.stages, flags)
    return g, o


def compare(g, o, flags, ctx):
    assert_same(g, o, flags, ctx)
    for k in ("dp", "mbs_index", "stages"):
        assert np.array_equal(g[k], o[k]), (ctx, k)


@pytest.mark.parametrize("flags", [0, CO, F32, DIST])
def test_fill_plans_random(H, flags):
    for seed in range(30):
        w = random_instance(3100 + seed, moe=seed % 2 == 0, n=37, cap_scale=float([1.0, 3.0, 100.0][seed % 3]))
        g, o = fill_both(H, w, [1, 2, 4], int([8, 13, 40][seed % 3]), int([2, 4, 16][seed % 3]), flags)
        compare(g, o, flags, f"seed {3100 + seed} flags {flags}")


@pytest.mark.parametrize("name,n", [("c3_70b_dense", 300), ("c4_moe", 1000), ("c2_7b_dense", 2000)])
def test_fill_plans_configs(H, name, n):
    w = sub_workload(make_workload(name, n=max(n, 2000)), np.arange(n))
    g, o = fill_both(H, w, [1, 2, 4], 64, 8, 0)
    compare(g, o, 0, name)
    say(name, "statuses", np.bincount(g["status"].ravel(), minlength=9).tolist(), "sizes",
        np.bincount(g["mbs_index"], minlength=3).tolist())


def test_fill_edges(H):
    """64-GPU nodes and TP 64, a cap of 65535, a type without nodes, a
    single-node cluster, and an empty batch"""
    import torch
    nn = np.array([1, 0, 3], np.int32)
    ng = np.array([64, 64, 2, 2], np.int32)
    S = np.array([1, 2, 3, 1, 2], np.uint8)
    rec = np.zeros((5, 3), np.uint32)
    rec[0, :1] = pack_stage(0, 6, 0, 1)                          # TP 64 on the 64-GPU node: 1 replica
    rec[1, :2] = pack_stage(np.array([0, 2]), np.array([0, 1]), 0, 1)
    rec[2, :3] = pack_stage(np.array([2, 2, 0]), np.array([0, 0, 2]), np.array([1, 0, 0]), 1)
    rec[3, :1] = pack_stage(1, 0, 0, 1)                          # type 1 has no nodes: D = 0
    rec[4, :2] = pack_stage(np.array([2, 2]), np.array([1, 1]), 0, 1)
    cl = H.heddle_load_cluster(nn, ng)
    for dp_cap in (1, 2, 65535):
        d_ns, d_st = H.to_device(S, rec)
        dp = H.heddle_fill_dp(cl, d_ns, d_st, dp_cap)
        torch.cuda.synchronize()
        o_dp, o_st = O.fill_dp(nn, ng, S, rec, dp_cap)
        assert np.array_equal(dp.cpu().numpy(), o_dp) and np.array_equal(d_st.cpu().numpy().view(np.uint32), o_st)
    assert o_dp[3] == 0
    d_ns, d_st = H.to_device(S[:0], rec[:0])
    H.heddle_fill_dp(cl, d_ns, d_st, 8)
    torch.cuda.synchronize()
