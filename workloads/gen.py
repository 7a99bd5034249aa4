"""Seeded synthetic inputs for batched plan pricing.

This module only *synthesises inputs*: a model/cluster profile (per-layer times
and byte counts, GPU-type properties, bandwidths) and a batch of structural
templates. It holds none of the pricing arithmetic (no prefix sums, no stage
costs, no partitioning, no iteration-time formula), so that the CPU oracle and
the GPU library, which both read its arrays, share nothing but their inputs.

Profile layout (all little-endian numpy arrays; names follow the cost model of
the paper's profile-based cost model section):

* ``layer_ns[g][k][l]``  int64, fwd+bwd ns of layer ``l`` for one micro-batch
  on GPU type ``g`` at the ``k``-th TP degree (computation + TP communication).
* ``profiled[g][k]``     uint8, 0 where no profile entry exists.
* ``is_moe[l]``          uint8, 1 for a mixture-of-experts layer.
* ``state_bytes[k][l]``  int64, per-GPU params + grads + optimizer state
  (dense part), ``xstate_bytes`` the expert part at EP = 1.
* ``act_bytes[k][l]``    int64, per-GPU activation bytes per micro-batch.
* ``grad_bytes[k][l]``   int64, per-GPU fp16 gradient bytes (dense part),
  ``xgrad_bytes`` the expert part at EP = 1.
* ``mem_cap_bytes[g]``, ``node_size[g]``, ``n_gpus[g]``, ``intra_bw_MBps[g]``,
  ``link_bw_MBps[g][h]``; scalars ``boundary_bytes``, ``a2a_bytes``.

Template layout: ``n_stages[n]`` uint8 and ``stages[n][s_max]`` uint32 with
one packed record per stage (see :func:`pack_stage`).
"""
from __future__ import annotations

import json
import math
import os
from dataclasses import dataclass, field

import numpy as np

CONFIG_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "configs")
CONFIG_NAMES = ["c1_tiny_dense", "c2_7b_dense", "c3_70b_dense", "c4_moe", "c5_stress"]

# packed stage record: bits 0-7 GPU type, 8-11 log2 TP, 12-15 log2 EP, 16-31 DP
TYPE_SHIFT, TP_SHIFT, EP_SHIFT, DP_SHIFT = 0, 8, 12, 16


def pack_stage(gtype, log2_tp, log2_ep, dp):
    """Pack one stage record (vectorised over numpy arrays)."""
    gtype = np.asarray(gtype, dtype=np.uint32)
    log2_tp = np.asarray(log2_tp, dtype=np.uint32)
    log2_ep = np.asarray(log2_ep, dtype=np.uint32)
    dp = np.asarray(dp, dtype=np.uint32)
    return ((gtype & 0xFF) << TYPE_SHIFT) | ((log2_tp & 0xF) << TP_SHIFT) | \
        ((log2_ep & 0xF) << EP_SHIFT) | ((dp & 0xFFFF) << DP_SHIFT)


def unpack_stage(rec):
    rec = np.asarray(rec, dtype=np.uint32)
    return ((rec >> TYPE_SHIFT) & 0xFF, (rec >> TP_SHIFT) & 0xF,
            (rec >> EP_SHIFT) & 0xF, (rec >> DP_SHIFT) & 0xFFFF)


@dataclass
class Profile:
    L: int
    tp_degrees: np.ndarray
    ep_degrees: np.ndarray
    layer_ns: np.ndarray
    profiled: np.ndarray
    is_moe: np.ndarray
    state_bytes: np.ndarray
    xstate_bytes: np.ndarray
    act_bytes: np.ndarray
    grad_bytes: np.ndarray
    xgrad_bytes: np.ndarray
    boundary_bytes: int
    a2a_bytes: int
    mem_cap_bytes: np.ndarray
    node_size: np.ndarray
    n_gpus: np.ndarray
    intra_bw_MBps: np.ndarray
    link_bw_MBps: np.ndarray
    layer_ns_f32: np.ndarray | None = None
    xlayer_ns: np.ndarray | None = None      # [N][K][L] expert part of each MoE layer's time at ETP = TP

    @property
    def n_types(self):
        return int(self.layer_ns.shape[0])

    def check(self):
        """Shape/dtype sanity of the arrays (format only, no pricing)."""
        N, K, L = self.layer_ns.shape
        assert L == self.L and K == len(self.tp_degrees)
        assert self.layer_ns.dtype == np.int64 and self.profiled.shape == (N, K)
        for a in (self.state_bytes, self.xstate_bytes, self.act_bytes, self.grad_bytes, self.xgrad_bytes):
            assert a.shape == (K, L) and a.dtype == np.int64
        assert self.is_moe.shape == (L,) and self.is_moe.dtype == np.uint8
        assert self.link_bw_MBps.shape == (N, N)
        for a in (self.mem_cap_bytes, self.intra_bw_MBps):
            assert a.shape == (N,) and a.dtype == np.int64
        for a in (self.node_size, self.n_gpus, self.tp_degrees, self.ep_degrees):
            assert a.dtype == np.int32
        if self.layer_ns_f32 is not None:
            assert self.layer_ns_f32.shape == self.layer_ns.shape and self.layer_ns_f32.dtype == np.float32
        if self.xlayer_ns is not None:
            assert self.xlayer_ns.shape == self.layer_ns.shape and self.xlayer_ns.dtype == np.int64
        return self


@dataclass
class Workload:
    name: str
    profile: Profile
    n_stages: np.ndarray          # uint8 [n]
    stages: np.ndarray            # uint32 [n][s_max]
    m: np.ndarray                 # int32 [n_m]
    s_max: int
    meta: dict = field(default_factory=dict)

    @property
    def n(self):
        return int(self.n_stages.shape[0])


def load_config(name):
    with open(os.path.join(CONFIG_DIR, name + ".json")) as f:
        return json.load(f)


def _round_half_even(x):
    return np.rint(x).astype(np.int64)          # numpy rint rounds half to even


def _ceil_div(a, b):
    return -((-a) // b)


def make_profile(cfg, rng):
    """Synthesise the profile of one config. Draw order: link bandwidths,
    intra-node bandwidths, then the base layer times."""
    types = cfg["types"]
    N, L = len(types), cfg["L"]
    tp = np.array(cfg["tp_degrees"], dtype=np.int32)
    K = len(tp)
    speed = np.array([t["speed"] for t in types], dtype=np.float64)
    node = np.array([t["node_size"] for t in types], dtype=np.int32)

    lo, hi = cfg["link_GBps"]
    link = rng.uniform(lo, hi, size=(N, N))
    link = np.triu(link) + np.triu(link, 1).T                       # symmetric
    link_MBps = _round_half_even(link * 1000.0)
    lo, hi = cfg["intra_GBps"]
    intra_MBps = _round_half_even(rng.uniform(lo, hi, size=N) * 1000.0)

    base = rng.lognormal(mean=math.log(cfg["base_ns_median"]), sigma=cfg["base_ns_sigma"], size=L)
    mult = np.ones(L)
    for k, v in cfg.get("time_multiplier", {}).items():
        mult[int(k)] = float(v)
    eff = np.array([cfg["tp_efficiency"] ** math.log2(k) for k in tp])
    denom = speed[:, None, None] * tp[None, :, None].astype(np.float64) * eff[None, :, None]
    layer_ns = np.maximum(_round_half_even((base * mult)[None, None, :] / denom), 1)
    profiled = (tp[None, :] <= node[:, None]).astype(np.uint8)

    moe = cfg.get("moe")
    is_moe = np.zeros(L, dtype=np.uint8)
    dense_params = np.full(L, cfg["dense_params_per_layer"], dtype=np.int64)
    expert_params = np.zeros(L, dtype=np.int64)
    a2a_bytes = 0
    if moe:
        is_moe[1::2] = 1
        dense_params[is_moe == 1] = moe["attention_params"]
        expert_params[is_moe == 1] = moe["n_experts"] * moe["expert_params"]
        a2a_bytes = int(moe["a2a_bytes"])
    # expert part of an MoE layer's time: the routed experts' share of the
    # layer's active parameters (top-k experts per token), at every TP degree
    xlayer_ns = None
    if moe:
        active = moe["top_k"] * moe["expert_params"]
        share = active / (moe["attention_params"] + active)
        xlayer_ns = np.ascontiguousarray(_round_half_even(layer_ns * share) * is_moe[None, None, :], dtype=np.int64)
    sbp, gbp = cfg["state_bytes_per_param"], cfg["grad_bytes_per_param"]
    kk = tp.astype(np.int64)[:, None]
    state = _ceil_div(sbp * dense_params[None, :], kk)
    xstate = _ceil_div(sbp * expert_params[None, :], kk)
    grad = _ceil_div(gbp * dense_params[None, :], kk)
    xgrad = _ceil_div(gbp * expert_params[None, :], kk)
    act = _ceil_div(np.full((1, L), cfg["act_bytes_per_layer"], dtype=np.int64), kk)
    return Profile(
        L=L, tp_degrees=tp, ep_degrees=np.array(cfg["ep_degrees"], dtype=np.int32),
        layer_ns=np.ascontiguousarray(layer_ns, dtype=np.int64), profiled=profiled, is_moe=is_moe,
        state_bytes=state, xstate_bytes=xstate, act_bytes=np.ascontiguousarray(act), grad_bytes=grad,
        xgrad_bytes=xgrad, boundary_bytes=int(cfg["boundary_bytes"]), a2a_bytes=a2a_bytes,
        mem_cap_bytes=np.array([t["mem_GiB"] * 2**30 for t in types], dtype=np.int64),
        node_size=node, n_gpus=np.array([t["n_gpus"] for t in types], dtype=np.int32),
        intra_bw_MBps=intra_MBps, link_bw_MBps=np.ascontiguousarray(link_MBps), xlayer_ns=xlayer_ns).check()


def _draw_templates(rng, n, s_max, N, tp_sets, dp_choices, ep_degrees):
    """One batch of draws, in this order: S, per-stage type, per-stage TP
    uniform, DP choice, per-stage EP uniform."""
    S = rng.integers(1, s_max + 1, size=n, dtype=np.int64)
    g = rng.integers(0, N, size=(n, s_max), dtype=np.uint8)
    tu = rng.random((n, s_max), dtype=np.float32)
    dsel = rng.integers(0, len(dp_choices), size=n, dtype=np.int64)
    eu = rng.random((n, s_max), dtype=np.float32)
    ntp = np.array([len(t) for t in tp_sets], dtype=np.int64)
    tp_tab = np.zeros((N, int(ntp.max())), dtype=np.int32)
    for i, t in enumerate(tp_sets):
        tp_tab[i, :len(t)] = t
    nt = ntp[g]
    tidx = np.minimum((tu * nt).astype(np.int64), nt - 1)
    tp = tp_tab[g, tidx]
    dps = np.asarray(dp_choices, dtype=np.int64)
    eps = np.asarray(ep_degrees, dtype=np.int64)
    # EP degrees allowed for each DP choice (those dividing it), ascending
    allowed = [eps[(d % eps) == 0] for d in dps]
    nok = np.array([len(a) for a in allowed], dtype=np.int64)
    ep_tab = np.zeros((len(dps), int(nok.max())), dtype=np.int32)
    for i, a in enumerate(allowed):
        ep_tab[i, :len(a)] = a
    nk = nok[dsel][:, None]
    pick = np.minimum((eu * nk).astype(np.int64), nk - 1)
    ep = ep_tab[dsel[:, None], pick]
    return S, g, tp, dps[dsel], ep


def _gpus_per_type(S, g, tp, D, N):
    n, s_max = g.shape
    used = np.arange(s_max)[None, :] < S[:, None]
    idx = (np.arange(n, dtype=np.int64)[:, None] * N + g.astype(np.int64))[used]
    w = (tp.astype(np.int64) * D[:, None])[used]
    return np.bincount(idx, weights=w, minlength=n * N).reshape(n, N)


TEMPLATE_CHUNK = 1 << 16


def make_templates(cfg, profile, rng, n=None):
    """Templates: S ~ U{1..s_max}; per stage a uniform GPU type and a uniform
    TP degree from that type's TP set (powers of two up to its node size);
    one DP degree per template copied into every stage; per stage a uniform EP
    degree among those dividing DP. Templates that use more GPUs of a type than
    the cluster holds are redrawn (the device mask of the planner).
    Drawn in chunks of TEMPLATE_CHUNK templates, each chunk's redraws right
    after its own draws."""
    n = cfg["n_templates"] if n is None else n
    s_max, N = cfg["s_max"], profile.n_types
    tp_sets = [[int(k) for k in profile.tp_degrees if k <= profile.node_size[g]] for g in range(N)]
    n_st = np.empty(n, dtype=np.uint8)
    out = np.empty((n, s_max), dtype=np.uint32)
    log2 = lambda a: np.log2(a).round().astype(np.uint32)
    for c0 in range(0, n, TEMPLATE_CHUNK):
        cn = min(TEMPLATE_CHUNK, n - c0)
        S, g, tp, D, ep = _draw_templates(rng, cn, s_max, N, tp_sets, cfg["dp_choices"], cfg["ep_degrees"])
        for _ in range(1000):
            bad = np.nonzero((_gpus_per_type(S, g, tp, D, N) > profile.n_gpus[None, :]).any(axis=1))[0]
            if bad.size == 0:
                break
            S2, g2, tp2, D2, ep2 = _draw_templates(rng, bad.size, s_max, N, tp_sets, cfg["dp_choices"],
                                                   cfg["ep_degrees"])
            S[bad], g[bad], tp[bad], D[bad], ep[bad] = S2, g2, tp2, D2, ep2
        else:
            raise RuntimeError("template rejection did not converge")
        used = np.arange(s_max)[None, :] < S[:, None]
        rec = pack_stage(g, log2(tp), log2(ep), D[:, None])
        out[c0:c0 + cn] = np.where(used, rec, np.uint32(0))
        n_st[c0:c0 + cn] = S
    return n_st, out


def make_workload(name, n=None):
    """Full workload of one config (``n`` overrides the template count; the
    first ``n`` templates of a smaller draw are not a prefix of a larger one)."""
    cfg = load_config(name)
    rng = np.random.Generator(np.random.PCG64(cfg["seed"]))
    prof = make_profile(cfg, rng)
    n_st, st = make_templates(cfg, prof, rng, n)
    return Workload(name=name, profile=prof, n_stages=n_st, stages=st,
                    m=np.array(cfg["m"], dtype=np.int32), s_max=cfg["s_max"], meta=cfg)


# --------------------------------------------------------------------------
# Random small instances for brute-force and property tests. Small integer
# tables make ties between splits common; caps are drawn so that memory both
# binds and does not; templates include every invalid-record kind.
# --------------------------------------------------------------------------

def random_instance(seed, L=None, n_types=None, s_max=6, n=40, max_cost=6, moe=None,
                    invalid_frac=0.15, cap_scale=None):
    rng = np.random.Generator(np.random.PCG64(seed))
    L = int(rng.integers(1, 15)) if L is None else L
    N = int(rng.integers(1, 4)) if n_types is None else n_types
    tp = np.array([1, 2, 4], dtype=np.int32)[: int(rng.integers(1, 4))]
    K = len(tp)
    moe = bool(rng.integers(0, 2)) if moe is None else moe
    ep = np.array([1, 2, 4], dtype=np.int32) if moe else np.array([1], dtype=np.int32)
    layer_ns = rng.integers(1, max_cost + 1, size=(N, K, L)).astype(np.int64)
    profiled = (rng.random((N, K)) < 0.9).astype(np.uint8)
    is_moe = (rng.random(L) < 0.5).astype(np.uint8) if moe else np.zeros(L, dtype=np.uint8)
    small = lambda: rng.integers(0, 7, size=(K, L)).astype(np.int64)
    state, xstate, act, grad, xgrad = small(), small() * is_moe[None, :], small(), small(), small() * is_moe[None, :]
    node = rng.choice(np.array([1, 2, 4, 8], dtype=np.int32), size=N)
    cap_scale = float(rng.choice([0.3, 1.0, 3.0, 100.0])) if cap_scale is None else cap_scale
    cap = np.maximum((rng.integers(5, 40, size=N) * cap_scale).astype(np.int64), 0)
    prof = Profile(
        L=L, tp_degrees=tp, ep_degrees=ep, layer_ns=layer_ns, profiled=profiled, is_moe=is_moe,
        state_bytes=state, xstate_bytes=xstate, act_bytes=act, grad_bytes=grad, xgrad_bytes=xgrad,
        boundary_bytes=int(rng.integers(0, 3000)), a2a_bytes=int(rng.integers(0, 3000)) if moe else 0,
        mem_cap_bytes=cap, node_size=node, n_gpus=rng.integers(4, 64, size=N).astype(np.int32),
        intra_bw_MBps=rng.integers(500, 4000, size=N).astype(np.int64),
        link_bw_MBps=rng.integers(100, 2000, size=(N, N)).astype(np.int64)).check()
    if moe:                                   # no draw: half of each MoE layer's time is its experts'
        prof.xlayer_ns = np.ascontiguousarray(layer_ns * is_moe[None, None, :] // 2, dtype=np.int64)
    S = rng.integers(1, min(s_max, max(L, 1)) + 1, size=n)
    g = rng.integers(0, N, size=(n, s_max))
    tpl = rng.integers(0, K, size=(n, s_max))
    D = rng.choice(np.array([1, 2, 3, 4]), size=n)
    epl = np.zeros((n, s_max), dtype=np.int64)
    if moe:
        for t in range(n):
            opts = [i for i, e in enumerate(ep) if D[t] % e == 0]
            epl[t] = rng.choice(opts, size=s_max)
    dp = np.broadcast_to(D[:, None], (n, s_max)).copy()
    S = S.astype(np.int64)
    # sprinkle invalid records of every kind
    for t in np.nonzero(rng.random(n) < invalid_frac)[0]:
        kind = int(rng.integers(0, 7))
        s = int(rng.integers(0, S[t]))
        if kind == 0:
            S[t] = int(rng.choice([0, L + 1, s_max + 1]))
        elif kind == 1:
            g[t, s] = N + int(rng.integers(0, 3))
        elif kind == 2:
            tpl[t, s] = int(rng.choice([3, 5, 7]))           # 8, 32, 128: not in the TP set
        elif kind == 3:
            dp[t, s] = 0
        elif kind == 4:
            dp[t, s] = dp[t, s] + 1                           # stages disagree on DP
        elif kind == 5:
            epl[t, s] = 3                                     # EP = 8: not in the EP set
        else:
            D[t] = 63
            dp[t, :] = 63                                     # oversubscribes small clusters
    log2tp = np.where(tpl < K, np.log2(np.where(tpl < K, tp[np.minimum(tpl, K - 1)], 1)), tpl).astype(np.uint32)
    log2ep = np.where(epl < len(ep), np.log2(ep[np.minimum(epl, len(ep) - 1)]), epl).astype(np.uint32)
    rec = pack_stage(np.minimum(g, 255), log2tp, log2ep, dp)
    used = np.arange(s_max)[None, :] < np.minimum(S, s_max)[:, None]
    rec = np.where(used, rec, np.uint32(0)).astype(np.uint32)
    m = np.unique(rng.integers(1, 20, size=int(rng.integers(1, 4)))).astype(np.int32)
    return Workload(name=f"random_{seed}", profile=prof, n_stages=np.minimum(S, 255).astype(np.uint8),
                    stages=np.ascontiguousarray(rec), m=m, s_max=s_max)


def mbs_profile(p, mbs, exponent=0.9):
    """The profile of the same model and cluster at micro-batch size `mbs`
    (the base profile is taken at size 1): per-layer times grow as
    mbs^exponent (a larger micro-batch uses the GPU better), activations,
    the boundary tensor and the MoE all-to-all grow with mbs, parameter,
    optimizer and gradient bytes do not. No random draws."""
    f = float(mbs) ** exponent
    scale = lambda a: np.maximum(_round_half_even(a * f), 1).astype(np.int64)
    q = Profile(**{k: getattr(p, k) for k in p.__dataclass_fields__})
    q.layer_ns = np.ascontiguousarray(scale(p.layer_ns))
    if p.xlayer_ns is not None:
        q.xlayer_ns = np.ascontiguousarray(np.minimum(_round_half_even(p.xlayer_ns * f), q.layer_ns), dtype=np.int64)
    q.layer_ns_f32 = None
    q.act_bytes = np.ascontiguousarray(p.act_bytes * int(mbs))
    q.boundary_bytes = int(p.boundary_bytes) * int(mbs)
    q.a2a_bytes = int(p.a2a_bytes) * int(mbs)
    return q.check()


def cluster_nodes(p):
    """A non-uniform node list per GPU type from a profile's largest node
    size and GPU count: about half of each type's GPUs in nodes of the
    largest size, the rest in nodes of half that size (one-GPU nodes for a
    type whose largest node has one GPU). Returns (n_nodes [N], node_gpus)."""
    n_nodes, gpus = [], []
    for g in range(p.n_types):
        k, total = int(p.node_size[g]), int(p.n_gpus[g])
        full = (total // 2) // k
        rest = total - full * k
        small = max(k // 2, 1)
        nodes = [k] * full + [small] * (rest // small) + ([rest % small] if rest % small else [])
        n_nodes.append(len(nodes))
        gpus += nodes
    return np.array(n_nodes, dtype=np.int32), np.array(gpus, dtype=np.int32)
