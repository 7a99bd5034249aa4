"""ctypes wrapper of the plain CPU oracle (heddle_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the test suite, by the smoke check and
by the CPU-baseline leg of the benchmark. The GPU library never imports it.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "heddle_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

F_FP32 = 1
F_COMPUTE_ONLY = 2
F_DISTRIBUTE = 4
STATUS = ["OK", "BAD_SHAPE", "BAD_TYPE", "BAD_TP", "UNPROFILED", "BAD_DP", "BAD_EP",
          "OVERSUBSCRIBED", "OOM"]


def build():
    """Compile the oracle with plain gcc (no SIMD flags)."""
    subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fPIC", "-shared", "-o", LIB, SRC, "-lm"])
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _lib = C.CDLL(LIB)
        P = C.c_void_p
        _lib.oracle_price_plans.argtypes = [P, C.c_int64, C.c_int64, C.c_int, P, P, P, C.c_int, C.c_uint32,
                                            P, P, P, P, P]
        _lib.oracle_price_plans.restype = C.c_int
        _lib.oracle_best_plan.argtypes = [C.c_int64, C.c_int, P, C.c_uint32, P, P,
                                          C.POINTER(C.c_int64), C.POINTER(C.c_int32)]
        _lib.oracle_best_plan.restype = C.c_int
        _lib.oracle_tile_plans.argtypes = [P, C.c_int64, C.c_int, P, P, P, C.c_int, C.c_uint32, P, P, P, P, P, P]
        _lib.oracle_tile_plans.restype = C.c_int
        _lib.oracle_fill_dp.argtypes = [C.c_int, P, P, C.c_int64, C.c_int, P, P, C.c_int, P]
        _lib.oracle_fill_dp.restype = C.c_int
        _lib.oracle_count_relaxations.argtypes = [P, C.c_int, P, C.c_int, C.c_int64, C.c_uint32]
        _lib.oracle_count_relaxations.restype = C.c_int64
        _lib.oracle_xfer_ns.argtypes = [C.c_int64, C.c_int64]
        _lib.oracle_xfer_ns.restype = C.c_int64
        _lib.oracle_allreduce_ns.argtypes = [C.c_int64, C.c_int64, C.c_int64]
        _lib.oracle_allreduce_ns.restype = C.c_int64
        _lib.oracle_round_sum_f32.argtypes = [P, C.c_int]
        _lib.oracle_round_sum_f32.restype = C.c_float
    return _lib


class _Desc(C.Structure):
    _fields_ = [("L", C.c_int32), ("n_types", C.c_int32), ("n_tp", C.c_int32), ("n_ep", C.c_int32),
                ("tp_degrees", C.c_void_p), ("ep_degrees", C.c_void_p),
                ("layer_ns", C.c_void_p), ("profiled", C.c_void_p), ("layer_ns_f32", C.c_void_p),
                ("is_moe", C.c_void_p),
                ("state_bytes", C.c_void_p), ("xstate_bytes", C.c_void_p), ("act_bytes", C.c_void_p),
                ("grad_bytes", C.c_void_p), ("xgrad_bytes", C.c_void_p),
                ("boundary_bytes", C.c_int64), ("a2a_bytes", C.c_int64),
                ("mem_cap_bytes", C.c_void_p), ("node_size", C.c_void_p), ("n_gpus", C.c_void_p),
                ("intra_bw_MBps", C.c_void_p), ("link_bw_MBps", C.c_void_p), ("xlayer_ns", C.c_void_p)]


class OracleProfile:
    """Holds the oracle's view of a profile (keeps the numpy arrays alive)."""

    def __init__(self, p):
        c = lambda a, dt: np.ascontiguousarray(a, dtype=dt)
        self._keep = {
            "tp": c(p.tp_degrees, np.int32), "ep": c(p.ep_degrees, np.int32),
            "layer_ns": c(p.layer_ns, np.int64), "profiled": c(p.profiled, np.uint8),
            "is_moe": c(p.is_moe, np.uint8),
            "state": c(p.state_bytes, np.int64), "xstate": c(p.xstate_bytes, np.int64),
            "act": c(p.act_bytes, np.int64), "grad": c(p.grad_bytes, np.int64),
            "xgrad": c(p.xgrad_bytes, np.int64), "cap": c(p.mem_cap_bytes, np.int64),
            "node": c(p.node_size, np.int32), "ngpu": c(p.n_gpus, np.int32),
            "intra": c(p.intra_bw_MBps, np.int64), "link": c(p.link_bw_MBps, np.int64),
        }
        if p.layer_ns_f32 is not None:
            self._keep["f32"] = c(p.layer_ns_f32, np.float32)
        if getattr(p, "xlayer_ns", None) is not None:
            self._keep["xlayer"] = c(p.xlayer_ns, np.int64)
        k = self._keep
        ptr = lambda a: a.ctypes.data
        self.desc = _Desc(
            L=p.L, n_types=p.layer_ns.shape[0], n_tp=len(p.tp_degrees), n_ep=len(p.ep_degrees),
            tp_degrees=ptr(k["tp"]), ep_degrees=ptr(k["ep"]), layer_ns=ptr(k["layer_ns"]),
            profiled=ptr(k["profiled"]), layer_ns_f32=ptr(k["f32"]) if "f32" in k else None,
            is_moe=ptr(k["is_moe"]), state_bytes=ptr(k["state"]), xstate_bytes=ptr(k["xstate"]),
            act_bytes=ptr(k["act"]), grad_bytes=ptr(k["grad"]), xgrad_bytes=ptr(k["xgrad"]),
            boundary_bytes=int(p.boundary_bytes), a2a_bytes=int(p.a2a_bytes),
            mem_cap_bytes=ptr(k["cap"]), node_size=ptr(k["node"]), n_gpus=ptr(k["ngpu"]),
            intra_bw_MBps=ptr(k["intra"]), link_bw_MBps=ptr(k["link"]),
            xlayer_ns=ptr(k["xlayer"]) if "xlayer" in k else None)
        self.L = p.L

    @property
    def ref(self):
        return C.byref(self.desc)


def price_plans(oprof, n_stages, stages, m, flags=0, t0=0, t1=None):
    """Price templates [t0, t1). Returns a dict of numpy arrays indexed
    [t - t0, k] (layers [t - t0, k, s])."""
    m = np.ascontiguousarray(m, dtype=np.int32)
    n, s_max = np.shape(stages)
    t1 = n if t1 is None else t1
    n_stages = np.ascontiguousarray(n_stages[t0:t1], dtype=np.uint8)
    stages = np.ascontiguousarray(stages[t0:t1], dtype=np.uint32)
    cnt, n_m = t1 - t0, len(m)
    f32 = bool(flags & F_FP32)
    it = np.empty((cnt, n_m), dtype=np.float32 if f32 else np.int64)
    bn = np.empty_like(it)
    pk = np.empty((cnt, n_m), dtype=np.int64)
    ly = np.empty((cnt, n_m, s_max), dtype=np.uint8)
    stt = np.empty((cnt, n_m), dtype=np.uint8)
    d = lambda a: a.ctypes.data
    rc = lib().oracle_price_plans(oprof.ref, 0, cnt, s_max, d(n_stages), d(stages), d(m), n_m, flags,
                                  d(it), d(bn), d(pk), d(ly), d(stt))
    assert rc == 0
    return {"iter": it, "bottleneck": bn, "peak_mem": pk, "layers": ly, "status": stt}


def tile_plans(oprof, n_stages, stages, m, flags, priced):
    """Re-tile priced plans (a dict from price_plans for the same templates,
    m and flags; int64 costs): returns a new dict with the re-tiled iter,
    bottleneck, peak_mem, status, the unchanged layers, and tiling [t, k, s]
    (log2 EP | log2 ETP << 4)."""
    m = np.ascontiguousarray(m, dtype=np.int32)
    n_stages = np.ascontiguousarray(n_stages, dtype=np.uint8)
    stages = np.ascontiguousarray(stages, dtype=np.uint32)
    n, s_max = stages.shape
    out = {k: np.array(v, copy=True) for k, v in priced.items()}
    out["tiling"] = np.zeros_like(out["layers"])
    d = lambda a: a.ctypes.data
    rc = lib().oracle_tile_plans(oprof.ref, n, s_max, d(n_stages), d(stages), d(m), len(m), flags, d(out["layers"]),
                                 d(out["status"]), d(out["iter"]), d(out["bottleneck"]), d(out["peak_mem"]),
                                 d(out["tiling"]))
    assert rc == 0, "tiling is defined for int64 costs"
    return out


def fill_dp(n_nodes, node_gpus, n_stages, stages, dp_cap):
    """DP degree of every template by packing (returns (dp [n], records with
    the DP field rewritten))."""
    n_nodes = np.ascontiguousarray(n_nodes, dtype=np.int32)
    node_gpus = np.ascontiguousarray(node_gpus, dtype=np.int32)
    n_stages = np.ascontiguousarray(n_stages, dtype=np.uint8)
    st = np.array(stages, dtype=np.uint32, copy=True)
    n, s_max = st.shape
    dp = np.zeros(n, dtype=np.int32)
    d = lambda a: a.ctypes.data
    lib().oracle_fill_dp(len(n_nodes), d(n_nodes), d(node_gpus), n, s_max, d(n_stages), d(st), int(dp_cap), d(dp))
    return dp, st


def fill_plans(oprofs, mbs, n_nodes, node_gpus, global_batch, dp_cap, n_stages, stages, flags=0):
    """BestFill: DP by packing, then every micro-batch size priced (profile
    oprofs[b] at m_b = ceil(global_batch / mbs[b]) micro-batches) and the
    fitting one with the shortest iteration time kept (smaller size on ties;
    the smallest size's results when none fits). Returns the outputs of
    price_plans (n_m = 1) plus dp, mbs_index and the rewritten records."""
    dp, st = fill_dp(n_nodes, node_gpus, n_stages, stages, dp_cap)
    outs = [price_plans(op, n_stages, st, np.array([-(-int(global_batch) // int(b))], dtype=np.int32), flags)
            for op, b in zip(oprofs, mbs)]
    n = len(n_stages)
    pick = np.zeros(n, dtype=np.uint8)
    for t in range(n):
        best = None
        for b, o in enumerate(outs):
            if o["status"][t, 0] != 0:
                continue
            if best is None or o["iter"][t, 0] < outs[best]["iter"][t, 0]:
                best = b
        pick[t] = 0 if best is None else best
    res = {k: np.stack([outs[pick[t]][k][t] for t in range(n)]) if n else outs[0][k] for k in outs[0]}
    res.update(dp=dp, mbs_index=pick, stages=st)
    return res


def best_plan(m, iter_, status, flags=0):
    """(template index, m index) of the best OK plan, or None."""
    iter_ = np.ascontiguousarray(iter_)
    status = np.ascontiguousarray(status, dtype=np.uint8)
    m = np.ascontiguousarray(m, dtype=np.int32)
    n, n_m = status.shape
    bt, bk = C.c_int64(-1), C.c_int32(-1)
    rc = lib().oracle_best_plan(n, n_m, m.ctypes.data, flags, iter_.ctypes.data, status.ctypes.data,
                                C.byref(bt), C.byref(bk))
    return None if rc != 0 else (int(bt.value), int(bk.value))


def count_relaxations(oprof, S, rec, s_max, m, flags=0):
    rec = np.ascontiguousarray(rec, dtype=np.uint32)
    return int(lib().oracle_count_relaxations(oprof.ref, int(S), rec.ctypes.data, s_max, int(m), flags))


def xfer_ns(b, bw):
    return int(lib().oracle_xfer_ns(int(b), int(bw)))


def allreduce_ns(b, n, bw):
    return int(lib().oracle_allreduce_ns(int(b), int(n), int(bw)))


def round_sum_f32(vals):
    v = np.ascontiguousarray(vals, dtype=np.float32)
    return np.float32(lib().oracle_round_sum_f32(v.ctypes.data, len(v)))
