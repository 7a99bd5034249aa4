"""Thin ctypes binding of libheddle.so (the gfx950 plan-pricing library).

Argument marshalling only: every step of pricing runs in the library's HIP
kernels. PyTorch supplies device memory (tensors' data pointers) and the
current HIP stream. Function names match the C ABI in include/heddle.h.
There is no fallback: if the library is not built, or no GPU is present,
the calls raise.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libheddle.so")

HEDDLE_OK, HEDDLE_E_INVAL, HEDDLE_E_NOMEM, HEDDLE_E_DEVICE, HEDDLE_E_RANGE, HEDDLE_E_NOFEASIBLE = 0, -1, -2, -3, -4, -5
HEDDLE_F_FP32, HEDDLE_F_COMPUTE_ONLY, HEDDLE_F_DISTRIBUTE = 1, 2, 4
HEDDLE_F_COUNT_EVALUATED = 8
NOALLOC_SCRATCH_BYTES = 64 << 20   # HEDDLE_NOALLOC_SCRATCH_BYTES
STATUS_NAMES = ["OK", "BAD_SHAPE", "BAD_TYPE", "BAD_TP", "UNPROFILED", "BAD_DP", "BAD_EP", "OVERSUBSCRIBED", "OOM"]
EXPORTS = ["heddle_load_profile", "heddle_free_profile", "heddle_price_plans", "heddle_price_plans_noalloc",
           "heddle_argmin_plans",
           "heddle_best_plan", "heddle_count_work", "heddle_profile_info_get", "heddle_last_error",
           "heddle_enum_count", "heddle_enum_templates", "heddle_best_enumerated", "heddle_tile_plans",
           "heddle_count_tile_work",
           "heddle_load_cluster", "heddle_free_cluster", "heddle_fill_dp", "heddle_fill_plans"]


class HeddleError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"heddle error {code}: {msg}")
        self.code = code


class heddle_profile_desc(C.Structure):
    _fields_ = [("L", C.c_int32), ("n_types", C.c_int32), ("n_tp", C.c_int32), ("n_ep", C.c_int32),
                ("tp_degrees", C.c_void_p), ("ep_degrees", C.c_void_p),
                ("layer_ns", C.c_void_p), ("profiled", C.c_void_p), ("layer_ns_f32", C.c_void_p),
                ("is_moe", C.c_void_p),
                ("state_bytes", C.c_void_p), ("xstate_bytes", C.c_void_p), ("act_bytes", C.c_void_p),
                ("grad_bytes", C.c_void_p), ("xgrad_bytes", C.c_void_p),
                ("boundary_bytes", C.c_int64), ("a2a_bytes", C.c_int64),
                ("mem_cap_bytes", C.c_void_p), ("node_size", C.c_void_p), ("n_gpus", C.c_void_p),
                ("intra_bw_MBps", C.c_void_p), ("link_bw_MBps", C.c_void_p), ("xlayer_ns", C.c_void_p)]


class heddle_enum_spec(C.Structure):
    _fields_ = [("d_max", C.c_int32), ("n_types", C.c_int32), ("types", C.c_void_p), ("n_tp", C.c_int32),
                ("log2_tp", C.c_void_p), ("n_dp", C.c_int32), ("dp", C.c_void_p), ("log2_ep", C.c_int32)]


class heddle_cluster_desc(C.Structure):
    _fields_ = [("n_types", C.c_int32), ("n_nodes", C.c_void_p), ("node_gpus", C.c_void_p)]


class heddle_profile_info(C.Structure):
    _fields_ = [("narrow", C.c_int32 * 2), ("fx_exp", C.c_int32), ("L", C.c_int32), ("n_types", C.c_int32),
                ("n_tp", C.c_int32), ("n_ep", C.c_int32), ("max_stage_ns", C.c_int64), ("scratch_bytes", C.c_int64),
                ("narrow_tile", C.c_int32)]


_lib = None


def lib():
    """Load libheddle.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run paper_2609_34244_amd.build.build()")
        L = C.CDLL(LIB_PATH)
        P, I32, I64, U32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32
        L.heddle_load_profile.argtypes = [C.POINTER(heddle_profile_desc), C.POINTER(C.c_void_p)]
        L.heddle_free_profile.argtypes = [P]
        L.heddle_free_profile.restype = None
        L.heddle_price_plans.argtypes = [P, I64, I32, P, P, P, I32, U32, P, P, P, P, P, P]
        L.heddle_price_plans_noalloc.argtypes = [P, I64, I32, P, P, P, I32, U32, P, P, P, P, P, P]
        L.heddle_argmin_plans.argtypes = [I64, P, I32, U32, P, P, C.POINTER(C.c_int64), C.POINTER(C.c_int32), P, P]
        L.heddle_best_plan.argtypes = [P, I64, I32, P, P, P, I32, U32, C.POINTER(C.c_int64), C.POINTER(C.c_int32),
                                       P, P]
        L.heddle_count_work.argtypes = [P, I64, I32, P, P, P, I32, U32, C.POINTER(C.c_int64), P]
        L.heddle_profile_info_get.argtypes = [P, C.POINTER(heddle_profile_info)]
        L.heddle_tile_plans.argtypes = [P, I64, I32, P, P, P, I32, U32, P, P, P, P, P, P, P]
        L.heddle_count_tile_work.argtypes = [P, I64, I32, P, P, P, I32, U32, P, P, C.POINTER(C.c_int64), P]
        L.heddle_load_cluster.argtypes = [C.POINTER(heddle_cluster_desc), C.POINTER(C.c_void_p)]
        L.heddle_free_cluster.argtypes = [P]
        L.heddle_free_cluster.restype = None
        L.heddle_fill_dp.argtypes = [P, I64, I32, P, P, I32, P, P]
        L.heddle_fill_plans.argtypes = [P, P, I32, P, I64, I32, I64, I32, P, P, U32, P, P, P, P, P, P, P, P]
        L.heddle_enum_count.argtypes = [C.POINTER(heddle_enum_spec), C.POINTER(C.c_int64)]
        L.heddle_enum_templates.argtypes = [C.POINTER(heddle_enum_spec), I64, I64, P, P, P]
        L.heddle_best_enumerated.argtypes = [P, C.POINTER(heddle_enum_spec), P, I32, U32, I64,
                                             C.POINTER(C.c_int64), C.POINTER(C.c_int32), P, C.POINTER(C.c_int64), P]
        L.heddle_last_error.restype = C.c_char_p
        for f in ("heddle_load_profile", "heddle_price_plans", "heddle_price_plans_noalloc", "heddle_argmin_plans",
                  "heddle_best_plan",
                  "heddle_count_work", "heddle_profile_info_get", "heddle_enum_count", "heddle_enum_templates",
                  "heddle_best_enumerated", "heddle_tile_plans", "heddle_count_tile_work", "heddle_load_cluster",
                  "heddle_fill_dp",
                  "heddle_fill_plans"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def heddle_last_error():
    return lib().heddle_last_error().decode()


def _check(rc):
    if rc != HEDDLE_OK:
        raise HeddleError(rc, heddle_last_error())
    return rc


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else None


class Profile:
    """Handle of a loaded profile (device-resident). Free with
    heddle_free_profile or let it be collected."""

    def __init__(self, handle):
        self.handle = C.c_void_p(handle)

    def __del__(self):
        if getattr(self, "handle", None) and self.handle.value and _lib is not None:
            _lib.heddle_free_profile(self.handle)
            self.handle = C.c_void_p(None)


def heddle_load_profile(p):
    """Load a profile given an object with the descriptor's fields as
    attributes (numpy arrays / ints; ``layer_ns_f32`` may be None)."""
    c = lambda a, dt: np.ascontiguousarray(a, dtype=dt)
    keep = [c(p.tp_degrees, np.int32), c(p.ep_degrees, np.int32), c(p.layer_ns, np.int64), c(p.profiled, np.uint8),
            None if getattr(p, "layer_ns_f32", None) is None else c(p.layer_ns_f32, np.float32),
            c(p.is_moe, np.uint8), c(p.state_bytes, np.int64), c(p.xstate_bytes, np.int64), c(p.act_bytes, np.int64),
            c(p.grad_bytes, np.int64), c(p.xgrad_bytes, np.int64), c(p.mem_cap_bytes, np.int64),
            c(p.node_size, np.int32), c(p.n_gpus, np.int32), c(p.intra_bw_MBps, np.int64),
            c(p.link_bw_MBps, np.int64),
            None if getattr(p, "xlayer_ns", None) is None else c(p.xlayer_ns, np.int64)]
    a = lambda x: None if x is None else x.ctypes.data
    d = heddle_profile_desc(
        L=int(p.L), n_types=int(np.shape(p.layer_ns)[0]), n_tp=len(p.tp_degrees), n_ep=len(p.ep_degrees),
        tp_degrees=a(keep[0]), ep_degrees=a(keep[1]), layer_ns=a(keep[2]), profiled=a(keep[3]),
        layer_ns_f32=a(keep[4]), is_moe=a(keep[5]), state_bytes=a(keep[6]), xstate_bytes=a(keep[7]),
        act_bytes=a(keep[8]), grad_bytes=a(keep[9]), xgrad_bytes=a(keep[10]),
        boundary_bytes=int(p.boundary_bytes), a2a_bytes=int(p.a2a_bytes), mem_cap_bytes=a(keep[11]),
        node_size=a(keep[12]), n_gpus=a(keep[13]), intra_bw_MBps=a(keep[14]), link_bw_MBps=a(keep[15]),
        xlayer_ns=a(keep[16]))
    h = C.c_void_p()
    _check(lib().heddle_load_profile(C.byref(d), C.byref(h)))
    return Profile(h.value)


def heddle_free_profile(prof):
    if prof.handle.value:
        lib().heddle_free_profile(prof.handle)
        prof.handle = C.c_void_p(None)


def heddle_profile_info_get(prof):
    info = heddle_profile_info()
    _check(lib().heddle_profile_info_get(prof.handle, C.byref(info)))
    return dict(narrow_i64=bool(info.narrow[0]), narrow_f32=bool(info.narrow[1]), fx_exp=info.fx_exp, L=info.L,
                n_types=info.n_types, n_tp=info.n_tp, n_ep=info.n_ep, max_stage_ns=info.max_stage_ns,
                scratch_bytes=info.scratch_bytes, narrow_tile=bool(info.narrow_tile))


def _mlist(m):
    m = np.ascontiguousarray(np.atleast_1d(m), dtype=np.int32)
    return m, m.ctypes.data


def alloc_outputs(n, n_m, s_max, flags=0, device="cuda"):
    """Caller-side output buffers for heddle_price_plans (torch tensors)."""
    import torch
    tdt = torch.float32 if flags & HEDDLE_F_FP32 else torch.int64
    return dict(iter=torch.empty((n, n_m), dtype=tdt, device=device),
                bottleneck=torch.empty((n, n_m), dtype=tdt, device=device),
                peak_mem=torch.empty((n, n_m), dtype=torch.int64, device=device),
                layers=torch.empty((n, n_m, s_max), dtype=torch.uint8, device=device),
                status=torch.empty((n, n_m), dtype=torch.uint8, device=device))


def heddle_price_plans(prof, n_stages, stages, m, flags, out, stream=None):
    """n_stages: uint8 [n] and stages: int32/uint32 [n, s_max] device tensors;
    m: host list of micro-batch counts; out: dict from alloc_outputs."""
    n, s_max = int(stages.shape[0]), int(stages.shape[1])
    mm, mp = _mlist(m)
    _check(lib().heddle_price_plans(prof.handle, n, s_max, _ptr(n_stages), _ptr(stages), mp, len(mm), flags,
                                    _ptr(out["iter"]), _ptr(out["bottleneck"]), _ptr(out["peak_mem"]),
                                    _ptr(out["layers"]), _ptr(out["status"]), _stream(stream)))
    return out


def heddle_price_plans_noalloc(prof, n_stages, stages, m, flags, out, stream=None):
    """heddle_price_plans with the window scratch in the library's fixed
    per-GPU buffer: no device allocation in the call."""
    n, s_max = int(stages.shape[0]), int(stages.shape[1])
    mm, mp = _mlist(m)
    _check(lib().heddle_price_plans_noalloc(prof.handle, n, s_max, _ptr(n_stages), _ptr(stages), mp, len(mm), flags,
                                            _ptr(out["iter"]), _ptr(out["bottleneck"]), _ptr(out["peak_mem"]),
                                            _ptr(out["layers"]), _ptr(out["status"]), _stream(stream)))
    return out


def noalloc_scratch_bytes(n, n_m, s_max, flags=0):
    """bytes of the fixed buffer a heddle_price_plans_noalloc call needs"""
    if n == 0 or flags & 4:
        return 0
    plans = n * n_m
    return (plans * 4 + 255) // 256 * 256 + plans * 2 * ((s_max + 3) // 4 * 4)


def heddle_tile_plans(prof, n_stages, stages, m, flags, out, stream=None):
    """Expert tiling of priced plans in place: out is the dict heddle_price_plans
    filled for the same templates, m and flags; adds out["tiling"] (uint8
    [n, n_m, s_max], log2 EP | log2 ETP << 4)."""
    import torch
    n, s_max = int(stages.shape[0]), int(stages.shape[1])
    mm, mp = _mlist(m)
    if "tiling" not in out:
        out["tiling"] = torch.empty_like(out["layers"])
    _check(lib().heddle_tile_plans(prof.handle, n, s_max, _ptr(n_stages), _ptr(stages), mp, len(mm), flags,
                                   _ptr(out["iter"]), _ptr(out["bottleneck"]), _ptr(out["peak_mem"]),
                                   _ptr(out["layers"]), _ptr(out["status"]), _ptr(out["tiling"]), _stream(stream)))
    return out


def heddle_count_tile_work(prof, n_stages, stages, m, flags, out, stream=None):
    """(layouts priced, dominance tests, bound tests) of tiling the plans in
    out (the dict heddle_price_plans filled)."""
    n, s_max = int(stages.shape[0]), int(stages.shape[1])
    mm, mp = _mlist(m)
    h = (C.c_int64 * 3)()
    _check(lib().heddle_count_tile_work(prof.handle, n, s_max, _ptr(n_stages), _ptr(stages), mp, len(mm), flags,
                                        _ptr(out["layers"]), _ptr(out["status"]), h, _stream(stream)))
    return int(h[0]), int(h[1]), int(h[2])


def heddle_argmin_plans(m, flags, iter_, status, stream=None):
    """(template, m index, iter) of the best OK plan; None if none is OK."""
    n = int(status.shape[0])
    mm, mp = _mlist(m)
    bt, bk = C.c_int64(-1), C.c_int32(-1)
    bi = (C.c_float if flags & HEDDLE_F_FP32 else C.c_int64)()
    rc = lib().heddle_argmin_plans(n, mp, len(mm), flags, _ptr(iter_), _ptr(status), C.byref(bt), C.byref(bk),
                                   C.cast(C.byref(bi), C.c_void_p), _stream(stream))
    if rc == HEDDLE_E_NOFEASIBLE:
        return None
    _check(rc)
    return int(bt.value), int(bk.value), bi.value


def heddle_best_plan(prof, n_stages, stages, m, flags, stream=None):
    n, s_max = int(stages.shape[0]), int(stages.shape[1])
    mm, mp = _mlist(m)
    bt, bk = C.c_int64(-1), C.c_int32(-1)
    bi = (C.c_float if flags & HEDDLE_F_FP32 else C.c_int64)()
    rc = lib().heddle_best_plan(prof.handle, n, s_max, _ptr(n_stages), _ptr(stages), mp, len(mm), flags,
                                C.byref(bt), C.byref(bk), C.cast(C.byref(bi), C.c_void_p), _stream(stream))
    if rc == HEDDLE_E_NOFEASIBLE:
        return None
    _check(rc)
    return int(bt.value), int(bk.value), bi.value


def heddle_count_work(prof, n_stages, stages, m, flags, stream=None):
    n, s_max = int(stages.shape[0]), int(stages.shape[1])
    mm, mp = _mlist(m)
    w = C.c_int64(0)
    _check(lib().heddle_count_work(prof.handle, n, s_max, _ptr(n_stages), _ptr(stages), mp, len(mm), flags,
                                   C.byref(w), _stream(stream)))
    return int(w.value)


def to_device(n_stages, stages, device="cuda"):
    """numpy templates -> device tensors (stages carried as int32 bits)."""
    import torch
    ns = torch.from_numpy(np.ascontiguousarray(n_stages, dtype=np.uint8)).to(device)
    st = torch.from_numpy(np.ascontiguousarray(stages, dtype=np.uint32).view(np.int32)).to(device)
    return ns, st


class EnumSpec:
    """Host description of an enumerated space (keeps its arrays alive)."""

    def __init__(self, d_max, types, log2_tp, dp=(1,), log2_ep=0):
        self.types = np.ascontiguousarray(types, dtype=np.uint8)
        self.log2_tp = np.ascontiguousarray(log2_tp, dtype=np.uint8)
        self.dp = np.ascontiguousarray(dp, dtype=np.int32)
        self.d_max, self.log2_ep = int(d_max), int(log2_ep)
        self.c = heddle_enum_spec(d_max=self.d_max, n_types=len(self.types), types=self.types.ctypes.data,
                                  n_tp=len(self.log2_tp), log2_tp=self.log2_tp.ctypes.data, n_dp=len(self.dp),
                                  dp=self.dp.ctypes.data, log2_ep=self.log2_ep)


def heddle_enum_count(spec):
    n = C.c_int64(0)
    _check(lib().heddle_enum_count(C.byref(spec.c), C.byref(n)))
    return int(n.value)


def heddle_enum_templates(spec, first, n, device="cuda", stream=None):
    """Templates first .. first + n - 1 of the space as device tensors
    (n_stages uint8 [n], stages int32 bits [n, d_max])."""
    import torch
    ns = torch.empty(n, dtype=torch.uint8, device=device)
    st = torch.empty((n, spec.d_max), dtype=torch.int32, device=device)
    _check(lib().heddle_enum_templates(C.byref(spec.c), int(first), int(n), _ptr(ns), _ptr(st), _stream(stream)))
    return ns, st


def heddle_best_enumerated(prof, spec, m, flags, chunk=0, stream=None):
    """(template index, m index, iter, OK plan count) of the best plan of the
    space; the index is None if no plan is OK."""
    mm, mp = _mlist(m)
    bt, bk, n_ok = C.c_int64(-1), C.c_int32(-1), C.c_int64(-1)
    bi = (C.c_float if flags & HEDDLE_F_FP32 else C.c_int64)()
    rc = lib().heddle_best_enumerated(prof.handle, C.byref(spec.c), mp, len(mm), flags, int(chunk), C.byref(bt),
                                      C.byref(bk), C.cast(C.byref(bi), C.c_void_p), C.byref(n_ok), _stream(stream))
    if rc == HEDDLE_E_NOFEASIBLE:
        return None, None, None, int(n_ok.value)
    _check(rc)
    return int(bt.value), int(bk.value), bi.value, int(n_ok.value)


class Cluster:
    """Handle of a loaded node list (device-resident)."""

    def __init__(self, handle):
        self.handle = C.c_void_p(handle)

    def __del__(self):
        if getattr(self, "handle", None) and self.handle.value and _lib is not None:
            _lib.heddle_free_cluster(self.handle)
            self.handle = C.c_void_p(None)


def heddle_load_cluster(n_nodes, node_gpus):
    """n_nodes: nodes per GPU type; node_gpus: GPUs per node, type 0's first."""
    nn = np.ascontiguousarray(n_nodes, dtype=np.int32)
    ng = np.ascontiguousarray(node_gpus, dtype=np.int32)
    d = heddle_cluster_desc(n_types=len(nn), n_nodes=nn.ctypes.data, node_gpus=ng.ctypes.data if ng.size else None)
    h = C.c_void_p()
    _check(lib().heddle_load_cluster(C.byref(d), C.byref(h)))
    return Cluster(h.value)


def heddle_free_cluster(cl):
    if cl.handle.value:
        lib().heddle_free_cluster(cl.handle)
        cl.handle = C.c_void_p(None)


def heddle_fill_dp(cl, n_stages, stages, dp_cap, stream=None):
    """DP degree by packing; rewrites the DP field of `stages` (device, in
    place) and returns d_dp (int32 [n])."""
    import torch
    n, s_max = int(stages.shape[0]), int(stages.shape[1])
    dp = torch.empty(n, dtype=torch.int32, device=stages.device)
    _check(lib().heddle_fill_dp(cl.handle, n, s_max, _ptr(n_stages), _ptr(stages), int(dp_cap), _ptr(dp),
                                _stream(stream)))
    return dp


def heddle_fill_plans(profiles, mbs, cl, global_batch, dp_cap, n_stages, stages, flags, stream=None):
    """BestFill: DP by packing (stages rewritten in place), then the best
    micro-batch size; returns the outputs of heddle_price_plans (n_m = 1)
    plus "dp" and "mbs_index"."""
    import torch
    n, s_max = int(stages.shape[0]), int(stages.shape[1])
    arr = (C.c_void_p * len(profiles))(*[p.handle.value for p in profiles])
    mb = np.ascontiguousarray(mbs, dtype=np.int32)
    out = alloc_outputs(n, 1, s_max, flags, device=stages.device)
    out["dp"] = torch.empty(n, dtype=torch.int32, device=stages.device)
    out["mbs_index"] = torch.empty(n, dtype=torch.uint8, device=stages.device)
    _check(lib().heddle_fill_plans(C.cast(arr, C.c_void_p), mb.ctypes.data, len(mb), cl.handle, int(global_batch),
                                   int(dp_cap), n, s_max, _ptr(n_stages), _ptr(stages), flags, _ptr(out["iter"]),
                                   _ptr(out["bottleneck"]), _ptr(out["peak_mem"]), _ptr(out["layers"]),
                                   _ptr(out["status"]), _ptr(out["dp"]), _ptr(out["mbs_index"]), _stream(stream)))
    return out
