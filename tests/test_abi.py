"""C-ABI checks that need no GPU: the library loads, exports every entry
point the header declares, the header compiles as C, and host-side argument
validation returns the documented codes before any device work."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2609_34244_amd import build as B
from paper_2609_34244_amd import heddle as H
from workloads.gen import make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "heddle.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(H.LIB_PATH):
        B.build()
    return H.lib()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(heddle_[a-z0-9_]+)\s*\(", src)) - {"heddle_profile_desc"})


def test_header_declares_the_entry_points():
    assert set(declared_functions()) == set(H.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", H.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\sT\s(heddle_\w+)", out))
    for f in declared_functions():
        assert f in exported, f
        assert hasattr(lib, f)


def test_header_compiles_as_c(tmp_path):
    src = tmp_path / "use.c"
    src.write_text('#include "heddle.h"\nint main(void){heddle_profile *p = 0; (void)p;'
                   ' return HEDDLE_STAGE(1, 2, 0, 4) == (1u | 2u << 8 | 4u << 16) ? 0 : 1;}\n')
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", os.path.dirname(HEADER),
                        "-I", "/opt/rocm/include", "-o", str(tmp_path / "use"), str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    assert subprocess.run([str(tmp_path / "use")]).returncode == 0


def test_stage_macro_matches_generator_packing():
    from workloads.gen import pack_stage
    assert int(pack_stage(3, 2, 1, 7)) == (3 | 2 << 8 | 1 << 12 | 7 << 16)


def _desc(p, **override):
    c = lambda a, dt: np.ascontiguousarray(a, dtype=dt)
    keep = dict(tp=c(p.tp_degrees, np.int32), ep=c(p.ep_degrees, np.int32), ns=c(p.layer_ns, np.int64),
                prof=c(p.profiled, np.uint8), moe=c(p.is_moe, np.uint8), st=c(p.state_bytes, np.int64),
                xst=c(p.xstate_bytes, np.int64), act=c(p.act_bytes, np.int64), gr=c(p.grad_bytes, np.int64),
                xgr=c(p.xgrad_bytes, np.int64), cap=c(p.mem_cap_bytes, np.int64), node=c(p.node_size, np.int32),
                ngpu=c(p.n_gpus, np.int32), intra=c(p.intra_bw_MBps, np.int64), link=c(p.link_bw_MBps, np.int64))
    keep.update(override)
    a = lambda k: keep[k].ctypes.data
    d = H.heddle_profile_desc(L=p.L, n_types=p.layer_ns.shape[0], n_tp=len(p.tp_degrees), n_ep=len(p.ep_degrees),
                              tp_degrees=a("tp"), ep_degrees=a("ep"), layer_ns=a("ns"), profiled=a("prof"),
                              layer_ns_f32=None, is_moe=a("moe"), state_bytes=a("st"), xstate_bytes=a("xst"),
                              act_bytes=a("act"), grad_bytes=a("gr"), xgrad_bytes=a("xgr"),
                              boundary_bytes=p.boundary_bytes, a2a_bytes=p.a2a_bytes, mem_cap_bytes=a("cap"),
                              node_size=a("node"), n_gpus=a("ngpu"), intra_bw_MBps=a("intra"), link_bw_MBps=a("link"))
    return d, keep


def test_load_profile_rejects_bad_descriptors(lib):
    p = make_workload("c1_tiny_dense", n=4).profile
    h = C.c_void_p(123)
    assert lib.heddle_load_profile(None, C.byref(h)) == H.HEDDLE_E_INVAL and h.value is None
    d, keep = _desc(p)
    assert lib.heddle_load_profile(C.byref(d), None) == H.HEDDLE_E_INVAL
    cases = [
        ("L", 0), ("L", 256), ("n_types", 0), ("n_tp", 0), ("n_ep", 17),
    ]
    for field, val in cases:
        d, keep = _desc(p)
        setattr(d, field, val)
        assert lib.heddle_load_profile(C.byref(d), C.byref(h)) == H.HEDDLE_E_INVAL, field
        assert h.value is None
    for name, arr in [("tp", np.array([1, 3], np.int32)), ("tp", np.array([2, 2], np.int32)),
                      ("ep", np.array([0], np.int32))]:
        d, keep = _desc(p, **{name: arr})
        if name == "tp":
            d.n_tp = 2
        assert lib.heddle_load_profile(C.byref(d), C.byref(h)) == H.HEDDLE_E_INVAL, (name, arr)
    bad = p.layer_ns.copy()
    bad[0, 0, 3] = 0
    d, keep = _desc(p, ns=bad)
    assert lib.heddle_load_profile(C.byref(d), C.byref(h)) == H.HEDDLE_E_INVAL
    assert "layer_ns" in H.heddle_last_error()
    d, keep = _desc(p, intra=np.zeros(p.layer_ns.shape[0], np.int64))
    assert lib.heddle_load_profile(C.byref(d), C.byref(h)) == H.HEDDLE_E_INVAL
    neg = p.act_bytes.copy()
    neg[0, 0] = -1
    d, keep = _desc(p, act=neg)
    assert lib.heddle_load_profile(C.byref(d), C.byref(h)) == H.HEDDLE_E_INVAL
    d, keep = _desc(p)
    d.layer_ns = None
    assert lib.heddle_load_profile(C.byref(d), C.byref(h)) == H.HEDDLE_E_INVAL


def test_load_profile_range_errors(lib):
    p = make_workload("c1_tiny_dense", n=4).profile
    h = C.c_void_p()
    big = np.full_like(p.layer_ns, 1 << 58)
    d, keep = _desc(p, ns=big)
    assert lib.heddle_load_profile(C.byref(d), C.byref(h)) == H.HEDDLE_E_RANGE
    d, keep = _desc(p)
    d.a2a_bytes = 1 << 62
    assert lib.heddle_load_profile(C.byref(d), C.byref(h)) == H.HEDDLE_E_RANGE


def test_price_calls_reject_null_profile(lib):
    m = (C.c_int32 * 1)(4)
    assert lib.heddle_price_plans(None, 0, 4, None, None, m, 1, 0, None, None, None, None, None, None) == H.HEDDLE_E_INVAL
    assert lib.heddle_price_plans_noalloc(None, 0, 4, None, None, m, 1, 0, None, None, None, None, None,
                                          None) == H.HEDDLE_E_INVAL
    cnt = (C.c_int64 * 3)()
    assert lib.heddle_count_tile_work(None, 0, 4, None, None, m, 1, 0, None, None, cnt, None) == H.HEDDLE_E_INVAL
    bt, bk = C.c_int64(), C.c_int32()
    assert lib.heddle_best_plan(None, 1, 4, None, None, m, 1, 0, C.byref(bt), C.byref(bk), None, None) == H.HEDDLE_E_INVAL
    w = C.c_int64()
    assert lib.heddle_count_work(None, 1, 4, None, None, m, 1, 0, C.byref(w), None) == H.HEDDLE_E_INVAL
    assert lib.heddle_argmin_plans(-1, m, 1, 0, None, None, C.byref(bt), C.byref(bk), None, None) == H.HEDDLE_E_INVAL
    assert lib.heddle_argmin_plans(1, m, 1, 8, None, None, C.byref(bt), C.byref(bk), None, None) == H.HEDDLE_E_INVAL
    assert lib.heddle_profile_info_get(None, None) == H.HEDDLE_E_INVAL
    lib.heddle_free_profile(None)          # no-op


def test_noalloc_scratch_size_rule():
    """the fixed buffer's size rule of the header: R(4 n n_m, 256) + 2 n n_m R(s_max, 4)"""
    assert H.noalloc_scratch_bytes(1_000_000, 1, 16) == 36_000_000
    assert H.noalloc_scratch_bytes(3, 2, 5) == 256 + 2 * 6 * 8
    assert H.noalloc_scratch_bytes(0, 2, 5) == 0 and H.noalloc_scratch_bytes(10, 1, 4, flags=4) == 0
    src = open(HEADER).read()
    assert "#define HEDDLE_NOALLOC_SCRATCH_BYTES (64u << 20)" in src and H.NOALLOC_SCRATCH_BYTES == 64 << 20


def _spec(d_max=3, types=(0, 1), tps=(0, 1), dps=(1,), ep=0):
    return H.EnumSpec(d_max, list(types), list(tps), list(dps), ep)


def test_enum_count_and_spec_errors(lib):
    from oracle import enumeration as EN
    for d, t, k, dp in [(1, (0,), (0,), (1,)), (3, (2, 0, 1), (1, 0), (1, 4)), (8, (0, 1, 2), (0, 1, 2), (1,))]:
        assert H.heddle_enum_count(_spec(d, t, k, dp)) == EN.space_size(d, len(t), len(k), len(dp))
    n = C.c_int64(0)
    bad = [_spec(d_max=0), _spec(d_max=65), _spec(types=()), _spec(types=(1, 1)), _spec(tps=(16,)),
           _spec(tps=(2, 2)), _spec(dps=(0,)), _spec(dps=(65536,)), _spec(dps=(2, 2)), _spec(ep=16), _spec(ep=-1)]
    for s in bad:
        assert lib.heddle_enum_count(C.byref(s.c), C.byref(n)) == H.HEDDLE_E_INVAL
    huge = _spec(d_max=64, types=range(255), tps=range(16))
    assert lib.heddle_enum_count(C.byref(huge.c), C.byref(n)) == H.HEDDLE_E_RANGE
    assert lib.heddle_enum_count(C.byref(_spec().c), None) == H.HEDDLE_E_INVAL


def test_enum_templates_range_errors(lib):
    s = _spec()                          # 4 + 16 + 64 = 84 templates
    p = C.c_void_p(16)
    call = lambda first, n, a=p, b=p: lib.heddle_enum_templates(C.byref(s.c), first, n, a, b, None)
    assert call(-1, 1) == H.HEDDLE_E_INVAL
    assert call(0, -1) == H.HEDDLE_E_INVAL
    assert call(80, 5) == H.HEDDLE_E_INVAL
    assert call(85, 0) == H.HEDDLE_E_INVAL
    assert call(0, 4, None, p) == H.HEDDLE_E_INVAL
    assert call(84, 0) == H.HEDDLE_OK           # empty range at the end: nothing enqueued


def test_cluster_and_fill_argument_errors(lib):
    h = C.c_void_p(5)
    nn = np.array([2], np.int32)
    for sizes in ([0, 4], [65, 4]):
        ng = np.array(sizes, np.int32)
        d = H.heddle_cluster_desc(n_types=1, n_nodes=nn.ctypes.data, node_gpus=ng.ctypes.data)
        assert lib.heddle_load_cluster(C.byref(d), C.byref(h)) == H.HEDDLE_E_INVAL and h.value is None
    d = H.heddle_cluster_desc(n_types=0, n_nodes=nn.ctypes.data, node_gpus=None)
    assert lib.heddle_load_cluster(C.byref(d), C.byref(h)) == H.HEDDLE_E_INVAL
    assert lib.heddle_load_cluster(None, C.byref(h)) == H.HEDDLE_E_INVAL
    p = C.c_void_p(16)
    assert lib.heddle_fill_dp(None, 4, 4, p, p, 8, p, None) == H.HEDDLE_E_INVAL
    mb = np.array([1], np.int32)
    assert lib.heddle_fill_plans(None, mb.ctypes.data, 0, p, 8, 8, 4, 4, p, p, 0, p, p, p, p, p, p, p,
                                 None) == H.HEDDLE_E_INVAL
    lib.heddle_free_cluster(None)
