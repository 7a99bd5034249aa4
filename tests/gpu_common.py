"""Shared helpers of the GPU tests: run the HIP library through its C ABI
binding, run the CPU oracle on the same seeded inputs, compare."""
from __future__ import annotations

import numpy as np

from oracle import oracle as O
from workloads.gen import Workload

F32 = 1
CO = 2
POISON = 0xAB


def sub_workload(w, idx):
    idx = np.asarray(idx)
    return Workload(name=w.name, profile=w.profile, n_stages=np.ascontiguousarray(w.n_stages[idx]),
                    stages=np.ascontiguousarray(w.stages[idx]), m=w.m, s_max=w.s_max, meta=w.meta)


def gpu_price(H, prof, w, flags, poison=True):
    """Price on the GPU; outputs pre-filled with a poison byte so that any
    slot the kernels do not write shows up."""
    import torch
    ns, st = H.to_device(w.n_stages, w.stages)
    out = H.alloc_outputs(w.n, len(w.m), w.s_max, flags)
    if poison:
        for v in out.values():
            v.view(torch.uint8).fill_(POISON)
    H.heddle_price_plans(prof, ns, st, [int(x) for x in w.m], flags, out)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def oracle_price(w, flags):
    return O.price_plans(O.OracleProfile(w.profile), w.n_stages, w.stages, w.m, flags)


def assert_same(g, o, flags, ctx=""):
    """Bit-exact comparison of every output."""
    for k in ("status", "layers", "peak_mem", "iter", "bottleneck"):
        a, b = g[k], o[k]
        if k in ("iter", "bottleneck") and flags & F32:
            a, b = a.view(np.uint32), b.view(np.uint32)
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)
            i = tuple(bad[0])
            t = i[0]
            raise AssertionError(
                f"{ctx}: {k} differs at {len(bad)} places, first {i}: gpu={a[i]} oracle={b[i]}; "
                f"template {t}: status gpu={g['status'][t]} oracle={o['status'][t]}, "
                f"layers gpu={g['layers'][t].tolist()} oracle={o['layers'][t].tolist()}, "
                f"iter gpu={g['iter'][t]} oracle={o['iter'][t]}")


def key_lt(it_a, m_a, it_b, m_b):
    """iter_a / m_a < iter_b / m_b, exactly"""
    from fractions import Fraction
    fa = Fraction(float(it_a)) if isinstance(it_a, (float, np.floating)) else int(it_a)
    fb = Fraction(float(it_b)) if isinstance(it_b, (float, np.floating)) else int(it_b)
    return fa * int(m_b) < fb * int(m_a)
