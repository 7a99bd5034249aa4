"""The allocation-free pricing entry point (heddle_price_plans_noalloc)
against heddle_price_plans, through the C ABI, bit for bit: the largest
batch its fixed buffer takes, then smaller batches of other shapes in the
same process, so that the second call runs over what the first left in the
buffer. Needs an MI355X."""
import sys

import numpy as np
import pytest

from gpu_common import CO, F32, POISON
from workloads.gen import make_workload

pytestmark = pytest.mark.gpu

OUTS = ("status", "layers", "peak_mem", "iter", "bottleneck")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def H():
    import torch
    assert torch.cuda.is_available(), "no GPU"
    from paper_2609_34244_amd import heddle
    heddle.lib()
    return heddle


@pytest.fixture(scope="module")
def c3():
    return make_workload("c3_70b_dense")


def _poisoned(H, n, n_m, s_max, flags):
    import torch
    out = H.alloc_outputs(n, n_m, s_max, flags)
    for v in out.values():
        v.view(torch.uint8).fill_(POISON)
    return out


def _both(H, prof, ns, st, m, flags):
    """(heddle_price_plans outputs, heddle_price_plans_noalloc outputs) as numpy"""
    import torch
    n, s_max = int(st.shape[0]), int(st.shape[1])
    ref = _poisoned(H, n, len(m), s_max, flags)
    H.heddle_price_plans(prof, ns, st, m, flags, ref)
    got = _poisoned(H, n, len(m), s_max, flags)
    H.heddle_price_plans_noalloc(prof, ns, st, m, flags, got)
    torch.cuda.synchronize()
    return ({k: ref[k].cpu().numpy() for k in OUTS}, {k: got[k].cpu().numpy() for k in OUTS})


def _same(ref, got, ctx):
    for k in OUTS:
        a, b = ref[k], got[k]
        if a.dtype.kind == "f":
            a, b = a.view(np.uint32), b.view(np.uint32)
        bad = np.argwhere(a != b)
        assert len(bad) == 0, f"{ctx}: {k} differs at {len(bad)} places, first {tuple(bad[0])}"


def _largest_n(H, n_m, s_max):
    """the largest template count (a multiple of 64) whose window scratch fits"""
    n = H.NOALLOC_SCRATCH_BYTES // (n_m * (4 + 2 * ((s_max + 3) // 4 * 4)))
    n -= n % 64
    while H.noalloc_scratch_bytes(n + 64, n_m, s_max) <= H.NOALLOC_SCRATCH_BYTES:
        n += 64
    assert H.noalloc_scratch_bytes(n, n_m, s_max) <= H.NOALLOC_SCRATCH_BYTES
    return n


@pytest.mark.parametrize("flags", [0, F32 | CO])
def test_noalloc_matches_price_plans_largest_then_smaller(H, c3, flags):
    """first call: the 70B-like templates repeated up to the largest batch the
    buffer takes; second call: a smaller batch of another model, s_max and m
    list; third: a ragged batch of the first profile"""
    w = c3
    n_max = _largest_n(H, len(w.m), w.s_max)
    idx = np.arange(n_max) % w.n
    say("noalloc flags", flags, "first call", n_max, "templates of", w.name,
        H.noalloc_scratch_bytes(n_max, len(w.m), w.s_max), "bytes of scratch")
    prof = H.heddle_load_profile(w.profile)
    ns, st = H.to_device(w.n_stages[idx], w.stages[idx])
    m = [int(x) for x in w.m]
    ref, got = _both(H, prof, ns, st, m, flags)
    _same(ref, got, f"{w.name} x{n_max} flags {flags}")
    assert (ref["status"] == 0).any() and (ref["status"] == 8).any()
    del ns, st, ref, got

    w2 = make_workload("c2_7b_dense", n=20000)
    say("noalloc flags", flags, "second call", w2.n, "templates of", w2.name, "m", list(w2.m))
    prof2 = H.heddle_load_profile(w2.profile)
    ns, st = H.to_device(w2.n_stages, w2.stages)
    ref, got = _both(H, prof2, ns, st, [int(x) for x in w2.m], flags)
    _same(ref, got, f"{w2.name} flags {flags}")
    assert (ref["status"] == 0).any()

    say("noalloc flags", flags, "third call", 1000 + 37, "templates of", w.name)
    ns, st = H.to_device(w.n_stages[:1037], w.stages[:1037])
    ref, got = _both(H, prof, ns, st, [64, 7, 64 * 16], flags)
    _same(ref, got, f"{w.name} 1037 templates, three m, flags {flags}")


def test_noalloc_distribute_and_empty(H, c3):
    """the speed-proportional split needs no scratch; n = 0 enqueues nothing"""
    w = c3
    prof = H.heddle_load_profile(w.profile)
    ns, st = H.to_device(w.n_stages[:50000], w.stages[:50000])
    ref, got = _both(H, prof, ns, st, [int(x) for x in w.m], 4)
    _same(ref, got, "distribute")
    ns0, st0 = H.to_device(w.n_stages[:0], w.stages[:0])
    out = H.alloc_outputs(0, 1, w.s_max)
    H.heddle_price_plans_noalloc(prof, ns0, st0, [64], 0, out)


def test_noalloc_rejects_a_batch_beyond_its_buffer(H, c3):
    """one plan row too many: HEDDLE_E_RANGE, nothing enqueued, outputs untouched"""
    import torch
    w = c3
    n = _largest_n(H, 2, w.s_max) + 64
    assert H.noalloc_scratch_bytes(n, 2, w.s_max) > H.NOALLOC_SCRATCH_BYTES
    idx = np.arange(n) % w.n
    prof = H.heddle_load_profile(w.profile)
    ns, st = H.to_device(w.n_stages[idx], w.stages[idx])
    out = _poisoned(H, n, 2, w.s_max, 0)
    with pytest.raises(H.HeddleError) as e:
        H.heddle_price_plans_noalloc(prof, ns, st, [64, 32], 0, out)
    assert e.value.code == H.HEDDLE_E_RANGE
    assert "HEDDLE_NOALLOC_SCRATCH_BYTES" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out["status"] == POISON).all())
    # the same batch goes through the allocating entry point
    H.heddle_price_plans(prof, ns, st, [64, 32], 0, out)
    torch.cuda.synchronize()
    assert int(out["status"].max()) <= 8


def test_noalloc_takes_no_device_memory(H, c3):
    """calls on two streams create no per-stream buffer in the profile, and
    once each stream has run the kernels (the runtime backs a kernel's
    private segment per hardware queue on its first launch there) they leave
    the device's free memory where it was"""
    import torch
    w = c3
    m = [int(x) for x in w.m]
    ns, st = H.to_device(w.n_stages, w.stages)
    out = H.alloc_outputs(w.n, len(w.m), w.s_max)
    s = torch.cuda.Stream()
    warm = H.heddle_load_profile(w.profile)
    H.heddle_price_plans_noalloc(warm, ns, st, m, 0, out)
    H.heddle_price_plans_noalloc(warm, ns, st, m, 0, out, stream=s)
    torch.cuda.synchronize()
    prof = H.heddle_load_profile(w.profile)
    free = [torch.cuda.mem_get_info()[0]]
    for i in range(4):
        H.heddle_price_plans_noalloc(prof, ns, st, m, 0, out, stream=s if i % 2 else None)
        torch.cuda.synchronize()
        free.append(torch.cuda.mem_get_info()[0])
    say("free device memory after each call", free)
    assert H.heddle_profile_info_get(prof)["scratch_bytes"] == 0
    # the allocating path would take 36 MB (the window scratch) on each stream
    assert free[0] - min(free) < 4 << 20
    # the allocating entry point does create the profile's buffer
    H.heddle_price_plans(prof, ns, st, m, 0, out)
    torch.cuda.synchronize()
    assert H.heddle_profile_info_get(prof)["scratch_bytes"] >= H.noalloc_scratch_bytes(w.n, len(m), w.s_max)
