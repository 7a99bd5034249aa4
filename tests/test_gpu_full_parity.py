"""Whole-configuration parity: the HIP library (through its C ABI) prices the
full batch of a configuration in one call, as the benchmark times it, and
every output byte of every plan is compared with the CPU oracle's through
per-chunk digests written by tests/golden/full_parity/make_digests.py from
the oracle alone (a seeded sample of the stress config's 4,000,000
templates). A chunk that differs is recomputed by the oracle here and
compared element by element to name the plan. Needs an MI355X."""
import json
import os
import sys
import time

import numpy as np
import pytest

import parity_digest as PD
from gpu_common import POISON, assert_same, gpu_price, oracle_price, sub_workload
from workloads.gen import make_workload

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(__file__), "golden", "full_parity")


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


_wl = {}


def workload(name):
    if name not in _wl:
        _wl.clear()
        _wl[name] = make_workload(name)
    return _wl[name]


@pytest.mark.parametrize("case", PD.CASES, ids=[f"{c[0]}-f{c[1]}" for c in PD.CASES])
def test_whole_config_matches_oracle(H, case):
    name, flags, n_sample = case
    with open(os.path.join(GOLD, PD.case_file(name, flags))) as f:
        rec = json.load(f)
    w = workload(name)
    assert PD.input_digest(w) == rec["input_digest"], "the seeded inputs differ from those the digests were made on"
    prof = H.heddle_load_profile(w.profile)
    t0 = time.time()
    g = gpu_price(H, prof, w, flags)
    assert not np.any(g["status"] == POISON)
    idx = PD.sample_index(w.n, n_sample)
    gs = g if n_sample is None else {k: v[idx] for k, v in g.items()}
    got = PD.chunk_digests(gs)
    assert len(got) == len(rec["chunk_digests"])
    bad = [c for c, (a, b) in enumerate(zip(got, rec["chunk_digests"])) if a != b]
    for c in bad[:1]:
        # name the first differing plans: the oracle on the start of that chunk
        lo = c * PD.CHUNK
        sel = idx[lo:lo + min(PD.CHUNK, 512)]
        o = oracle_price(sub_workload(w, sel), flags)
        assert_same({k: v[lo:lo + len(sel)] for k, v in gs.items()}, o, flags, f"{name} flags {flags} chunk {c}")
    assert not bad, f"{name} flags {flags}: {len(bad)} of {len(got)} chunks differ (first {bad[:5]})"
    st = np.bincount(gs["status"].ravel(), minlength=9).tolist()
    assert st == rec["statuses"]
    say(f"{name} flags {flags}: {len(idx)} templates x {len(w.m)} m bit-exact "
        f"({len(got)} chunks), statuses {st}, {time.time() - t0:.1f}s")
