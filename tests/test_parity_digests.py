"""The stored whole-configuration parity digests (tests/golden/full_parity/)
against what they claim to be: every case has its file, the seeded inputs
regenerate to the recorded input digest, the chunk count matches the batch,
and for the cases the oracle prices in seconds the first chunk's digest is
recomputed here from the oracle. No GPU."""
import json
import os

import numpy as np
import pytest

import parity_digest as PD
from gpu_common import oracle_price, sub_workload
from workloads.gen import make_workload

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "full_parity")
# cases whose first chunk of 8,192 templates the oracle prices in a few seconds
FIRST_CHUNK = {("c2_7b_dense", 0), ("c2_7b_dense", 2), ("c2_7b_dense", 1), ("c2_7b_dense", 3),
               ("c3_70b_dense", 0), ("c4_moe", 0), ("c4_moe", 2)}

_wl = {}


def workload(name):
    if name not in _wl:
        _wl.clear()
        _wl[name] = make_workload(name)
    return _wl[name]


def test_every_case_has_its_file():
    files = sorted(f for f in os.listdir(GOLD) if f.endswith(".json"))
    assert files == sorted(PD.case_file(n, f) for n, f, _ in PD.CASES)


@pytest.mark.parametrize("case", PD.CASES, ids=[f"{n}-f{f}" for n, f, _ in PD.CASES])
def test_digest_file_matches_its_inputs(case):
    name, flags, n_sample = case
    with open(os.path.join(GOLD, PD.case_file(name, flags))) as f:
        rec = json.load(f)
    sample = None if n_sample is None else {"n": n_sample, "seed": PD.SAMPLE_SEED}
    assert (rec["config"], rec["flags"], rec["sample"], rec["chunk"]) == (name, flags, sample, PD.CHUNK)
    w = workload(name)
    assert PD.input_digest(w) == rec["input_digest"]
    idx = PD.sample_index(w.n, n_sample)
    assert rec["n_templates"] == w.n and list(rec["m"]) == [int(x) for x in w.m]
    assert len(rec["chunk_digests"]) == -(-len(idx) // PD.CHUNK)
    assert sum(rec["statuses"]) == len(idx) * len(w.m)
    if (name, flags) in FIRST_CHUNK:
        o = oracle_price(sub_workload(w, idx[:PD.CHUNK]), flags)
        assert PD.chunk_digests(o)[0] == rec["chunk_digests"][0]
