"""Writes the expected whole-configuration parity digests.

Runs the plain CPU oracle (and nothing else) over every template of each
case in tests/parity_digest.py (a seeded sample for the stress config), one
process per host core over disjoint chunks, and stores per-chunk digests of
its outputs with the digest of the inputs. Usage, from the repository root:

    python tests/golden/full_parity/make_digests.py [case names ...]
"""
from __future__ import annotations

import json
import multiprocessing as mp
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

import parity_digest as PD  # noqa: E402
from oracle import oracle as O  # noqa: E402
from workloads.gen import make_workload  # noqa: E402

_W = {}


def _price(task):
    lo, hi = task
    w, flags, idx = _W["w"], _W["flags"], _W["idx"]
    sel = idx[lo:hi]
    op = O.OracleProfile(w.profile)
    return O.price_plans(op, w.n_stages[sel], w.stages[sel], w.m, flags)


def run_case(name, flags, n_sample, w):
    idx = PD.sample_index(w.n, n_sample)
    _W.update(w=w, flags=flags, idx=idx)
    step = 2048
    tasks = [(lo, min(lo + step, len(idx))) for lo in range(0, len(idx), step)]
    t0 = time.time()
    with mp.get_context("fork").Pool(len(os.sched_getaffinity(0))) as pool:
        parts = pool.map(_price, tasks, chunksize=1)
    dt = time.time() - t0
    out = {k: np.concatenate([p[k] for p in parts]) for k in PD.OUTPUTS}
    rec = {
        "_what": "digests of the CPU oracle's outputs (status, layers, peak_mem, iter, bottleneck bytes) per chunk of "
                 f"{PD.CHUNK} templates, in template order over the "
                 + ("whole batch" if n_sample is None else f"seeded sample of {len(idx)} templates"),
        "config": name, "flags": flags, "n_templates": int(w.n), "m": [int(x) for x in w.m],
        "sample": None if n_sample is None else {"n": len(idx), "seed": PD.SAMPLE_SEED},
        "chunk": PD.CHUNK, "input_digest": PD.input_digest(w), "chunk_digests": PD.chunk_digests(out),
        "statuses": np.bincount(out["status"].ravel(), minlength=9).tolist(),
        "written_by": "python tests/golden/full_parity/make_digests.py (CPU oracle only)",
        "oracle_wall_s": round(dt, 1), "oracle_processes": len(os.sched_getaffinity(0)),
    }
    with open(os.path.join(HERE, PD.case_file(name, flags)), "w") as f:
        json.dump(rec, f, indent=1)
    print(f"{name} flags {flags}: {len(idx)} templates x {len(w.m)} m in {dt:.1f}s, statuses {rec['statuses']}",
          flush=True)


def main():
    want = set(sys.argv[1:])
    cache = {}
    for name, flags, n_sample in PD.CASES:
        if want and name not in want and PD.case_file(name, flags) not in want:
            continue
        if name not in cache:
            cache.clear()
            cache[name] = make_workload(name)
        run_case(name, flags, n_sample, cache[name])


if __name__ == "__main__":
    main()
