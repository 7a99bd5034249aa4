"""Digests of pricing outputs for whole-configuration parity.

The expected digests under tests/golden/full_parity/ are written by
tests/golden/full_parity/make_digests.py from the CPU oracle only; the GPU
test recomputes them from the library's outputs of the same seeded inputs.
This module only serialises arrays and hashes bytes: it holds none of the
pricing arithmetic and imports neither the oracle nor the library.
"""
from __future__ import annotations

import hashlib

import numpy as np

CHUNK = 8192                       # templates per digest
OUTPUTS = ("status", "layers", "peak_mem", "iter", "bottleneck")
# (config, flags, templates sampled or None for the whole batch); flags: 1 fp32, 2 compute-only
CASES = [
    ("c2_7b_dense", 0, None), ("c2_7b_dense", 2, None), ("c2_7b_dense", 1, None), ("c2_7b_dense", 3, None),
    ("c3_70b_dense", 0, None),
    ("c4_moe", 0, None), ("c4_moe", 2, None), ("c4_moe", 1, None),
    ("c5_stress", 0, 40000), ("c5_stress", 1, 20000),
]
SAMPLE_SEED = 2026


def case_file(name, flags):
    return f"{name}_f{flags}.json"


def sample_index(n, n_sample):
    """sorted seeded sample of template indices (the whole batch for None)"""
    if n_sample is None or n_sample >= n:
        return np.arange(n)
    return np.sort(np.random.default_rng(SAMPLE_SEED).choice(n, size=n_sample, replace=False))


def _h():
    return hashlib.blake2b(digest_size=16)


def input_digest(w):
    """the seeded inputs both sides price: profile arrays, templates, m"""
    h = _h()
    p = w.profile
    for k in sorted(p.__dataclass_fields__):
        v = getattr(p, k)
        h.update(k.encode())
        if v is None:
            h.update(b"-")
        elif isinstance(v, np.ndarray):
            h.update(str(v.dtype).encode() + str(v.shape).encode())
            h.update(np.ascontiguousarray(v).tobytes())
        else:
            h.update(repr(int(v)).encode())
    for a in (w.n_stages, w.stages, w.m):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def chunk_digests(out):
    """one digest per CHUNK consecutive rows (templates) of every output,
    over their exact bytes (fp32 values by their bit patterns)"""
    n = out["status"].shape[0]
    res = []
    for c in range(0, n, CHUNK):
        h = _h()
        for k in OUTPUTS:
            h.update(np.ascontiguousarray(out[k][c:c + CHUNK]).tobytes())
        res.append(h.hexdigest())
    return res
