#!/usr/bin/env python3
"""Benchmark of batched plan pricing on one MI355X.

A step is one pass of the whole hot path over the batch: template decode and
validation, PartitionLayers (min-max layer split), Evaluate (1F1B iteration
time, peak memory) for every (template, m) plan -- one launch of the pricing
kernel -- followed by the argmin over all plans. Inputs are resident in HBM
before the timed region. Prints one JSON line.

Default workload: the 70B-like dense config (L = 80 layers, 6 GPU types,
1,000,000 templates of up to 16 stages, m = 64 micro-batches, int64 costs).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_LANE_OPS = 256 * 4 * 16 * 2.4e9       # CUs x SIMDs x lanes x clock: 32-bit VALU lane-ops/s
HBM_PEAK = 8e12                             # MI355X HBM3E bytes/s (context: the path is not memory bound)
K_MIN = 3                                   # sub, max, min per relaxation (32-bit DP)
# Distribute: 32-bit lane-ops of one stage-cost evaluation counted from its
# integer arithmetic, leaving out the two all-reduce divisions: time
# difference + p2p (4), state and activation differences, activation x
# in-flight count, sum and compare with capacity (12), dense and expert
# gradient differences (4), and the 64-bit max / sum / max folds into the
# split's bottleneck, total and peak memory (6)
K_EVAL = 26
WORKLOAD_TEXT = {
    "c1_tiny_dense": "tiny dense: L=24, 2 GPU types, 1k templates S<=4, m=16",
    "c2_7b_dense": "7B-like dense: L=32, 4 GPU types, 100k templates S<=8, m in {8,32}",
    "c3_70b_dense": "70B-like dense: L=80, 6 GPU types, 1M templates S<=16, m=64",
    "c4_moe": "MoE: L=48 alternating dense/MoE, 5 GPU types, 500k templates S<=12, EP<=8, m=32",
    "c5_stress": "stress: L=128 MoE pattern, 8 GPU types, 4M templates S<=32, m in {8..256}",
}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# sources of the kernels a traffic measurement covers (and of the tables they read)
COMMON_SOURCES = ["heddle_internal.h", "device_common.h", "exact_math.h", "stage_cost.h", "profile.cpp"]
MEASURED_SOURCES = {"": ["windows.hip", "validate.h", "price.hip", "decode.h", "dp_common.h", "evaluate.hip"],
                    "_distribute": ["distribute.hip", "validate.h"]}


def source_hash(mode=""):
    """hash of the code (comments and spacing dropped) of the device sources
    the traffic counters were taken on"""
    import re
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_34244_amd", "csrc")
    for f in sorted(COMMON_SOURCES + MEASURED_SOURCES[mode]):
        with open(os.path.join(csrc, f)) as fh:
            code = re.sub(r"/\*.*?\*/|//[^\n]*", " ", fh.read(), flags=re.S)
        h.update(f.encode() + b"\0" + " ".join(code.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(config, flags, n_plans, distribute=False):
    """HBM bytes per launch from the committed rocprofv3 counter summary,
    valid only for the kernel source it was measured on."""
    mode = "_distribute" if distribute else ""
    path = os.path.join(ROOT, "profiles", f"price_plans_{config}{mode}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_sha") != source_hash(mode) or t.get("flags") != flags or t.get("plans") != n_plans:
        return None
    return t.get("bytes_per_launch")


def host_cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


_ALL_CORES = {}


def _oracle_chunk(task):
    lo, hi = task
    from oracle import oracle as O
    w, flags, idx = _ALL_CORES["w"], _ALL_CORES["flags"], _ALL_CORES["idx"]
    op = O.OracleProfile(w.profile)
    if idx is None:
        return O.price_plans(op, w.n_stages, w.stages, w.m, flags, lo, hi)   # templates [lo, hi)
    sel = idx[lo:hi]
    return O.price_plans(op, w.n_stages[sel], w.stages[sel], w.m, flags)


def cpu_baseline_all_cores(w, flags, budget_s):
    """The same unmodified oracle, one process per host core (the cores this
    process may run on) over disjoint chunks: the whole batch when it fits the
    budget, else a seeded sample of templates. Forked before the GPU is
    initialised. Returns the rate and the oracle's outputs with the template
    indices they cover, for the parity check of the GPU's outputs."""
    import multiprocessing as mp

    import numpy as np

    from oracle import oracle as O
    op = O.OracleProfile(w.profile)
    probe = min(20, w.n)
    t0 = time.perf_counter()
    O.price_plans(op, w.n_stages, w.stages, w.m, flags, 0, probe)
    per = (time.perf_counter() - t0) / probe
    cores = len(os.sched_getaffinity(0))
    n_fit = int(budget_s * cores / max(per, 1e-9))
    if n_fit >= w.n:
        idx, what = None, f"all {w.n} templates"
        n_done = w.n
    else:
        idx = np.sort(np.random.default_rng(0).choice(w.n, size=max(n_fit, 1), replace=False))
        n_done, what = len(idx), f"a seeded sample of {len(idx)} of {w.n} templates"
    step = max(1, min(4096, -(-n_done // (4 * cores))))
    tasks = [(lo, min(lo + step, n_done)) for lo in range(0, n_done, step)]
    _ALL_CORES.update(w=w, flags=flags, idx=idx)
    with mp.get_context("fork").Pool(cores) as pool:
        t0 = time.perf_counter()
        parts = pool.map(_oracle_chunk, tasks, chunksize=1)
        dt = time.perf_counter() - t0
    _ALL_CORES.clear()
    outs = {k: np.concatenate([p[k] for p in parts]) for k in parts[0]}
    rate = {"value": n_done * len(w.m) / dt, "unit": "plans/s", "cores": cores, "kind": "oracle",
            "sample": f"{what} x {len(w.m)} m in {len(tasks)} chunks over {cores} oracle processes "
                      f"(one per host core), {dt:.1f} s wall"}
    return rate, outs, (np.arange(w.n) if idx is None else idx)


def parity_check(gpu, oracle_out, idx, flags):
    """element-by-element comparison of the GPU's outputs (status, layers,
    peak memory, iteration time, bottleneck) with the oracle's"""
    import numpy as np
    bad = np.zeros(oracle_out["status"].shape, dtype=bool)
    fields = {}
    for k in ("status", "layers", "peak_mem", "iter", "bottleneck"):
        a, b = gpu[k][idx], oracle_out[k]
        if a.dtype == np.float32:
            a, b = a.view(np.uint32), b.view(np.uint32)
        d = a != b
        if d.ndim == 3:
            d = d.any(axis=2)
        fields[k] = int(d.sum())
        bad |= d
    return {"compared_templates": int(len(idx)), "compared_plans": int(bad.size),
            "mismatching_plans": int(bad.sum()), "mismatches_by_output": fields,
            "method": "all-core oracle run, every output of every compared plan compared exactly"}


def cpu_baseline(w, flags, budget_s):
    from oracle import oracle as O
    op = O.OracleProfile(w.profile)
    t0 = time.perf_counter()
    probe = min(20, w.n)
    O.price_plans(op, w.n_stages, w.stages, w.m, flags, 0, probe)
    per = (time.perf_counter() - t0) / probe
    n = int(max(probe, min(w.n, budget_s / max(per, 1e-9))))
    t0 = time.perf_counter()
    O.price_plans(op, w.n_stages, w.stages, w.m, flags, 0, n)
    dt = time.perf_counter() - t0
    return {"value": n * len(w.m) / dt, "unit": "plans/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} of {w.n} templates x {len(w.m)} m, single-threaded plain C oracle, {dt:.1f} s",
            "host_cores_available": len(os.sched_getaffinity(0)), "host_cpu": host_cpu_model()}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c3_70b_dense", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--fp32", action="store_true", help="fp32 cost variant")
    ap.add_argument("--compute-only", action="store_true", help="split ignores memory; fit checked after")
    ap.add_argument("--distribute", action="store_true",
                    help="Heddle's speed-proportional split with its fallback list instead of the min-max split")
    ap.add_argument("--tiling", action="store_true",
                    help="re-tile every priced plan's expert layouts (heddle_tile_plans) inside the step")
    ap.add_argument("--fill", action="store_true",
                    help="BestFill: DP degree from node lists, micro-batch size 1, 2 or 4 from per-size profiles "
                         "(global batch = the config's m micro-batches of size 1)")
    ap.add_argument("--enumerate", action="store_true",
                    help="price the whole space of the search backbone (every stage count up to --enum-depth, "
                         "every type and TP per stage) on the config's profile instead of its template batch")
    ap.add_argument("--enum-types", type=int, default=3, help="GPU types 0..n-1 of the enumerated space")
    ap.add_argument("--enum-tps", type=int, default=3, help="TP degrees 1, 2, 4, ... of the enumerated space")
    ap.add_argument("--enum-depth", type=int, default=8, help="largest stage count of the enumerated space")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the single-core oracle baseline")
    ap.add_argument("--parity-seconds", type=float, default=90.0,
                    help="budget of the all-core oracle run whose outputs are compared with the GPU's (the whole "
                         "batch when it fits, else a seeded sample)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES (reference for HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py prices on one GPU only; plans are independent, so a multi-GPU run would shard "
              "the batch by estimated work and reduce the argmin keys. Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_34244_amd import heddle as H
    from workloads.gen import make_workload

    flags = (H.HEDDLE_F_FP32 if args.fp32 else 0) | (H.HEDDLE_F_COMPUTE_ONLY if args.compute_only else 0) | \
        (H.HEDDLE_F_DISTRIBUTE if args.distribute else 0)
    w = None
    cpu_all = None
    if not (args.copy_calibration or args.enumerate or args.fill):
        t0 = time.perf_counter()
        w = make_workload(args.config)
        log(f"workload {args.config}: {w.n} templates x {len(w.m)} m generated in {time.perf_counter() - t0:.1f}s")
        if not args.no_cpu_baseline:
            log(f"oracle on every host core, at most about {args.parity_seconds:.0f} s (before the GPU is initialised)")
            cpu_all = cpu_baseline_all_cores(w, flags, args.parity_seconds)
            log(f"oracle all-core leg: {cpu_all[0]['sample']}")

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        src = torch.ones(args.copy_calibration, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": args.copy_calibration}))
        return
    k_unit, unit_name = (K_EVAL, "stage-cost evaluation") if args.distribute else (K_MIN, "DP relaxation")
    if args.enumerate:
        return run_enumerate(args, H, flags, k_unit, unit_name)
    if args.fill:
        return run_fill(args, H, flags)
    t0 = time.perf_counter()
    prof = H.heddle_load_profile(w.profile)
    load_ms = (time.perf_counter() - t0) * 1e3
    info = H.heddle_profile_info_get(prof)
    h2d = []
    for _ in range(3):                     # host-to-device copy of the template records (pageable host memory)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ns, st = H.to_device(w.n_stages, w.stages)
        torch.cuda.synchronize()
        h2d.append((time.perf_counter() - t0) * 1e3)
    h2d_ms = float(np.median(h2d))
    # the same copy from page-locked host buffers (a caller that keeps its
    # templates in pinned memory): DMA only, no staging through pageable pages
    pin_ns = torch.from_numpy(np.ascontiguousarray(w.n_stages, dtype=np.uint8)).pin_memory()
    pin_st = torch.from_numpy(np.ascontiguousarray(w.stages, dtype=np.uint32).view(np.int32)).pin_memory()
    h2d_pin = []
    for _ in range(3):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ns.copy_(pin_ns, non_blocking=True)
        st.copy_(pin_st, non_blocking=True)
        torch.cuda.synchronize()
        h2d_pin.append((time.perf_counter() - t0) * 1e3)
    h2d_pin_ms = float(np.median(h2d_pin))
    del pin_ns, pin_st
    m = [int(x) for x in w.m]
    out = H.alloc_outputs(w.n, len(m), w.s_max, flags)
    torch.cuda.synchronize()
    # work: the pairs the split kernel relaxes (its exit rule skips part of the
    # window pairs); the window count is kept as context
    relax_win = H.heddle_count_work(prof, ns, st, m, flags)
    relax = relax_win if args.distribute else H.heddle_count_work(prof, ns, st, m, flags | H.HEDDLE_F_COUNT_EVALUATED)
    n_plans = w.n * len(m)
    log(f"profile loaded in {load_ms:.1f} ms; work per step {relax:,} x {unit_name} ({relax / w.n:.0f} per template; "
        f"{relax_win:,} over the windows); 32-bit DP: {info['narrow_f32' if args.fp32 else 'narrow_i64']}")

    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        H.heddle_price_plans(prof, ns, st, m, flags, out)
        if ev:
            ev[1].record(stream)
        if args.tiling:
            H.heddle_tile_plans(prof, ns, st, m, flags, out)
            if ev:
                ev[2].record(stream)
        return H.heddle_argmin_plans(m, flags, out["iter"], out["status"])

    for i in range(args.warmup):
        step()
        log(f"warmup {i + 1}/{args.warmup} done")
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    best = None
    for i in range(args.steps):
        best = step(evs[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kern_ms = [e[0].elapsed_time(e[1]) for e in evs]
    tile_ms = [e[1].elapsed_time(e[2]) for e in evs] if args.tiling else None
    log(f"timed {args.steps} steps in {elapsed:.3f}s; price kernel {np.mean(kern_ms):.3f} ms avg "
        f"(min {np.min(kern_ms):.3f}); best plan {best}")
    status_np = out["status"].cpu().numpy()
    statuses = np.bincount(status_np.ravel(), minlength=9).tolist()
    parity = None
    if cpu_all is not None and not args.tiling:
        gpu_np = {k: v.cpu().numpy() for k, v in out.items()}
        parity = parity_check(gpu_np, cpu_all[1], cpu_all[2], flags)
        log(f"parity: {parity['mismatching_plans']} of {parity['compared_plans']} plans differ from the oracle")
    # the unpruned recurrence's work, (S-1)(L-S+1)(L-S+2)/2 per distinct split
    # of every plan whose split was computed: context only, the kernel relaxes
    # far fewer pairs (row windows), so this is not an achieved rate
    lay_np = out["layers"].cpu().numpy()[:, :, 0]
    valid = ((status_np == 0) | ((status_np == 8) & (lay_np > 0))).any(axis=1)
    S_np = w.n_stages.astype(np.int64)
    L = w.profile.L
    r_np = (S_np - 1) * (L - S_np + 1) * (L - S_np + 2) // 2
    D_np = np.maximum((w.stages[:, 0] >> 16).astype(np.int64), 1)
    if args.compute_only:
        n_splits = np.ones_like(S_np)
    else:
        keys = np.minimum(-(-np.array(m, dtype=np.int64)[None, :] // D_np[:, None]), S_np[:, None])
        keys.sort(axis=1)
        n_splits = 1 + (np.diff(keys, axis=1) != 0).sum(axis=1)
    dense_r = int((r_np * n_splits * valid).sum())

    kern_s = float(np.mean(kern_ms)) / 1e3
    achieved = relax * k_unit / kern_s
    traffic = measured_traffic(args.config, flags, n_plans, args.distribute)
    if args.distribute:
        roof = {"kernel": "distribute_kernel (one heddle_price_plans launch)",
                "work_per_launch": relax, "work_unit": unit_name, "ops_per_unit": k_unit}
        # context: the same plans under the min-max split (one launch outside the timed region)
        ref = H.alloc_outputs(w.n, len(m), w.s_max, flags & ~H.HEDDLE_F_DISTRIBUTE)
        H.heddle_price_plans(prof, ns, st, m, flags & ~H.HEDDLE_F_DISTRIBUTE, ref)
        torch.cuda.synchronize()
        rs = ref["status"].cpu().numpy()
        both = (status_np == 0) & (rs == 0)
        bd = out["bottleneck"].cpu().numpy().astype(np.float64)
        br = ref["bottleneck"].cpu().numpy().astype(np.float64)
        it_d = out["iter"].cpu().numpy().astype(np.float64)
        it_r = ref["iter"].cpu().numpy().astype(np.float64)
        roof["vs_min_max"] = {"plans_ok": int((status_np == 0).sum()), "min_max_plans_ok": int((rs == 0).sum()),
                              "mean_bottleneck_ratio": float(np.mean(bd[both] / br[both])) if both.any() else None,
                              "mean_iter_ratio": float(np.mean(it_d[both] / it_r[both])) if both.any() else None}
    else:
        roof = {"kernel": "window_kernel + split_kernel + evaluate_kernel (one heddle_price_plans call)",
                "work_per_launch": relax, "work_unit": unit_name + " (pairs the split kernel relaxes)",
                "ops_per_unit": k_unit,
                "context_window": {
                    "per_launch": relax_win,
                    "note": "pairs of the recurrence over the row windows; the row loop's exit rule leaves "
                            "per_launch - work_per_launch of them unrelaxed, so this is context, not an achieved rate",
                    "equivalent_frac": relax_win * K_MIN / kern_s / PEAK_LANE_OPS},
                "context_dense_R": {
                    "per_launch": dense_r,
                    "note": "relaxations of the unpruned suffix recurrence over the plans whose split was computed; "
                            "the kernel performs work_per_launch of them, so this is context, not an achieved rate",
                    "equivalent_frac": dense_r * K_MIN / kern_s / PEAK_LANE_OPS}}
    result = {
        "metric": "candidate plans priced/sec (partition+evaluate) on 1 MI355X; % VALU roofline",
        "value": n_plans * args.steps / elapsed,
        "unit": "plans/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("fp32" if args.fp32 else "int64") +
                 (" (exact 32-bit DP)" if info["narrow_f32" if args.fp32 else "narrow_i64"] and not args.distribute else ""),
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.config], "name": args.config, "templates": w.n, "m": m,
                   "plans": n_plans, "memory_aware": not args.compute_only, "seed": w.meta["seed"],
                   "partition": ("distribute" if args.distribute else "min-max") +
                                (" + expert tiling" if args.tiling else "")},
        "roofline": dict({"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_LANE_OPS / 1e12,
                          "unit": "Tlane-op/s", "frac": achieved / PEAK_LANE_OPS, "traffic": traffic,
                          "traffic_GBps": None if traffic is None else traffic / kern_s / 1e9,
                          "hbm_frac": None if traffic is None else traffic / kern_s / HBM_PEAK,
                          "kernel_ms": float(np.mean(kern_ms))}, **roof),
        "statuses": statuses,
        "tiling": None if not args.tiling else dict({
            "tile_kernel_ms": float(np.mean(tile_ms)),
            "note": "heddle_tile_plans re-tiles every plan's expert layouts after pricing, inside the timed step"},
            **tiling_gain(H, prof, ns, st, m, flags, w, out, float(np.mean(tile_ms)))),
        "best_plan": {"template": best[0], "m_index": best[1], "iter": best[2]} if best else None,
        "profile_load_ms": load_ms,
        "template_h2d_ms": h2d_ms,
        "plans_per_s_with_h2d": n_plans / (elapsed / args.steps + h2d_ms / 1e3),
        "template_h2d_pinned_ms": h2d_pin_ms,
        "plans_per_s_with_pinned_h2d": n_plans / (elapsed / args.steps + h2d_pin_ms / 1e3),
        "parity": parity,
    }
    if not args.no_cpu_baseline:
        log(f"oracle baseline, about {args.cpu_seconds:.0f} s on one host core")
        result["cpu_baseline"] = cpu_baseline(w, flags, args.cpu_seconds)
        result["cpu_baseline"]["all_cores"] = cpu_all[0]
    print(json.dumps(result), flush=True)


# lane-ops per unit of the tile kernel's work: a priced layout (time 8:
# prefix difference, all-to-all product, two sums; memory 10: prefix
# difference, in-flight product, two sums, capacity compare; synchronisation
# 12: prefix difference, the ring formula's two products, quotient and
# ceiling, sum), a dominance test (two compares and the tie rule's two) and a
# bound test (a kept layout under a bound: two compares, two selects; or a
# stage fold: two maxima and a 64-bit sum); 64-bit values count two lane-ops
TILE_OPS = {"layouts_priced": 30, "dominance_tests": 4, "bound_tests": 4}


def tiling_gain(H, prof, ns, st, m, flags, w, tiled, tile_ms):
    """the same plans priced without tiling (one launch outside the timed
    region) against the tiled outputs, and the tile kernel's rate in lane-ops
    over the work heddle_count_tile_work counts on those priced plans"""
    import numpy as np
    import torch
    ref = H.alloc_outputs(w.n, len(m), w.s_max, flags)
    H.heddle_price_plans(prof, ns, st, m, flags, ref)
    torch.cuda.synchronize()
    counts = dict(zip(TILE_OPS, H.heddle_count_tile_work(prof, ns, st, m, flags, ref)))
    ops = sum(TILE_OPS[k] * v for k, v in counts.items())
    achieved = ops / (tile_ms / 1e3)
    s0, s1 = ref["status"].cpu().numpy(), tiled["status"].cpu().numpy()
    i0, i1 = ref["iter"].cpu().numpy().astype(np.float64), tiled["iter"].cpu().numpy().astype(np.float64)
    both = (s0 == 0) & (s1 == 0)
    return {"plans_ok_untiled": int((s0 == 0).sum()), "plans_ok_tiled": int((s1 == 0).sum()),
            "faster_after_tiling": int((i1[both] < i0[both]).sum()),
            "mean_iter_ratio": float(np.mean(i1[both] / i0[both])) if both.any() else None,
            "tile_roofline": {"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_LANE_OPS / 1e12,
                              "unit": "Tlane-op/s", "frac": achieved / PEAK_LANE_OPS, "kernel_ms": tile_ms,
                              "work_per_launch": counts, "ops_per_unit": TILE_OPS}}


def run_fill(args, H, flags):
    """A step is one heddle_fill_plans call over the config's batch (DP by
    packing, every template priced at each micro-batch size, the best size
    kept) followed by the argmin."""
    import numpy as np
    import torch

    from workloads.gen import cluster_nodes, make_workload, mbs_profile

    w = make_workload(args.config)
    mbs, G, dp_cap = [1, 2, 4], int(w.m[0]), 8
    nn, ng = cluster_nodes(w.profile)
    cl = H.heddle_load_cluster(nn, ng)
    profs = [H.heddle_load_profile(mbs_profile(w.profile, b)) for b in mbs]
    ns, st = H.to_device(w.n_stages, w.stages)
    torch.cuda.synchronize()
    out = None
    for i in range(args.warmup):
        out = H.heddle_fill_plans(profs, mbs, cl, G, dp_cap, ns, st, flags)
        log(f"warmup {i + 1}/{args.warmup} done")
    times, best = [], None
    for i in range(args.steps):
        t0 = time.perf_counter()
        out = H.heddle_fill_plans(profs, mbs, cl, G, dp_cap, ns, st, flags)
        best = H.heddle_argmin_plans([G], flags, out["iter"], out["status"])
        times.append(time.perf_counter() - t0)
    step_s = float(np.mean(times))
    status = out["status"].cpu().numpy().ravel()
    dp = out["dp"].cpu().numpy()
    pick = out["mbs_index"].cpu().numpy()
    log(f"timed {args.steps} steps: {step_s * 1e3:.2f} ms each; best {best}")
    result = {
        "metric": "candidate plans priced/sec (partition+evaluate) on 1 MI355X; % VALU roofline",
        "value": w.n / step_s,
        "unit": "plans/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("fp32" if args.fp32 else "int64"),
        "data": "synthetic",
        "config": {"workload": f"BestFill on {WORKLOAD_TEXT[args.config]}: DP by packing (cap {dp_cap}) into "
                               f"node lists of full and half-size nodes, micro-batch size in {mbs}, global batch "
                               f"{G} samples",
                   "name": args.config, "templates": w.n, "plans": w.n, "pricings_per_step": w.n * len(mbs),
                   "memory_aware": not args.compute_only,
                   "partition": "distribute" if args.distribute else "min-max"},
        "roofline": None,
        "fill": {"dp_histogram": np.bincount(dp, minlength=dp_cap + 1).tolist(),
                 "size_chosen": {str(b): int((pick[status == 0] == i).sum()) for i, b in enumerate(mbs)},
                 "statuses": np.bincount(status, minlength=9).tolist()},
        "best_plan": {"template": best[0], "iter": best[2]} if best else None,
    }
    print(json.dumps(result), flush=True)


def run_enumerate(args, H, flags, k_unit, unit_name):
    """A step is one heddle_best_enumerated call: every template of the space
    generated on the device, priced, and the best plan of the space found."""
    import numpy as np
    import torch

    from workloads.gen import make_workload

    w = make_workload(args.config, n=16)           # the config's profile; its template batch is not used
    n_types = w.profile.layer_ns.shape[0]
    tp_log2 = [int(np.log2(t)) for t in w.profile.tp_degrees]
    assert args.enum_types <= n_types and args.enum_tps <= len(tp_log2), "space larger than the profile"
    types, tps = list(range(args.enum_types)), tp_log2[:args.enum_tps]
    spec = H.EnumSpec(args.enum_depth, types, tps, [1], 0)
    m = [int(x) for x in w.m]
    total = H.heddle_enum_count(spec)
    prof = H.heddle_load_profile(w.profile)
    n_plans = total * len(m)
    # algorithmic work of one pass over the space, counted chunk by chunk outside the timed region
    relax, chunk = 0, 1 << 22
    for first in range(0, total, chunk):
        ns, st = H.heddle_enum_templates(spec, first, min(chunk, total - first))
        relax += H.heddle_count_work(prof, ns, st, m, flags if args.distribute else flags | H.HEDDLE_F_COUNT_EVALUATED)
    del ns, st
    torch.cuda.synchronize()
    log(f"space: {total:,} templates x {len(m)} m (types {types}, log2 TP {tps}, S <= {args.enum_depth}); "
        f"work {relax:,} x {unit_name}")
    for i in range(args.warmup):
        H.heddle_best_enumerated(prof, spec, m, flags)
        log(f"warmup {i + 1}/{args.warmup} done")
    times, best = [], None
    for i in range(args.steps):
        t0 = time.perf_counter()
        best = H.heddle_best_enumerated(prof, spec, m, flags)
        times.append(time.perf_counter() - t0)
    step_s = float(np.mean(times))
    log(f"timed {args.steps} passes over the space: {step_s * 1e3:.1f} ms each; best {best}")
    achieved = relax * k_unit / step_s
    result = {
        "metric": "candidate plans priced/sec (partition+evaluate) on 1 MI355X; % VALU roofline",
        "value": n_plans / step_s,
        "unit": "plans/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("fp32" if args.fp32 else "int64"),
        "data": "synthetic",
        "config": {"workload": f"search-backbone enumeration on the {WORKLOAD_TEXT[args.config].split(':')[0]} "
                               f"profile (L={w.profile.L}): {args.enum_types} GPU types x {args.enum_tps} TP degrees "
                               f"per stage, S <= {args.enum_depth}, DP 1, m={m}: {n_plans:,} plans",
                   "name": args.config, "templates": total, "m": m, "plans": n_plans,
                   "memory_aware": not args.compute_only,
                   "partition": "distribute" if args.distribute else "min-max"},
        "roofline": {"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_LANE_OPS / 1e12, "unit": "Tlane-op/s",
                     "frac": achieved / PEAK_LANE_OPS, "traffic": None,
                     "kernel": "whole pass (generator, split, evaluate and argmin kernels, per-chunk host syncs)",
                     "kernel_ms": step_s * 1e3, "work_per_launch": relax,
                     "work_unit": unit_name if args.distribute else unit_name + " (pairs the split kernel relaxes)",
                     "ops_per_unit": k_unit},
        "best_plan": {"template": best[0], "m_index": best[1], "iter": best[2], "ok_plans": best[3]},
    }
    if not args.no_cpu_baseline:
        log(f"oracle baseline, about {args.cpu_seconds:.0f} s on one host core")
        result["cpu_baseline"] = cpu_baseline_enumerate(w, spec, m, flags, total, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def cpu_baseline_enumerate(w, spec, m, flags, total, budget_s):
    import numpy as np

    from oracle import enumeration as EN
    from oracle import oracle as O
    op = O.OracleProfile(w.profile)
    rng = np.random.default_rng(0)
    pick = lambda n: EN.as_arrays([EN.template_at(spec.d_max, spec.types.tolist(), spec.log2_tp.tolist(),
                                                  spec.dp.tolist(), spec.log2_ep, int(u))
                                   for u in rng.integers(0, total, size=n)], spec.d_max)
    ns, st = pick(20)
    t0 = time.perf_counter()
    O.price_plans(op, ns, st, m, flags)
    per = (time.perf_counter() - t0) / 20
    n = int(max(20, min(total, budget_s / max(per, 1e-9))))
    ns, st = pick(n)
    t0 = time.perf_counter()
    O.price_plans(op, ns, st, m, flags)
    dt = time.perf_counter() - t0
    return {"value": n * len(m) / dt, "unit": "plans/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} templates drawn uniformly from the {total:,} of the space x {len(m)} m, "
                      f"single-threaded plain C oracle, {dt:.1f} s",
            "host_cores_available": len(os.sched_getaffinity(0)), "host_cpu": host_cpu_model()}


if __name__ == "__main__":
    main()
