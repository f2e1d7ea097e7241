"""Benchmark of the EZ-SP partition step on one MI355X.

One step = the whole path on one synthetic driving tile already resident in
HBM: exact kNN (k = 10) of 3,000,000 points, graph build, and the merge
ladder over lambda = {0.05, 0.2, 0.8} with D = 16 embeddings, down to the
canonical per-level labels.  Prints one JSON line:
  value        points partitioned per second (n / seconds per step)
  roofline     the stage that takes the most time: its algorithmic bytes per
               launch over its mean launch duration (HIP events on the
               library's stream), against the 8 TB/s HBM peak
  cpu_baseline the CPU oracle (one thread) on a bounded slab of the same tile
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
WORKLOAD = "driving-3m"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--no-cpu", action="store_true",
                    help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-points", type=int, default=400_000)
    return ap.parse_args()


def cpu_baseline(sc, n_sample):
    """Oracle (single-threaded C) on the slab of the tile around x = 0 that
    holds n_sample points: full density profile of the scene, sensor
    included."""
    import numpy as np
    import oracle
    order = np.argsort(np.abs(sc.xyz[:, 0]), kind="stable")[:n_sample]
    idx = np.sort(order)
    xyz = np.ascontiguousarray(sc.xyz[idx])
    emb = np.ascontiguousarray(sc.emb[idx])
    oracle.build()
    t0 = time.perf_counter()
    nbr, _ = oracle.knn(xyz, sc.k)
    t1 = time.perf_counter()
    lo, hi, w = oracle.graph(nbr)
    oracle.partition_graph(emb, lo, hi, w, sc.lambdas, want_energy=False)
    t2 = time.perf_counter()
    return {
        "value": n_sample / (t2 - t0), "unit": "points/s", "cores": 1,
        "kind": "oracle",
        "sample": (f"{n_sample} points of the {sc.name} tile nearest the "
                   f"x = 0 plane (sensor slab), k={sc.k}, ladder "
                   f"{sc.lambdas}; kNN {t1 - t0:.2f} s, graph+ladder "
                   f"{t2 - t1:.2f} s; host {platform.processor() or 'cpu'} "
                   f"with {os.cpu_count()} logical cores"),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}):"
              " this build has no multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2512_00385_amd import ezsp, scenes

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    ezsp.load()
    print(f"[bench] generating {args.workload}", file=sys.stderr, flush=True)
    sc = scenes.load(args.workload)
    dev = torch.device("cuda:0")
    xyz = torch.from_numpy(sc.xyz).to(dev)
    emb = torch.from_numpy(sc.emb).to(dev)
    part = ezsp.Partitioner(sc.n, sc.d, sc.k, sc.lambdas, device=dev)
    print(f"[bench] n={sc.n} d={sc.d} k={sc.k} ws={part.nbytes / 2**30:.2f} "
          "GiB; warmup", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        part(xyz, emb)
    torch.cuda.synchronize()
    ezsp.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        labels, n_comp, _ = part(xyz, emb)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    stages = {}
    for s in ezsp.STAGES:
        launches, ms, nbytes = ezsp.profile_read(s)
        stages[s] = {"launches": launches, "ms": ms, "bytes": nbytes}
    ezsp.profile_enable(False)
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = sc.n / (ms_per_step / 1e3)
    print(f"[bench] {ms_per_step:.3f} ms/step, n_comp {n_comp.tolist()}",
          file=sys.stderr, flush=True)

    dom = max(stages, key=lambda s: stages[s]["ms"])
    d = stages[dom]
    per_launch_ms = d["ms"] / max(d["launches"], 1)
    per_launch_bytes = d["bytes"] / max(d["launches"], 1)
    achieved = per_launch_bytes / (per_launch_ms * 1e-3) / 1e9 \
        if per_launch_ms > 0 else 0.0
    alg_total = sum(v["bytes"] for v in stages.values()) / args.steps
    roofline = {
        "bound": "hbm", "kernel": dom, "achieved": round(achieved, 2),
        "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": None,
        "launch_ms": round(per_launch_ms, 5),
        "alg_bytes_per_launch": per_launch_bytes,
        "step_alg_bytes": alg_total,
        "step_alg_frac": round(alg_total / (ms_per_step * 1e-3) / 1e9 /
                               HBM_PEAK_GBS, 5),
    }
    split = {s: round(v["ms"] / args.steps, 4) for s, v in stages.items()}

    out = {
        "metric": "points/sec partitioned (kNN+merge) on 3M-pt tile",
        "value": round(value, 1), "unit": "points/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"{sc.name}: synthetic driving tile, "
                               f"{sc.n} points, D={sc.d}, k={sc.k}, "
                               f"lambda ladder {sc.lambdas}",
                   "n_points": sc.n, "d": sc.d, "k": sc.k,
                   "lambdas": sc.lambdas},
        "roofline": roofline,
        "stage_ms_per_step": split,
        "n_comp": [int(x) for x in n_comp],
    }
    if not args.no_cpu:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(sc, min(args.cpu_points, sc.n))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
