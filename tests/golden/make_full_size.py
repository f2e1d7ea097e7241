"""Writes tests/golden/full_size.json: the oracle's results on whole
workloads too large to recompute inside a GPU test run.

For each case the CPU oracle (``oracle/``, single thread) runs on the seeded
scene (``paper_2512_00385_amd.scenes``, draws only) and the script stores
- for kNN cases: the SHA-256 of the neighbour table (int32, row-major) and of
  the squared distances (fp32), plus a few rows in clear;
- for partition cases: per level the SHA-256 of the canonical labels
  (int32), the superpoint count and the energy of Eq. gmpp, and the round
  count of the oracle's log.

Nothing here comes from the HIP path.  Run from the repository root:
    python tests/golden/make_full_size.py [case ...]
(about an hour of CPU for every case; the aerial tile dominates).
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(
    os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2512_00385_amd import scenes  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)),
                   "full_size.json")

# (kind, workload, link)
CASES = {
    "knn:room-1m": ("knn", "room-1m", False),
    "knn:driving-3m": ("knn", "driving-3m", False),
    "knn:aerial-10m": ("knn", "aerial-10m", False),
    "partition:aerial-10m": ("partition", "aerial-10m", False),
    "partition:aerial-10m-paper": ("partition", "aerial-10m-paper", False),
    "partition:aerial-10m-paper+link": ("partition", "aerial-10m-paper",
                                        True),
}


def sha(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def run(case):
    kind, name, link = CASES[case]
    sc = scenes.load(name)
    t0 = time.time()
    if kind == "knn":
        nbr, d2 = oracle.knn(sc.xyz, sc.k)
        rows = [0, sc.n // 2, sc.n - 1]
        return {"n": sc.n, "k": sc.k, "scene": sc.digest(),
                "nbr_sha256": sha(nbr.astype("<i4")),
                "d2_sha256": sha(d2.astype("<f4")),
                "rows": {str(r): nbr[r].tolist() for r in rows},
                "oracle_s": round(time.time() - t0, 1)}
    labels, nc, en, log = oracle.partition(sc.xyz, sc.emb, sc.k, sc.lambdas,
                                           sc.min_size, want_log=True,
                                           link=link)
    rounds = [sum(1 for r in log if r["level"] == l)
              for l in range(len(sc.lambdas))]
    return {"n": sc.n, "d": sc.d, "k": sc.k, "scene": sc.digest(),
            "lambdas": sc.lambdas, "min_size": sc.min_size, "link": link,
            "n_comp": [int(x) for x in nc],
            "energy": [float(x) for x in en],
            "labels_sha256": [sha(labels[l].astype("<i4"))
                              for l in range(labels.shape[0])],
            "rounds_per_level": rounds,
            "oracle_s": round(time.time() - t0, 1)}


def main(argv):
    todo = argv or list(CASES)
    data = {}
    if os.path.exists(OUT):
        with open(OUT) as fh:
            data = json.load(fh)
    for case in todo:
        print(f"[golden] {case}", flush=True)
        data[case] = run(case)
        print(f"[golden] {case}: {data[case]}", flush=True)
        with open(OUT + ".tmp", "w") as fh:
            json.dump(data, fh, indent=1, sort_keys=True)
        os.replace(OUT + ".tmp", OUT)


if __name__ == "__main__":
    main(sys.argv[1:])
