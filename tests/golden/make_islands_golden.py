"""Write the oracle's island construction of the largest node cluster the
library takes (4096 nodes) as digests: the per-node island list and the
island-to-island bandwidth matrix (little-endian int32 / float64 bytes, SHA-256),
the island count and the island attributes.

Run from the repository root:  python -m tests.golden.make_islands_golden
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle.oracle import build, build_islands  # noqa: E402
from workloads import node_cluster  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
CASE = {"seed": 11, "n_nodes": 4096}
PATH = os.path.join(HERE, "islands_4096.json")


def digests(r):
    isl = np.ascontiguousarray(np.array(r["island_of"], dtype="<i4")).tobytes()
    e = np.ascontiguousarray(np.array(r["inter_bw"], dtype="<f8")).tobytes()
    return hashlib.sha256(isl).hexdigest(), hashlib.sha256(e).hexdigest()


def main():
    build(force=False)
    cl = node_cluster(CASE["seed"], CASE["n_nodes"])
    t = time.time()
    r = build_islands(cl)
    d_isl, d_e = digests(r)
    out = dict(CASE, K=r["K"], island_of_sha256=d_isl, inter_bw_sha256=d_e, islands=r["islands"],
               oracle_seconds=round(time.time() - t, 1))
    with open(PATH, "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)
        fh.write("\n")
    print(CASE, "K", r["K"], out["oracle_seconds"], "s")


if __name__ == "__main__":
    main()
