"""Write the expected plan-search results of the five named instances.

Every stored value comes from the CPU oracle (oracle/tangram_oracle.c) and
nothing else: counts, the surviving set (count, SHA-256 of the ascending int64
little-endian index list, and its first/last entries), the per-b (P*, F*, T)
table, the chosen plan, the plan and per-b (P*, bound, F, T) table of the
composition with the step-(4) relaxation, for instances of at most 16 islands
the plan and per-b (P*, F*, T) table of the composition over every island
order, and a seeded sample of per-candidate scores.

With --imbalance the same records (survivors, plan, per-b table) are
written for the instance with imbalance pruning at IMBALANCE_EPS, to
<name>_imbalance.json; with --extended for the instance with the extended
config space (context parallelism {1, 2, 4}, recomputation, offloading), to
<name>_extended.json, plus a seeded sample of candidate scores.

Run from the repository root:
    python -m tests.golden.make_golden [--imbalance | --extended] [names...]
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

from oracle.oracle import Oracle, build  # noqa: E402
from workloads import CONFIG_NAMES, load_instance  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
N_SAMPLE = 4096
IMBALANCE_EPS = 1.0


def sample_indices(N, NS, seed=1234):
    """Seeded sample of candidate indices: random picks plus both ends of the
    space and of the first and last config rows."""
    rng = np.random.default_rng(seed)
    picks = set(int(x) for x in rng.integers(0, N, size=min(N_SAMPLE, N)))
    for x in (0, 1, NS - 1, NS, N - NS, N - 2, N - 1):
        if 0 <= x < N:
            picks.add(x)
    return np.array(sorted(picks), dtype=np.int64)


def survivors_digest(s):
    return hashlib.sha256(np.ascontiguousarray(s, dtype="<i8").tobytes()).hexdigest()


def golden(name):
    inst = load_instance(name)
    o = Oracle(inst)
    t0 = time.time()
    surv = o.prune()
    t1 = time.time()
    st, plan, per_b = o.compose(surv)
    t2 = time.time()
    rst, rplan, rper_b = o.compose_relaxed(surv)
    t3 = time.time()
    all_orders = None
    if o.K <= 16:
        ast, aplan, aper_b = o.compose_all_orders(surv)
        all_orders = {"status": ast, "plan": aplan, "per_b": [[float(v) for v in row] for row in aper_b]}
    t4 = time.time()
    idx = sample_indices(o.N, o.NS)
    cost, dmax = o.score_list(idx)
    return {
        "name": name,
        "counts": {"NS": o.NS, "n_configs": o.n_configs, "N": o.N, "n_b": o.n_b},
        "bvalues": o.bvalues,
        "survivors": {"count": int(len(surv)), "sha256": survivors_digest(surv),
                      "head": [int(x) for x in surv[:16]], "tail": [int(x) for x in surv[-16:]]},
        "status": st,
        "plan": plan,
        "per_b": [[float(v) for v in row] for row in per_b],
        "relaxed": {"status": rst, "plan": rplan,
                    "per_b": [[float(v) for v in row] for row in rper_b]},
        "all_orders": all_orders,
        "sample": {"idx": [int(x) for x in idx], "cost": [float(x) for x in cost],
                   "dmax": [int(x) for x in dmax]},
        "oracle_seconds": {"prune": round(t1 - t0, 3), "compose": round(t2 - t1, 3),
                           "compose_relaxed": round(t3 - t2, 3), "compose_all_orders": round(t4 - t3, 3)},
    }


def golden_imbalance(name):
    inst = load_instance(name)
    inst["space"]["imbalance_eps"] = IMBALANCE_EPS
    o = Oracle(inst)
    t0 = time.time()
    surv = o.prune()
    t1 = time.time()
    st, plan, per_b = o.compose(surv)
    t2 = time.time()
    return {
        "name": name, "imbalance_eps": IMBALANCE_EPS,
        "survivors": {"count": int(len(surv)), "sha256": survivors_digest(surv),
                      "head": [int(x) for x in surv[:16]], "tail": [int(x) for x in surv[-16:]]},
        "status": st, "plan": plan, "per_b": [[float(v) for v in row] for row in per_b],
        "oracle_seconds": {"prune": round(t1 - t0, 3), "compose": round(t2 - t1, 3)},
    }


def golden_extended(name):
    from workloads import extended
    inst = extended(load_instance(name))
    o = Oracle(inst)
    t0 = time.time()
    surv = o.prune()
    t1 = time.time()
    st, plan, per_b = o.compose(surv)
    t2 = time.time()
    idx = sample_indices(o.N, o.NS)
    cost, dmax = o.score_list(idx)
    return {
        "name": name, "space": "extended",
        "counts": {"NS": o.NS, "n_configs": o.n_configs, "N": o.N, "n_b": o.n_b},
        "survivors": {"count": int(len(surv)), "sha256": survivors_digest(surv),
                      "head": [int(x) for x in surv[:16]], "tail": [int(x) for x in surv[-16:]]},
        "status": st, "plan": plan, "per_b": [[float(v) for v in row] for row in per_b],
        "sample": {"idx": [int(x) for x in idx], "cost": [float(x) for x in cost],
                   "dmax": [int(x) for x in dmax]},
        "oracle_seconds": {"prune": round(t1 - t0, 3), "compose": round(t2 - t1, 3)},
    }


def path(name):
    return os.path.join(HERE, f"{name}.json")


def load(name):
    with open(path(name)) as fh:
        return json.load(fh)


def main(names):
    build(force=False)
    if names and names[0] == "--extended":
        for name in names[1:] or list(CONFIG_NAMES):
            g = golden_extended(name)
            with open(path(name + "_extended"), "w") as fh:
                json.dump(g, fh, indent=1, sort_keys=True)
                fh.write("\n")
            print(name, "extended", g["counts"], "survivors", g["survivors"]["count"], "T", g["plan"]["T"],
                  g["oracle_seconds"], flush=True)
        return
    if names and names[0] == "--imbalance":
        for name in names[1:] or list(CONFIG_NAMES):
            g = golden_imbalance(name)
            with open(path(name + "_imbalance"), "w") as fh:
                json.dump(g, fh, indent=1, sort_keys=True)
                fh.write("\n")
            print(name, "imbalance", "survivors", g["survivors"]["count"], "T", g["plan"]["T"],
                  g["oracle_seconds"], flush=True)
        return
    for name in names:
        g = golden(name)
        with open(path(name), "w") as fh:
            json.dump(g, fh, indent=1, sort_keys=True)
            fh.write("\n")
        print(name, g["counts"], "survivors", g["survivors"]["count"], "T", g["plan"]["T"],
              g["oracle_seconds"], flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or list(CONFIG_NAMES))
