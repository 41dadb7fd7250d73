"""Benchmark of the plan search on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload large]
                    [--space named|extended] [--other-steps 10]

A step is one whole plan search over a resident instance: score every
model-slice/island/config candidate (tg_score_pairs), prune to the surviving
set (tg_prune), compose the pipeline (tg_compose_pipeline, plan returned to
the host).  The instance's tables and the score buffers are on the device
before the timed region.  Prints one JSON line:
  value        candidates per second of whole plan search: N * steps / the
               host-clock time of the K timed steps (score + prune + compose,
               plan on the host); `score_kernel_pairs_per_s` is N over the
               score call alone
  ms_per_step  end-to-end plan-search milliseconds (host clock, mean of the K
               steps); `ms_per_step_median` the median of the per-step HIP
               event spans
  roofline     the score kernel: algorithmic bytes (8 B cost + 1 B depth per
               candidate) per launch / its mean HIP-event duration, against
               the 8 TB/s HBM peak; `write_ceiling` is what torch's fill_
               reaches over as many bytes (at most 16 GiB) in the same run
  cpu_baseline the CPU oracle, single thread, on the same workload, whole:
               score every candidate, prune, compose, in the same run on the
               GPU machine's host (CPU model, logical CPUs, the all-cores
               projection); its surviving set and plan are compared with the
               GPU's bit for bit.  `workloads` times the oracle (median of 3)
               on each smaller cluster and compares its plan with the GPU's
  workloads    the same plan search timed on each of the five synthetic
               clusters (fewer steps), after the main measurement; for those
               with at most 16 islands also the composition over every
               island order (tg_compose_pipeline_all_orders)
  redundancy_pruned  the same plan search with redundancy pruning: each
               (config, slice class) scored once, survivors expanded to slices
  island_construction  tg_build_islands on node clusters of 1024 and 4096
               nodes (the oracle beside it at 1024)
--space extended adds context parallelism {1,2,4}, recomputation and
offloading to the chosen workload's config space.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
SCORE_BYTES_PER_CANDIDATE = 9  # 8-byte cost + 1-byte depth written; inputs stay in registers/L2
METRIC = "slice/island pairs scored/sec; end-to-end plan-search seconds (1 GPU)"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "score_kernel_large_traffic.txt")
SCORE_SOURCES = [os.path.join(ROOT, "paper_2606_16907_amd", "csrc", f) for f in ("score.hip", "tg_device.h")]

WORKLOADS = {
    "large": "128-layer dense decoder (h 12288, FFN 49152 GeLU, 96 heads, s 8192, global batch "
             "4096) on 128 islands of 8-64 GPUs, 5 GPU types, 3-level fabric 400/100/25 GB/s; "
             "TP{1,2,4,8} x DP 1..n/tp x ZeRO 0-3 x MB{1,2,4,8}",
    "tiny": "8-layer dense (h 1024, 16 heads, s 2048, global batch 64) on 2 islands of 4 GPUs",
    "dense8b": "32-layer dense (h 4096, FFN 14336 SwiGLU, GQA 32/8, s 4096, global batch 512) "
               "on 4 islands of 8 GPUs",
    "dense70b": "80-layer dense (h 8192, FFN 28672 SwiGLU, GQA 64/8, s 8192, global batch 1024) "
                "on 16 islands of 8-64 GPUs",
    "moe": "48-layer MoE (h 6144, 64 experts top-2, expert FFN 4096, s 4096, global batch 2048) "
           "on 32 islands of 8-32 GPUs, EP{1,2,4,8,16}",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="large", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-islands", type=int, default=0,
                    help="time the CPU baseline on the workload's first islands only (0: the whole "
                         "workload)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-baseline leg")
    ap.add_argument("--relaxed-steps", type=int, default=5,
                    help="also time the composition with the step-(4) relaxation this many times "
                         "(0 skips it); reported beside the main metric, not in it")
    ap.add_argument("--space", default="named", choices=("named", "extended"),
                    help="config space: the workload's own, or extended with context parallelism "
                         "{1,2,4}, recomputation and offloading")
    ap.add_argument("--imbalance-eps", type=float, default=0.0,
                    help="imbalance-pruning tolerance for every workload (0: off)")
    ap.add_argument("--other-steps", type=int, default=10,
                    help="timed plan searches per workload in the five-workload table (0 skips it)")
    ap.add_argument("--redundancy-steps", type=int, default=10,
                    help="also time the plan search with redundancy pruning (scores per slice class) this "
                         "many times (0 skips it); reported beside the main metric")
    ap.add_argument("--island-nodes", type=int, nargs="*", default=[1024, 4096],
                    help="time island construction (tg_build_islands) on generated node clusters of "
                         "these sizes (none: skip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="before the steps, copy BYTES between two device buffers (a plain copy of "
                         "known size that scales profiler byte counters)")
    return ap.parse_args()


def host_info():
    """The CPU the oracle runs on: model name, logical CPUs of the machine and
    of this process's affinity set."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count() or 1
    return {"cpu_model": model, "nproc": os.cpu_count() or 1, "affinity_cpus": usable, "cores_used": 1}


def oracle_search(o):
    """One whole plan search by the oracle: score every candidate, prune,
    compose.  Returns (seconds per phase, survivors, status, plan)."""
    t0 = time.perf_counter()
    cost, dmax = o.score()
    t1 = time.perf_counter()
    del cost, dmax
    t1b = time.perf_counter()
    surv = o.prune()
    t2 = time.perf_counter()
    st, plan, _ = o.compose(surv)
    t3 = time.perf_counter()
    return {"score_s": t1 - t0, "prune_s": t2 - t1b, "compose_s": t3 - t2}, surv, st, plan


def same_plan(gpu_status, gpu_plan, st, plan):
    """The oracle's plan equals the GPU's: status, b, m, S, P, F, T bit for
    bit and every stage field."""
    if gpu_status != st:
        return False
    if st != 0:
        return True
    if any(gpu_plan[f] != plan[f] for f in ("b", "m", "S", "P", "F", "T")):
        return False
    return all(all(a[f] == b[f] for f in a) for a, b in zip(gpu_plan["stages"], plan["stages"]))


def cpu_baseline(inst, n_islands, gpu):
    """The oracle, as it stands, on the workload (or, with n_islands, on its
    first islands only): score every candidate, prune, compose, one thread,
    timed once (the whole 128-island search takes tens of seconds).  `gpu`
    holds the GPU's survivors digest, plan and ms per step from this run."""
    import hashlib
    import numpy as np
    from oracle.oracle import Oracle
    K = len(inst["island_order"])
    whole = n_islands <= 0 or n_islands >= K
    sub = inst
    if not whole:
        sub = dict(inst)
        keep = list(range(n_islands))
        sub["islands"] = {f: [v[k] for k in keep] for f, v in inst["islands"].items()}
        sub["inter_bw"] = [[inst["inter_bw"][a][b] for b in keep] for a in keep]
        sub["island_order"] = [k for k in inst["island_order"] if k < n_islands]
    print(f"bench: CPU baseline, the oracle on {'the whole workload' if whole else f'{n_islands} islands'}",
          file=sys.stderr, flush=True)
    o = Oracle(sub)
    ph, surv, st, plan = oracle_search(o)
    el = sum(ph.values())
    host = host_info()
    out = {"value": o.N / el, "unit": "pairs/s", "cores": 1, "kind": "oracle",
           "sample": (f"the whole workload ({K} islands, N={o.N} candidates)" if whole else
                      f"same workload on its first {n_islands} of {K} islands (N={o.N} candidates)")
                     + ": score every candidate, prune, compose; single thread, timed once",
           "seconds": round(el, 3), "score_s": round(ph["score_s"], 3), "prune_s": round(ph["prune_s"], 3),
           "compose_s": round(ph["compose_s"], 3), "candidates": o.N, "survivors": int(len(surv)),
           "plan_status": st, "host": host,
           "all_cores_projection_s": el / host["affinity_cpus"]}
    if whole and gpu is not None:
        digest = hashlib.sha256(np.ascontiguousarray(surv, dtype=np.int64).tobytes()).hexdigest()
        out["same_survivors_as_gpu"] = bool(digest == gpu["survivors_sha256"] and len(surv) == gpu["survivors"])
        out["same_plan_as_gpu"] = same_plan(gpu["status"], gpu["plan"], st, plan)
        out["gpu_speedup"] = el / (gpu["ms_per_step"] / 1e3)
        out["gpu_speedup_vs_all_cores_projection"] = out["all_cores_projection_s"] / (gpu["ms_per_step"] / 1e3)
    return out


def cpu_baseline_workloads(load_instance, space, imbalance_eps, gpu_rows, skip, reps=3):
    """The oracle on each smaller synthetic cluster, whole: score every
    candidate, prune, compose (single thread, median of `reps` runs), and
    whether its surviving set and plan equal the GPU's from the same run."""
    from oracle.oracle import Oracle
    out = {}
    for name in ("tiny", "dense8b", "dense70b", "moe"):
        if name == skip:
            continue
        inst = load_instance(name)
        if space == "extended":
            from workloads import extended
            inst = extended(inst)
        inst["space"]["imbalance_eps"] = imbalance_eps
        o = Oracle(inst)
        runs = []
        for _ in range(reps):
            ph, surv, st, plan = oracle_search(o)
            runs.append((sum(ph.values()), ph))
        runs.sort(key=lambda r: r[0])
        el, ph = runs[len(runs) // 2]
        row = {"candidates": o.N, "seconds": round(el, 4), "runs": reps, "pairs_per_s": o.N / el,
               "score_s": round(ph["score_s"], 4), "prune_s": round(ph["prune_s"], 4),
               "compose_s": round(ph["compose_s"], 4), "survivors": int(len(surv)), "plan_status": st}
        g = (gpu_rows or {}).get(name)
        if g is not None:
            row["gpu_speedup"] = el / (g["ms_per_step"] / 1e3)
            row["same_plan_as_gpu"] = bool(g["survivors"] == len(surv) and same_plan(
                g["plan"]["status"], g["plan_full"], st, plan))
        out[name] = row
    return out


def write_ceiling(torch, nbytes, reps=5):
    """GB/s of torch's fill_ over a buffer of the score arrays' size: the
    practical ceiling of a kernel that only writes that many bytes."""
    buf = torch.empty(max(nbytes // 8, 1), dtype=torch.float64, device="cuda")
    stream = torch.cuda.current_stream()
    buf.fill_(1.0)
    ts = []
    for r in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        buf.fill_(float(r))
        b.record(stream)
        b.synchronize()
        ts.append(a.elapsed_time(b))
    ts.sort()
    gbs = buf.numel() * 8 / (ts[len(ts) // 2] / 1e3) / 1e9
    del buf
    torch.cuda.empty_cache()
    return gbs


def time_search(torch, T, inst, steps, warmup, relaxed_steps=0):
    """Create the problem, size the buffers (untimed), then run `warmup` and
    `steps` whole plan searches (score, prune, compose with the plan on the
    host), with HIP events between the three calls of every timed step."""
    t_create = time.perf_counter()
    p = T.Problem(inst)
    torch.cuda.synchronize()
    t_create = time.perf_counter() - t_create
    N = p.N
    cost = torch.empty(N, dtype=torch.float64, device="cuda")
    dmax = torch.empty(N, dtype=torch.uint8, device="cuda")
    pws = p.prune_workspace()

    # size the survivor buffer and composition workspace once (untimed)
    p.tg_score_pairs(0, N, cost, dmax)
    surv0 = p.tg_prune(cost, dmax, workspace=pws)
    n_surv = int(surv0.numel())
    surv_buf = torch.empty(max(n_surv, 1), dtype=torch.int64, device="cuda")
    cws = p.compose_workspace(n_surv)
    del surv0

    stream = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]

    def step(e=None):
        if e:
            e[0].record(stream)
        p.tg_score_pairs(0, N, cost, dmax)
        if e:
            e[1].record(stream)
        s = p.tg_prune(cost, dmax, survivors=surv_buf, workspace=pws)
        if e:
            e[2].record(stream)
        st, plan = p.tg_compose_pipeline(s, cost, dmax, workspace=cws)
        if e:
            e[3].record(stream)
        return st, plan, s

    for _ in range(warmup):
        st, plan, s = step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        st, plan, s = step(ev[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    orders = None
    if p.K <= 16 and steps > 0:
        # composition over every island order on the same survivors (host
        # clock around each call: it synchronises once)
        ows = p.compose_all_orders_workspace(int(s.numel()))
        p.tg_compose_pipeline_all_orders(s, cost, dmax, workspace=ows)  # warm-up
        torch.cuda.synchronize()
        times = []
        for _ in range(min(steps, 5)):
            t1 = time.perf_counter()
            ost, oplan = p.tg_compose_pipeline_all_orders(s, cost, dmax, workspace=ows)
            times.append((time.perf_counter() - t1) * 1e3)
        times.sort()
        orders = {"compose_ms_median": times[len(times) // 2], "status": ost, "b": oplan["b"],
                  "stages": oplan["S"], "T": oplan["T"],
                  "islands": [x["island"] for x in oplan["stages"]]}
        del ows
    relaxed = None
    if relaxed_steps > 0 and steps > 0:
        # the composition with the step-(4) relaxation on the same survivors
        # (host clock around each call: it synchronises per search round)
        rws = p.compose_relaxed_workspace(int(s.numel()))
        p.tg_compose_pipeline_relaxed(s, cost, dmax, workspace=rws)  # warm-up
        torch.cuda.synchronize()
        times = []
        for _ in range(relaxed_steps):
            t1 = time.perf_counter()
            rst, rplan = p.tg_compose_pipeline_relaxed(s, cost, dmax, workspace=rws)
            times.append((time.perf_counter() - t1) * 1e3)
        times.sort()
        relaxed = {"compose_ms_median": times[len(times) // 2], "status": rst, "b": rplan["b"],
                   "stages": rplan["S"], "T": rplan["T"]}
        del rws
    return {"problem": p, "all_orders": orders, "relaxed": relaxed, "N": N, "cost": cost, "dmax": dmax, "survivors": s, "status": st,
            "plan": plan, "elapsed": elapsed, "create_s": t_create,
            "score_ms": [ev[k][0].elapsed_time(ev[k][1]) for k in range(steps)],
            "prune_ms": [ev[k][1].elapsed_time(ev[k][2]) for k in range(steps)],
            "compose_ms": [ev[k][2].elapsed_time(ev[k][3]) for k in range(steps)]}


def five_workloads(torch, T, load_instance, space, steps, main_name, main_row, imbalance_eps=0.0):
    """The plan search on each synthetic cluster: candidates, survivors,
    milliseconds per whole search, candidates per second, the score kernel's
    share of the HBM peak, the chosen plan's b, stages and T."""
    out = {}
    for name in ("tiny", "dense8b", "dense70b", "moe", "large"):
        if name == main_name:
            out[name] = main_row
            continue
        inst = load_instance(name)
        if space == "extended":
            from workloads import extended
            inst = extended(inst)
        inst["space"]["imbalance_eps"] = imbalance_eps
        run = time_search(torch, T, inst, steps, 2, relaxed_steps=min(steps, 5))
        out[name] = workload_row(run, steps)
        del run
        torch.cuda.empty_cache()
    return out


def workload_row(run, steps):
    sc = sum(run["score_ms"]) / steps
    return {"candidates": run["N"], "survivors": int(run["survivors"].numel()),
            "ms_per_step": run["elapsed"] / steps * 1e3,
            "pairs_per_s": run["N"] * steps / run["elapsed"],
            "score_ms": sc, "prune_ms": sum(run["prune_ms"]) / steps,
            "compose_ms": sum(run["compose_ms"]) / steps,
            "score_hbm_frac": SCORE_BYTES_PER_CANDIDATE * run["N"] / (sc / 1e3) / 1e9 / HBM_PEAK_GBS,
            "plan": {"status": run["status"], "b": run["plan"]["b"], "stages": run["plan"]["S"],
                     "T": run["plan"]["T"]},
            "plan_full": run["plan"],
            "all_orders_compose": run["all_orders"],
            "relaxed_compose": run.get("relaxed")}


def redundancy_search(torch, T, p, steps, order=None):
    """The plan search with redundancy pruning on a created problem: score
    each (config, slice class) once, the surviving set from class scores,
    composition reading them; HIP events between the three calls."""
    nc = p.n_configs * p.NC
    cost = torch.empty(max(nc, 1), dtype=torch.float64, device="cuda")
    dmax = torch.empty(max(nc, 1), dtype=torch.uint8, device="cuda")
    pws = p.prune_classes_workspace()
    p.tg_score_classes(0, nc, cost, dmax)
    s0 = p.tg_prune_classes(cost, dmax, workspace=pws)
    surv_buf = torch.empty(max(int(s0.numel()), 1), dtype=torch.int64, device="cuda")
    cws = p.compose_workspace(int(s0.numel()))
    stream = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for k in range(-2, steps):
        e = ev[k] if k >= 0 else None
        if e:
            e[0].record(stream)
        p.tg_score_classes(0, nc, cost, dmax)
        if e:
            e[1].record(stream)
        s = p.tg_prune_classes(cost, dmax, survivors=surv_buf, workspace=pws)
        if e:
            e[2].record(stream)
        st, plan = p.tg_compose_pipeline_classes(s, cost, dmax, workspace=cws)
        if e:
            e[3].record(stream)
        if k == -1:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    mean = lambda a, b: sum(ev[k][a].elapsed_time(ev[k][b]) for k in range(steps)) / steps
    return {"slice_classes": p.NC, "class_candidates": nc, "survivors": int(s.numel()),
            "ms_per_step": elapsed / steps * 1e3,
            "breakdown_ms": {"score_classes": mean(0, 1), "prune_classes": mean(1, 2), "compose": mean(2, 3)},
            "plan": {"status": st, "b": plan["b"], "stages": plan["S"], "T": plan["T"]}}


def island_construction(T, sizes, with_cpu):
    """Island construction on generated node clusters (GPU types bought in
    runs on a leaf/pod fabric): milliseconds per call (host arrays in and
    out, so the node bandwidth matrix upload is inside), islands found, and
    the oracle on the clusters of at most 1024 nodes."""
    from workloads import node_cluster
    out = []
    for n in sizes:
        cl = node_cluster(11, n)
        ws = None
        r = T.build_islands(cl)  # warm-up
        times = []
        for _ in range(3):
            t0 = time.perf_counter()
            r = T.build_islands(cl, workspace=ws)
            times.append((time.perf_counter() - t0) * 1e3)
        times.sort()
        row = {"nodes": n, "islands": r["K"], "gpu_ms_median": times[1]}
        if with_cpu and n <= 1024:
            from oracle.oracle import build_islands
            t0 = time.perf_counter()
            o = build_islands(cl)
            row["oracle_s"] = round(time.perf_counter() - t0, 3)
            row["oracle_cores"] = 1
            row["same_islands"] = o["island_of"] == r["island_of"]
        out.append(row)
    return out


def score_source_digest():
    import hashlib
    h = hashlib.sha256()
    for f in SCORE_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload, N):
    """HBM bytes per score-kernel launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known size), or None
    when it was taken on another workload or the kernel source has changed."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    with open(TRAFFIC_FILE) as fh:
        for line in fh:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    if kv.get("workload") != workload or kv.get("candidates") != str(N):
        return None
    if kv.get("score_source_sha256") != score_source_digest():
        return None
    return float(kv["hbm_bytes_per_launch"])


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the plan search is a "
              f"single-GPU path", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_16907_amd import tangram as T
    from workloads import load_instance

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    inst = load_instance(args.workload)
    if args.space == "extended":
        from workloads import extended
        inst = extended(inst)
    inst["space"]["imbalance_eps"] = args.imbalance_eps
    if args.copy_calibration > 0:
        a = torch.ones(args.copy_calibration // 8, dtype=torch.float64, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    run = time_search(torch, T, inst, args.steps, args.warmup)
    p, N, s, st, plan = run["problem"], run["N"], run["survivors"], run["status"], run["plan"]
    cost, dmax = run["cost"], run["dmax"]
    elapsed, t_create = run["elapsed"], run["create_s"]
    score_ms, prune_ms, compose_ms = run["score_ms"], run["prune_ms"], run["compose_ms"]

    mean = lambda xs: sum(xs) / len(xs)
    # composition with the step-(4) relaxation, timed after the main loop on
    # the same survivors (host clock around the call: it synchronises per round)
    relaxed = None
    if args.relaxed_steps > 0:
        rws = p.compose_relaxed_workspace(int(s.numel()))
        p.tg_compose_pipeline_relaxed(s, cost, dmax, workspace=rws)  # warm-up
        torch.cuda.synchronize()
        times = []
        for _ in range(args.relaxed_steps):
            t1 = time.perf_counter()
            rst, rplan = p.tg_compose_pipeline_relaxed(s, cost, dmax, workspace=rws)
            times.append((time.perf_counter() - t1) * 1e3)
        times.sort()
        relaxed = {"compose_ms_median": times[len(times) // 2], "status": rst, "b": rplan["b"],
                   "stages": rplan["S"], "P": rplan["P"], "T": rplan["T"]}
        del rws
    score_s = mean(score_ms) / 1e3
    achieved = SCORE_BYTES_PER_CANDIDATE * N / score_s / 1e9
    step_ms = sorted(a + b + c for a, b, c in zip(score_ms, prune_ms, compose_ms))
    # what the CPU baseline compares with: the GPU's surviving set (digest) and plan
    import hashlib
    gpu_result = {"survivors": int(s.numel()), "status": st, "plan": plan,
                  "survivors_sha256": hashlib.sha256(s.cpu().numpy().astype("int64").tobytes()).hexdigest(),
                  "ms_per_step": elapsed / args.steps * 1e3}
    ceiling = write_ceiling(torch, min(SCORE_BYTES_PER_CANDIDATE * N, 16 << 30))
    traffic = measured_traffic(args.workload if args.space == "named" else args.workload + "+extended", N)
    if args.imbalance_eps > 0:
        traffic = None  # the counters were taken without imbalance pruning
    out = {
        "metric": METRIC,
        "value": N * args.steps / elapsed,
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {WORKLOADS[args.workload]}"
                               + ("" if args.space == "named" else
                                  "; extended with CP{1,2,4} x recomputation x offloading")
                               + ("" if args.imbalance_eps == 0 else
                                  f"; imbalance pruning eps {args.imbalance_eps}"),
                   "candidates": N, "survivors": int(s.numel()), "islands": p.K, "layers": p.L,
                   "plan": {"status": st, "b": plan["b"], "stages": plan["S"], "T": plan["T"]}},
        "roofline": {"kernel": "score_kernel", "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic,
                     "write_ceiling": {"what": "torch fill_ of as many bytes (at most 16 GiB), same run", "achieved": ceiling,
                                       "frac": achieved / ceiling}},
        "ms_per_step_median": step_ms[len(step_ms) // 2],
        "breakdown_ms": {"score": mean(score_ms), "prune": mean(prune_ms),
                         "compose": mean(compose_ms), "create": t_create * 1e3},
        "breakdown_ms_median": {k: sorted(v)[len(v) // 2] for k, v in
                                (("score", score_ms), ("prune", prune_ms), ("compose", compose_ms))},
        "score_kernel_pairs_per_s": N / score_s,
        "relaxed_compose": relaxed,
        "end_to_end_s": elapsed / args.steps,
    }
    if args.other_steps > 0:
        main_row = workload_row(run, args.steps)
        main_row["relaxed_compose"] = relaxed
        del run, cost, dmax, s
        torch.cuda.empty_cache()
        out["workloads"] = five_workloads(torch, T, load_instance, args.space, args.other_steps,
                                          args.workload, main_row, args.imbalance_eps)
    if args.redundancy_steps > 0:
        out["redundancy_pruned"] = redundancy_search(torch, T, p, args.redundancy_steps)
    if args.island_nodes:
        out["island_construction"] = island_construction(T, args.island_nodes, not args.no_cpu)
    if not args.no_cpu:
        cb = cpu_baseline(inst, args.cpu_islands, gpu_result)
        cb["workloads"] = cpu_baseline_workloads(load_instance, args.space, args.imbalance_eps,
                                                 out.get("workloads"), args.workload)
        out["cpu_baseline"] = cb
    for row in (out.get("workloads") or {}).values():
        row.pop("plan_full", None)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
