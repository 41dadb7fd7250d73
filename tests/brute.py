"""Exhaustive reference searches used to pin the oracle on tiny instances.

These walk every pipeline plan (micro-batch size b, ordered subsequence of
islands, cut set, per-stage config) with no dynamic programming and no pruning:
the objective of Sec. 5.2 evaluated plan by plan.  They take the per-candidate
(cost, d_max) scores as given; the scores are pinned separately by closed forms.
"""
from __future__ import annotations

import itertools
import math


def candidate_table(orc):
    """Every candidate of an oracle instance: list of dicts with its tuple,
    group key and score."""
    cost, dmax = orc.score()
    B = orc.inst["space"]["global_batch"]
    rows = []
    for idx in range(orc.N):
        t = orc.decode(idx)
        t["idx"] = idx
        t["b"] = t["dp"] * t["mb"]
        t["compatible"] = B % t["b"] == 0
        t["cost"] = float(cost[idx])
        t["dmax"] = int(dmax[idx])
        rows.append(t)
    return rows


def key(r):
    return (r["cost"], -r["dmax"], r["idx"])


def groups_of(rows):
    g = {}
    for r in rows:
        if r["compatible"]:
            g.setdefault((r["i"], r["j"], r["island"], r["b"]), []).append(r)
    return g


def survivors_by_reps(rows, K):
    """Union over groups and depths d = 1..K of rep(G, d), the least-key member
    whose d_max reaches d."""
    out = set()
    for members in groups_of(rows).values():
        for d in range(1, K + 1):
            fit = [r for r in members if r["dmax"] >= d]
            if fit:
                out.add(min(fit, key=key)["idx"])
    return sorted(out)


def survivors_by_dominance(rows):
    """p survives iff no member q of its group has key_q < key_p and
    d_max_q >= d_max_p (quadratic Pareto definition), and d_max_p >= 1."""
    out = []
    for members in groups_of(rows).values():
        for p in members:
            if p["dmax"] < 1:
                continue
            if not any(key(q) < key(p) and q["dmax"] >= p["dmax"] for q in members):
                out.append(p["idx"])
    return sorted(out)


def transfer(inst, b, j, ka, kb):
    """Activations forward plus gradients backward of one micro-batch across the
    boundary after layer j-1 (Sec. 5.2: stages exchange only activations)."""
    E = inst["inter_bw"][ka][kb]
    if E == 0.0:
        return math.inf
    return ((2.0 * float(b)) * float(inst["layers"]["out_act_bytes"][j - 1])) / E


def right_fold(f, x):
    acc = f[-1]
    for t in range(len(f) - 2, -1, -1):
        acc = f[t] + (x[t] + acc)
    return acc


def enumerate_plans(orc, rows, order=None, allowed=None):
    """Every feasible plan per b: dict b -> list of plans, each with its
    bottleneck P, fill F, lexicographic key (o_1, S, j_1, o_2, j_2, ...) and
    the chosen candidate per stage (the group's least-key member fitting at
    the stage's depth).

    `allowed`: optional set of candidate indices that may be used (default:
    every compatible candidate)."""
    inst = orc.inst
    if order is None:
        order = inst["island_order"]
    L, K = orc.L, orc.K
    B = inst["space"]["global_batch"]
    groups = groups_of(rows)

    def stage_choice(i, j, k, b, d):
        fit = [r for r in groups.get((i, j, k, b), [])
               if r["dmax"] >= d and (allowed is None or r["idx"] in allowed)]
        return min(fit, key=key) if fit else None

    out = {}
    for b in orc.bvalues:
        m = B // b
        plans = []
        for S in range(1, min(K, L) + 1):
            for posn in itertools.combinations(range(K), S):
                for cuts in itertools.combinations(range(1, L), S - 1):
                    bounds = (0,) + cuts + (L,)
                    f, x, picks = [], [], []
                    ok = True
                    for t in range(S):
                        pick = stage_choice(bounds[t], bounds[t + 1], order[posn[t]], b, S - t)
                        if pick is None:
                            ok = False
                            break
                        f.append(pick["cost"])
                        picks.append(pick)
                        if t < S - 1:
                            x.append(transfer(inst, b, bounds[t + 1], order[posn[t]],
                                              order[posn[t + 1]]))
                    if not ok:
                        continue
                    P = max(f + x)
                    if P == math.inf:
                        continue
                    F = right_fold(f, x)
                    pk = [posn[0], S]
                    for t in range(S - 1):
                        pk += [cuts[t], posn[t + 1]]
                    plans.append({"P": P, "F": F, "key": tuple(pk), "posn": posn, "cuts": cuts,
                                  "picks": picks, "f": f, "x": x, "b": b, "m": m, "L": L})
        out[b] = plans
    return out


def brute_force_compose(orc, rows, order=None, allowed=None):
    """Exhaustive composition with the objective of steps (1)-(3): per b the
    least bottleneck P*, then the least fill among plans attaining it.
    Returns per-b (P*, F*, T) and the optimum."""
    per_b = {}
    best = None
    for b, plans in enumerate_plans(orc, rows, order, allowed).items():
        if not plans:
            per_b[b] = (math.inf, math.inf, math.inf)
            continue
        m = plans[0]["m"]
        Pst = min(p["P"] for p in plans)
        at = [p for p in plans if p["P"] == Pst]
        Fst = min(p["F"] for p in at)
        opt = [p for p in at if p["F"] == Fst]
        T = (float(m - 1) * Pst) + Fst
        per_b[b] = (Pst, Fst, T)
        lexmin = min(opt, key=lambda p: p["key"])
        if best is None or T < best["T"]:
            best = {"T": T, "b": b, "P": Pst, "F": Fst, "lexmin": lexmin, "optimal": opt}
    return per_b, best


def brute_force_relaxed(orc, rows, order=None, allowed=None):
    """Exhaustive composition with the iteration time itself as the objective
    (step (4) relaxes the bottleneck bound until T stops improving): per b the
    least T = (m-1) * P + F over every plan; among plans attaining it the
    least P is the bound tau; the plan is then the least-fill plan among those
    whose every stage and link is within tau, lexicographically least key.
    Returns per-b (P*, tau, F, T) and the optimum."""
    per_b = {}
    best = None
    for b, plans in enumerate_plans(orc, rows, order, allowed).items():
        if not plans:
            per_b[b] = (math.inf, math.inf, math.inf, math.inf)
            continue
        m = plans[0]["m"]
        Pst = min(p["P"] for p in plans)
        for p in plans:
            p["T"] = (float(m - 1) * p["P"]) + p["F"]
        T = min(p["T"] for p in plans)
        tau = min(p["P"] for p in plans if p["T"] == T)
        within = [p for p in plans if p["P"] <= tau]
        F = min(p["F"] for p in within)
        opt = [p for p in within if p["F"] == F]
        assert (float(m - 1) * tau) + F == T
        per_b[b] = (Pst, tau, F, T)
        lexmin = min(opt, key=lambda p: p["key"])
        if best is None or T < best["T"]:
            best = {"T": T, "b": b, "P": tau, "F": F, "lexmin": lexmin, "optimal": opt}
    return per_b, best


def suffix_values(p):
    """Fill of each suffix of a plan (stage t .. S)."""
    f, x = p["f"], p["x"]
    return [right_fold(f[t:], x[t:]) for t in range(len(f))]


def plan_signature(plan_dict):
    """(positions..., cuts...) of an oracle/GPU plan dictionary, comparable with
    brute-force plans."""
    st = plan_dict["stages"]
    return tuple((s["island"], s["first_layer"], s["end_layer"], s["depth"], s["pair_index"])
                 for s in st)


def brute_signature(p, order):
    S = len(p["posn"])
    bounds = (0,) + p["cuts"] + (p["L"],)
    return tuple((order[p["posn"][t]], bounds[t], bounds[t + 1], S - t, p["picks"][t]["idx"])
                 for t in range(S))


def linear_partition_minmax(values, parts):
    """Least possible largest part sum when splitting `values` into at most
    `parts` contiguous non-empty runs (binary search on the answer + greedy)."""
    lo, hi = max(values), sum(values)
    while lo < hi:
        mid = (lo + hi) // 2
        runs, acc = 1, 0
        for v in values:
            if acc + v > mid:
                runs += 1
                acc = v
            else:
                acc += v
        if runs <= parts:
            hi = mid
        else:
            lo = mid + 1
    return lo


def enumerate_plans_all_orders(orc, rows, allowed=None):
    """Every feasible plan per b over every island subset and order: dict
    b -> list of plans with P, F and the key (k_1, S, set mask, j_1, k_2, j_2,
    ..., k_S) that orders ties (first island, stage count, set, then cuts and
    islands front to back)."""
    inst = orc.inst
    L, K = orc.L, orc.K
    B = inst["space"]["global_batch"]
    groups = groups_of(rows)

    def stage_choice(i, j, k, b, d):
        fit = [r for r in groups.get((i, j, k, b), [])
               if r["dmax"] >= d and (allowed is None or r["idx"] in allowed)]
        return min(fit, key=key) if fit else None

    out = {}
    for b in orc.bvalues:
        m = B // b
        plans = []
        for S in range(1, min(K, L) + 1):
            for isl in itertools.permutations(range(K), S):
                mask = sum(1 << k for k in isl)
                for cuts in itertools.combinations(range(1, L), S - 1):
                    bounds = (0,) + cuts + (L,)
                    f, x, picks = [], [], []
                    ok = True
                    for t in range(S):
                        pick = stage_choice(bounds[t], bounds[t + 1], isl[t], b, S - t)
                        if pick is None:
                            ok = False
                            break
                        f.append(pick["cost"])
                        picks.append(pick)
                        if t < S - 1:
                            x.append(transfer(inst, b, bounds[t + 1], isl[t], isl[t + 1]))
                    if not ok:
                        continue
                    P = max(f + x)
                    if P == math.inf:
                        continue
                    pk = [isl[0], S, mask]
                    for t in range(S - 1):
                        pk += [cuts[t], isl[t + 1]]
                    plans.append({"P": P, "F": right_fold(f, x), "key": tuple(pk), "islands": isl,
                                  "cuts": cuts, "picks": picks, "f": f, "x": x, "b": b, "m": m, "L": L})
        out[b] = plans
    return out


def brute_force_all_orders(orc, rows, allowed=None):
    """Exhaustive steps (1)-(3) over every island subset and order: per b the
    least bottleneck, then the least fill at it.  Returns per-b (P*, F*, T)
    and the optimum with its optimal plans and the least-key one."""
    per_b = {}
    best = None
    for b, plans in enumerate_plans_all_orders(orc, rows, allowed).items():
        if not plans:
            per_b[b] = (math.inf, math.inf, math.inf)
            continue
        m = plans[0]["m"]
        Pst = min(p["P"] for p in plans)
        at = [p for p in plans if p["P"] == Pst]
        Fst = min(p["F"] for p in at)
        opt = [p for p in at if p["F"] == Fst]
        T = (float(m - 1) * Pst) + Fst
        per_b[b] = (Pst, Fst, T)
        if best is None or T < best["T"]:
            best = {"T": T, "b": b, "P": Pst, "F": Fst, "lexmin": min(opt, key=lambda p: p["key"]),
                    "optimal": opt}
    return per_b, best


def all_orders_signature(p):
    S = len(p["islands"])
    bounds = (0,) + p["cuts"] + (p["L"],)
    return tuple((p["islands"][t], bounds[t], bounds[t + 1], S - t, p["picks"][t]["idx"]) for t in range(S))
