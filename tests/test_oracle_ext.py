"""Pins of the oracle's extra configuration dimensions: context parallelism
(cp), activation recomputation (rc) and activation offloading (of), the
parallelism and memory-saving techniques of Sec. 2.1 as intra-island config
dimensions.  The stated readings, each checked in closed form on power-of-two
inputs (exact in binary64):

  cp: tp*cp*dp GPUs; compute, TP traffic and stashed activations split over
      tp*cp; ring attention moves (cp-1)/(cp*tp) of each layer's key/value
      bytes once forward and twice backward; the data-parallel group is dp*cp.
  rc: the forward pass runs twice (compute 4x instead of 3x forward FLOPs,
      forward collectives 3 passes instead of 2); only each layer's boundary
      activation (its output) is stashed.
  of: the stash travels to host memory and back (2 transfers at the island's
      host bandwidth per GPU); only one micro-batch is on the device at any
      depth; needs a host link.
With cp = 1, no rc and no of every extra term is an exact +0 and the candidate
order reduces to the original one.
"""
import itertools

import numpy as np
import pytest

from oracle.oracle import Oracle, OracleError, EINVAL, ENOPLAN
from workloads import extended, make_instance, random_tiny
from tests import brute
from tests.inst_util import instance, scaled

P30 = 2.0 ** 30


def rows_of(inst):
    o = Oracle(inst)
    cost, dmax = o.score()
    rows = []
    for idx in range(o.N):
        t = o.decode(idx)
        t.update(idx=idx, cost=float(cost[idx]), dmax=int(dmax[idx]))
        rows.append(t)
    return o, rows


def rand_ext(seed):
    return extended(random_tiny(seed, L_range=(2, 5), K_range=(1, 3), tight=(seed % 2 == 1)),
                    cp=(1, 2), recompute=(0, 1), offload=(0, 1))


# ---------------------------------------------------------------------------
# candidate space
# ---------------------------------------------------------------------------
def admissible(inst):
    sp = inst["space"]
    out = []
    for k, n in enumerate(inst["islands"]["n_gpus"]):
        host = inst["islands"].get("host_bw", [0.0] * len(inst["islands"]["n_gpus"]))[k]
        for tp, cp, dp, ep, z, rc, of, mb in itertools.product(
                sp["tp"], sp["cp"], range(1, n + 1), sp["ep"], sp["zero"], sp["recompute"],
                sp["offload"], sp["mb"]):
            if tp * cp * dp > n or dp % ep:
                continue
            if (sp["n_experts"] == 0 and ep != 1) or (sp["n_experts"] > 0 and sp["n_experts"] % ep):
                continue
            if of and not host > 0:
                continue
            out.append((k, tp, cp, dp, ep, z, rc, of, mb))
    return out


@pytest.mark.parametrize("seed", range(8))
def test_decode_is_the_ordered_product(seed):
    inst = rand_ext(seed)
    if seed % 3 == 0:  # an island without a host link admits no offloading
        inst["islands"]["host_bw"][0] = 0.0
    o = Oracle(inst)
    slices = [(i, j) for i in range(o.L) for j in range(i + 1, o.L + 1)]
    cfgs = sorted(admissible(inst))
    assert o.N == len(cfgs) * o.NS
    seen = []
    for idx in range(o.N):
        t = o.decode(idx)
        seen.append(((t["island"], t["tp"], t["cp"], t["dp"], t["ep"], t["zero"], t["recompute"],
                      t["offload"], t["mb"]), (t["i"], t["j"])))
    assert seen == [(c, s) for c in cfgs for s in slices]


@pytest.mark.parametrize("make", [lambda: make_instance("tiny"), lambda: make_instance("moe")] +
                         [lambda s=s: random_tiny(s) for s in range(6)])
def test_default_options_are_an_exact_no_op(make):
    # in the extended space, every config with cp = 1, no rc and no of scores
    # bit for bit like the same config of the original space
    base = make()
    if base["name"] == "moe":  # keep the oracle fast: two islands, 4 layers
        base["islands"] = {f: v[:2] for f, v in base["islands"].items()}
        base["inter_bw"] = [row[:2] for row in base["inter_bw"][:2]]
        base["island_order"] = [k for k in base["island_order"] if k < 2]
        base["layers"] = {f: v[:4] for f, v in base["layers"].items()}
    a = Oracle(base)
    b = Oracle(extended(base, cp=(1, 2), recompute=(0, 1), offload=(0, 1)))
    ca, da = a.score()
    cb, db = b.score()
    key_b = {}
    for g in range(b.n_configs):
        t = b.decode(g * b.NS)
        if t["cp"] == 1 and not t["recompute"] and not t["offload"]:
            key_b[(t["island"], t["tp"], t["dp"], t["ep"], t["zero"], t["mb"])] = g
    assert len(key_b) == a.n_configs
    for g in range(a.n_configs):
        t = a.decode(g * a.NS)
        gb = key_b[(t["island"], t["tp"], t["dp"], t["ep"], t["zero"], t["mb"])]
        sa = slice(g * a.NS, (g + 1) * a.NS)
        sb = slice(gb * b.NS, (gb + 1) * b.NS)
        assert np.array_equal(ca[sa].view(np.uint64), cb[sb].view(np.uint64))
        assert np.array_equal(da[sa], db[sb])


# ---------------------------------------------------------------------------
# terms in isolation
# ---------------------------------------------------------------------------
def test_context_parallel_splits_compute():
    # 3x forward FLOPs over tp*cp GPUs (6 * mb / (tp cp) seconds at 2^41 FLOP, 2^40 FLOP/s)
    inst = instance(layer={"fwd_flops": 2 ** 41}, n_gpus=8, peak=2.0 ** 40, B=8, tp=(1, 2),
                    cp=(1, 2, 4), mb=(1, 2))
    o, rows = rows_of(inst)
    assert {r["cp"] for r in rows} == {1, 2, 4}
    for r in rows:
        assert r["tp"] * r["cp"] * r["dp"] <= 8
        assert r["cost"] == 6.0 * r["mb"] / (r["tp"] * r["cp"]), r


def test_ring_attention_term():
    # (cp-1)/(cp tp) of the key/value bytes per pass; 3 passes, 4 with recomputation
    inst = instance(layer={"cp_comm_bytes": 2 ** 30}, n_gpus=8, intra=P30, B=8, tp=(1, 2),
                    cp=(1, 2, 4), recompute=(0, 1), mb=(1, 2))
    o, rows = rows_of(inst)
    for r in rows:
        c, t = r["cp"], r["tp"]
        passes = 4 if r["recompute"] else 3
        want = passes * r["mb"] * (c - 1) / (c * t)
        assert r["cost"] == want, r


def test_tp_collectives_with_cp_and_recompute():
    inst = instance(layer={"tp_comm_bytes": 2 ** 30}, n_gpus=8, intra=P30, B=8, tp=(1, 2, 4),
                    cp=(1, 2), recompute=(0, 1), mb=(1, 2))
    o, rows = rows_of(inst)
    for r in rows:
        t, c = r["tp"], r["cp"]
        passes = 3 if r["recompute"] else 2
        assert r["cost"] == 2.0 * passes * r["mb"] * (t - 1) / (t * c), r


def test_all_to_all_with_recompute():
    inst = instance(layer={"a2a_bytes": 2 ** 30}, n_gpus=8, intra=P30, B=8, tp=(1,), cp=(1, 2),
                    ep=(1, 2), recompute=(0, 1), mb=(1,), n_experts=2)
    o, rows = rows_of(inst)
    for r in rows:
        e, c = r["ep"], r["cp"]
        passes = 3 if r["recompute"] else 2
        assert r["cost"] == passes * (e - 1) / (e * c), r


def test_recompute_compute_term():
    inst = instance(layer={"fwd_flops": 2 ** 41}, n_gpus=4, peak=2.0 ** 40, B=4, tp=(1, 2),
                    recompute=(0, 1), mb=(1, 2))
    o, rows = rows_of(inst)
    for r in rows:
        assert r["cost"] == (8.0 if r["recompute"] else 6.0) * r["mb"] / r["tp"], r


def test_sync_group_spans_context_parallel_ranks():
    # ZeRO-3 over D = dp * cp: 6 (D-1)/D bytes per param per micro-batch, / tp
    inst = instance(layer={"dense_params": 2 ** 30}, n_gpus=8, intra=P30, B=2, tp=(1, 2),
                    cp=(1, 2, 4), mb=(1,), zero=(3,))
    o, rows = rows_of(inst)
    checked = set()
    for r in rows:
        D = r["dp"] * r["cp"]
        if D & (D - 1):  # exact closed form at powers of two
            continue
        assert r["cost"] == 6.0 * (D - 1) / D / r["tp"], r
        checked.add((r["dp"], r["cp"]))
    assert {(2, 2), (1, 4), (4, 2), (2, 1)} <= checked


def test_memory_with_cp_recompute_offload():
    # 2^30 params, ZeRO-3 over D = dp*cp = 4: 4 B/param = 2^32 B of state; a
    # micro-batch stashes 2^22 B of activations (2^20 of layer output) per GPU
    # at tp*cp = 1; HBM = 2^32 + 5 * 2^22.
    K = 16
    lay = {"dense_params": 2 ** 30, "act_stash_bytes": 2 ** 22, "out_act_bytes": 2 ** 20}
    H = 2.0 ** 32 + 5 * 2.0 ** 22
    inst = instance(K=K, layer=lay, n_gpus=4, hbm=H, B=64, tp=(1,), cp=(1, 2), mb=(1,),
                    zero=(3,), recompute=(0, 1), offload=(0, 1), host=2.0 ** 30)
    o, rows = rows_of(inst)
    for r in rows:
        if r["i"] != 0:
            continue
        D = r["dp"] * r["cp"]
        if D != 4:
            continue
        # state 2^32 (D = 4); stash per micro-batch: act / cp, or out_act / cp with rc
        stash = (2.0 ** 20 if r["recompute"] else 2.0 ** 22) / r["cp"]
        room = H - 2.0 ** 32
        if r["offload"]:
            want = K if stash <= room else 0  # one micro-batch on the device at any depth
        else:
            want = min(K, int(room // stash))
        assert r["dmax"] == want, r


def test_offload_term_and_host_link():
    # 2 transfers of the stash at the host bandwidth: 2 * mb * S / (tp cp Hb)
    lay = {"act_stash_bytes": 2 ** 30, "out_act_bytes": 2 ** 28}
    inst = instance(layer=lay, n_gpus=4, host=2.0 ** 30, B=4, tp=(1, 2), cp=(1, 2),
                    recompute=(0, 1), offload=(0, 1), mb=(1, 2))
    o, rows = rows_of(inst)
    assert any(r["offload"] for r in rows)
    for r in rows:
        S = 2.0 ** 28 if r["recompute"] else 2.0 ** 30
        want = (2.0 * r["mb"] * S / (r["tp"] * r["cp"] * 2.0 ** 30)) if r["offload"] else 0.0
        assert r["cost"] == want, r
    # no host link: offloading is not a candidate
    o2 = Oracle(instance(layer=lay, n_gpus=4, host=0.0, B=4, tp=(1,), offload=(0, 1)))
    assert all(not o2.decode(g * o2.NS)["offload"] for g in range(o2.n_configs))


# ---------------------------------------------------------------------------
# search over the extended space
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(24))
def test_survivors_and_plans_on_extended_instances(seed):
    o = Oracle(rand_ext(seed))
    rows = brute.candidate_table(o)
    s = o.prune().tolist()
    assert s == brute.survivors_by_reps(rows, o.K) == brute.survivors_by_dominance(rows)
    st, plan, per_b = o.compose(s)
    bf, best = brute.brute_force_compose(o, rows)
    if best is None:
        assert st == ENOPLAN
        return
    assert (plan["b"], plan["P"], plan["F"], plan["T"]) == (best["b"], best["P"], best["F"], best["T"])
    st, plan, per_b = o.compose_relaxed(s)
    bf, best = brute.brute_force_relaxed(o, rows)
    assert (plan["b"], plan["P"], plan["F"], plan["T"]) == (best["b"], best["P"], best["F"], best["T"])


def test_extended_space_never_worse():
    # a superset of configs can only lower the least iteration time
    for seed in range(10):
        base = random_tiny(seed, tight=True)
        a = Oracle(base)
        b = Oracle(extended(base, cp=(1, 2), recompute=(0, 1), offload=(0, 1)))
        pa = a.compose(a.prune())[1]
        pb = b.compose_relaxed(b.prune())[1]
        pr = a.compose_relaxed(a.prune())[1]
        assert pb["T"] <= pr["T"] <= pa["T"]


@pytest.mark.parametrize("seed", [1, 2, 5])
def test_power_of_two_rate_scaling_extended(seed):
    inst = rand_ext(seed)
    a = Oracle(inst)
    b = Oracle(scaled(inst, compute=8.0, bandwidth=8.0))
    ca, da = a.score()
    cb, db = b.score()
    assert np.array_equal(da, db) and np.array_equal(ca, cb * 8.0)


@pytest.mark.parametrize("bad", [dict(cp=(2, 1)), dict(cp=(0,)), dict(recompute=(2,)),
                                 dict(offload=(3,)), dict(host=-1.0), dict(host=float("nan"))])
def test_invalid_extended_inputs_rejected(bad):
    kw = dict(K=2, layer={"fwd_flops": 10})
    kw.update(bad)
    with pytest.raises(OracleError) as e:
        Oracle(instance(**kw))
    assert e.value.status == EINVAL
