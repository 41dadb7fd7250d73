"""Pins of the oracle's candidate space and per-candidate cost / memory model.

Expected values come from closed forms of the stated model on inputs chosen as
powers of two so every expected number is exact in binary64: forward+backward
compute of 3x the forward FLOPs, ring collectives moving 2(t-1)/t (all-reduce)
or (t-1)/t (reduce-scatter, all-gather, all-to-all) of the data, textbook ZeRO
state sizes 16 : 4+12/D : 2+14/D : 16/D bytes per parameter, and 1F1B holding
min(d, m) micro-batches of activations at depth d (Sec. 5.2).
"""
import itertools

import numpy as np
import pytest

from oracle.oracle import Oracle, OracleError, EINVAL
from workloads import make_instance, random_tiny
from workloads.gen import layer_ints
from tests.inst_util import instance, scaled

P30 = 2.0 ** 30


def single(inst):
    """Oracle over an instance and its candidate list with decoded tuples."""
    o = Oracle(inst)
    cost, dmax = o.score()
    rows = []
    for idx in range(o.N):
        t = o.decode(idx)
        t.update(idx=idx, cost=float(cost[idx]), dmax=int(dmax[idx]))
        rows.append(t)
    return o, rows


# ---------------------------------------------------------------------------
# candidate space
# ---------------------------------------------------------------------------
def admissible_tuples(inst):
    """Every (island, tp, dp, ep, z, mb) the space admits, by its definition:
    tp*dp GPUs of the island, ep dividing dp and the expert count (dense: 1)."""
    sp = inst["space"]
    out = []
    for k, n in enumerate(inst["islands"]["n_gpus"]):
        for tp, dp, ep, z, mb in itertools.product(sp["tp"], range(1, n + 1), sp["ep"],
                                                   sp["zero"], sp["mb"]):
            if tp * dp > n or dp % ep:
                continue
            if sp["n_experts"] == 0 and ep != 1:
                continue
            if sp["n_experts"] > 0 and sp["n_experts"] % ep:
                continue
            out.append((k, tp, dp, ep, z, mb))
    return out


@pytest.mark.parametrize("make", [lambda: make_instance("tiny")] +
                         [lambda s=s: random_tiny(s) for s in range(12)])
def test_decode_is_the_ordered_product(make):
    inst = make()
    o = Oracle(inst)
    L = o.L
    slices = [(i, j) for i in range(L) for j in range(i + 1, L + 1)]
    assert o.NS == L * (L + 1) // 2 == len(slices)
    cfgs = sorted(admissible_tuples(inst))
    assert o.N == len(cfgs) * o.NS
    seen = []
    for idx in range(o.N):
        t = o.decode(idx)
        seen.append(((t["island"], t["tp"], t["dp"], t["ep"], t["zero"], t["mb"]), (t["i"], t["j"])))
    # idx order: configs lexicographic (island, tp, dp, ep, z, mb), slices innermost
    assert seen == [(c, s) for c in cfgs for s in slices]
    with pytest.raises(OracleError):
        o.decode(o.N)


def test_published_candidate_counts():
    # hand counts: 4-GPU islands admit 7 (tp, dp) pairs for tp in {1,2,4};
    # 8-GPU islands admit 15 for tp in {1,2,4,8}
    assert Oracle(make_instance("tiny")).N == 2 * 7 * 4 * 3 * 36 == 6048
    assert Oracle(make_instance("dense8b")).N == 4 * 15 * 4 * 4 * 528 == 506880


def test_gpt_layer_shape_textbook():
    s, h = 2048, 1024
    t = layer_ints(s=s, h=h, n_heads=16, n_kv=16, ffn=4 * h, act="gelu")
    assert t["act_stash_bytes"] == 34 * s * h        # Korthikanti et al. per-layer stash
    assert t["fwd_flops"] == 24 * s * h * h + 4 * s * s * h
    assert t["dense_params"] == 12 * h * h + 2 * h


# ---------------------------------------------------------------------------
# cost terms in isolation
# ---------------------------------------------------------------------------
def test_compute_term():
    # 3x forward FLOPs per sample, mb samples per micro-batch, split over tp GPUs
    inst = instance(layer={"fwd_flops": 2 ** 41}, n_gpus=8, peak=2.0 ** 40, B=8,
                    tp=(1, 2, 4, 8), mb=(1, 2, 4), zero=(0, 1, 2, 3))
    o, rows = single(inst)
    for r in rows:
        assert r["cost"] == 6.0 * r["mb"] / r["tp"], r


def test_efficiency_scales_compute():
    inst = instance(layer={"fwd_flops": 2 ** 41}, peak=2.0 ** 40, eta=0.5)
    o, rows = single(inst)
    assert rows[0]["cost"] == 12.0


def test_tp_collectives_term():
    # two passes of a ring all-reduce-sized exchange of the TP bytes: 2 * 2(t-1)/t
    inst = instance(layer={"tp_comm_bytes": 2 ** 30}, n_gpus=8, intra=P30, B=8,
                    tp=(1, 2, 4, 8), mb=(1, 2))
    o, rows = single(inst)
    for r in rows:
        t = r["tp"]
        assert r["cost"] == 4.0 * r["mb"] * (t - 1) / t, r


def test_all_to_all_term():
    # forward + backward all-to-all; (e-1)/e of the tokens leave each GPU and
    # sequence-parallel TP splits the tokens over tp GPUs
    inst = instance(layer={"a2a_bytes": 2 ** 30}, n_gpus=8, intra=P30, B=8,
                    tp=(1, 2), ep=(1, 2, 4), mb=(1, 2), n_experts=4)
    o, rows = single(inst)
    assert {r["ep"] for r in rows} == {1, 2, 4}
    for r in rows:
        e, t = r["ep"], r["tp"]
        assert r["cost"] == 2.0 * r["mb"] * (e - 1) / (e * t), r


@pytest.mark.parametrize("D", [1, 2, 4, 8])
def test_data_parallel_sync_term(D):
    # per parameter, bf16: ZeRO-0/1 all-reduce grads once per iteration
    # (2 B x 2r); ZeRO-2 reduce-scatters grads every micro-batch (2 B x r) and
    # all-gathers params once (2 B x r); ZeRO-3 all-gathers fwd and bwd and
    # reduce-scatters every micro-batch (3 x 2 B x r).  r = (D-1)/D; per-
    # iteration traffic is spread over the m micro-batches of the iteration.
    m = 4
    inst = instance(layer={"dense_params": 2 ** 30}, n_gpus=16, intra=P30, B=D * m,
                    tp=(1, 2), mb=(1,), zero=(0, 1, 2, 3))
    o, rows = single(inst)
    r = (D - 1) / D
    want = {0: 4 * r / m, 1: 4 * r / m, 2: 2 * r + 2 * r / m, 3: 6 * r}
    got = [x for x in rows if x["dp"] == D]
    assert len(got) == 2 * 4
    for x in got:
        assert x["cost"] == want[x["zero"]] / x["tp"], x


def test_expert_sync_uses_expert_data_parallel_degree():
    # expert parameters are replicated over dp/ep GPUs and sharded over tp*ep
    inst = instance(layer={"expert_params": 2 ** 30}, n_gpus=8, intra=P30, B=4,
                    tp=(1,), ep=(1, 2, 4), mb=(1,), zero=(3,), n_experts=4)
    o, rows = single(inst)
    for x in rows:
        if x["dp"] != 4:
            continue
        De = x["dp"] // x["ep"]
        assert x["cost"] == 6 * (De - 1) / De / x["ep"], x


def test_zero_ties_when_dp_is_one():
    # with one replica there is nothing to synchronise and nothing to shard:
    # all ZeRO stages cost and weigh the same, and only stage 0 (least index)
    # can survive
    inst = make_instance("tiny")
    o, rows = single(inst)
    by = {}
    for r in rows:
        if r["dp"] == 1:
            by.setdefault((r["island"], r["tp"], r["ep"], r["mb"], r["i"], r["j"]), []).append(r)
    assert by
    for v in by.values():
        assert len({(x["cost"], x["dmax"]) for x in v}) == 1
    surv = set(o.prune().tolist())
    assert all(rows[i]["zero"] == 0 for i in surv if rows[i]["dp"] == 1)


# ---------------------------------------------------------------------------
# memory and depth
# ---------------------------------------------------------------------------
def test_state_bytes_and_depth_closed_form():
    # 2^30 parameters on dp = 4: ZeRO-3 keeps 16/4 = 4 B/param = 2^32 B; one
    # micro-batch of stash is 2^20 B.  With HBM = 2^32 + 5 * 2^20 the stage fits
    # five in-flight micro-batches: d_max = 5 when m >= 5 (ZeRO 0-2 need
    # 16, 7 and 5.5 B/param and never fit).
    K = 8
    H = 2.0 ** 32 + 5 * 2.0 ** 20
    inst = instance(K=K, layer={"dense_params": 2 ** 30, "act_stash_bytes": 2 ** 20},
                    n_gpus=4, hbm=H, B=64, tp=(1,), mb=(1,), zero=(0, 1, 2, 3))
    o, rows = single(inst)
    for r in rows:
        if r["dp"] == 4 and r["i"] == 0:
            assert r["dmax"] == (5 if r["zero"] == 3 else 0), r
    # m = 12 / 4 = 3 micro-batches: at most 3 are ever in flight, so every depth fits
    inst = instance(K=K, layer={"dense_params": 2 ** 30, "act_stash_bytes": 2 ** 20},
                    n_gpus=4, hbm=H, B=12, tp=(1,), mb=(1,), zero=(3,))
    o, rows = single(inst)
    assert all(r["dmax"] == K for r in rows if r["dp"] == 4)
    # tp = 2 halves both state and stash per GPU
    inst = instance(K=K, layer={"dense_params": 2 ** 30, "act_stash_bytes": 2 ** 20},
                    n_gpus=8, hbm=2.0 ** 31 + 3 * 2.0 ** 19, B=64, tp=(2,), mb=(1,), zero=(3,))
    o, rows = single(inst)
    assert all(r["dmax"] == 3 for r in rows if r["dp"] == 4)


def test_memory_fraction_and_extremes():
    base = dict(K=4, layer={"dense_params": 2 ** 30, "act_stash_bytes": 2 ** 20}, n_gpus=4,
                B=64, tp=(1,), mb=(1,), zero=(3,))
    o, rows = single(instance(hbm=2.0 ** 60, **base))
    assert all(r["dmax"] == 4 for r in rows)
    o, rows = single(instance(hbm=1.0, **base))
    assert all(r["dmax"] == 0 for r in rows)
    # mem_frac halves the usable HBM: 2 * (2^32 + 2 * 2^20) usable -> depth 2 on dp=4
    o, rows = single(instance(hbm=2.0 * (2.0 ** 32 + 2 * 2.0 ** 20), mem_frac=0.5, **base))
    assert all(r["dmax"] == 2 for r in rows if r["dp"] == 4)


def test_depth_monotone_in_memory_and_cost_monotone_in_work():
    inst = random_tiny(7)
    o1, r1 = single(inst)
    o2, r2 = single(scaled(inst, memory=1.5))
    assert all(b["dmax"] >= a["dmax"] for a, b in zip(r1, r2))
    heavier = scaled(inst)
    heavier["layers"]["fwd_flops"] = [2 * x for x in heavier["layers"]["fwd_flops"]]
    o3, r3 = single(heavier)
    assert all(b["cost"] >= a["cost"] for a, b in zip(r1, r3))


# ---------------------------------------------------------------------------
# metamorphic: exact power-of-two rescaling of every rate
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", [1, 2, 3, 11])
def test_power_of_two_rate_scaling(seed):
    inst = random_tiny(seed)
    a = Oracle(inst)
    b = Oracle(scaled(inst, compute=8.0, bandwidth=8.0))
    ca, da = a.score()
    cb, db = b.score()
    assert np.array_equal(da, db)
    assert np.array_equal(ca, cb * 8.0)
    sa, sb = a.prune(), b.prune()
    assert np.array_equal(sa, sb)
    st_a, pa, _ = a.compose(sa)
    st_b, pb, _ = b.compose(sb)
    assert st_a == st_b
    if st_a == 0:
        assert (pa["P"], pa["F"], pa["T"]) == (pb["P"] * 8.0, pb["F"] * 8.0, pb["T"] * 8.0)
        assert [s["pair_index"] for s in pa["stages"]] == [s["pair_index"] for s in pb["stages"]]


# ---------------------------------------------------------------------------
# input validation
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("bad", [
    dict(n_gpus=0), dict(peak=0.0), dict(hbm=-1.0), dict(intra=float("nan")),
    dict(tp=(2, 1)), dict(tp=()), dict(mb=(0,)), dict(zero=()), dict(B=0),
    dict(inter=-1.0), dict(eta=0.0), dict(mem_frac=float("inf")),
    dict(tp=(1, 2, 3, 4, 5, 6, 7, 8, 9)),
])
def test_invalid_inputs_rejected(bad):
    kw = dict(K=2, layer={"fwd_flops": 10})
    kw.update(bad)
    with pytest.raises(OracleError) as e:
        Oracle(instance(**kw))
    assert e.value.status == EINVAL


def test_invalid_layers_rejected():
    with pytest.raises(OracleError):
        Oracle(instance(layer={"fwd_flops": -1}))
    with pytest.raises(OracleError):
        Oracle(instance(L=4, layer={"fwd_flops": 2 ** 61}))   # whole-model sum >= 2^62
    with pytest.raises(OracleError):
        Oracle(instance(L=513))
