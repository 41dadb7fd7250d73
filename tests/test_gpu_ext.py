"""GPU parity over the extended configuration space (context parallelism,
activation recomputation, activation offloading): decoding, every score bit
for bit, the surviving set and both compositions against the live oracle."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from workloads import extended, load_instance, random_tiny  # noqa: E402
from tests.inst_util import instance  # noqa: E402
from tests.test_gpu_parity import bits, plan_equal  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402


def _closed_form():
    lay = {"dense_params": 2 ** 30, "act_stash_bytes": 2 ** 22, "out_act_bytes": 2 ** 20,
           "fwd_flops": 2 ** 41, "tp_comm_bytes": 2 ** 30, "cp_comm_bytes": 2 ** 30}
    return instance(L=3, K=2, layer=lay, n_gpus=[4, 8], hbm=2.0 ** 32 + 5 * 2.0 ** 22, B=64,
                    tp=(1, 2), cp=(1, 2, 4), mb=(1, 2), zero=(0, 3), recompute=(0, 1),
                    offload=(0, 1), host=[2.0 ** 30, 0.0], peak=2.0 ** 40, intra=2.0 ** 30)


def _no_offload_island():
    inst = extended(random_tiny(3, L_range=(4, 4), K_range=(3, 3)), cp=(1, 2), recompute=(0, 1),
                    offload=(0, 1))
    inst["islands"]["host_bw"][1] = 0.0
    return inst


CASES = ([("closed_form", _closed_form), ("tiny_ext", lambda: extended(load_instance("tiny"))),
          ("dense8b_ext", lambda: extended(load_instance("dense8b"))),
          ("no_offload_island", _no_offload_island)]
         + [(f"rand_ext{s}", lambda s=s: extended(random_tiny(s, tight=(s % 2 == 1)), cp=(1, 2, 4),
                                                   recompute=(0, 1), offload=(0, 1)))
            for s in range(12)])


@pytest.mark.parametrize("name,make", CASES, ids=[n for n, _ in CASES])
def test_extended_parity(name, make):
    inst = make()
    print("case", name, flush=True)
    sys.stdout.flush()
    o = Oracle(inst)
    p = T.Problem(inst)
    assert (p.N, p.NS, p.n_configs, p.n_b) == (o.N, o.NS, o.n_configs, o.n_b)
    pairs = p.tg_enumerate_pairs().cpu().numpy()
    for idx in range(0, o.N, max(1, o.N // 1999)):
        d = o.decode(idx)
        assert tuple(pairs[idx]) == (d["i"], d["j"], d["island"], d["tp"], d["cp"], d["dp"], d["ep"],
                                     d["zero"], d["recompute"], d["offload"], d["mb"], 0)
    cost, dmax = p.tg_score_pairs()
    oc, od = o.score()
    torch.cuda.synchronize()
    assert np.array_equal(bits(cost.cpu().numpy()), bits(oc))
    assert np.array_equal(dmax.cpu().numpy(), od)
    surv = p.tg_prune(cost, dmax)
    osurv = o.prune()
    assert np.array_equal(surv.cpu().numpy(), osurv)
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    ost, oplan, _ = o.compose(osurv)
    assert st == ost
    if st == 0:
        plan_equal(plan, oplan)
    st, plan = p.tg_compose_pipeline_relaxed(surv, cost, dmax)
    ost, oplan, _ = o.compose_relaxed(osurv)
    assert st == ost
    if st == 0:
        plan_equal(plan, oplan)


def test_extended_plans_use_the_new_dimensions():
    # on the extended 8B instance the chosen plan is no slower than the
    # original and the space really contains cp > 1, recomputed and offloaded
    # candidates that survive
    base = load_instance("dense8b")
    p0 = T.Problem(base)
    c0, d0 = p0.tg_score_pairs()
    s0 = p0.tg_prune(c0, d0)
    t0 = p0.tg_compose_pipeline(s0, c0, d0)[1]["T"]
    p = T.Problem(extended(base))
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    plan = p.tg_compose_pipeline(surv, cost, dmax)[1]
    assert plan["T"] <= t0
    pairs = p.tg_enumerate_pairs().cpu().numpy()[surv.cpu().numpy()]
    assert (pairs[:, 4] > 1).any() and (pairs[:, 8] == 1).any() and (pairs[:, 9] == 1).any()


@pytest.mark.parametrize("name", ["dense70b", "moe", "large"])
def test_extended_named_against_stored(name):
    """The extended named instances against the oracle's stored results: on
    the 128-island one N = 7,881,904,128 candidates (more than 2^32, 71 GB of
    scores) in the launch configuration bench.py times."""
    import hashlib
    from tests.golden.make_golden import load as load_golden
    g = load_golden(name + "_extended")
    print("case", name, "extended", g["counts"], flush=True)
    p = T.Problem(extended(load_instance(name)))
    assert (p.N, p.NS, p.n_configs) == (g["counts"]["N"], g["counts"]["NS"], g["counts"]["n_configs"])
    cost, dmax = p.tg_score_pairs()
    idx = torch.tensor(g["sample"]["idx"], dtype=torch.int64, device="cuda")
    assert np.array_equal(bits(cost[idx].cpu().numpy()), bits(g["sample"]["cost"]))
    assert np.array_equal(dmax[idx].cpu().numpy(), np.array(g["sample"]["dmax"], dtype=np.uint8))
    surv = p.tg_prune(cost, dmax)
    s = surv.cpu().numpy()
    assert len(s) == g["survivors"]["count"]
    assert s[:16].tolist() == g["survivors"]["head"] and s[-16:].tolist() == g["survivors"]["tail"]
    assert hashlib.sha256(np.ascontiguousarray(s, dtype="<i8").tobytes()).hexdigest() == g["survivors"]["sha256"]
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    assert st == g["status"] == 0
    g["plan"]["status"] = 0
    plan_equal(plan, g["plan"])
    del cost, dmax, surv
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,ext", [("large", False), ("large", True), ("moe", False), ("dense70b", True)])
def test_full_size_scores_against_the_oracle(name, ext):
    """Per-candidate scores at full size in the launch configuration bench.py
    times, against the oracle one candidate at a time: 48 whole config rows
    (every slice of configs spread over the islands, the first and the last
    included), 250,000 seeded random candidates and the last 4,096 (on the
    extended 128-island instance N > 2^32, so the 64-bit index path is
    covered end to end)."""
    import zlib
    inst = load_instance(name)
    if ext:
        inst = extended(inst)
    print("case", name, "extended" if ext else "", flush=True)
    p = T.Problem(inst)
    N, NS, C = p.N, p.NS, p.n_configs
    rng = np.random.default_rng(zlib.crc32(f"{name}/{ext}".encode()))
    rows = np.unique(np.r_[0, C - 1, np.linspace(0, C - 1, 46).astype(np.int64)])
    idx = np.unique(np.r_[(rows[:, None] * NS + np.arange(NS)[None, :]).ravel(),
                          rng.integers(0, N, size=250_000), np.arange(max(0, N - 4096), N)])
    cost, dmax = p.tg_score_pairs()
    t = torch.from_numpy(idx).cuda()
    gc, gd = cost[t].cpu().numpy(), dmax[t].cpu().numpy()
    del cost, dmax, t
    torch.cuda.empty_cache()
    oc, od = Oracle(inst).score_list(idx)
    bad = np.nonzero((bits(gc) != bits(oc)) | (gd != od))[0]
    assert bad.size == 0, [(int(idx[b]), float(gc[b]), float(oc[b]), int(gd[b]), int(od[b])) for b in bad[:5]]
    assert len(idx) >= 250_000 and (idx >= 2 ** 32).any() == (N > 2 ** 32)
