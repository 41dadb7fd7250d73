"""Parity of the HIP plan search (through the C ABI) with the CPU oracle.

Bit-exact everywhere: candidate decoding, per-candidate cost (binary64,
compared bitwise) and d_max, the ascending surviving set, and the composed
plan (b, stages, cuts, islands, configs, pair indices, P, F, T and per-stage
cost, memory and link times).  The oracle runs live for the four smaller
instances and random ones; the 128-island instance is compared with the
oracle's stored results (tests/golden, written by make_golden.py) plus
per-candidate samples the oracle scores one by one.
"""
import ctypes
import hashlib
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from workloads import load_instance, random_tiny  # noqa: E402
from tests.inst_util import deep_staircase, instance, longest_staircase, scaled, tiny_tight  # noqa: E402
from tests.golden.make_golden import load as load_golden  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402


# decoded pair columns (tg_pair), named like the oracle's decode
PAIR_COLS = ("i", "j", "island", "tp", "cp", "dp", "ep", "zero", "recompute", "offload", "mb")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bits(x):
    return np.asarray(x, dtype=np.float64).view(np.uint64)


def plan_equal(gpu_plan, orc_plan):
    assert orc_plan["status"] == 0
    for f in ("b", "m", "S"):
        assert gpu_plan[f] == orc_plan[f], f
    for f in ("P", "F", "T"):
        assert bits(gpu_plan[f]) == bits(orc_plan[f]), (f, gpu_plan[f], orc_plan[f])
    assert len(gpu_plan["stages"]) == len(orc_plan["stages"])
    for a, b in zip(gpu_plan["stages"], orc_plan["stages"]):
        for f in ("island", "first_layer", "end_layer", "tp", "dp", "ep", "zero", "mb", "depth",
                  "pair_index"):
            assert a[f] == b[f], (f, a, b)
        for f in ("cp", "recompute", "offload"):
            assert a[f] == b[f], (f, a, b)
        for f in ("cost", "mem_bytes", "link_out"):
            assert bits(a[f]) == bits(b[f]), (f, a[f], b[f])


SMALL = ["tiny", "dense8b"]
MEDIUM = ["dense70b", "moe"]


def _instances():
    out = [(n, lambda n=n: load_instance(n)) for n in SMALL]
    out.append(("tiny_tight", tiny_tight))
    out += [(f"rand{s}", lambda s=s: random_tiny(s, tight=(s % 2 == 1))) for s in range(16)]
    out += [(f"randL{s}", lambda s=s: random_tiny(1000 + s, L_range=(9, 14), K_range=(3, 6)))
            for s in range(6)]
    return out


INSTANCES = _instances()


@pytest.mark.parametrize("name,make", INSTANCES, ids=[n for n, _ in INSTANCES])
def test_full_path_parity(name, make):
    inst = make()
    say("case", name)
    o = Oracle(inst)
    p = T.Problem(inst)
    assert (p.N, p.NS, p.n_configs, p.n_b) == (o.N, o.NS, o.n_configs, o.n_b)
    assert p.bvalues == o.bvalues
    # decode
    pairs = p.tg_enumerate_pairs().cpu().numpy()
    for idx in range(0, o.N, max(1, o.N // 997)):
        d = o.decode(idx)
        assert tuple(pairs[idx]) == tuple(d[f] for f in PAIR_COLS) + (0,)
    # score
    cost, dmax = p.tg_score_pairs()
    oc, od = o.score()
    torch.cuda.synchronize()
    assert np.array_equal(bits(cost.cpu().numpy()), bits(oc))
    assert np.array_equal(dmax.cpu().numpy(), od)
    # prune
    surv = p.tg_prune(cost, dmax)
    osurv = o.prune()
    assert np.array_equal(surv.cpu().numpy(), osurv)
    # compose, in the instance's order and reversed
    for order in (inst["island_order"], list(reversed(inst["island_order"]))):
        st, plan = p.tg_compose_pipeline(surv, cost, dmax, order)
        ost, oplan, _ = o.compose(osurv, order)
        assert st == ost
        if st == 0:
            plan_equal(plan, oplan)
        else:
            assert st == T.TG_ENOPLAN and plan["S"] == 0 and np.isinf(plan["T"])


@pytest.mark.parametrize("seed", [105, 111, 123, 135])
def test_staircases_longer_than_a_pass_keeps(seed):
    # groups of at most 64 configs keep four staircase entries per lane and
    # pass; these instances have groups with five or six survivors, so the
    # frontier needs a second pass for them
    inst = deep_staircase(seed)
    say("case deep_staircase", seed)
    o = Oracle(inst)
    osurv = o.prune()
    longest, members = longest_staircase(o, osurv)
    assert longest > 4 and members <= 64
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    assert np.array_equal(surv.cpu().numpy(), osurv)
    cost_c, dmax_c = p.tg_score_classes()
    assert np.array_equal(p.tg_prune_classes(cost_c, dmax_c).cpu().numpy(), osurv)
    st, plan = p.tg_compose_pipeline(surv, cost, dmax, inst["island_order"])
    ost, oplan, _ = o.compose(osurv, inst["island_order"])
    assert st == ost
    if st == 0:
        plan_equal(plan, oplan)


@pytest.mark.parametrize("name", MEDIUM)
def test_medium_instances_parity(name):
    inst = load_instance(name)
    say("case", name)
    o = Oracle(inst)
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    torch.cuda.synchronize()
    step = 8_000_000
    for first in range(0, o.N, step):
        cnt = min(step, o.N - first)
        oc, od = o.score(first, cnt)
        assert np.array_equal(bits(cost[first:first + cnt].cpu().numpy()), bits(oc)), first
        assert np.array_equal(dmax[first:first + cnt].cpu().numpy(), od), first
    surv = p.tg_prune(cost, dmax)
    g = load_golden(name)
    s = surv.cpu().numpy()
    assert len(s) == g["survivors"]["count"]
    assert hashlib.sha256(np.ascontiguousarray(s, dtype="<i8").tobytes()).hexdigest() == \
        g["survivors"]["sha256"]
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    ost, oplan, _ = o.compose(s)
    assert st == ost == 0
    plan_equal(plan, oplan)
    g["plan"]["status"] = g["status"]
    plan_equal(plan, g["plan"])


@pytest.mark.parametrize("first,count", [(0, 1), (37, 1000), (527, 530), (1055, 64 * 33 + 5),
                                         (100000, 0), (506879, 1), (3, 506877)])
def test_score_windows(first, count):
    inst = load_instance("dense8b")
    say("window", first, count)
    o = Oracle(inst)
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs(first, count)
    oc, od = o.score(first, count)
    torch.cuda.synchronize()
    assert np.array_equal(bits(cost.cpu().numpy()), bits(oc))
    assert np.array_equal(dmax.cpu().numpy(), od)
    pairs = p.tg_enumerate_pairs(first, count).cpu().numpy()
    for t in range(0, count, max(1, count // 50)):
        d = o.decode(first + t)
        assert tuple(pairs[t]) == tuple(d[f] for f in PAIR_COLS) + (0,)


def test_prune_safety_on_gpu():
    inst = load_instance("dense8b")
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    B = inst["space"]["global_batch"]
    pairs = p.tg_enumerate_pairs().cpu().numpy()
    col = {f: c for c, f in enumerate(PAIR_COLS)}
    compatible = (B % (pairs[:, col["dp"]] * pairs[:, col["mb"]]) == 0)
    allc = torch.from_numpy(np.nonzero(compatible)[0].astype(np.int64)).cuda()
    a = p.tg_compose_pipeline(surv, cost, dmax)
    b = p.tg_compose_pipeline(allc, cost, dmax)
    assert a[0] == b[0] == 0
    assert a[1] == b[1]


def test_large_instance_against_stored_oracle_results():
    """The 128-island, 128-layer instance at full size, in the configuration
    the benchmark times."""
    inst = load_instance("large")
    g = load_golden("large")
    say("case large: create")
    p = T.Problem(inst)
    assert (p.N, p.NS, p.n_configs) == (g["counts"]["N"], g["counts"]["NS"], g["counts"]["n_configs"])
    say("case large: score", p.N)
    cost, dmax = p.tg_score_pairs()
    idx = torch.tensor(g["sample"]["idx"], dtype=torch.int64, device="cuda")
    gc = cost[idx].cpu().numpy()
    gd = dmax[idx].cpu().numpy()
    assert np.array_equal(bits(gc), bits(g["sample"]["cost"]))
    assert np.array_equal(gd, np.array(g["sample"]["dmax"], dtype=np.uint8))
    say("case large: prune")
    surv = p.tg_prune(cost, dmax)
    s = surv.cpu().numpy()
    assert len(s) == g["survivors"]["count"]
    assert s[:16].tolist() == g["survivors"]["head"] and s[-16:].tolist() == g["survivors"]["tail"]
    assert hashlib.sha256(np.ascontiguousarray(s, dtype="<i8").tobytes()).hexdigest() == \
        g["survivors"]["sha256"]
    say("case large: compose")
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    assert st == g["status"] == 0
    g["plan"]["status"] = 0
    plan_equal(plan, g["plan"])
    # a second, independent sample scored by the oracle one candidate at a time
    rng = np.random.default_rng(77)
    extra = np.unique(rng.integers(0, p.N, size=2000))
    o = Oracle(inst)
    oc, od = o.score_list(extra)
    t = torch.from_numpy(extra).cuda()
    assert np.array_equal(bits(cost[t].cpu().numpy()), bits(oc))
    assert np.array_equal(dmax[t].cpu().numpy(), od)


# ---------------------------------------------------------------------------
# error paths and determinism
# ---------------------------------------------------------------------------
def test_errors_and_capacity():
    inst = load_instance("tiny")
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    with pytest.raises(T.TangramError) as e:
        p.tg_score_pairs(first=p.N - 1, count=2)
    assert e.value.status == T.TG_EINVAL
    small = torch.empty(3, dtype=torch.int64, device="cuda")
    with pytest.raises(T.TangramError) as e:
        p.tg_prune(cost, dmax, survivors=small)
    assert e.value.status == T.TG_ECAPACITY and e.value.required == 360
    surv = p.tg_prune(cost, dmax)
    with pytest.raises(T.TangramError) as e:
        p.tg_compose_pipeline(surv.flip(0).contiguous(), cost, dmax)
    assert e.value.status == T.TG_EINVAL
    with pytest.raises(T.TangramError) as e:
        p.tg_compose_pipeline(surv, cost, dmax, island_order=[0, 0])
    assert e.value.status == T.TG_EINVAL
    tiny_ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(T.TangramError) as e:
        p.tg_compose_pipeline(surv, cost, dmax, workspace=tiny_ws)
    assert e.value.status == T.TG_ENOMEM


def test_binding_refuses_short_or_mistyped_buffers_before_any_launch():
    """Plain pointers carry no length: the binding refuses a buffer shorter
    than the call reads or writes, of another dtype, or not contiguous,
    before the library is called."""
    p = T.Problem(load_instance("tiny"))
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    short_c = torch.empty(p.N - 1, dtype=torch.float64, device="cuda")
    short_d = torch.empty(p.N - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError, match="at least"):
        p.tg_score_pairs(0, p.N, short_c, dmax)
    with pytest.raises(ValueError, match="dtype"):
        p.tg_score_pairs(0, p.N, cost.float(), dmax)
    with pytest.raises(ValueError, match="at least"):
        p.tg_enumerate_pairs(0, 4, torch.empty((3, 12), dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError, match="at least"):
        p.tg_prune(cost, short_d)
    with pytest.raises(ValueError, match="dtype"):
        p.tg_prune(cost, dmax, survivors=torch.empty(p.N, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError, match="contiguous"):
        p.tg_compose_pipeline(torch.stack([surv, surv], 1)[:, 0], cost, dmax)
    with pytest.raises(ValueError, match="at least"):
        p.tg_compose_pipeline_relaxed(surv, short_c, dmax)
    with pytest.raises(ValueError, match="dtype"):
        p.tg_compose_pipeline_all_orders(surv.int(), cost, dmax)
    with pytest.raises(ValueError, match="device buffer"):
        p.tg_compose_pipeline(surv, cost.cpu(), dmax)
    # the checked calls still give the plan
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    assert st == T.TG_OK and plan["S"] >= 1


def test_library_refuses_misaligned_buffers_before_any_launch():
    """Workspaces are carved at 256-byte offsets and hold atomic counters;
    score and survivor arrays hold 8-byte values.  A misaligned base is
    refused before any launch."""
    p = T.Problem(load_instance("tiny"))
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    lib, vp = T.load_library(), ctypes.c_void_p
    raw = torch.empty(p.prune_workspace().numel() + 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(T.TangramError) as e:
        p.tg_prune(cost, dmax, workspace=raw[8:])
    assert e.value.status == T.TG_EINVAL and "aligned" in str(e.value)
    raw = torch.empty(p.compose_workspace(surv.numel()).numel() + 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(T.TangramError) as e:
        p.tg_compose_pipeline(surv, cost, dmax, workspace=raw[64:])
    assert e.value.status == T.TG_EINVAL
    assert lib.tg_score_pairs(p.h, 0, 1, vp(cost.data_ptr() + 4), vp(dmax.data_ptr()), None) == T.TG_EINVAL
    out = torch.empty(24, dtype=torch.int32, device="cuda")
    n = ctypes.c_int64(0)
    assert lib.tg_enumerate_pairs(p.h, ctypes.byref(n), 0, 1, vp(out.data_ptr() + 2), None) == T.TG_EINVAL
    # aligned views of the same memory still work
    st, plan = p.tg_compose_pipeline(surv, cost, dmax, workspace=raw[256:])
    assert st == T.TG_OK


def test_two_streams_share_one_problem():
    """A problem is read-only after create: two streams with their own
    buffers and workspaces, issued so that one's scoring overlaps the
    other's pruning, give the one-stream results bit for bit."""
    p = T.Problem(load_instance("dense8b"))
    c0, d0 = p.tg_score_pairs()
    s0 = p.tg_prune(c0, d0)
    st0, plan0 = p.tg_compose_pipeline(s0, c0, d0)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    scores, survs = [], []
    for st in streams:
        with torch.cuda.stream(st):
            scores.append(p.tg_score_pairs())
    for st, (c, d) in zip(streams, scores):
        with torch.cuda.stream(st):
            survs.append(p.tg_prune(c, d))
    plans = []
    for st, (c, d), sv in zip(streams, scores, survs):
        with torch.cuda.stream(st):
            plans.append(p.tg_compose_pipeline(sv, c, d))
    torch.cuda.synchronize()
    for (c, d), sv, (st, plan) in zip(scores, survs, plans):
        assert torch.equal(c.view(torch.int64), c0.view(torch.int64)) and torch.equal(d, d0)
        assert torch.equal(sv, s0)
        assert st == st0 and plan == plan0


def test_invalid_instances_rejected_like_the_oracle():
    from oracle.oracle import OracleError
    for bad in (dict(n_gpus=0), dict(tp=(2, 1)), dict(zero=()), dict(B=0), dict(inter=-1.0),
                dict(mem_frac=0.0)):
        kw = dict(K=2, layer={"fwd_flops": 10})
        kw.update(bad)
        inst = instance(**kw)
        with pytest.raises(OracleError):
            Oracle(inst)
        with pytest.raises(T.TangramError) as e:
            T.Problem(inst)
        assert e.value.status == T.TG_EINVAL


def test_no_plan_and_empty_list():
    inst = scaled(load_instance("tiny"), memory=1e-6)
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    assert surv.numel() == 0
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    assert st == T.TG_ENOPLAN and plan["S"] == 0 and np.isinf(plan["T"])


def test_repeatable_bit_for_bit():
    inst = load_instance("dense8b")
    p = T.Problem(inst)
    r1 = p.plan_search()
    r2 = p.plan_search()
    assert r1[1] == r2[1]
    assert torch.equal(r1[2], r2[2])
    assert torch.equal(r1[3].view(torch.int64), r2[3].view(torch.int64))
    assert torch.equal(r1[4], r2[4])
