"""Three-way pin of the per-candidate model: the plain-Python evaluation of
tests/cost_ref.py against the C oracle, bit for bit (the GPU tests compare the
HIP path with the same oracle bit for bit, which closes the triangle).

The two implementations share nothing but the instance dictionaries: the
Python one builds its own config order, slice order, prefix sums,
coefficients and depth search.  A dropped term, a swapped operand order, a
wrong ring factor or ZeRO share, a wrong decode or a depth rule off by one in
either shows up as a differing bit pattern or depth at some sampled index."""
import zlib

import numpy as np
import pytest

from oracle.oracle import Oracle
from tests.cost_ref import CostRef
from workloads import extended, load_instance, random_tiny
from tests.inst_util import deep_staircase, tiny_tight

SAMPLES = 12_000  # per named instance; the random ones are checked whole


def _check(inst, idx):
    ref, o = CostRef(inst), Oracle(inst)
    assert ref.N == o.N and ref.NS == o.NS
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64))
    oc, od = o.score_list(idx)
    got_c = np.empty(len(idx), dtype=np.float64)
    got_d = np.empty(len(idx), dtype=np.uint8)
    for t, x in enumerate(idx.tolist()):
        got_c[t], got_d[t] = ref.score(x)
    bad = np.nonzero((got_c.view(np.uint64) != oc.view(np.uint64)) | (got_d != od))[0]
    assert bad.size == 0, [(int(idx[b]), ref.decode(int(idx[b])), float(got_c[b]), float(oc[b]),
                            int(got_d[b]), int(od[b])) for b in bad[:5]]
    # the decoded tuple as well: island, degrees, ZeRO stage, recompute, offload, micro-batch, slice
    for x in idx[:: max(1, len(idx) // 300)].tolist():
        (k, tp, cp, dp, ep, z, rc, of, mb), (i, j) = ref.decode(x)
        d = o.decode(x)
        assert (d["island"], d["tp"], d["cp"], d["dp"], d["ep"], d["zero"], d["recompute"], d["offload"],
                d["mb"], d["i"], d["j"]) == (k, tp, cp, dp, ep, z, rc, of, mb, i, j)
    return len(idx)


def _sample(N, n, seed):
    """n distinct indices: the two ends of the space and a uniform sample
    between them."""
    rng = np.random.default_rng(seed)
    if N <= n:
        return np.arange(N)
    out = np.unique(np.r_[np.arange(64), np.arange(N - 64, N)])
    while len(out) < n:
        out = np.unique(np.r_[out, rng.integers(0, N, size=n - len(out))])
    return out


@pytest.mark.parametrize("seed", range(16))
def test_random_instances_whole(seed):
    inst = random_tiny(seed, tight=seed % 2 == 1)
    assert _check(inst, np.arange(CostRef(inst).N)) > 0


@pytest.mark.parametrize("seed", range(6))
def test_random_extended_instances_whole(seed):
    inst = extended(random_tiny(100 + seed))
    assert _check(inst, np.arange(CostRef(inst).N)) > 0


@pytest.mark.parametrize("make", [tiny_tight, lambda: deep_staircase(105), lambda: deep_staircase(123)])
def test_handmade_instances_whole(make):
    inst = make()
    assert _check(inst, np.arange(CostRef(inst).N)) > 0


@pytest.mark.parametrize("name", ["tiny", "dense8b", "dense70b", "moe", "large"])
@pytest.mark.parametrize("space", ["named", "extended"])
def test_named_instances_sampled(name, space):
    inst = load_instance(name)
    if space == "extended":
        inst = extended(inst)
    N = CostRef(inst).N
    seed = zlib.crc32(f"{name}/{space}".encode())
    assert _check(inst, _sample(N, SAMPLES, seed)) >= min(N, SAMPLES)


def test_total_sampled_count():
    """At least 1e5 indices are compared over the named instances."""
    total = 0
    for name in ["tiny", "dense8b", "dense70b", "moe", "large"]:
        for space in ["named", "extended"]:
            inst = load_instance(name)
            if space == "extended":
                inst = extended(inst)
            total += min(CostRef(inst).N, SAMPLES)
    assert total >= 100_000
