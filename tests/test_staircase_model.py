"""The frontier's counting argument, checked on random groups in plain
Python (no GPU): a member survives iff no other member at least as deep has
a smaller key (cost, -d_max, idx) -- the union of rep(G, d) over d -- and a
lane that keeps only R staircase entries, drops the shallowest when full,
ignores members at or above that depth for the rest of the pass, and settles
the shallower survivors in later passes capped by the least settled cost,
finds exactly that set.  The HIP frontier follows these steps; its output
is compared with the oracle's surviving set by the GPU tests."""
import random

import pytest

MB = 23  # an entry packs depth << MB | member


def survivors_by_definition(costs, depths):
    n = len(costs)
    key = lambda m: (costs[m], -depths[m], m)
    out = set()
    for d in range(1, max(depths + [0]) + 1):  # rep(G, d): least key with d_max >= d
        cands = [m for m in range(n) if depths[m] >= d]
        if cands:
            out.add(min(cands, key=key))
    return out


def offer(cv, pk, c, d, m, floor):
    dk = d << MB
    if any(pk[r] >= dk and cv[r] <= c for r in range(len(pk))):
        return floor
    dk1 = (d + 1) << MB
    x = dk | m
    for r in range(len(pk)):
        if pk[r] < dk1 and cv[r] >= c:
            pk[r] = 0
    for r in range(len(pk)):
        if pk[r] == 0:
            pk[r], cv[r] = x, c
            return floor
    lo = min([x] + pk)
    floor = lo >> MB
    if lo != x:
        r = pk.index(lo)
        pk[r], cv[r] = x, c
    return floor


def survivors_by_passes(costs, depths, R):
    hi, cap, capped, out, passes = 1 << 30, 0.0, False, set(), 0
    while True:
        passes += 1
        cv, pk, floor = [0.0] * R, [0] * R, 0
        for m in range(len(costs)):  # ascending idx
            d = depths[m]
            if floor < d <= hi and not (capped and cap <= costs[m]):
                floor = offer(cv, pk, costs[m], d, m, floor)
        settled = [(p, c) for p, c in zip(pk, cv) if p]
        out |= {p & ((1 << MB) - 1) for p, _ in settled}
        if floor == 0:
            return out, passes
        hi, cap, capped = floor, min(settled)[1], True


@pytest.mark.parametrize("seed", range(40))
def test_bounded_staircase_passes_find_the_survivors(seed):
    rng = random.Random(seed)
    for _ in range(200):
        n = rng.randint(0, 40)
        ncost = rng.choice([2, 4, 16, 1000])  # few distinct costs force ties
        costs = [float(rng.randint(0, ncost)) for _ in range(n)]
        depths = [rng.choice([0, 0, 1, 2, 3, 4, 5, 6, 7, 8, 12, 20, 255]) for _ in range(n)]
        want = survivors_by_definition(costs, depths)
        for R in (1, 2, 3, 4, 8):
            got, passes = survivors_by_passes(costs, depths, R)
            assert got == want, (seed, R, costs, depths)
            # each further pass lowers the depth bound: at most one per distinct depth
            assert passes <= len(set(depths)) + 1


def test_survival_depends_only_on_deeper_members():
    rng = random.Random(7)
    for _ in range(500):
        n = rng.randint(1, 30)
        costs = [float(rng.randint(0, 6)) for _ in range(n)]
        depths = [rng.randint(0, 9) for _ in range(n)]
        full = survivors_by_definition(costs, depths)
        t = rng.randint(0, 9)
        deep = [m for m in range(n) if depths[m] > t]
        sub = survivors_by_definition([costs[m] for m in deep], [depths[m] for m in deep])
        assert {deep[k] for k in sub} == {m for m in full if depths[m] > t}
