"""A third, independent evaluation of the per-candidate model: plain Python.

TEST INFRASTRUCTURE ONLY.  It pins the C oracle's candidate order, cost and
deepest-fitting-position arithmetic bit for bit (the GPU path is compared with
the oracle by the GPU tests, so the three agree pairwise).

Written from the stated model, not from either implementation: the paper
delegates a pair's cost to the homogeneous parallelizer's profile() and
parallelize() queries (Tab. 2, Sec. 5.1); this project's reading replaces them
with an analytic step time per micro-batch and the 1F1B memory rule that a
stage d positions from the pipeline end holds min(d, m) micro-batches of
stashed activations (Sec. 5.2: memory depends on the stage's position).

Python floats are IEEE binary64 and every arithmetic operator rounds once;
Python never contracts a*b+c into a fused multiply-add, so writing each
operation as a separate expression in the stated order evaluates exactly the
parenthesised formula.  Slice sums are exact Python integers, converted once.
"""
from __future__ import annotations

from workloads import LAYER_FIELDS

# per-layer fields in the order the slice sums are taken
FL, PD, PE, ACT, TB, AB, OA, CB = range(8)


class CostRef:
    """Candidate decoding and scoring of one instance dictionary."""

    def __init__(self, inst):
        lay = inst["layers"]
        L = len(lay["fwd_flops"])
        self.L = L
        self.NS = L * (L + 1) // 2
        cols = [[int(v) for v in lay.get(f, [0] * L)] for f in LAYER_FIELDS]
        self.pre = []
        for col in cols:
            acc, p = 0, [0]
            for v in col:
                acc += v
                p.append(acc)
            self.pre.append(p)
        isl = inst["islands"]
        self.K = len(isl["n_gpus"])
        self.n = [int(x) for x in isl["n_gpus"]]
        self.F = [float(x) for x in isl["peak_flops"]]
        self.M = [float(x) for x in isl["hbm_bytes"]]
        self.W = [float(x) for x in isl["intra_bw"]]
        self.Hb = [float(x) for x in isl.get("host_bw", [0.0] * self.K)]
        sp = inst["space"]
        self.B = int(sp["global_batch"])
        self.eta = float(sp["eta"])
        self.mem_frac = float(sp["mem_frac"])
        n_exp = int(sp["n_experts"])
        cps = list(sp.get("cp", [1]))
        rcs = sorted(set(sp.get("recompute", [0])))
        ofs = sorted(set(sp.get("offload", [0])))
        # configs of each island in lexicographic (tp, cp, dp, ep, z, rc, of, mb)
        # order; tp cp dp GPUs of the island; ep divides dp and the expert
        # count (a dense model admits ep = 1 only); offloading needs a host link
        self.cfg = []
        for k in range(self.K):
            for tp in sp["tp"]:
                for cp in cps:
                    if tp * cp > self.n[k]:
                        continue
                    for dp in range(1, self.n[k] // (tp * cp) + 1):
                        for ep in sp["ep"]:
                            if dp % ep:
                                continue
                            if (ep != 1) if n_exp == 0 else (n_exp % ep):
                                continue
                            for z in sorted(sp["zero"]):
                                for rc in rcs:
                                    for of in ofs:
                                        if of and not self.Hb[k] > 0.0:
                                            continue
                                        for mb in sp["mb"]:
                                            self.cfg.append((k, tp, cp, dp, ep, z, rc, of, mb))
        self.N = self.NS * len(self.cfg)
        self._coef = {}

    # -- decoding ------------------------------------------------------------
    def slice_ij(self, s):
        """Slices are every [i, j), 0 <= i < j <= L, ordered by i then j."""
        i, left = 0, s
        while left >= self.L - i:
            left -= self.L - i
            i += 1
        return i, i + 1 + left

    def decode(self, idx):
        g, s = divmod(idx, self.NS)
        return self.cfg[g], self.slice_ij(s)

    # -- the model -------------------------------------------------------------
    def coef(self, g):
        if g in self._coef:
            return self._coef[g]
        k, tp, cp, dp, ep, z, rc, of, mb = self.cfg[g]
        F, W, Hb = self.F[k], self.W[k], self.Hb[k]
        b = dp * mb
        m = float(self.B) / float(b)
        q = tp * cp                       # GPUs sharing one micro-batch's tokens
        Dd, De = dp * cp, (dp // ep) * cp  # data-parallel groups of dense / expert parameters
        qd, qe = float(tp), float(tp * ep)
        nc = 4.0 if rc else 3.0           # compute passes: forward (twice with recomputation) + backward
        nt = 3 if rc else 2               # passes over the forward collectives

        def r(D):
            return float(D - 1) / float(D)

        def per_microbatch(D):            # bf16 bytes per parameter synchronised each micro-batch
            return (0.0, 0.0, 2.0 * r(D), 6.0 * r(D))[z]

        def per_iteration(D):             # ... and once per iteration
            return (4.0 * r(D), 4.0 * r(D), 2.0 * r(D), 0.0)[z]

        def state(D):                     # model-state bytes per parameter on one GPU
            if z == 0:
                return 16.0
            if z == 1:
                return 4.0 + 12.0 / float(D)
            if z == 2:
                return 2.0 + 14.0 / float(D)
            return 16.0 / float(D)

        fmb = float(mb)
        alpha = (nc * fmb) / ((float(q) * F) * self.eta)
        beta = ((float(2 * nt) * fmb) * float(tp - 1)) / (float(q) * W) if tp > 1 else 0.0
        gamma = ((float(nt) * fmb) * float(ep - 1)) / ((float(ep) * float(q)) * W) if ep > 1 else 0.0
        kappa = ((float(nt + 1) * fmb) * float(cp - 1)) / ((float(cp) * float(tp)) * W) if cp > 1 else 0.0
        omega = (2.0 * fmb) / (float(q) * Hb) if of else 0.0
        dd = ((per_microbatch(Dd) / qd) / W) + (((per_iteration(Dd) / qd) / W) / m)
        de = ((per_microbatch(De) / qe) / W) + (((per_iteration(De) / qe) / W) / m)
        mud = state(Dd) / qd
        mue = state(De) / qe
        rho = fmb / float(q)
        H = self.M[k] * self.mem_frac
        c = (alpha, beta, gamma, kappa, omega, dd, de, mud, mue, rho, H, m, rc, of)
        self._coef[g] = c
        return c

    def score(self, idx):
        """(cost in seconds per micro-batch, deepest fitting position) of one
        candidate index."""
        g, s = divmod(idx, self.NS)
        i, j = self.slice_ij(s)
        alpha, beta, gamma, kappa, omega, dd, de, mud, mue, rho, H, m, rc, of = self.coef(g)
        x = [float(p[j] - p[i]) for p in self.pre]
        S = x[OA] if rc else x[ACT]       # recomputation stashes only the layer outputs
        v = alpha * x[FL]
        v = v + beta * x[TB]
        v = v + gamma * x[AB]
        v = v + dd * x[PD]
        v = v + de * x[PE]
        v = v + kappa * x[CB]
        v = v + omega * S
        st = mud * x[PD]
        st = st + mue * x[PE]
        A1 = rho * S

        def fits(d):
            inflight = min(1.0 if of else float(d), m)
            return st + inflight * A1 <= H

        # fits() only loses depth as d grows: the largest fitting d by bisection
        lo, hi = 0, self.K  # fits(lo) holds (lo = 0 means none); answer in [lo, hi]
        if not fits(1):
            return v, 0
        lo = 1
        while lo < hi:
            mid = (lo + hi + 1) // 2
            if fits(mid):
                lo = mid
            else:
                hi = mid - 1
        return v, lo
