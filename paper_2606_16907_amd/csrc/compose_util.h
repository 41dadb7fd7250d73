// compose_util.h -- pieces shared by the two composition drivers: grouping
// of the candidate list and the resolution of a plan stage's candidate.
#pragma once

#include "tg_device.h"

#pragma clang fp contract(off)

namespace tg {

// Groups (slice, island position, b) are numbered position-major, then b,
// then slice: the candidate list runs through each config's slices in
// ascending order, so building the groups touches consecutive counters
// (their atomics stay within few cache lines).
__host__ __device__ inline int64_t group_id(const DevProblem &P, int64_t o, int64_t bi, int64_t s) {
    return (o * P.nb + bi) * P.NS + s;
}

// Candidate order within a group: least cost, then deepest fit, then least
// index; idx < 0 marks "none".
__device__ inline bool cand_less(double c1, int d1, int64_t i1, double c2, int d2, int64_t i2) {
    if (i1 < 0) return false;
    if (i2 < 0) return true;
    return c1 < c2 || (c1 == c2 && (d1 > d2 || (d1 == d2 && i1 < i2)));
}

// Grouped candidate entries, CSR by group id: after grouping, gcnt[G] is the
// end of group G's entries and its start is gcnt[G - 1] (0 for G = 0).
struct Groups {
    int32_t *rec_g;  // [n] group of list entry r, -1 if unused
    double *rec_c;   // [n] its cost
    uint8_t *rec_d;  // [n] its d_max
    int32_t *gcnt;   // [n_groups] counts -> offsets -> ends
    double *ent_c;   // [n] grouped entries: cost
    uint8_t *ent_d;  // [n] d_max
    int64_t *ent_i;  // [n] candidate index
    int64_t *tmp;    // scan tiles, at least group_scan_tiles(n_groups) entries
};
int64_t group_scan_tiles(int64_t n);
// Clears the counts, validates the list (res->err bits 1: not ascending or out
// of range, 2: incompatible) and groups the entries with d_max >= 1.
// pos[k] is island k's position in the group numbering.  Asynchronous on s.
void launch_grouping(const DevProblem &P, const int64_t *surv, int64_t n, const double *cost,
                     const uint8_t *dmax, const int32_t *pos, const Groups &g, ComposeResult *res,
                     hipStream_t s);

// One wave resolves a plan stage: layers [i, j) on island `island` (group
// position o) at depth d for micro-batch index bb: the group's least
// candidate fitting at d, its config and memory, written to sg by lane 0.
// `link` is the transfer time to the next stage (0 for the last).  A group
// with no fitting candidate sets res->err = 4 (the stage table said one fits).
// G is the group's index in the grouped entries (callers number groups their
// own way).
__device__ inline void resolve_stage(const DevProblem &P, const int32_t *gcnt, const double *ent_c,
                                     const uint8_t *ent_d, const int64_t *ent_i, int64_t G, int i, int j,
                                     int island, int d, double link, tg_stage &sg, ComposeResult *res) {
    const int L = P.L;
    const int lane = threadIdx.x % kWave;
    const int32_t st = G ? gcnt[G - 1] : 0, en = gcnt[G];
    int64_t best = -1;
    double bc = kInf;
    int bd = 0;
    for (int32_t e = st + lane; e < en; e += kWave) {
        const int dd = ent_d[e];
        if (dd < d) continue;
        const double c = ent_c[e];
        const int64_t ie = ent_i[e];
        if (cand_less(c, dd, ie, bc, bd, best)) {
            best = ie;
            bc = c;
            bd = dd;
        }
    }
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double c2 = __shfl_xor(bc, off);
        const int d2 = __shfl_xor(bd, off);
        const int64_t i2 = __shfl_xor(best, off);
        if (cand_less(c2, d2, i2, bc, bd, best)) {
            best = i2;
            bc = c2;
            bd = d2;
        }
    }
    if (lane != 0) return;
    if (best < 0) {
        res->err = 4;
        res->status = TG_ENOPLAN;
        return;
    }
    const int64_t g = best / P.NS;
    const Coef &c = P.coef[g];
    const int64_t Lp = L + 1;
    const double Pd = (double)(P.pre[Lp + j] - P.pre[Lp + i]);
    const double Pe = (double)(P.pre[2 * Lp + j] - P.pre[2 * Lp + i]);
    // stash per sample: layer outputs with recomputation, else all activations
    const int sq = c.rc ? 6 : 3;
    const double S = (double)(P.pre[sq * Lp + j] - P.pre[sq * Lp + i]);
    const double state = (c.mud * Pd) + (c.mue * Pe);
    const double A1 = c.rho * S;
    sg.island = island;
    sg.first_layer = i;
    sg.end_layer = j;
    sg.tp = c.tp;
    sg.cp = c.cp;
    sg.dp = c.dp;
    sg.ep = c.ep;
    sg.zero = c.z;
    sg.recompute = c.rc;
    sg.offload = c.of;
    sg.mb = c.mb;
    sg.depth = d;
    sg.pair_index = best;
    sg.cost = bc;
    // in flight: min(d, m) micro-batches, one when offloaded
    sg.mem_bytes = state + (fmin(c.of ? 1.0 : (double)d, c.m_real) * A1);
    sg.link_out = link;
}

}  // namespace tg
