// islands.hip -- GPU island construction from nodes (Sec. 4.1).
//
// An island holds nodes with the same GPU count whose compute, memory
// (Eq. 1) and intra-node bandwidth (Eq. 2) differ by at most a factor 1 + eps
// pairwise, and every member's links inside the island are at least as fast
// as its links leaving it (Eq. 3).  Steps (1)-(2): one block splits the nodes
// by GPU count, compute, memory and intra-node bandwidth, each split a block
// bitonic sort by (group, value, node) followed by a sweep that opens a new
// group at the first value above the group's smallest times (1 + eps).  Step
// (3): agglomerative clustering per group: the pair of clusters with the
// highest complete linkage (the least bandwidth between their nodes, a node
// pair counted by its slower direction; ties to the least pair of smallest
// node ids) is merged if the union satisfies Eq. 3 against every node outside
// it, else marked, until every pair is marked.  A union's Eq. 3 outcome
// depends only on its own nodes, so a failed pair stays failed while both
// clusters last, and the next merge is the highest pair whose union passes.
// One block per group runs it in rounds: each cluster's row keeps its best
// unmarked partner, known to pass (clean) or untested (dirty); when the best
// clean pair is above every dirty one it is merged, else every dirty pair
// above it is tested at once (a wave each) and the failures marked.  The
// group's linkage, marks and per-cluster least links (for each cluster and
// node, the node's slowest link into the cluster) sit in matrices over the
// group's own node numbering; a cluster's members are one contiguous range
// of a permutation, so a test gives each lane a member: its slowest link
// inside the union from its own cluster's value and the other cluster's
// entry, its fastest link leaving from its bandwidth row sorted once (the
// first entry outside the union, from where its own cluster ends).  A finish
// pass numbers islands by their smallest node and reduces the island
// attributes and island-to-island bandwidths (least over node pairs).
#include <stdint.h>

#include <vector>

#include "tg_device.h"

#pragma clang fp contract(off)

namespace tg {

constexpr int kMaxNodes = 4096;
constexpr int kGroupThreads = 1024;
constexpr int kMergeThreads = 1024;
constexpr int kMergeWaves = kMergeThreads / 64;
constexpr double kNoPair = -__builtin_huge_val();

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct IslandWs {
    int32_t *gpus;      // [n]
    double *val;        // [4][n] compute, memory, intra, host per node
    double *e;          // [n][n] node bandwidth, row = source
    int32_t *srt;       // [n][n] row u: the other nodes by bandwidth from u, fastest first
    int32_t *grp;       // [n] group after steps (1)-(2)
    int32_t *gstart;    // [n + 1] group g's nodes are gnodes[gstart[g] .. gstart[g + 1])
    int32_t *gnodes;    // [n]
    int32_t *ngroups;   // [1]
    int32_t *lq;        // [n] a node's number inside its group (its place in gnodes)
    int64_t *goff;      // [n + 1] where group g's nm x nm matrices start (sum of nm^2 before it)
    double *L;          // per group [nm][nm]: complete linkage between clusters (-inf: no pair)
    uint8_t *M;         // per group [nm][nm]: pairs whose union breaks Eq. 3
    double *XT;         // per group [nm][nm]: row c, column m: slowest link from node m into cluster c
    double *inown;      // [n] a node's slowest link into its own cluster (+inf alone)
    int32_t *pos;       // [n] first entry of the node's sorted row outside its own cluster
    int32_t *nxl;       // [n] that entry's number inside the group (-1: another group, or none)
    double *outv;       // [n] the node's bandwidth to it (-inf: none)
    int32_t *cl;        // [n] cluster (its smallest node) of each node
    int32_t *err;       // [2] a merge loop overran its round bound (an internal error); first bad node_bw entry
    int32_t *island_of; // [n]
    int32_t *out_k;     // [1]
    int32_t *isl_gpus;  // [n]
    double *isl_val;    // [4][n] least compute, memory, intra, host
    double *isl_e;      // [n][n] (K x K used)
    size_t bytes;
};

static IslandWs carve_islands(int64_t n, void *base) {
    IslandWs w{};
    char *p = (char *)base;
    size_t off = 0;
    auto take = [&](size_t bytes) -> void * {
        void *r = base ? (void *)(p + off) : nullptr;
        off += align256(bytes > 0 ? bytes : 1);
        return r;
    };
    w.gpus = (int32_t *)take(4 * n);
    w.val = (double *)take(8 * 4 * n);
    w.e = (double *)take(8 * n * n);
    w.srt = (int32_t *)take(4 * n * n);
    w.grp = (int32_t *)take(4 * n);
    w.gstart = (int32_t *)take(4 * (n + 1));
    w.gnodes = (int32_t *)take(4 * n);
    w.ngroups = (int32_t *)take(4);
    w.lq = (int32_t *)take(4 * n);
    w.goff = (int64_t *)take(8 * (n + 1));
    w.L = (double *)take(8 * n * n);  // the groups' matrices together hold at most n^2 entries
    w.M = (uint8_t *)take(n * n);
    w.XT = (double *)take(8 * n * n);
    w.inown = (double *)take(8 * n);
    w.pos = (int32_t *)take(4 * n);
    w.nxl = (int32_t *)take(4 * n);
    w.outv = (double *)take(8 * n);
    w.cl = (int32_t *)take(4 * n);
    w.err = (int32_t *)take(8);
    w.island_of = (int32_t *)take(4 * n);
    w.out_k = (int32_t *)take(4);
    w.isl_gpus = (int32_t *)take(4 * n);
    w.isl_val = (double *)take(8 * 4 * n);
    w.isl_e = (double *)take(8 * n * n);
    w.bytes = off;
    return w;
}

size_t islands_ws_bytes(int n) { return carve_islands(n, nullptr).bytes; }

// Node bandwidths must be finite and non-negative: the first entry that is not
// into *bad (INT32_MAX if none; n^2 <= 2^24 entries).
__global__ __launch_bounds__(256) void islands_check(int64_t nn, const double *__restrict__ e, int32_t *bad) {
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nn; t += (int64_t)gridDim.x * blockDim.x) {
        const double x = e[t];
        if (!(x >= 0.0) || !(x < __builtin_huge_val())) atomicMin(bad, (int32_t)t);
    }
}

// ---------------------------------------------------------------------------
// steps (1)-(2): groups
// ---------------------------------------------------------------------------
// Order of nodes u, v by (group, value, node id); padding slots (>= n) last.
__device__ inline bool node_before(int u, int v, int n, const int32_t *g, const double *x) {
    if (u >= n) return false;
    if (v >= n) return true;
    if (g[u] != g[v]) return g[u] < g[v];
    if (x[u] != x[v]) return x[u] < x[v];
    return u < v;
}

__global__ __launch_bounds__(kGroupThreads) void islands_groups(int n, const int32_t *__restrict__ gpus,
                                                                const double *__restrict__ val, double eps_c,
                                                                double eps_m, double eps_i, int32_t *grp,
                                                                int32_t *gstart, int32_t *gnodes, int32_t *ngroups,
                                                                int32_t *lq, int64_t *goff) {
    __shared__ int32_t ord[kMaxNodes];
    __shared__ int32_t g[kMaxNodes];
    __shared__ double x[kMaxNodes];
    __shared__ int32_t ng[kMaxNodes];      // new group of the t-th node in sorted order
    __shared__ int32_t gs[kMaxNodes + 1];  // group starts after the last split
    __shared__ int32_t nx[kMaxNodes];      // next opening position after an opening at t
    __shared__ int32_t scan_lds[kGroupThreads / 64 + 1];
    __shared__ int32_t s_groups;
    int np = 1;
    while (np < n) np <<= 1;
    for (int u = threadIdx.x; u < n; u += blockDim.x) g[u] = 0;
    // the split keys: GPU count (exact), compute, memory, intra-node bandwidth
    for (int f = 0; f < 4; ++f) {
        const double eps = f == 0 ? 0.0 : (f == 1 ? eps_c : (f == 2 ? eps_m : eps_i));
        for (int u = threadIdx.x; u < np; u += blockDim.x) {
            ord[u] = u;
            if (u < n) x[u] = f == 0 ? (double)gpus[u] : val[(int64_t)(f - 1) * n + u];
        }
        __syncthreads();
        for (int k = 2; k <= np; k <<= 1)
            for (int j = k >> 1; j > 0; j >>= 1) {
                for (int t = threadIdx.x; t < np; t += blockDim.x) {
                    const int q = t ^ j;
                    if (q > t) {
                        const int a = ord[t], b = ord[q];
                        const bool up = (t & k) == 0;
                        const bool swap = up ? node_before(b, a, n, g, x) : node_before(a, b, n, g, x);
                        if (swap) {
                            ord[t] = b;
                            ord[q] = a;
                        }
                    }
                }
                __syncthreads();
            }
        // the sweep: a new group opens at the first node of an old group and
        // at the first node whose value exceeds the opening node's times
        // (1 + eps).  From an opening position t the next one is the first
        // t' > t whose (old group, value) passes (g, x (1 + eps)) of t, found
        // by bisection in the sorted order; the openings are the chain of
        // such positions from 0, which thread 0 follows (one hop per group).
        for (int t = threadIdx.x; t < n; t += blockDim.x) {
            const int u = ord[t];
            const int gu = g[u];
            const double thr = x[u] * (1.0 + eps);
            int lo = t + 1, hi = n;  // first position past the run, in [t + 1, n]
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                const int v = ord[mid];
                if (g[v] > gu || (g[v] == gu && !(x[v] <= thr)))
                    hi = mid;
                else
                    lo = mid + 1;
            }
            nx[t] = lo;
            ng[t] = 0;
        }
        __syncthreads();
        if (threadIdx.x == 0)
            for (int t = 0; t < n; t = nx[t]) ng[t] = 1;
        __syncthreads();
        {  // new group of each position: openings up to it, less one
            int32_t carry = 0;
            for (int base = 0; base < n; base += blockDim.x) {
                const int t = base + (int)threadIdx.x;
                const int32_t f = t < n ? ng[t] : 0;
                int32_t tot;
                const int32_t ex = block_excl_scan<int32_t>(f, scan_lds, &tot);
                __syncthreads();
                if (t < n) ng[t] = carry + ex + f - 1;
                carry += tot;
            }
            if (threadIdx.x == 0) s_groups = carry;
        }
        __syncthreads();
        for (int t = threadIdx.x; t < n; t += blockDim.x) g[ord[t]] = ng[t];
        __syncthreads();
    }
    // group starts and member lists in sorted order (groups are numbered in it)
    const int G = s_groups;
    for (int t = threadIdx.x; t < n; t += blockDim.x)
        if (t == 0 || ng[t] != ng[t - 1]) gs[ng[t]] = t;
    if (threadIdx.x == 0) gs[G] = n;
    __syncthreads();
    if (threadIdx.x == 0) {
        *ngroups = G;
        int64_t off = 0;
        for (int gg = 0; gg < G; ++gg) {
            goff[gg] = off;
            const int64_t nm = gs[gg + 1] - gs[gg];
            off += nm * nm;
        }
        goff[G] = off;
    }
    for (int gg = threadIdx.x; gg <= G; gg += blockDim.x) gstart[gg] = gs[gg];
    for (int t = threadIdx.x; t < n; t += blockDim.x) {
        const int u = ord[t];
        gnodes[t] = u;
        grp[u] = ng[t];
        lq[u] = t - gs[ng[t]];
    }
}

// Row u of the node bandwidth sorted, fastest first (ties to the lesser
// node), u itself left out: the fastest link from u to a node outside a
// cluster is then the first entry outside it, a few entries in for a cluster
// whose own links are its fastest, as Eq. 3 asks.
__global__ __launch_bounds__(1024) void islands_sort_rows(int n, const double *__restrict__ e, int32_t *srt) {
    __shared__ double x[kMaxNodes];
    __shared__ int32_t id[kMaxNodes];
    const int u = blockIdx.x;
    int np = 1;
    while (np < n) np <<= 1;
    for (int t = threadIdx.x; t < np; t += blockDim.x) {
        id[t] = (t < n && t != u) ? t : n;  // n: after every real entry
        x[t] = t < n ? e[(int64_t)u * n + t] : 0.0;
    }
    __syncthreads();
    auto before = [&](int p, int q) {  // entry p sorts before entry q
        if (id[p] >= n) return false;
        if (id[q] >= n) return true;
        if (x[p] != x[q]) return x[p] > x[q];
        return id[p] < id[q];
    };
    for (int k = 2; k <= np; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int t = threadIdx.x; t < np; t += blockDim.x) {
                const int o = t ^ j;
                if (o > t) {
                    const bool up = (t & k) == 0;
                    if (up ? before(o, t) : before(t, o)) {
                        const double tx = x[t];
                        x[t] = x[o];
                        x[o] = tx;
                        const int32_t ti = id[t];
                        id[t] = id[o];
                        id[o] = ti;
                    }
                }
            }
            __syncthreads();
        }
    for (int t = threadIdx.x; t < n - 1; t += blockDim.x) srt[(int64_t)u * n + t] = id[t];
}

// The groups' matrices over their own node numbering: linkage of node pairs
// (the slower direction), no marks, and each node's slowest link into each
// single-node cluster; every node its own cluster.  Thread per node pair of
// the whole cluster; pairs in different groups do nothing.
__global__ __launch_bounds__(256) void islands_link_init(int n, const double *__restrict__ e,
                                                         const int32_t *__restrict__ grp,
                                                         const int32_t *__restrict__ gstart,
                                                         const int32_t *__restrict__ lq,
                                                         const int64_t *__restrict__ goff, double *L, uint8_t *M,
                                                         double *XT, double *inown, int32_t *cl) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n * n) return;
    const int u = (int)(t / n), v = (int)(t - (int64_t)u * n);
    if (v == 0) {
        cl[u] = u;
        inown[u] = __builtin_huge_val();
    }
    const int g = grp[u];
    if (grp[v] != g) return;
    const int64_t nm = gstart[g + 1] - gstart[g];
    const int64_t qu = lq[u], qv = lq[v], base = goff[g];
    double l = kNoPair, x = __builtin_huge_val();
    if (u != v) {
        x = e[t];
        const double y = e[(int64_t)v * n + u];
        l = x < y ? x : y;
    }
    L[base + qu * nm + qv] = l;
    M[base + qu * nm + qv] = 0;
    XT[base + qv * nm + qu] = x;
}

// ---------------------------------------------------------------------------
// step (3): agglomerative clustering, one block per group
// ---------------------------------------------------------------------------
// Pairs are ordered by linkage (higher first), then by the smaller node id of
// the pair's two clusters, then by the larger one: key (l, x, y), x < y the
// two ids.  No pair is (-inf, INT_MAX, INT_MAX), after every pair.
__device__ inline bool key_before(double l1, int x1, int y1, double l2, int x2, int y2) {
    return l1 > l2 || (l1 == l2 && (x1 < x2 || (x1 == x2 && y1 < y2)));
}

__device__ inline bool pair_before(double l1, int x1, int y1, double l2, int x2, int y2) {
    return key_before(l1, min(x1, y1), max(x1, y1), l2, min(x2, y2), max(x2, y2));
}

// The group's state in LDS, by node number inside the group (q < nm).  A
// cluster is named by its representative, its node with the least id; its
// members are perm[st[c] .. st[c] + sz[c]).
struct MergeLds {
    int32_t gid[kMaxNodes];  // node id of q
    int16_t rep[kMaxNodes];  // representative of q's cluster
    int16_t perm[kMaxNodes];
    int16_t tmp[kMaxNodes];  // rotation buffer of perm
    int16_t st[kMaxNodes];
    int16_t sz[kMaxNodes];
    double rb[kMaxNodes];    // row c: linkage of its best unmarked partner
    int16_t ra[kMaxNodes];   // row c: that partner (-1: none)
    int16_t vp[kMaxNodes];   // row c: a partner whose union is known to pass (-1: none)
    uint8_t ok[kMaxNodes];   // row c: ra[c] is known to pass
    uint8_t redo[kMaxNodes]; // row c: its best partner was just marked
    int16_t list[kMaxNodes]; // rows to work on this round
    double wv_l[kMergeWaves];
    int32_t wv_x[kMergeWaves], wv_y[kMergeWaves], wv_q[kMergeWaves];
    int32_t cnt;
};

// Row c's best unmarked partner among the group's clusters, by one wave.
__device__ inline void merge_row_best(MergeLds &S, int c, int nm, const double *__restrict__ L,
                                      const uint8_t *__restrict__ M, int lane) {
    const double *Lr = L + (int64_t)c * nm;
    const uint8_t *Mr = M + (int64_t)c * nm;
    constexpr int kBatch = 16;  // row entries per lane with their loads in flight together
    double b = kNoPair;
    int a = -1;
    for (int v0 = lane; v0 < nm; v0 += kBatch * kWave) {
        double l[kBatch];
        uint8_t mk[kBatch];
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            const int v = v0 + k * kWave;
            l[k] = v < nm ? Lr[v] : kNoPair;
            mk[k] = v < nm ? Mr[v] : 1;
        }
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            const int v = v0 + k * kWave;
            if (v < nm && v != c && S.rep[v] == v && !mk[k] && l[k] != kNoPair &&
                (a < 0 || l[k] > b || (l[k] == b && S.gid[v] < S.gid[a]))) {
                b = l[k];
                a = v;
            }
        }
    }
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double b2 = __shfl_xor(b, off);
        const int a2 = __shfl_xor(a, off);
        if (a2 >= 0 && (a < 0 || b2 > b || (b2 == b && S.gid[a2] < S.gid[a]))) {
            b = b2;
            a = a2;
        }
    }
    if (lane == 0) {
        S.rb[c] = b;
        S.ra[c] = (int16_t)a;
        S.ok[c] = a >= 0 && a == S.vp[c];
    }
}

// Eq. 3 for the union of clusters c and d, by one wave: a lane per member.
__device__ inline bool merge_eq3(const MergeLds &S, int c, int d, int g, int n, int nm, const double *__restrict__ e,
                                 const int32_t *__restrict__ srt, const int32_t *__restrict__ grp,
                                 const int32_t *__restrict__ lq, const double *__restrict__ XT,
                                 const double *__restrict__ inown, const int32_t *__restrict__ pos,
                                 const int32_t *__restrict__ nxl, const double *__restrict__ outv, int lane) {
    bool pass = true;
    for (int side = 0; side < 2; ++side) {
        const int own = side ? d : c, oth = side ? c : d;
        const int t0 = S.st[own], t1 = t0 + S.sz[own];
        for (int t = t0 + lane; t < t1; t += kWave) {
            const int m = S.perm[t];
            const int gm = S.gid[m];
            const double x = XT[(int64_t)oth * nm + m];
            const double io = inown[gm];
            const double in = x < io ? x : io;
            // the fastest link leaving the union: the first entry past the own
            // cluster, unless it is in the other cluster (then scan on, past
            // both: an own node can follow an outside one of equal speed)
            const int x1 = nxl[gm];
            double out = outv[gm];
            if (x1 >= 0 && S.rep[x1] == oth) {
                const int32_t *row = srt + (int64_t)gm * n;
                out = kNoPair;
                for (int p = pos[gm] + 1; p < n - 1; ++p) {
                    const int w = row[p];
                    if (grp[w] != g) {
                        out = e[(int64_t)gm * n + w];
                        break;
                    }
                    const int r = S.rep[lq[w]];
                    if (r != oth && r != own) {
                        out = e[(int64_t)gm * n + w];
                        break;
                    }
                }
            }
            if (!(in >= out)) pass = false;
        }
    }
    return __ballot(!pass) == 0;
}

__global__ __launch_bounds__(kMergeThreads) void islands_merge(int n, const double *__restrict__ e,
                                                               const int32_t *__restrict__ srt,
                                                               const int32_t *__restrict__ grp,
                                                               const int32_t *__restrict__ lq,
                                                               const int32_t *__restrict__ gstart,
                                                               const int32_t *__restrict__ gnodes,
                                                               const int32_t *__restrict__ ngroups,
                                                               const int64_t *__restrict__ goff, double *Lg,
                                                               uint8_t *Mg, double *XTg, double *inown, int32_t *pos,
                                                               int32_t *nxl, double *outv, int32_t *cl, int32_t *err) {
    __shared__ MergeLds S;
    const int g = blockIdx.x;
    if (g >= *ngroups) return;
    const int nm = gstart[g + 1] - gstart[g];
    if (nm < 2) return;
    double *L = Lg + goff[g];
    uint8_t *M = Mg + goff[g];
    double *XT = XTg + goff[g];
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    for (int q = threadIdx.x; q < nm; q += kMergeThreads) {
        const int gm = gnodes[gstart[g] + q];
        S.gid[q] = gm;
        S.rep[q] = (int16_t)q;
        S.perm[q] = (int16_t)q;
        S.st[q] = (int16_t)q;
        S.sz[q] = 1;
        S.vp[q] = -1;
        S.redo[q] = 0;
        // alone in its cluster: the first entry of its sorted row (which
        // leaves the node itself out) is outside
        const int w = srt[(int64_t)gm * n];
        pos[gm] = 0;
        nxl[gm] = grp[w] == g ? lq[w] : -1;
        outv[gm] = e[(int64_t)gm * n + w];
    }
    __syncthreads();
    for (int q = wv; q < nm; q += kMergeWaves) merge_row_best(S, q, nm, L, M, lane);
    __syncthreads();
    // every round merges two clusters, or marks a pair or finds one that
    // passes (a row then stays clean until a merge touches it): at most nm - 1
    // merges, each followed by at most nm^2 marks and nm clean rows
    const int64_t max_rounds = (int64_t)nm * ((int64_t)nm * nm + nm + 1) + nm * (int64_t)nm + 1;
    for (int64_t round = 0;; ++round) {
        if (round >= max_rounds) {  // a broken invariant, not an input case
            if (threadIdx.x == 0) atomicExch(err, 1);
            break;
        }
        // the best clean pair: keys in registers, wave results in LDS, which
        // every thread then reduces itself
        double bl = kNoPair;
        int bx = INT_MAX, by = INT_MAX, bq = -1;
        for (int q = threadIdx.x; q < nm; q += kMergeThreads)
            if (S.rep[q] == q && S.ra[q] >= 0 && S.ok[q]) {
                const int a = S.gid[q], b = S.gid[S.ra[q]];
                const int x = min(a, b), y = max(a, b);
                if (key_before(S.rb[q], x, y, bl, bx, by)) {
                    bl = S.rb[q];
                    bx = x;
                    by = y;
                    bq = q;
                }
            }
        for (int off = kWave / 2; off > 0; off >>= 1) {
            const double l2 = __shfl_xor(bl, off);
            const int x2 = __shfl_xor(bx, off), y2 = __shfl_xor(by, off), q2 = __shfl_xor(bq, off);
            if (key_before(l2, x2, y2, bl, bx, by)) {
                bl = l2;
                bx = x2;
                by = y2;
                bq = q2;
            }
        }
        if (lane == 0) {
            S.wv_l[wv] = bl;
            S.wv_x[wv] = bx;
            S.wv_y[wv] = by;
            S.wv_q[wv] = bq;
        }
        if (threadIdx.x == 0) S.cnt = 0;
        __syncthreads();
#pragma unroll
        for (int w = 0; w < kMergeWaves; ++w)
            if (key_before(S.wv_l[w], S.wv_x[w], S.wv_y[w], bl, bx, by)) {
                bl = S.wv_l[w];
                bx = S.wv_x[w];
                by = S.wv_y[w];
                bq = S.wv_q[w];
            }
        const int bc = bq;
        // the dirty pairs above it
        for (int q = threadIdx.x; q < nm; q += kMergeThreads)
            if (S.rep[q] == q && S.ra[q] >= 0 && !S.ok[q]) {
                const int a = S.gid[q], b = S.gid[S.ra[q]];
                if (key_before(S.rb[q], min(a, b), max(a, b), bl, bx, by)) S.list[atomicAdd(&S.cnt, 1)] = (int16_t)q;
            }
        __syncthreads();
        const int nl = S.cnt;
        if (nl > 0) {
            for (int k = wv; k < nl; k += kMergeWaves) {
                const int c = S.list[k], d = S.ra[c];
                const bool pass = merge_eq3(S, c, d, g, n, nm, e, srt, grp, lq, XT, inown, pos, nxl, outv, lane);
                if (lane == 0) {
                    if (pass) {
                        S.ok[c] = 1;
                        S.vp[c] = (int16_t)d;
                    } else {
                        M[(int64_t)c * nm + d] = 1;
                        M[(int64_t)d * nm + c] = 1;
                        // the rows whose best partner this pair was look again
                        S.redo[c] = 1;
                        if (S.ra[d] == c) S.redo[d] = 1;
                    }
                }
            }
            if (threadIdx.x == 0) S.cnt = 0;
            __syncthreads();
            for (int q = threadIdx.x; q < nm; q += kMergeThreads)
                if (S.redo[q]) {
                    S.redo[q] = 0;
                    S.list[atomicAdd(&S.cnt, 1)] = (int16_t)q;
                }
            __syncthreads();
            const int nr = S.cnt;
            for (int k = wv; k < nr; k += kMergeWaves) merge_row_best(S, S.list[k], nm, L, M, lane);
            __syncthreads();
            continue;
        }
        if (bc < 0) break;  // no pair left
        // merge d into c, the cluster with the smaller representative id
        int c = bc, d = S.ra[bc];
        if (S.gid[d] < S.gid[c]) {
            const int x = c;
            c = d;
            d = x;
        }
        const int sc = S.st[c], zc = S.sz[c], sd = S.st[d], zd = S.sz[d];
        // slowest links into the grown cluster, before its column of XT changes
        for (int t = threadIdx.x; t < zc + zd; t += kMergeThreads) {
            const int m = S.perm[t < zc ? sc + t : sd + t - zc];
            const double x = XT[(int64_t)(t < zc ? d : c) * nm + m];
            const int gm = S.gid[m];
            if (x < inown[gm]) inown[gm] = x;
        }
        // complete linkage is the lesser of the two rows; pairs with the grown
        // cluster are new pairs
        for (int v = threadIdx.x; v < nm; v += kMergeThreads) {
            if (v == c || v == d) continue;
            const double lc = L[(int64_t)c * nm + v], ld = L[(int64_t)d * nm + v];
            const double l = lc < ld ? lc : ld;
            L[(int64_t)c * nm + v] = l;
            L[(int64_t)v * nm + c] = l;
            M[(int64_t)c * nm + v] = 0;
            M[(int64_t)v * nm + c] = 0;
        }
        __syncthreads();
        for (int v = threadIdx.x; v < nm; v += kMergeThreads) {
            const double xc = XT[(int64_t)c * nm + v], xd = XT[(int64_t)d * nm + v];
            XT[(int64_t)c * nm + v] = xc < xd ? xc : xd;
        }
        for (int t = threadIdx.x; t < zd; t += kMergeThreads) S.rep[S.perm[sd + t]] = (int16_t)c;
        // the two member ranges side by side: rotate the stretch between them
        const int lo = sd > sc ? sc + zc : sd, hi = sd > sc ? sd + zd : sc + zc;
        for (int t = lo + (int)threadIdx.x; t < hi; t += kMergeThreads) S.tmp[t] = S.perm[t];
        __syncthreads();
        if (sd > sc) {  // d's range moves down to just after c's
            for (int t = lo + (int)threadIdx.x; t < hi; t += kMergeThreads)
                S.perm[t] = t < lo + zd ? S.tmp[sd + (t - lo)] : S.tmp[t - zd];
            for (int q = threadIdx.x; q < nm; q += kMergeThreads)
                if (S.rep[q] == q && q != c && S.st[q] >= lo && S.st[q] < sd) S.st[q] += zd;
        } else {  // d's range moves up to just after c's, which moves down
            for (int t = lo + (int)threadIdx.x; t < hi; t += kMergeThreads)
                S.perm[t] = t < hi - zd ? S.tmp[t + zd] : S.tmp[sd + (t - (hi - zd))];
            for (int q = threadIdx.x; q < nm; q += kMergeThreads)
                if (S.rep[q] == q && q != c && S.st[q] > sd && S.st[q] < sc) S.st[q] -= zd;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            if (sd < sc) S.st[c] = (int16_t)(sc - zd);
            S.sz[c] = (int16_t)(zc + zd);
            S.cnt = 0;
        }
        __syncthreads();
        // each member's first sorted-row entry outside the grown cluster,
        // kScan entries' loads in flight at a time
        for (int t = threadIdx.x; t < zc + zd; t += kMergeThreads) {
            constexpr int kScan = 8;
            const int gm = S.gid[S.perm[S.st[c] + t]];
            const int32_t *row = srt + (int64_t)gm * n;
            int p = pos[gm], w = -1;
            while (p < n - 1) {
                int ws[kScan], gg[kScan], ll[kScan];
#pragma unroll
                for (int k = 0; k < kScan; ++k) ws[k] = p + k < n - 1 ? row[p + k] : -1;
#pragma unroll
                for (int k = 0; k < kScan; ++k) {
                    gg[k] = ws[k] >= 0 ? grp[ws[k]] : -1;
                    ll[k] = ws[k] >= 0 ? lq[ws[k]] : 0;
                }
                int hit = -1;
#pragma unroll
                for (int k = 0; k < kScan; ++k)
                    if (hit < 0 && ws[k] >= 0 && (gg[k] != g || S.rep[ll[k]] != c)) hit = k;
                if (hit >= 0) {
                    w = ws[hit];
                    p += hit;
                    break;
                }
                p += kScan;  // all in the cluster, or past the row's end
            }
            if (p > n - 1) p = n - 1;
            pos[gm] = p;
            if (p < n - 1) {
                nxl[gm] = grp[w] == g ? lq[w] : -1;
                outv[gm] = e[(int64_t)gm * n + w];
            } else {
                nxl[gm] = -1;
                outv[gm] = kNoPair;
            }
        }
        // rows to look again: the grown cluster's, and those whose best partner
        // was one of the two; the others may now prefer the grown cluster
        for (int q = threadIdx.x; q < nm; q += kMergeThreads) {
            if (S.rep[q] != q) continue;
            if (q == c || S.vp[q] == c || S.vp[q] == d) S.vp[q] = -1;
            if (q == c || S.ra[q] == c || S.ra[q] == d) {
                S.list[atomicAdd(&S.cnt, 1)] = (int16_t)q;
            } else {
                const double l = L[(int64_t)q * nm + c];
                if (l != kNoPair &&
                    (S.ra[q] < 0 || pair_before(l, S.gid[q], S.gid[c], S.rb[q], S.gid[q], S.gid[S.ra[q]]))) {
                    S.rb[q] = l;
                    S.ra[q] = (int16_t)c;
                    S.ok[q] = 0;
                }
            }
        }
        __syncthreads();
        const int nr = S.cnt;
        for (int k = wv; k < nr; k += kMergeWaves) merge_row_best(S, S.list[k], nm, L, M, lane);
        __syncthreads();
    }
    for (int q = threadIdx.x; q < nm; q += kMergeThreads) cl[S.gid[q]] = S.gid[S.rep[q]];
}

// ---------------------------------------------------------------------------
// numbering and island attributes
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void islands_number(int n, const int32_t *__restrict__ cl,
                                                       const int32_t *__restrict__ gpus,
                                                       const double *__restrict__ val, int32_t *island_of,
                                                       int32_t *out_k, int32_t *isl_gpus, double *isl_val) {
    __shared__ int32_t lds[1024 / kWave + 1];
    __shared__ int32_t id[kMaxNodes];
    // island id of a representative: representatives before it
    int32_t carry = 0;
    for (int base = 0; base < n; base += blockDim.x) {
        const int u = base + threadIdx.x;
        const int32_t rep = (u < n && cl[u] == u) ? 1 : 0;
        int32_t tot;
        const int32_t ex = block_excl_scan<int32_t>(rep, lds, &tot);
        if (u < n) id[u] = carry + ex;
        carry += tot;
    }
    __syncthreads();
    const int K = carry;
    for (int k = threadIdx.x; k < K; k += blockDim.x) {
        isl_gpus[k] = 0;
        for (int f = 0; f < 4; ++f) isl_val[(int64_t)f * n + k] = __builtin_huge_val();
    }
    __syncthreads();
    // GPU sums and least values: integer sums and minima do not depend on the
    // order of the updates; the values are non-negative (a zero taken as +0),
    // so their bit patterns order like the values
    for (int u = threadIdx.x; u < n; u += blockDim.x) {
        const int k = id[cl[u]];
        island_of[u] = k;
        atomicAdd(&isl_gpus[k], gpus[u]);
        for (int f = 0; f < 4; ++f) {
            const double v = val[(int64_t)f * n + u];
            atomicMin((unsigned long long *)&isl_val[(int64_t)f * n + k],
                      (unsigned long long)__double_as_longlong(v == 0.0 ? 0.0 : v));
        }
    }
    if (threadIdx.x == 0) *out_k = K;
}

// Island-to-island bandwidth: block u reduces its row per destination island
// in LDS, then one atomic per (u, island) into the K x K matrix.  The values
// are non-negative, so their bit patterns order like the values.
__global__ __launch_bounds__(256) void islands_inter_init(int64_t kk, int K, double *isl_e) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < kk) isl_e[t] = (t / K == t % K) ? 0.0 : __builtin_huge_val();
}

__global__ __launch_bounds__(256) void islands_inter(int n, const int32_t *__restrict__ out_k,
                                                     const double *__restrict__ e,
                                                     const int32_t *__restrict__ island_of, double *isl_e) {
    __shared__ unsigned long long m[kMaxNodes];
    const int u = blockIdx.x;
    const int K = *out_k;
    const int a = island_of[u];
    for (int k = threadIdx.x; k < K; k += blockDim.x) m[k] = 0x7FF0000000000000ull;  // +inf
    __syncthreads();
    for (int v = threadIdx.x; v < n; v += blockDim.x) {
        const int b = island_of[v];
        if (b != a) atomicMin(&m[b], (unsigned long long)__double_as_longlong(e[(int64_t)u * n + v]));
    }
    __syncthreads();
    for (int k = threadIdx.x; k < K; k += blockDim.x)
        if (k != a && m[k] != 0x7FF0000000000000ull)
            atomicMin((unsigned long long *)&isl_e[(int64_t)a * K + k], m[k]);
}

hipError_t launch_build_islands(int n, const tg_island *nodes_host, const double *e_host, double eps_c,
                                double eps_m, double eps_i, void *ws, hipStream_t s, int32_t *island_of,
                                tg_island *islands, double *inter_bw, int32_t *n_islands, int64_t *bad_bw) {
    const IslandWs w = carve_islands(n, ws);
    // node columns, uploaded from the caller's arrays
    std::vector<int32_t> hg(n);
    std::vector<double> hv((size_t)4 * n);
    for (int u = 0; u < n; ++u) {
        hg[u] = nodes_host[u].n_gpus;
        hv[u] = nodes_host[u].peak_flops;
        hv[n + u] = nodes_host[u].hbm_bytes;
        hv[2 * n + u] = nodes_host[u].intra_bw;
        hv[3 * n + u] = nodes_host[u].host_bw;
    }
    hipError_t e = hipMemcpyAsync(w.gpus, hg.data(), 4 * (size_t)n, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(w.val, hv.data(), 8 * 4 * (size_t)n, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(w.e, e_host, 8 * (size_t)n * n, hipMemcpyHostToDevice, s);
    const int32_t none[2] = {0, INT32_MAX};
    if (e == hipSuccess) e = hipMemcpyAsync(w.err, none, sizeof(none), hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return e;
    const int64_t nn = (int64_t)n * n;
    islands_check<<<dim3((unsigned)std::min<int64_t>((nn + 255) / 256, 2048)), dim3(256), 0, s>>>(nn, w.e, w.err + 1);
    int32_t bad = INT32_MAX;
    e = hipMemcpyAsync(&bad, w.err + 1, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);  // the host staging arrays go away
    if (e != hipSuccess) return e;
    *bad_bw = bad == INT32_MAX ? -1 : bad;
    if (bad != INT32_MAX) return hipSuccess;
    islands_groups<<<dim3(1), dim3(kGroupThreads), 0, s>>>(n, w.gpus, w.val, eps_c, eps_m, eps_i, w.grp, w.gstart,
                                                           w.gnodes, w.ngroups, w.lq, w.goff);
    islands_link_init<<<dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, s>>>(
        n, w.e, w.grp, w.gstart, w.lq, w.goff, w.L, w.M, w.XT, w.inown, w.cl);
    islands_sort_rows<<<dim3((unsigned)n), dim3(1024), 0, s>>>(n, w.e, w.srt);
    islands_merge<<<dim3((unsigned)n), dim3(kMergeThreads), 0, s>>>(n, w.e, w.srt, w.grp, w.lq, w.gstart, w.gnodes,
                                                                     w.ngroups, w.goff, w.L, w.M, w.XT, w.inown,
                                                                     w.pos, w.nxl, w.outv, w.cl, w.err);
    islands_number<<<dim3(1), dim3(1024), 0, s>>>(n, w.cl, w.gpus, w.val, w.island_of, w.out_k, w.isl_gpus,
                                                  w.isl_val);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    int32_t K = 0, merr = 0;
    e = hipMemcpyAsync(&K, w.out_k, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&merr, w.err, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
    if (merr) return hipErrorUnknown;
    const int64_t kk = (int64_t)K * K;
    islands_inter_init<<<dim3((unsigned)((kk + 255) / 256)), dim3(256), 0, s>>>(kk, K, w.isl_e);
    islands_inter<<<dim3((unsigned)n), dim3(256), 0, s>>>(n, w.out_k, w.e, w.island_of, w.isl_e);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    std::vector<int32_t> og(K > 0 ? K : 1);
    std::vector<double> ov((size_t)4 * n);
    e = hipMemcpyAsync(island_of, w.island_of, 4 * (size_t)n, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(og.data(), w.isl_gpus, 4 * (size_t)K, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(ov.data(), w.isl_val, 8 * 4 * (size_t)n, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(inter_bw, w.isl_e, 8 * (size_t)kk, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess) {
        for (int k = 0; k < K; ++k) {
            islands[k].n_gpus = og[k];
            islands[k].reserved = 0;
            islands[k].peak_flops = ov[k];
            islands[k].hbm_bytes = ov[n + k];
            islands[k].intra_bw = ov[2 * n + k];
            islands[k].host_bw = ov[3 * n + k];
        }
        *n_islands = K;
    }
    return e;
}

}  // namespace tg
