// compose.hip -- pipeline composition (Sec. 5.2) on the GPU.
//
// A plan picks a micro-batch size b, an ordered subsequence of islands (in the
// caller's island order; skipped islands are eliminated), cuts of the layers
// into contiguous stages and, per stage, a candidate fitting at the stage's
// depth (stages from it to the pipeline end).  Per b the plan minimises the
// bottleneck P (composition steps (1)-(2): least achievable largest stage or
// link time), then the fill F at that bottleneck (step (3)).  Plans are built
// by adding stages in front, so each stage's depth is known when it is added.
//
// Tables (o = island position in the order, d = depth):
//   T_d(s, o)  least cost in group (s, island o, b) among candidates fitting at d
//   V_d(i, o)  least bottleneck covering [i, L) with d stages, first on o
//   W_d(j, o)  least bottleneck of a continuation after a stage on o ending at j
//   F_d, G_d   the same for the fill, restricted to stages and links <= P*
// Work: one launch per depth level and phase; block (i, b) owns row i of V/W
// (or F/G) for every position o (one thread per o).  T_d changes only where a
// group's least fitting candidate changes; those changes are precomputed as
// events bucketed by (level, b, first layer i) and applied by the block that
// reads them, so the table is never rebuilt.
//
// T_d(i, j, o) never decreases as j grows (a longer slice costs at least as
// much under every config and fits in memory under fewer), so a row's scan
// over j stops at the first T not below the running best: no later j can
// improve it.  This holds whenever the candidate list contains the surviving
// set, since then T_d equals the least cost over all group members.
#include <algorithm>
#include <cmath>
#include <vector>
#include <climits>
#include <cstddef>
#include <type_traits>

#include "compose_util.h"

#pragma clang fp contract(off)

namespace tg {

constexpr int kScanThreads = 256;
constexpr int kScanPerThread = 16;  // four 16-byte loads of consecutive counts per thread
constexpr int kScanTile = kScanThreads * kScanPerThread;

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---------------------------------------------------------------------------
// generic helpers
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void fill_kernel(T *a, int64_t n, T v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        a[i] = v;
}

template <typename T>
static void fill(T *a, int64_t n, T v, hipStream_t s) {
    if (n <= 0) return;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    fill_kernel<T><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a, n, v);
}

// A thread's kScanPerThread consecutive int32 counts (zeros past n); the
// array base is 16-byte aligned (workspace offsets are multiples of 256).
__device__ inline void load_counts(const int32_t *a, int64_t n, int64_t first, int32_t (&v)[kScanPerThread]) {
    if (first + kScanPerThread <= n) {
        const int4 *q = (const int4 *)(a + first);
#pragma unroll
        for (int u = 0; u < kScanPerThread / 4; ++u) {
            const int4 x = q[u];
            v[4 * u] = x.x;
            v[4 * u + 1] = x.y;
            v[4 * u + 2] = x.z;
            v[4 * u + 3] = x.w;
        }
    } else {
#pragma unroll
        for (int u = 0; u < kScanPerThread; ++u) v[u] = first + u < n ? a[first + u] : 0;
    }
}

__global__ __launch_bounds__(kScanThreads) void scan_reduce_i32(const int32_t *a, int64_t n, int64_t *tile_sum) {
    __shared__ int64_t lds[kScanThreads / kWave + 1];
    const int64_t first = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPerThread;
    int32_t v[kScanPerThread];
    load_counts(a, n, first, v);
    int64_t c = 0;
#pragma unroll
    for (int u = 0; u < kScanPerThread; ++u) c += v[u];
    int64_t total;
    block_excl_scan<int64_t>(c, lds, &total);
    if (threadIdx.x == 0) tile_sum[blockIdx.x] = total;
}

__global__ __launch_bounds__(1024) void scan_tiles_i64(int64_t *a, int64_t n) {
    __shared__ int64_t lds[1024 / kWave + 1];
    int64_t carry = 0;
    for (int64_t base = 0; base < n; base += blockDim.x) {
        const int64_t i = base + threadIdx.x;
        const int64_t v = i < n ? a[i] : 0;
        int64_t sum;
        const int64_t ex = block_excl_scan<int64_t>(v, lds, &sum);
        if (i < n) a[i] = carry + ex;
        carry += sum;
    }
}

__global__ __launch_bounds__(kScanThreads) void scan_apply_i32(int32_t *a, int64_t n, const int64_t *tile_off) {
    __shared__ int64_t lds[kScanThreads / kWave + 1];
    const int64_t first = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPerThread;
    int32_t v[kScanPerThread];
    load_counts(a, n, first, v);
    int64_t c = 0;
#pragma unroll
    for (int u = 0; u < kScanPerThread; ++u) c += v[u];
    int64_t total;
    int64_t run = tile_off[blockIdx.x] + block_excl_scan<int64_t>(c, lds, &total);
    int32_t out[kScanPerThread];
#pragma unroll
    for (int u = 0; u < kScanPerThread; ++u) {
        out[u] = (int32_t)run;
        run += v[u];
    }
    if (first + kScanPerThread <= n) {
        int4 *q = (int4 *)(a + first);
#pragma unroll
        for (int u = 0; u < kScanPerThread / 4; ++u) q[u] = make_int4(out[4 * u], out[4 * u + 1], out[4 * u + 2], out[4 * u + 3]);
    } else {
#pragma unroll
        for (int u = 0; u < kScanPerThread; ++u)
            if (first + u < n) a[first + u] = out[u];
    }
}

// In-place exclusive scan of an int32 array; tmp holds >= tiles int64.
static void scan_i32(int32_t *a, int64_t n, int64_t *tmp, hipStream_t s) {
    if (n <= 0) return;
    const int64_t tiles = (n + kScanTile - 1) / kScanTile;
    scan_reduce_i32<<<dim3((unsigned)tiles), dim3(kScanThreads), 0, s>>>(a, n, tmp);
    scan_tiles_i64<<<dim3(1), dim3(1024), 0, s>>>(tmp, tiles);
    scan_apply_i32<<<dim3((unsigned)tiles), dim3(kScanThreads), 0, s>>>(a, n, tmp);
}

// ---------------------------------------------------------------------------
// workspace
// ---------------------------------------------------------------------------
struct Ws {
    ComposeResult *res;
    int32_t *order;    // [K] copy of the caller's order
    int32_t *pos;      // [K] island -> position
    double *EoT;       // [K*K] EoT[o2*K + o] = E[order[o]][order[o2]]
    uint8_t *EiT;      // [K(K-1)/2] index of E[order[o]][order[o2]] (o < o2) in the distinct list
    int32_t *rec_g;    // [n] group of list entry r, -1 if unused
    double *rec_c;     // [n] its cost
    uint8_t *rec_d;    // [n] its d_max
    int32_t *gcnt;     // [n_groups] counts -> offsets -> ends (group order)
    double *ent_c;     // [n] grouped entries: cost
    uint8_t *ent_d;    // [n] d_max
    int64_t *ent_i;    // [n] candidate index
    int32_t *rowev;    // [nb][L][D+1] per row (b, i): where the events of each level start (last = end)
    int32_t *ev_total; // [1] events reserved so far
    int32_t *ev_cell;  // [2n]
    double *ev_val;    // [2n]
    double *T;         // [n_groups] current stage table of phase 1, layout [b][s][o] (= group order)
    double *T0;        // [n_groups] the same starting table for phase 2
    double *T1;        // [nb][L][K] depth-1 table of the slices (i, L)
    int32_t *jlo_pos;  // [K][L] first balanced cut by island position (imbalance pruning)
    double *Wb[2];     // [nb][L+1][K] continuation rows, double-buffered by level
    uint16_t *argF;    // [D][nb][L][K]
    uint8_t *argG;     // [D][nb][L+1][K]
    double *Pst;       // [nb]
    double *rootF;     // [nb]
    int32_t *root_o;   // [nb]
    int32_t *root_d;   // [nb]
    double *Rv;        // [D][nb] least bottleneck of a whole plan with d stages (phase 1, per level)
    double *RF;        // [D][nb] least root fill with d stages (phase 2, per level)
    int32_t *RO;       // [D][nb] its first position (least on ties), -1 if none
    int32_t *dlim;     // [nb] deepest level whose root bottleneck reaches P* (0: no plan)
    int64_t *tmp;      // scan tiles
    size_t bytes;
};

__host__ __device__ inline int64_t n_groups(const DevProblem &P) { return (int64_t)P.nb * P.NS * P.K; }
static int levels(const DevProblem &P) { return P.K < P.L ? P.K : P.L; }
static int64_t n_rowev(const DevProblem &P) { return (int64_t)P.nb * P.L * (levels(P) + 1); }

static Ws carve(const DevProblem &P, int64_t n, void *base) {
    Ws w{};
    char *p = (char *)base;
    size_t off = 0;
    auto take = [&](size_t bytes) -> void * {
        void *r = base ? (void *)(p + off) : nullptr;
        off += align256(bytes > 0 ? bytes : 1);
        return r;
    };
    const int64_t G = n_groups(P), D = levels(P);
    const int64_t rows = (int64_t)P.nb * (P.L + 1) * P.K;
    const int64_t tiles = (G + kScanTile - 1) / kScanTile + 1;
    const int64_t K2 = (int64_t)P.K * P.K;
    w.res = (ComposeResult *)take(sizeof(ComposeResult));
    w.order = (int32_t *)take(sizeof(int32_t) * P.K);
    w.pos = (int32_t *)take(sizeof(int32_t) * P.K);
    w.EoT = (double *)take(sizeof(double) * K2);
    w.EiT = (uint8_t *)take((size_t)K2 / 2 + 4);
    w.rec_g = (int32_t *)take(sizeof(int32_t) * n);
    w.rec_c = (double *)take(sizeof(double) * n);
    w.rec_d = (uint8_t *)take(n);
    w.gcnt = (int32_t *)take(sizeof(int32_t) * G);
    w.ent_c = (double *)take(sizeof(double) * n);
    w.ent_d = (uint8_t *)take(n);
    w.ent_i = (int64_t *)take(sizeof(int64_t) * n);
    w.rowev = (int32_t *)take(sizeof(int32_t) * n_rowev(P));
    w.ev_total = (int32_t *)take(sizeof(int32_t));
    w.ev_cell = (int32_t *)take(sizeof(int32_t) * 2 * n);
    w.ev_val = (double *)take(sizeof(double) * 2 * n);
    w.T = (double *)take(sizeof(double) * G);
    w.T0 = (double *)take(sizeof(double) * G);
    w.T1 = (double *)take(sizeof(double) * P.nb * P.L * P.K);
    w.jlo_pos = (int32_t *)take(P.imb ? sizeof(int32_t) * P.K * P.L : 1);
    w.Wb[0] = (double *)take(sizeof(double) * rows);
    w.Wb[1] = (double *)take(sizeof(double) * rows);
    w.argF = (uint16_t *)take(sizeof(uint16_t) * D * P.nb * P.L * P.K);
    w.argG = (uint8_t *)take(sizeof(uint8_t) * D * rows);
    w.Pst = (double *)take(sizeof(double) * P.nb);
    w.rootF = (double *)take(sizeof(double) * P.nb);
    w.root_o = (int32_t *)take(sizeof(int32_t) * P.nb);
    w.root_d = (int32_t *)take(sizeof(int32_t) * P.nb);
    w.Rv = (double *)take(sizeof(double) * D * P.nb);
    w.RF = (double *)take(sizeof(double) * D * P.nb);
    w.RO = (int32_t *)take(sizeof(int32_t) * D * P.nb);
    w.dlim = (int32_t *)take(sizeof(int32_t) * P.nb);
    w.tmp = (int64_t *)take(sizeof(int64_t) * tiles);
    w.bytes = off;
    return w;
}

size_t compose_ws_bytes(const DevProblem &P, int64_t n_surv) { return carve(P, n_surv, nullptr).bytes; }
size_t compose_order_offset(const DevProblem &P, int64_t n_surv) {
    (void)P;
    (void)n_surv;
    return align256(sizeof(ComposeResult));
}

// The stage table keeps the DP's layout [b][slice][position].
__host__ __device__ inline int64_t cell_id(const DevProblem &P, int64_t bi, int64_t s, int64_t o) {
    return (bi * P.NS + s) * P.K + o;
}

// Index of the pair of positions (o, o2), o < o2, in a packed triangle.
__host__ __device__ inline int tri(int o, int o2) { return o2 * (o2 - 1) / 2 + o; }

__global__ __launch_bounds__(256) void prep_kernel(DevProblem P, const int32_t *order, int32_t *pos, double *EoT,
                                                   uint8_t *EiT, ComposeResult *res, int32_t *ev_total) {
    const int K = P.K;
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t < K) pos[order[t]] = t;
    if (t < K * K) {
        const int o2 = t / K, o = t - o2 * K;
        const int64_t e = (int64_t)order[o] * K + order[o2];
        EoT[t] = P.E[e];
        if (o < o2) EiT[tri(o, o2)] = P.n_ev ? (uint8_t)P.Eidx[e] : 0;
    }
    if (t == 0) {
        res->err = 0;
        res->status = TG_ENOPLAN;
        *ev_total = 0;
    }
}

// First balanced cut of each first layer, by island position of this call.
__global__ __launch_bounds__(256) void jlo_kernel(DevProblem P, const int32_t *order, int32_t *jlo_pos) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= P.K * P.L) return;
    const int o = t / P.L, i = t - o * P.L;
    jlo_pos[t] = P.jlo[order[o] * P.L + i];
}

// ---------------------------------------------------------------------------
// grouping: candidate list -> per-group entry records -> per-level events
// ---------------------------------------------------------------------------
// Reads each listed candidate's score once (the list is ascending, so the
// reads walk the score arrays forward) and counts the group sizes.  A thread
// takes kGatherPer entries, a block's threads apart, with all their loads in
// flight together.
constexpr int kGatherPer = 4;
constexpr int kGatherBlock = 256 * kGatherPer;

__global__ __launch_bounds__(256) void gather_kernel(DevProblem P, const int64_t *surv, int64_t n,
                                                     const double *cost, const uint8_t *dmax, const int32_t *pos,
                                                     int32_t *rec_g, double *rec_c, uint8_t *rec_d, int32_t *gcnt,
                                                     ComposeResult *res) {
    const int64_t r0 = (int64_t)blockIdx.x * kGatherBlock + threadIdx.x;
    int64_t idx[kGatherPer], prev[kGatherPer];
#pragma unroll
    for (int u = 0; u < kGatherPer; ++u) {
        const int64_t r = r0 + u * 256;
        idx[u] = r < n ? surv[r] : 0;
        prev[u] = (r < n && r > 0) ? surv[r - 1] : -1;
    }
    int32_t G[kGatherPer];
    int64_t si[kGatherPer];
    int err = 0;
#pragma unroll
    for (int u = 0; u < kGatherPer; ++u) {
        const int64_t r = r0 + u * 256;
        G[u] = -1;
        si[u] = -1;
        if (r >= n) continue;
        if (idx[u] < 0 || idx[u] >= P.N || prev[u] >= idx[u]) {
            err |= 1;
            continue;
        }
        const int64_t g = idx[u] / P.NS, s = idx[u] - g * P.NS;
        const Coef &c = P.coef[g];
        const uint32_t ij = P.sij[s];
        if (c.b_idx < 0 || !slice_balanced(P, P.pre, (int)(ij & 0xFFFFu), (int)(ij >> 16), c.k)) {
            err |= 2;
            continue;
        }
        G[u] = (int32_t)group_id(P, pos[c.k], c.b_idx, s);
        // scores by candidate, or by class candidate (equal on every slice of the class)
        si[u] = P.class_scores ? g * P.NC + P.cls[s] : idx[u];
    }
    uint8_t d[kGatherPer];
    double cv[kGatherPer];
#pragma unroll
    for (int u = 0; u < kGatherPer; ++u) {
        d[u] = si[u] >= 0 ? dmax[si[u]] : 0;
        cv[u] = si[u] >= 0 ? cost[si[u]] : 0.0;
    }
#pragma unroll
    for (int u = 0; u < kGatherPer; ++u) {
        const int64_t r = r0 + u * 256;
        if (r >= n) continue;
        if (d[u] == 0) G[u] = -1;  // fits nowhere: not a group entry
        if (G[u] >= 0) {
            rec_c[r] = cv[u];
            rec_d[r] = d[u];
            atomicAdd(&gcnt[G[u]], 1);
        }
        rec_g[r] = G[u];
    }
    if (err) atomicOr(&res->err, err);
}

__global__ __launch_bounds__(256) void scatter_kernel(const int64_t *surv, int64_t n, const int32_t *rec_g,
                                                      const double *rec_c, const uint8_t *rec_d, int32_t *gcnt,
                                                      double *ent_c, uint8_t *ent_d, int64_t *ent_i) {
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x) {
        const int32_t G = rec_g[r];
        if (G < 0) continue;
        const int32_t slot = atomicAdd(&gcnt[G], 1);
        ent_c[slot] = rec_c[r];
        ent_d[slot] = rec_d[r];
        ent_i[slot] = surv[r];
    }
}

int64_t group_scan_tiles(int64_t n) { return (n + kScanTile - 1) / kScanTile + 1; }

void launch_grouping(const DevProblem &P, const int64_t *surv, int64_t n, const double *cost,
                     const uint8_t *dmax, const int32_t *pos, const Groups &g, ComposeResult *res,
                     hipStream_t s) {
    const int64_t G = n_groups(P);
    fill<int32_t>(g.gcnt, G, 0, s);
    if (n > 0) {
        const int64_t blocks = (n + kGatherBlock - 1) / kGatherBlock;
        gather_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, surv, n, cost, dmax, pos, g.rec_g, g.rec_c,
                                                                    g.rec_d, g.gcnt, res);
        scan_i32(g.gcnt, G, g.tmp, s);
        const int64_t sblocks = std::min<int64_t>((n + 255) / 256, 65536);
        scatter_kernel<<<dim3((unsigned)sblocks), dim3(256), 0, s>>>(surv, n, g.rec_g, g.rec_c, g.rec_d, g.gcnt,
                                                                      g.ent_c, g.ent_d, g.ent_i);
    } else {
        scan_i32(g.gcnt, G, g.tmp, s);  // all zeros: offsets stay zero
    }
}

// Per group: entry e is the least fitting candidate at depths (D_e, d_e],
// D_e = the largest d_max among entries with a smaller key; it sets T at
// level D_e + 1.  After the group's largest d_max M nothing fits: T = +inf
// from level M + 1.  At most one change per (group, level).  Levels 1 and 2
// come from the starting tables, so only changes at levels >= 3 become
// events.  Also returns the starting values: v1 the least cost of the group
// (depth 1), v2 the least cost fitting at depth 2.
constexpr int kGroupRegs = 4;

template <typename Emit>
__device__ inline void cell_events(const int32_t *__restrict__ gcnt, const double *__restrict__ ent_c,
                                   const uint8_t *__restrict__ ent_d, const int64_t *__restrict__ ent_i, int64_t G,
                                   int D, double &v1, double &v2, Emit emit) {
    v1 = kInf;
    v2 = kInf;
    const int32_t st = G ? gcnt[G - 1] : 0, en = gcnt[G];
    if (st == en) return;
    int M = 0;
    if (en - st <= kGroupRegs) {
        // small group (the usual staircase): entries in registers, compared
        // there; the indices only break cost ties, so they load only when
        // two entries cost the same (never among a surviving set's entries of
        // one group, where the deeper or earlier of two equal costs dominates)
        double c[kGroupRegs];
        int d[kGroupRegs];
        int64_t id[kGroupRegs];
        const int n = en - st;
#pragma unroll
        for (int e = 0; e < kGroupRegs; ++e) {
            c[e] = e < n ? ent_c[st + e] : kInf;
            d[e] = e < n ? (int)ent_d[st + e] : 0;
        }
        bool tie = false;
#pragma unroll
        for (int e = 0; e < kGroupRegs; ++e)
#pragma unroll
            for (int q = e + 1; q < kGroupRegs; ++q) tie = tie || (q < n && c[q] == c[e]);
#pragma unroll
        for (int e = 0; e < kGroupRegs; ++e) id[e] = (tie && e < n) ? ent_i[st + e] : 0;
#pragma unroll
        for (int e = 0; e < kGroupRegs; ++e) {
            if (e >= n) break;
            M = max(M, d[e]);
            v1 = fmin(v1, c[e]);
            if (d[e] >= 2) v2 = fmin(v2, c[e]);
            int De = 0;
#pragma unroll
            for (int q = 0; q < kGroupRegs; ++q) {
                const bool less =
                    q < n && (c[q] < c[e] || (c[q] == c[e] && (d[q] > d[e] || (d[q] == d[e] && id[q] < id[e]))));
                if (less) De = max(De, d[q]);
            }
            if (De >= 2 && De < d[e] && De + 1 <= D) emit(De + 1, c[e]);
        }
    } else {
        for (int32_t e = st; e < en; ++e) {
            const double ce = ent_c[e];
            const int de = ent_d[e];
            M = max(M, de);
            v1 = fmin(v1, ce);
            if (de >= 2) v2 = fmin(v2, ce);
            int De = 0;
            for (int32_t q = st; q < en; ++q) {
                const double cq = ent_c[q];
                const int dq = ent_d[q];
                // indices only for an exact tie in cost and depth
                const bool less = cq < ce || (cq == ce && (dq > de || (dq == de && ent_i[q] < ent_i[e])));
                if (less) De = max(De, dq);
            }
            if (De >= 2 && De < de && De + 1 <= D) emit(De + 1, ce);
        }
    }
    if (M >= 2 && M + 1 <= D) emit(M + 1, kInf);
}

// Starting tables and events, one block per row (b, first layer i): its
// cells are the slices starting at i times the positions, taken in tiles of
// 64 slices x 16 positions.  A wave reads the offsets and entries of 64
// consecutive groups (the group order runs along slices) and the block writes
// the tile through LDS along positions (the table order), 128-byte runs.  A
// first sweep writes the starting stage table (depth 2; two copies, one per
// phase) and, for the slice (i, L), the depth-1 table T1[b][i][o], and counts
// the row's events per level in LDS; the block then reserves one range for
// all of them (one atomic) and records where each level's events start in
// rowev[b][i][.]; a second sweep (whose reads hit the caches) writes the
// events grouped by level.  The level kernel that owns row i at level d then
// applies the events of level d + 1 from one contiguous range.
constexpr int kRowThreads = 1024;
constexpr int kRowTileS = 64, kRowTileO = kRowThreads / kRowTileS;

// 16-wave blocks at 8 waves per SIMD: two blocks per CU (64 VGPRs), so one
// block's tile barriers overlap the other's loads
__global__ __launch_bounds__(kRowThreads, 8) void row_tables(DevProblem P, const int32_t *__restrict__ gcnt,
                                                             const double *__restrict__ ent_c,
                                                             const uint8_t *__restrict__ ent_d,
                                                             const int64_t *__restrict__ ent_i,
                                                             double *__restrict__ T, double *__restrict__ T0,
                                                             double *__restrict__ T1, int32_t *rowev,
                                                             int32_t *ev_total, int32_t *__restrict__ ev_cell,
                                                             double *__restrict__ ev_val) {
    __shared__ int32_t hist[256];
    __shared__ int64_t scan_lds[kRowThreads / kWave + 1];
    __shared__ double tile[kRowTileO][kRowTileS + 1];
    __shared__ int32_t base;
    const int i = blockIdx.x, bi = blockIdx.y;
    const int L = P.L, K = P.K;
    const int D = K < L ? K : L;
    const int64_t s0 = slice_of(L, i, i + 1);
    const int n_sl = L - i;
    const int64_t t1row = ((int64_t)bi * L + i) * K;
    const int ol = threadIdx.x / kRowTileS, jl = threadIdx.x % kRowTileS;  // reading: 64 slices per wave
    const int ow = threadIdx.x % kRowTileO, jw = threadIdx.x / kRowTileO;  // writing: 16 positions per run
    for (int lev = threadIdx.x; lev < 256; lev += kRowThreads) hist[lev] = 0;
    __syncthreads();
    for (int j0 = 0; j0 < n_sl; j0 += kRowTileS)
        for (int o0 = 0; o0 < K; o0 += kRowTileO) {
            const int js = j0 + jl, o = o0 + ol;
            double v2 = kInf;
            if (js < n_sl && o < K) {
                double v1;
                cell_events(gcnt, ent_c, ent_d, ent_i, group_id(P, o, bi, s0 + js), D, v1, v2,
                            [&](int level, double) { atomicAdd(&hist[level - 1], 1); });
                if (js == n_sl - 1) T1[t1row + o] = v1;  // the slice (i, L)
            }
            tile[ol][jl] = v2;
            __syncthreads();
            const int jo = j0 + jw, oo = o0 + ow;
            if (jo < n_sl && oo < K) {
                const int64_t c = cell_id(P, bi, s0 + jo, oo);
                const double v = tile[ow][jw];
                T[c] = v;
                T0[c] = v;
            }
            __syncthreads();
        }
    // the row's event range and the start of each level in it
    const int lev = threadIdx.x;
    const int64_t cnt = lev < D ? hist[lev] : 0;
    int64_t total;
    const int64_t off = block_excl_scan<int64_t>(cnt, scan_lds, &total);
    if (threadIdx.x == 0) base = total ? atomicAdd(ev_total, (int32_t)total) : 0;
    __syncthreads();
    int32_t *re = rowev + ((int64_t)bi * L + i) * (D + 1);
    if (lev < D) {
        hist[lev] = base + (int32_t)off;
        re[lev] = base + (int32_t)off;
    }
    if (lev == D) re[D] = base + (int32_t)total;
    __syncthreads();
    if (total == 0) return;
    for (int j0 = 0; j0 < n_sl; j0 += kRowTileS)
        for (int o0 = 0; o0 < K; o0 += kRowTileO) {
            const int js = j0 + jl, o = o0 + ol;
            if (js >= n_sl || o >= K) continue;
            const int64_t c = cell_id(P, bi, s0 + js, o);
            double v1, v2;
            cell_events(gcnt, ent_c, ent_d, ent_i, group_id(P, o, bi, s0 + js), D, v1, v2, [&](int level, double v) {
                const int32_t slot = atomicAdd(&hist[level - 1], 1);
                ev_cell[slot] = (int32_t)c;
                ev_val[slot] = v;
            });
        }
}

// ---------------------------------------------------------------------------
// dynamic program, one launch per level
// ---------------------------------------------------------------------------
// Block (i, b) owns row i of one level for every position o; each cell (i, o)
// is served by SPLIT threads (sub-threads 0..SPLIT-1), and LDS combines them.
// The level kernels are latency chains, so each block starts its row's table
// and continuation reads and its link loads at once.  It also applies the next
// level's table changes for its row (bucket (d+1, b, i)): they touch only
// slices starting at layer i, which no other block reads, so they are loaded
// once the block's own table reads are done and written at its end.
constexpr int kEvRegs = 2;
constexpr int kEvBatch = 8;
constexpr int kAhead = 4;  // scan steps read at a time
// cut steps a bottleneck scan reads at a time: a scan stops at its first
// stage cost not below its running best, mostly within the first two steps,
// so two loads a round keep the rows' reads down (the light levels took
// 6.7 -> 6.4 µs; four a round stay better for the fill's scans)
constexpr int kCutAhead = 2;

// Waves per SIMD the level kernels are compiled for: the most a SIMD holds (8,
// so at most 64 VGPRs) rounded down to whole blocks.
constexpr int level_waves(int threads) {
    const int per_simd = (threads / kWave + 3) / 4;
    return (8 / per_simd) * per_simd;
}

struct RowEvents {
    int32_t st, en;
    int32_t c[kEvRegs];
    double v[kEvRegs];
};

// The events of level d + 1 in row (b, i): rowev[b][i][d] .. rowev[b][i][d + 1].
__device__ inline void event_bounds(RowEvents &R, const DevProblem &P, int d, int bi, int i, const int32_t *rowev) {
    const int D = P.K < P.L ? P.K : P.L;
    R.st = 0;
    R.en = 0;
    if (d < D) {
        const int32_t *re = rowev + ((int64_t)bi * P.L + i) * (D + 1);
        R.st = re[d];
        R.en = re[d + 1];
    }
}

template <int THREADS>
__device__ inline void load_events(RowEvents &R, const int32_t *__restrict__ ev_cell,
                                   const double *__restrict__ ev_val) {
#pragma unroll
    for (int k = 0; k < kEvRegs; ++k) {
        const int32_t e = R.st + (int32_t)threadIdx.x + k * THREADS;
        R.c[k] = e < R.en ? ev_cell[e] : -1;
        R.v[k] = e < R.en ? ev_val[e] : 0.0;
    }
}

template <int THREADS>
__device__ inline void store_events(const RowEvents &R, const int32_t *__restrict__ ev_cell,
                                    const double *__restrict__ ev_val, double *__restrict__ T) {
#pragma unroll
    for (int k = 0; k < kEvRegs; ++k)
        if (R.c[k] >= 0) T[R.c[k]] = R.v[k];
    // large buckets (the first levels): the rest in batches of loads in flight
    const int32_t step = THREADS;
    for (int32_t base = R.st + (int32_t)threadIdx.x + kEvRegs * step; base < R.en; base += kEvBatch * step) {
        int32_t c[kEvBatch];
        double v[kEvBatch];
#pragma unroll
        for (int k = 0; k < kEvBatch; ++k) {
            const int32_t e = base + k * step;
            c[k] = e < R.en ? ev_cell[e] : -1;
            v[k] = e < R.en ? ev_val[e] : 0.0;
        }
#pragma unroll
        for (int k = 0; k < kEvBatch; ++k)
            if (c[k] >= 0) T[c[k]] = v[k];
    }
}

// Link times of the boundary after layer i-1 for this block's b.  With few
// distinct bandwidths (the usual case) the block divides once per distinct
// value and keeps the per-pair index triangle in LDS; otherwise it divides
// per pair.  The link data is loaded into registers first and written to LDS
// after the row scan, so the loads overlap it.
struct Links {
    const double *xs;      // LDS [n_ev]
    const uint8_t *tri_s;  // LDS triangle of indices
    const double *EoT;     // global, used without a table
    double num;
    bool table;
    __device__ inline double tab(int o, int o2) const { return xs[tri_s[tri(o, o2)]]; }
    __device__ inline double direct(int o, int o2, int K) const {
        const double E = EoT[(int64_t)o2 * K + o];
        return E == 0.0 ? kInf : num / E;
    }
};

template <int THREADS, int KP>
struct LinkRegs {
    // triangle words (rows o2 <= KP-1) and distinct bandwidths per thread
    static constexpr int kWords = (((KP - 1) * KP / 2 + 3) / 4 + THREADS - 1) / THREADS;
    static constexpr int kE = (kMaxDistinctE + THREADS - 1) / THREADS;
    double E[kE];
    uint32_t w[kWords];
};

template <int THREADS, int KP>
__device__ inline Links load_links(LinkRegs<THREADS, KP> &R, const DevProblem &P, int i, int bi, int top,
                                   const uint8_t *EiT, const double *EoT, double *xs, uint8_t *tri_s) {
    Links X{xs, tri_s, EoT, 0.0, P.n_ev > 0};
    if (i == 0) return X;
    X.num = (2.0 * (double)P.bvals[bi]) * (double)P.outact[i - 1];
    if (X.table) {
#pragma unroll
        for (int k = 0; k < LinkRegs<THREADS, KP>::kE; ++k) {
            const int u = (int)threadIdx.x + k * THREADS;
            R.E[k] = u < P.n_ev ? P.Ev[u] : 0.0;
        }
        const int nwords = (top * (top + 1) / 2 + 3) / 4;  // rows o2 <= top
        const uint32_t *src = (const uint32_t *)EiT;
#pragma unroll
        for (int k = 0; k < LinkRegs<THREADS, KP>::kWords; ++k) {
            const int t = (int)threadIdx.x + k * THREADS;
            R.w[k] = t < nwords ? src[t] : 0u;
        }
    }
    return X;
}

template <int THREADS, int KP>
__device__ inline void store_links(const LinkRegs<THREADS, KP> &R, const Links &X, const DevProblem &P, int i,
                                   int top, double *xs, uint8_t *tri_s) {
    if (i == 0 || !X.table) return;
#pragma unroll
    for (int k = 0; k < LinkRegs<THREADS, KP>::kE; ++k) {
        const int u = (int)threadIdx.x + k * THREADS;
        if (u < P.n_ev) xs[u] = R.E[k] == 0.0 ? kInf : X.num / R.E[k];
    }
    const int nwords = (top * (top + 1) / 2 + 3) / 4;
    uint32_t *dst = (uint32_t *)tri_s;
#pragma unroll
    for (int k = 0; k < LinkRegs<THREADS, KP>::kWords; ++k) {
        const int t = (int)threadIdx.x + k * THREADS;
        if (t < nwords) dst[t] = R.w[k];
    }
}

// Next-position scan.  Only positions with a finite value can give the
// minimum, so when fewer than half of them are finite the block lists those
// positions (ascending) and the scan walks the list; otherwise it walks the
// positions directly.  The threads that combined the values (sub-thread 0,
// whole waves) publish one ballot mask per wave.
__device__ inline void publish_live(bool live, uint64_t *lmask) {
    const uint64_t bal = __ballot(live);
    if ((threadIdx.x & (kWave - 1)) == 0) lmask[threadIdx.x / kWave] = bal;
}

struct LiveList {
    int32_t start;  // finite positions <= o: o's successors start here in the list
    int32_t total;
    bool sparse;
};

// After the barrier that follows publish_live; a sparse list needs one more
// barrier (taken here, uniformly) before it is read.
template <int KP>
__device__ inline LiveList build_live(int o, int sub, int top, const uint64_t *lmask, int32_t *list) {
    const int w = o / kWave, b = o % kWave;
    int before = 0, total = 0;
#pragma unroll
    for (int u = 0; u < KP / kWave; ++u) {
        const int c = (int)__popcll(lmask[u]);
        if (u < w) before += c;
        total += c;
    }
    const uint64_t mw = lmask[w];
    const uint64_t below = b == 0 ? 0ull : (mw & (~0ull >> (kWave - b)));
    const int rank = before + (int)__popcll(below);
    const int self = (int)((mw >> b) & 1ull);
    const bool sparse = 2 * total <= top + 1;
    if (sparse) {
        if (sub == 0 && self) list[rank] = o;
        __syncthreads();
    }
    return LiveList{rank + self, total, sparse};
}

// Visits this sub-thread's share of the positions after o in ascending order:
// take(link time, value, position).
template <int SPLIT, typename Link, typename Take>
__device__ inline void scan_next(int o, int sub, int top, const LiveList &lv, const int32_t *list,
                                 const double *vals, Link link, Take take) {
    if (lv.sparse) {
        int r = lv.start + sub;
        for (; r + (kAhead - 1) * SPLIT < lv.total; r += kAhead * SPLIT) {
            int q[kAhead];
            double x[kAhead], y[kAhead];
#pragma unroll
            for (int u = 0; u < kAhead; ++u) q[u] = list[r + u * SPLIT];
#pragma unroll
            for (int u = 0; u < kAhead; ++u) {
                x[u] = link(q[u]);
                y[u] = vals[q[u]];
            }
#pragma unroll
            for (int u = 0; u < kAhead; ++u) take(x[u], y[u], q[u]);
        }
        for (; r < lv.total; r += SPLIT) {
            const int q = list[r];
            take(link(q), vals[q], q);
        }
    } else {
        int o2 = o + 1 + sub;
        for (; o2 + (kAhead - 1) * SPLIT <= top; o2 += kAhead * SPLIT) {
            double x[kAhead], y[kAhead];
#pragma unroll
            for (int u = 0; u < kAhead; ++u) {
                x[u] = link(o2 + u * SPLIT);
                y[u] = vals[o2 + u * SPLIT];
            }
#pragma unroll
            for (int u = 0; u < kAhead; ++u) take(x[u], y[u], o2 + u * SPLIT);
        }
        for (; o2 <= top; o2 += SPLIT) take(link(o2), vals[o2], o2);
    }
}

// Least value over a wave.
__device__ inline double wave_min(double v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v = fmin(v, __shfl_xor(v, off));
    return v;
}

// Least (value, index) pair over a wave: the smaller value, ties to the
// smaller index.
__device__ inline void wave_min_arg(double &v, int &a) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double v2 = __shfl_xor(v, off);
        const int a2 = __shfl_xor(a, off);
        if (v2 < v || (v2 == v && a2 < a)) {
            v = v2;
            a = a2;
        }
    }
}

// Sub-thread k of a cell scans j = i+1+k, i+1+k+SPLIT, ...  It may stop at
// its own first T not below its own running best: everything it skips is no
// smaller than that best, which it reached at a smaller j, so neither the
// minimum nor the least j attaining it can be among the skipped ones.

// Phase 1: bottleneck values.  KP = K padded to whole waves.
template <int KP, int SPLIT>
__global__ __launch_bounds__(SPLIT * KP, level_waves(SPLIT * KP)) void level_bottleneck(
    DevProblem P, int d, const int32_t *rowev, const int32_t *ev_cell, const double *ev_val, double *T,
    const double *T1, const double *Wprev, double *Wnext, const double *EoT, const uint8_t *EiT, double *Rv) {
    constexpr int THREADS = SPLIT * KP;
    extern __shared__ uint32_t tri_w[];
    uint8_t *tri_s = (uint8_t *)tri_w;
    __shared__ double part[SPLIT][KP];
    __shared__ double Vs[KP];
    __shared__ double wred[KP / kWave];
    __shared__ double xs[kMaxDistinctE];
    __shared__ uint64_t lmask[KP / kWave];
    __shared__ int32_t list[KP];
    const int i = blockIdx.x, bi = blockIdx.y;
    const int L = P.L, K = P.K;
    const int o = threadIdx.x % KP, sub = threadIdx.x / KP;
    const int top = K - d;
    RowEvents ev;
    event_bounds(ev, P, d, bi, i, rowev);
    LinkRegs<SPLIT * KP, KP> lr;
    const Links X = load_links(lr, P, i, bi, top, EiT, EoT, xs, tri_s);
    const int64_t srow = (int64_t)bi * P.NS + slice_of(L, i, i + 1);  // slice (i, j) is srow + j-i-1
    double v = kInf;
    if (o < K && o <= top) {
        if (d == 1) {
            if (sub == 0) v = T1[((int64_t)bi * L + i) * K + o];  // the slice (i, L)
        } else {
            const double *Wp = Wprev + (int64_t)bi * (L + 1) * K + o;
            const double *Tp = T + srow * K + o;
            const int jmax = L - d + 1;
            // with imbalance pruning the cuts before the first balanced one have no
            // stage; from there on T again never decreases in j
            const int js = P.jlo_pos ? max(i + 1, P.jlo_pos[o * L + i]) : i + 1;
            bool go = true;
            for (int j0 = js + sub; go && j0 <= jmax; j0 += kCutAhead * SPLIT) {
                double t[kCutAhead], w[kCutAhead];
#pragma unroll
                for (int u = 0; u < kCutAhead; ++u) {  // unconditional loads, all in flight at once
                    const int j = min(j0 + u * SPLIT, jmax);
                    t[u] = Tp[(int64_t)(j - i - 1) * K];
                    w[u] = Wp[(int64_t)j * K];
                }
#pragma unroll
                for (int u = 1; u < kCutAhead; ++u)
                    if (j0 + u * SPLIT > jmax) t[u] = kInf;
#pragma unroll
                for (int u = 0; u < kCutAhead; ++u) {
                    if (go && !(t[u] < v)) go = false;  // T never decreases in j
                    if (go) v = fmin(v, fmax(t[u], w[u]));
                }
            }
        }
    }
    part[sub][o] = v;
    store_links(lr, X, P, i, top, xs, tri_s);
    __syncthreads();
    // every read of this row's table is done
    load_events<THREADS>(ev, ev_cell, ev_val);
    if (sub == 0) {
        double m = part[0][o];
#pragma unroll
        for (int k = 1; k < SPLIT; ++k) m = fmin(m, part[k][o]);
        Vs[o] = m;
        publish_live(o <= top && m < kInf, lmask);
        if (i == 0) {  // the whole-plan bottleneck at this depth: least over first positions
            const double r = wave_min(m);
            if ((threadIdx.x & (kWave - 1)) == 0) wred[threadIdx.x / kWave] = r;
        }
    }
    __syncthreads();
    if (i == 0) {
        if (threadIdx.x == 0) {
            double m = wred[0];
#pragma unroll
            for (int u = 1; u < KP / kWave; ++u) m = fmin(m, wred[u]);
            Rv[(int64_t)(d - 1) * P.nb + bi] = m;
        }
        store_events<THREADS>(ev, ev_cell, ev_val, T);
        return;
    }
    const LiveList lv = build_live<KP>(o, sub, top, lmask, list);
    double w = kInf;
    if (o < K) {
        auto take = [&](double x, double y, int) { w = fmin(w, fmax(x, y)); };
        if (X.table)
            scan_next<SPLIT>(o, sub, top, lv, list, Vs, [&](int q) { return X.tab(o, q); }, take);
        else
            scan_next<SPLIT>(o, sub, top, lv, list, Vs, [&](int q) { return X.direct(o, q, K); }, take);
    }
    part[sub][o] = w;
    __syncthreads();
    if (sub == 0 && o < K) {
        double m = part[0][o];
#pragma unroll
        for (int k = 1; k < SPLIT; ++k) m = fmin(m, part[k][o]);
        Wnext[((int64_t)bi * (L + 1) + i) * K + o] = m;
    }
    store_events<THREADS>(ev, ev_cell, ev_val, T);
}

// (value, index) pairs: the smaller value, ties to the smaller index.
__device__ inline bool lex_less(double v1, int a1, double v2, int a2) {
    return v1 < v2 || (v1 == v2 && a1 < a2);
}

// Phase 2: fill values and argmins at a bound on every stage and link (the
// bottleneck P* of phase 1, or a relaxed bound).  Block (i, b) with b's bound
// bound[b]; a b whose bound is +inf is skipped, and so is a level deeper than
// dlim[b] when dlim is given (no whole plan of that depth stays within the
// bound).  The first row's blocks record the level's least root fill and its
// first position in RF/RO[d][b].
// With kJobs, block (i, job)
// computes fill values only for job = (job_b, job_tau) up to its depth limit
// dlim[job]: its own continuation rows (Gprev/Gnext indexed by job), its least
// root fill in rootF[job], no argmins.  Several jobs may share one b's table,
// so the row's table changes are applied by the last of its jobs' blocks to
// finish reading: each block counts itself on row_cnt[b][i] after its reads
// (jobs_of_b[d-1][b] blocks in all: the jobs of b at least d deep), and the
// last one writes the changes and resets the counter.
template <int KP, int SPLIT, bool kJobs>
__global__ __launch_bounds__(SPLIT * KP, level_waves(SPLIT * KP)) void level_fill(
    DevProblem P, int d, const int32_t *rowev, const int32_t *ev_cell, const double *ev_val, double *T,
    const double *T1, const double *Gprev, double *Gnext, const double *EoT, const uint8_t *EiT, const double *bound,
    const int32_t *job_b, const double *job_tau, const int32_t *jobs_of_b, int32_t *row_cnt, uint16_t *argF,
    uint8_t *argG, double *rootF, const int32_t *dlim, double *RF, int32_t *RO) {
    constexpr int THREADS = SPLIT * KP;
    extern __shared__ uint32_t tri_w[];
    uint8_t *tri_s = (uint8_t *)tri_w;
    __shared__ double part[SPLIT][KP];
    __shared__ int32_t parg[SPLIT][KP];
    __shared__ double Fs[KP];
    __shared__ double wred[KP / kWave];
    __shared__ int32_t wreo[KP / kWave];
    __shared__ double xs[kMaxDistinctE];
    __shared__ uint64_t lmask[KP / kWave];
    __shared__ int32_t list[KP];
    __shared__ int32_t last_reader;
    const int i = blockIdx.x, row = blockIdx.y;  // row: b, or the job
    const int bi = kJobs ? job_b[row] : row;
    const int L = P.L, K = P.K;
    const int o = threadIdx.x % KP, sub = threadIdx.x / KP;
    const int top = K - d;
    const double Ps = kJobs ? job_tau[row] : bound[bi];
    const int dl = !dlim ? INT_MAX : dlim[kJobs ? row : bi];
    if (!(Ps < kInf) || d > dl) return;
    RowEvents ev;
    event_bounds(ev, P, d, bi, i, rowev);
    LinkRegs<SPLIT * KP, KP> lr;
    const Links X = load_links(lr, P, i, bi, top, EiT, EoT, xs, tri_s);
    const int64_t srow = (int64_t)bi * P.NS + slice_of(L, i, i + 1);
    double v = kInf;
    int arg = 0xFFFF;
    if (o < K && o <= top) {
        if (d == 1) {
            if (sub == 0) {
                const double t = T1[((int64_t)bi * L + i) * K + o];  // the slice (i, L)
                if (t <= Ps) {
                    v = t;
                    arg = L;
                }
            }
        } else {
            const double *Gp = Gprev + (int64_t)row * (L + 1) * K + o;
            const double *Tp = T + srow * K + o;
            const int jmax = L - d + 1;
            const int js = P.jlo_pos ? max(i + 1, P.jlo_pos[o * L + i]) : i + 1;
            bool go = true;
            for (int j0 = js + sub; go && j0 <= jmax; j0 += kAhead * SPLIT) {
                double t[kAhead], g[kAhead];
#pragma unroll
                for (int u = 0; u < kAhead; ++u) {  // unconditional loads, all in flight at once
                    const int j = min(j0 + u * SPLIT, jmax);
                    t[u] = Tp[(int64_t)(j - i - 1) * K];
                    g[u] = Gp[(int64_t)j * K];
                }
#pragma unroll
                for (int u = 1; u < kAhead; ++u)
                    if (j0 + u * SPLIT > jmax) t[u] = kInf;
#pragma unroll
                for (int u = 0; u < kAhead; ++u) {
                    if (go && (!(t[u] <= Ps) || !(t[u] < v))) go = false;  // T never decreases in j
                    if (go) {
                        const double c = t[u] + g[u];
                        if (c < v) {
                            v = c;
                            arg = j0 + u * SPLIT;
                        }
                    }
                }
            }
        }
    }
    part[sub][o] = v;
    parg[sub][o] = arg;
    store_links(lr, X, P, i, top, xs, tri_s);
    __syncthreads();
    // every read of this row's table is done
    // (every read of the block has returned its value before the barrier above,
    // so counting needs no fence; the next level reads the table after the
    // kernel boundary)
    bool apply = true;
    if (kJobs) {
        if (threadIdx.x == 0)
            last_reader =
                atomicAdd(&row_cnt[(int64_t)bi * L + i], 1) == jobs_of_b[(int64_t)(d - 1) * P.nb + bi] - 1;
        __syncthreads();
        apply = last_reader != 0;
    }
    if (apply) load_events<THREADS>(ev, ev_cell, ev_val);
    if (sub == 0) {
        double m = part[0][o];
        int a = parg[0][o];
#pragma unroll
        for (int k = 1; k < SPLIT; ++k)
            if (lex_less(part[k][o], parg[k][o], m, a)) {
                m = part[k][o];
                a = parg[k][o];
            }
        Fs[o] = m;
        if (!kJobs && o < K)
            argF[(((int64_t)(d - 1) * P.nb + bi) * L + i) * K + o] = (uint16_t)(m < kInf ? a : 0xFFFF);
        publish_live(o <= top && m < kInf, lmask);
        if (i == 0) {  // the level's least root fill, ties to the least first position
            double r = m;
            int ro = m < kInf ? o : INT_MAX;
            wave_min_arg(r, ro);
            if ((threadIdx.x & (kWave - 1)) == 0) {
                wred[threadIdx.x / kWave] = r;
                wreo[threadIdx.x / kWave] = ro;
            }
        }
    }
    __syncthreads();
    if (i == 0) {
        if (threadIdx.x == 0) {
            double m = wred[0];
            int mo = wreo[0];
#pragma unroll
            for (int u = 1; u < KP / kWave; ++u)
                if (wred[u] < m || (wred[u] == m && wreo[u] < mo)) {
                    m = wred[u];
                    mo = wreo[u];
                }
            if (kJobs) {
                if (m < rootF[row]) rootF[row] = m;
            } else {
                RF[(int64_t)(d - 1) * P.nb + bi] = m;
                RO[(int64_t)(d - 1) * P.nb + bi] = m < kInf ? mo : -1;
            }
        }
        if (apply) store_events<THREADS>(ev, ev_cell, ev_val, T);
        if (kJobs && apply && threadIdx.x == 0) atomicExch(&row_cnt[(int64_t)bi * L + i], 0);
        return;
    }
    const LiveList lv = build_live<KP>(o, sub, top, lmask, list);
    double w = kInf;
    int a = 0xFF;
    if (o < K) {
        auto take = [&](double x, double f, int o2) {
            if (!(x <= Ps)) return;
            const double c = x + f;
            if (c < w) {
                w = c;
                a = o2;
            }
        };
        if (X.table)
            scan_next<SPLIT>(o, sub, top, lv, list, Fs, [&](int q) { return X.tab(o, q); }, take);
        else
            scan_next<SPLIT>(o, sub, top, lv, list, Fs, [&](int q) { return X.direct(o, q, K); }, take);
    }
    part[sub][o] = w;
    parg[sub][o] = a;
    __syncthreads();
    if (sub == 0 && o < K) {
        double m = part[0][o];
        int aa = parg[0][o];
#pragma unroll
        for (int k = 1; k < SPLIT; ++k)
            if (lex_less(part[k][o], parg[k][o], m, aa)) {
                m = part[k][o];
                aa = parg[k][o];
            }
        Gnext[((int64_t)row * (L + 1) + i) * K + o] = m;
        if (!kJobs) argG[(((int64_t)(d - 1) * P.nb + bi) * (L + 1) + i) * K + o] = (uint8_t)(m < kInf ? aa : 0xFF);
    }
    if (apply) store_events<THREADS>(ev, ev_cell, ev_val, T);
    if (kJobs && apply && threadIdx.x == 0) atomicExch(&row_cnt[(int64_t)bi * L + i], 0);
}

// P*_b = least whole-plan bottleneck over the levels; dlim[b] = the deepest
// level whose whole-plan bottleneck reaches P*_b (the fill of step (3) has
// no plan deeper than that), 0 when b has no plan.  Then the b that cannot
// win skip the fill: T_b = (m - 1) P*_b + F_b with F_b at least P*_b (the
// fill adds non-negative stage and link times, one of them at least P*_b),
// so T_b >= LB_b = (m - 1) P*_b + P*_b, rounded as T_b is.  The
// least-bottleneck plan of the shallowest level d reaching P*_b has d stages
// and d - 1 links, each within P*_b, so F_b <= (2 d - 1) P*_b and T_b <= UB_b
// (with a margin far above the rounding of a sum of at most 2D terms).  A b
// with LB_b above the least UB can neither win nor tie: its depth limit
// becomes 0.  One block; a wave per b searches the levels.
constexpr int kPstThreads = 1024;

__global__ __launch_bounds__(kPstThreads) void pst_kernel(DevProblem P, int D, const double *__restrict__ Rv,
                                                          double *Pst, int32_t *dlim, int32_t *dlim_host) {
    __shared__ double red[kPstThreads / kWave];
    const int wv = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
    double ub = kInf;
    for (int bi = wv; bi < P.nb; bi += kPstThreads / kWave) {
        double m = kInf;
        for (int d = lane; d < D; d += kWave) m = fmin(m, Rv[(int64_t)d * P.nb + bi]);
        m = wave_min(m);
        int top = 0, first = INT_MAX;
        for (int d = lane; d < D; d += kWave)
            if (m < kInf && Rv[(int64_t)d * P.nb + bi] <= m) {
                top = d + 1;
                first = min(first, d + 1);
            }
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) {
            top = max(top, __shfl_xor(top, off));
            first = min(first, __shfl_xor(first, off));
        }
        if (lane == 0) {
            Pst[bi] = m;
            dlim[bi] = top;
        }
        if (m < kInf) {
            const double mm1 = (double)(P.B / P.bvals[bi] - 1);
            ub = fmin(ub, ((mm1 * m) + ((double)(2 * first - 1) * m)) * (1.0 + 1e-12));
        }
    }
    if (lane == 0) red[wv] = ub;
    __syncthreads();
    ub = red[0];
#pragma unroll
    for (int u = 1; u < kPstThreads / kWave; ++u) ub = fmin(ub, red[u]);
    for (int bi = threadIdx.x; bi < P.nb; bi += kPstThreads) {
        const double ps = Pst[bi];
        int32_t lim = dlim[bi];
        if (ps < kInf && ((double)(P.B / P.bvals[bi] - 1) * ps) + ps > ub) {
            lim = 0;
            dlim[bi] = 0;
        }
        if (dlim_host) dlim_host[bi] = lim;
    }
}

// The root of each b: the least fill over the levels, ties to the least first
// position, then the least depth.  One wave per b.
__global__ __launch_bounds__(256) void roots_kernel(DevProblem P, int D, const double *RF, const int32_t *RO,
                                                    double *rootF, int32_t *root_o, int32_t *root_d) {
    const int bi = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    if (bi >= P.nb) return;
    double v = kInf;
    int key = INT_MAX;  // position * 2^16 + level: (position, depth) in that order
    for (int d = lane; d < D; d += kWave) {
        const double f = RF[(int64_t)d * P.nb + bi];
        const int o = RO[(int64_t)d * P.nb + bi];
        const int k = o >= 0 ? (o << 16) | d : INT_MAX;
        if (f < kInf && (f < v || (f == v && k < key))) {
            v = f;
            key = k;
        }
    }
    wave_min_arg(v, key);
    if (lane == 0) {
        rootF[bi] = v;
        root_o[bi] = v < kInf ? key >> 16 : -1;
        root_d[bi] = v < kInf ? (key & 0xFFFF) + 1 : -1;
    }
}

// Threads per cell for a level of `blocks` blocks: the most (up to 4) whose
// blocks all fit on the device at once, else 2.  When the device size or the
// occupancy cannot be queried, four.
template <int KP>
struct LevelKernels {
    template <int SPLIT>
    static int capacity(int n_cu, size_t lds) {
        if (n_cu <= 0) return INT_MAX;  // unknown device size: keep four threads per cell
        int per_cu = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, level_bottleneck<KP, SPLIT>, SPLIT * KP, lds) !=
            hipSuccess)
            return INT_MAX;
        int per_cu2 = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu2, level_fill<KP, SPLIT, false>, SPLIT * KP, lds) !=
            hipSuccess)
            return INT_MAX;
        return std::min(per_cu, per_cu2) * n_cu;
    }
};

// ---------------------------------------------------------------------------
// choose b, walk the argmins, resolve each stage's candidate
// ---------------------------------------------------------------------------
// The walk is serial (a stage's argmins give the next stage's first layer and
// position), so one wave follows it and records the stages in LDS; then one
// wave per stage (16 waves) finds the stage's candidate in its group.
constexpr int kFinishThreads = 1024;


__global__ __launch_bounds__(kFinishThreads) void finish_kernel(DevProblem P, const int32_t *gcnt,
                                                                const double *ent_c, const uint8_t *ent_d,
                                                                const int64_t *ent_i, const int32_t *order,
                                                                const double *EoT, const double *Pst,
                                                                const double *rootF, const int32_t *root_o,
                                                                const int32_t *root_d, const uint16_t *argF,
                                                                const uint8_t *argG, ComposeResult *res,
                                                                ComposeResult *res_host) {
    __shared__ int32_t st_i[256], st_j[256], st_o[256], st_on[256];
    __shared__ int32_t sh_S, sh_bb;
    const int L = P.L, K = P.K;
    tg_plan &plan = res->plan;
    if (threadIdx.x == 0) {
        sh_S = 0;
        plan.b = 0;
        plan.m = 0;
        plan.S = 0;
        plan.reserved = 0;
        plan.P = kInf;
        plan.F = kInf;
        plan.T = kInf;
        double bestT = kInf;
        int bb = -1;
        if (!res->err)
            for (int bi = 0; bi < P.nb; ++bi) {
                if (!(Pst[bi] < kInf) || root_o[bi] < 0) continue;
                const int64_t m = P.B / P.bvals[bi];
                const double T = ((double)(m - 1) * Pst[bi]) + rootF[bi];
                if (T < bestT) {
                    bestT = T;
                    bb = bi;
                }
            }
        if (bb >= 0) {
            const int64_t b = P.bvals[bb];
            const int S = root_d[bb];
            plan.b = (int32_t)b;
            plan.m = (int32_t)(P.B / b);
            plan.S = S;
            plan.P = Pst[bb];
            plan.F = rootF[bb];
            plan.T = bestT;
            res->status = TG_OK;
            sh_S = S;
            sh_bb = bb;
        }
    }
    __syncthreads();
    // The walk, by wave 0: once a stage's cut j is known, the next stage's
    // whole argmin row argF[d-2][b][j][.] is loaded with argG[d-2][b][j][o],
    // so the next cut needs no further load (one dependent load per stage).
    if (threadIdx.x < kWave && sh_S > 0) {
        const int lane = threadIdx.x;
        const int S = sh_S, bb = sh_bb;
        int i = 0, o = root_o[bb];
        bool ok = S >= 1 && S <= 255;
        int j = L;
        if (ok && S > 1) j = argF[(((int64_t)(S - 1) * P.nb + bb) * L + i) * K + o];
        for (int t = 0; ok && t < S; ++t) {
            const int d = S - t;
            int o_next = -1, jn = L;
            if (d > 1) {
                // an argmin on the optimal path is always set
                ok = j > i && j <= L - d + 1;
                if (ok) {
                    const uint16_t *row = argF + (((int64_t)(d - 2) * P.nb + bb) * L + j) * K;
                    uint16_t rv[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int oo = lane + q * kWave;
                        rv[q] = (d > 2 && oo < K) ? row[oo] : 0;
                    }
                    o_next = argG[(((int64_t)(d - 2) * P.nb + bb) * (L + 1) + j) * K + o];
                    ok = o_next > o && o_next < K;
                    if (ok && d > 2) {
                        const int q = o_next / kWave;
                        const int pick = q == 0 ? rv[0] : (q == 1 ? rv[1] : (q == 2 ? rv[2] : rv[3]));
                        jn = __shfl(pick, o_next % kWave);
                    }
                }
            }
            if (lane == 0) {
                st_i[t] = i;
                st_j[t] = j;
                st_o[t] = o;
                st_on[t] = o_next;
            }
            i = j;
            o = o_next;
            j = jn;
        }
        if (!ok && lane == 0) {
            sh_S = 0;
            res->err = 4;
            res->status = TG_ENOPLAN;
        }
    }
    __syncthreads();
    const int S = sh_S;
    const int wv = threadIdx.x / kWave;
    if (S > 0) {
        const int bb = sh_bb;
        const int64_t b = P.bvals[bb];
        for (int t = wv; t < S; t += kFinishThreads / kWave) {
            const int d = S - t, i = st_i[t], j = st_j[t], o = st_o[t], o_next = st_on[t];
            double link = 0.0;
            if (d > 1) {
                const double E = EoT[(int64_t)o_next * K + o];
                link = E == 0.0 ? kInf : ((2.0 * (double)b) * (double)P.outact[j - 1]) / E;
            }
            resolve_stage(P, gcnt, ent_c, ent_d, ent_i, group_id(P, o, bb, slice_of(L, i, j)), i, j, order[o], d,
                          link, plan.stage[t], res);
        }
    }
    if (!res_host) return;
    // the header and the S stages into host memory (8-byte words)
    __syncthreads();
    static_assert(offsetof(ComposeResult, plan) % 8 == 0 && offsetof(tg_plan, stage) % 8 == 0 &&
                      sizeof(tg_stage) % 8 == 0, "result words");
    const int n = (int)((offsetof(ComposeResult, plan) + offsetof(tg_plan, stage) + sizeof(tg_stage) * S) / 8);
    const uint64_t *src = (const uint64_t *)res;
    uint64_t *dst = (uint64_t *)res_host;
    for (int k = threadIdx.x; k < n; k += kFinishThreads) dst[k] = src[k];
}

// ---------------------------------------------------------------------------
// host-side sequencing
// ---------------------------------------------------------------------------
// Workspace of the relaxed search, after the composition workspace.
constexpr int kMaxJobs = 128;  // fill evaluations per launch

constexpr int64_t kSpecBounds = 4096;  // collected bounds read back with the phase results

// Byte offsets of the relaxed search's packed transfers.  The device read-back
// and upload regions and the pinned host buffer share the layout, so each
// transfer is one copy: `down` (after phase 2: phase results, the collected
// bound count and the first kSpecBounds bounds), `up` (before each fill run:
// its jobs; before the last fill: its bound and depth limit).  The host
// buffer holds down, then up, then the fill results of a run and m - 1 per b.
struct RelaxXfer {
    size_t pst, f0, rv, thv, err, cnt, thb, down;
    size_t mm1, tau, bound, jb, jd, fdl, njob, up;
    size_t h_up, h_jf, h_mm1, h_res, host;
};

static RelaxXfer xfer_layout(const DevProblem &P) {
    const size_t nb = P.nb, D = levels(P), J = kMaxJobs, S = kSpecBounds;
    RelaxXfer x{};
    size_t o = 0;
    auto put = [&](size_t bytes) {
        const size_t at = o;
        o += (bytes + 15) & ~(size_t)15;
        return at;
    };
    x.pst = put(8 * nb);
    x.f0 = put(8 * nb);
    x.rv = put(8 * D * nb);
    x.thv = put(8 * S);
    x.err = put(4);
    x.cnt = put(4);
    x.thb = put(4 * S);
    x.down = o;
    o = 0;
    x.tau = put(8 * J);
    x.bound = put(8 * nb);
    x.jb = put(4 * J);
    x.jd = put(4 * J);
    x.fdl = put(4 * nb);
    x.njob = put(4 * D * nb);
    x.up = o;
    o = x.down;
    x.h_up = put(x.up);
    x.h_jf = put(8 * J);
    x.h_mm1 = put(8 * nb);
    x.h_res = put(sizeof(ComposeResult));
    x.host = o;
    return x;
}

size_t compose_relaxed_stage_bytes(const DevProblem &P) { return xfer_layout(P).host; }

struct RelaxWs {
    double *th_val;   // [n_surv] collected stage-cost bounds
    int32_t *th_b;    // [n_surv] their b
    int32_t *th_cnt;  // [1]
    double *lo;       // [nb] P* per b (bounds must exceed it)
    double *hi;       // [nb] the best T found so far
    double *mm1;      // [nb] m - 1 per b
    char *down;       // packed read-back (RelaxXfer)
    char *up;         // packed uploads (RelaxXfer): the arrays below point into it
    double *job_tau;     // [kMaxJobs]
    double *bound;       // [nb] the last fill's bound per b
    int32_t *job_b;      // [kMaxJobs]
    int32_t *job_dlim;   // [kMaxJobs] deepest level with a whole plan within the job's bound
    int32_t *fdl;        // [nb] the last fill's depth limit per b
    int32_t *jobs_of_b;  // [D][nb] jobs of each b at least d deep in the current run
    int32_t *row_cnt;    // [nb][L] readers done per row (job runs)
    double *job_F;    // [kMaxJobs]
    double *job_G;    // [2][kMaxJobs][L+1][K]
    double *Tp;       // [n_groups] pristine starting stage table (each fill run starts from it)
    size_t bytes;
};

static RelaxWs carve_relax(const DevProblem &P, int64_t n, void *base) {
    RelaxWs r{};
    char *p = (char *)base;
    size_t off = 0;
    auto take = [&](size_t bytes) -> void * {
        void *x = base ? (void *)(p + off) : nullptr;
        off += align256(bytes > 0 ? bytes : 1);
        return x;
    };
    const RelaxXfer X = xfer_layout(P);
    const int64_t jrows = (int64_t)kMaxJobs * (P.L + 1) * P.K;
    r.th_val = (double *)take(sizeof(double) * n);
    r.th_b = (int32_t *)take(sizeof(int32_t) * n);
    r.th_cnt = (int32_t *)take(sizeof(int32_t));
    r.lo = (double *)take(sizeof(double) * P.nb);
    r.hi = (double *)take(sizeof(double) * P.nb);
    r.mm1 = (double *)take(sizeof(double) * P.nb);
    r.down = (char *)take(X.down);
    r.up = (char *)take(X.up);
    if (base) {
        r.job_tau = (double *)(r.up + X.tau);
        r.bound = (double *)(r.up + X.bound);
        r.job_b = (int32_t *)(r.up + X.jb);
        r.job_dlim = (int32_t *)(r.up + X.jd);
        r.fdl = (int32_t *)(r.up + X.fdl);
        r.jobs_of_b = (int32_t *)(r.up + X.njob);
    }
    r.row_cnt = (int32_t *)take(sizeof(int32_t) * P.nb * P.L);
    r.job_F = (double *)take(sizeof(double) * kMaxJobs);
    r.job_G = (double *)take(sizeof(double) * 2 * jrows);
    r.Tp = (double *)take(sizeof(double) * n_groups(P));
    r.bytes = off;
    return r;
}

// The phase results, the collected bound count and the first `spec` collected
// bounds into the packed read-back region.
__global__ __launch_bounds__(256) void pack_readback(int nb, int D, const double *__restrict__ Pst,
                                                     const double *__restrict__ F0, const double *__restrict__ Rv,
                                                     const ComposeResult *__restrict__ res,
                                                     const int32_t *__restrict__ cnt,
                                                     const double *__restrict__ thv, const int32_t *__restrict__ thb,
                                                     int64_t spec, char *__restrict__ down, RelaxXfer X) {
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = t0; t < nb; t += step) {
        ((double *)(down + X.pst))[t] = Pst[t];
        ((double *)(down + X.f0))[t] = F0[t];
    }
    for (int64_t t = t0; t < (int64_t)D * nb; t += step) ((double *)(down + X.rv))[t] = Rv[t];
    for (int64_t t = t0; t < spec; t += step) {
        ((double *)(down + X.thv))[t] = thv[t];
        ((int32_t *)(down + X.thb))[t] = thb[t];
    }
    if (t0 == 0) {
        *(int32_t *)(down + X.err) = res->err;
        *(int32_t *)(down + X.cnt) = *cnt;
    }
}

size_t compose_relaxed_ws_bytes(const DevProblem &P, int64_t n_surv) {
    return compose_ws_bytes(P, n_surv) + carve_relax(P, n_surv, nullptr).bytes;
}

// Stage costs that can serve as relaxed bounds for their b: above P*_b and
// with (m-1) * cost not above hi[b], the best iteration time found so far (a
// plan bounded by a larger value cannot reach it, its fill being
// non-negative).  Every listed
// candidate that fits somewhere (a grouped record) is a candidate bound; one
// thread per record, duplicates removed on the host.
constexpr int kBoundRecs = 8;  // records per thread, loads in flight together
constexpr int kMaxB = 512;     // b values staged in LDS (more are read from global memory)

__global__ __launch_bounds__(256) void collect_bounds(DevProblem P, const int32_t *__restrict__ rec_g,
                                                      const double *__restrict__ rec_c, int64_t n,
                                                      const double *lo, const double *hi, const double *mm1,
                                                      double *th_val, int32_t *th_b, int32_t *th_cnt, int32_t cap) {
    __shared__ double slo[kMaxB], shi[kMaxB], smm[kMaxB];
    for (int t = threadIdx.x; t < P.nb && t < kMaxB; t += blockDim.x) {
        slo[t] = lo[t];
        shi[t] = hi[t];
        smm[t] = mm1[t];
    }
    __syncthreads();
    const int64_t r0 = ((int64_t)blockIdx.x * blockDim.x * kBoundRecs) + threadIdx.x;
    int32_t g[kBoundRecs];
    double c[kBoundRecs];
#pragma unroll
    for (int k = 0; k < kBoundRecs; ++k) {
        const int64_t r = r0 + (int64_t)k * blockDim.x;
        g[k] = r < n ? rec_g[r] : -1;
        c[k] = r < n ? rec_c[r] : 0.0;  // unused when the group is -1
    }
    int bi[kBoundRecs];
    int cnt = 0;
#pragma unroll
    for (int k = 0; k < kBoundRecs; ++k) {
        bi[k] = -1;
        if (g[k] >= 0) {
            // G = (position * nb + b) * NS + slice < 2^31 (checked at the boundary)
            const int b = (int)(((uint32_t)g[k] / (uint32_t)P.NS) % (uint32_t)P.nb);
            const double l = b < kMaxB ? slo[b] : lo[b];
            const double h = b < kMaxB ? shi[b] : hi[b];
            const double f = b < kMaxB ? smm[b] : mm1[b];
            if (c[k] > l && c[k] < kInf && (f * c[k]) <= h) {
                bi[k] = b;
                ++cnt;
            }
        }
    }
    // one counter update per block: same-address atomics serialise
    __shared__ int32_t scan_lds[256 / kWave + 1];
    __shared__ int32_t block_base;
    int32_t total;
    int32_t slot = block_excl_scan<int32_t>(cnt, scan_lds, &total);
    if (threadIdx.x == 0) block_base = total ? atomicAdd(th_cnt, total) : 0;
    __syncthreads();
    slot += block_base;
#pragma unroll
    for (int k = 0; k < kBoundRecs; ++k)
        if (bi[k] >= 0) {
            if (slot < cap) {
                th_val[slot] = c[k];
                th_b[slot] = bi[k];
            }
            ++slot;
        }
}

// The relaxed search's starting incumbent, the least (T, b) with T = (m-1)
// P*_b + F(P*_b) (its bound is P*_b), and the window of stage costs worth
// collecting: lo[b] = P*_b for a b still in the race ((m-1) P*_b not above the
// incumbent, a fill being non-negative), +inf for the rest; hi[b] = the
// incumbent T.  One block; the host repeats the same arithmetic on the values
// it reads back.
constexpr int kInitThreads = 256;

__global__ __launch_bounds__(kInitThreads) void relax_init(DevProblem P, const double *__restrict__ Pst,
                                                           const double *__restrict__ F0,
                                                           const double *__restrict__ mm1, double *lo, double *hi) {
    __shared__ double sT[kInitThreads];
    __shared__ int32_t sb[kInitThreads];
    double bt = kInf;
    int bb = INT_MAX;
    for (int b = threadIdx.x; b < P.nb; b += kInitThreads)
        if (Pst[b] < kInf && F0[b] < kInf) {
            const double t = (mm1[b] * Pst[b]) + F0[b];
            if (t < bt || (t == bt && b < bb)) {
                bt = t;
                bb = b;
            }
        }
    sT[threadIdx.x] = bt;
    sb[threadIdx.x] = bb;
    __syncthreads();
    for (int h = kInitThreads / 2; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) {
            const double t = sT[threadIdx.x + h];
            const int b = sb[threadIdx.x + h];
            if (t < sT[threadIdx.x] || (t == sT[threadIdx.x] && b < sb[threadIdx.x])) {
                sT[threadIdx.x] = t;
                sb[threadIdx.x] = b;
            }
        }
        __syncthreads();
    }
    const double inc = sT[0];
    for (int b = threadIdx.x; b < P.nb; b += kInitThreads) {
        const bool live = Pst[b] < kInf && F0[b] < kInf && (mm1[b] * Pst[b]) <= inc;
        lo[b] = live ? Pst[b] : kInf;
        hi[b] = inc;
    }
}

// Pipelines of at least this many levels read the fill's depth limits back
// before phase 2 and launch only the levels some b needs.
constexpr int kSyncLevels = 64;
// Fill levels queued ahead of the read-back of the depth limits when they go
// through pinned memory, so the GPU is not idle while the host waits.
constexpr int kLeadLevels = 8;

// Sequencing of the composition kernels on one workspace.
struct Driver {
    DevProblem P;  // this call's copy: carries the table of first balanced cuts by position
    Ws w;
    hipStream_t s;
    int D;
    int64_t rows;
    size_t tri_lds;
    int n_cu = 0;

    Driver(const DevProblem &P_, int64_t n_surv, void *ws, hipStream_t s_)
        : P(P_), w(carve(P_, n_surv, ws)), s(s_), D(levels(P_)), rows((int64_t)P_.nb * (P_.L + 1) * P_.K) {
        tri_lds = P.n_ev ? (size_t)(P.K * (P.K - 1) / 2 + 4) : 0;
        P.jlo_pos = P.imb ? w.jlo_pos : nullptr;
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            n_cu = 0;
    }

    // candidate list -> grouped entries -> starting tables (one copy per
    // phase) and per-row, per-level table changes
    void setup(const int64_t *surv, int64_t n_surv, const double *cost, const uint8_t *dmax) {
        prep_kernel<<<dim3((unsigned)((P.K * P.K + 255) / 256)), dim3(256), 0, s>>>(P, w.order, w.pos, w.EoT,
                                                                                     w.EiT, w.res, w.ev_total);
        if (P.imb)
            jlo_kernel<<<dim3((unsigned)((P.K * P.L + 255) / 256)), dim3(256), 0, s>>>(P, w.order, w.jlo_pos);
        const Groups g{w.rec_g, w.rec_c, w.rec_d, w.gcnt, w.ent_c, w.ent_d, w.ent_i, w.tmp};
        launch_grouping(P, surv, n_surv, cost, dmax, w.pos, g, w.res, s);
        row_tables<<<dim3((unsigned)P.L, (unsigned)P.nb), dim3(kRowThreads), 0, s>>>(
            P, w.gcnt, w.ent_c, w.ent_d, w.ent_i, w.T, w.T0, w.T1, w.rowev, w.ev_total, w.ev_cell, w.ev_val);
    }

    template <typename F>
    void with_kp(F f) {
        if (P.K <= 64)
            f(std::integral_constant<int, 64>{});
        else if (P.K <= 128)
            f(std::integral_constant<int, 128>{});
        else if (P.K <= 192)
            f(std::integral_constant<int, 192>{});
        else
            f(std::integral_constant<int, 256>{});
    }

    template <int KP>
    int split_for(int blocks) {
        using LK = LevelKernels<KP>;
        const int cap4 = LK::template capacity<4>(n_cu, tri_lds);
        if (blocks <= cap4) return 4;
        const int cap3 = LK::template capacity<3>(n_cu, tri_lds);
        return blocks <= cap3 ? 3 : 2;
    }

    // The continuation rows need no clearing: level d reads rows j of level
    // d - 1 only for i < j <= L - d + 1 (the cut scan stops there), and level
    // d - 1 wrote every row 1..L - d + 1 at every position (a b or job that
    // skips a level skips every deeper one too).

    // phase 1: least bottleneck per b into w.Pst, the fill's depth limit per b
    // into w.dlim
    void phase1(int32_t *dlim_host = nullptr) {
        with_kp([&](auto kp) {
            constexpr int KP = decltype(kp)::value;
            for (int d = 1; d <= D; ++d) {
                const dim3 grid((unsigned)(P.L - d + 1), (unsigned)P.nb);
                const int sp = split_for<KP>((int)(grid.x * grid.y));
                const double *Wp = w.Wb[(d - 1) & 1];
                double *Wn = w.Wb[d & 1];
                auto go = [&](auto spc) {
                    constexpr int SP = decltype(spc)::value;
                    level_bottleneck<KP, SP><<<grid, dim3(SP * KP), tri_lds, s>>>(
                        P, d, w.rowev, w.ev_cell, w.ev_val, w.T, w.T1, Wp, Wn, w.EoT, w.EiT, w.Rv);
                };
                if (sp == 4)
                    go(std::integral_constant<int, 4>{});
                else if (sp == 3)
                    go(std::integral_constant<int, 3>{});
                else
                    go(std::integral_constant<int, 2>{});
            }
        });
        pst_kernel<<<dim3(1), dim3(kPstThreads), 0, s>>>(P, D, w.Rv, w.Pst, w.dlim, dlim_host);
    }

    // The deepest fill level any b needs.  Reading w.dlim back costs one host
    // synchronisation (tens of microseconds of idle GPU), which pays only when
    // many levels may be skipped: with fewer than kSyncLevels levels every
    // level is launched and the blocks of a b past its limit leave at once.
    hipError_t fill_levels(int *nlev) {
        if (D < kSyncLevels) {
            *nlev = D;
            return hipSuccess;
        }
        std::vector<int32_t> dl(P.nb);
        hipError_t e = hipMemcpyAsync(dl.data(), w.dlim, sizeof(int32_t) * P.nb, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return e;
        int n = 0;
        for (int v : dl) n = std::max(n, std::min(v, D));
        *nlev = n;
        return hipSuccess;
    }

    // phase 2 at bound[b] (+inf skips b), levels 1..nlev, each b up to
    // dlim[b] when given: fills, argmins and roots per b, from the starting
    // stage table in `table` (phase 2's own copy unless given).
    void phase2(const double *bound, const int32_t *dlim, int nlev, double *table = nullptr) {
        phase2_begin();
        phase2_levels(bound, dlim, 1, nlev, table);
        phase2_end();
    }
    // Phase 2 at P* with the depth limits that phase1(dlim_dev) stored into
    // the pinned host words `dlim` (at least nb int32), read once the event
    // `ev` has passed: the event is recorded right after phase 1, the first
    // kLeadLevels fill levels are queued behind it, and the host waits for
    // the event alone before queueing the levels some b still needs, so the
    // GPU keeps busy meanwhile.
    hipError_t phase2_read_back(const int32_t *dlim, hipEvent_t ev) {
        hipError_t e = hipEventRecord(ev, s);
        if (e != hipSuccess) return e;
        const int lead = std::min(D, kLeadLevels);
        phase2_begin();
        phase2_levels(w.Pst, w.dlim, 1, lead);
        e = hipEventSynchronize(ev);
        if (e != hipSuccess) return e;
        int nlev = 0;
        for (int b = 0; b < P.nb; ++b) nlev = std::max(nlev, std::min((int)dlim[b], D));
        phase2_levels(w.Pst, w.dlim, lead + 1, nlev);
        phase2_end();
        return hipSuccess;
    }
    void phase2_begin() {
        fill<double>(w.RF, (int64_t)D * P.nb, kInf, s);
        fill<int32_t>(w.RO, (int64_t)D * P.nb, -1, s);
    }
    // levels d0..d1 (a level past a b's limit costs only its early return)
    void phase2_levels(const double *bound, const int32_t *dlim, int d0, int d1, double *table = nullptr) {
        if (!table) table = w.T0;
        with_kp([&](auto kp) {
            constexpr int KP = decltype(kp)::value;
            for (int d = d0; d <= d1; ++d) {
                const dim3 grid((unsigned)(P.L - d + 1), (unsigned)P.nb);
                const int sp = split_for<KP>((int)(grid.x * grid.y));
                const double *Gp = w.Wb[(d - 1) & 1];
                double *Gn = w.Wb[d & 1];
                auto go = [&](auto spc) {
                    constexpr int SP = decltype(spc)::value;
                    level_fill<KP, SP, false><<<grid, dim3(SP * KP), tri_lds, s>>>(
                        P, d, w.rowev, w.ev_cell, w.ev_val, table, w.T1, Gp, Gn, w.EoT, w.EiT, bound, nullptr,
                        nullptr, nullptr, nullptr, w.argF, w.argG, nullptr, dlim, w.RF, w.RO);
                };
                if (sp == 4)
                    go(std::integral_constant<int, 4>{});
                else if (sp == 3)
                    go(std::integral_constant<int, 3>{});
                else
                    go(std::integral_constant<int, 2>{});
            }
        });
    }
    void phase2_end() {
        roots_kernel<<<dim3((unsigned)((P.nb + 3) / 4)), dim3(256), 0, s>>>(P, D, w.RF, w.RO, w.rootF, w.root_o,
                                                                            w.root_d);
    }

    // the starting stage table of the b with used[b] back into w.T from the
    // pristine copy (layout [b][s][o]: one contiguous run per b)
    hipError_t restore_tables(const double *Tp, const std::vector<char> &used) {
        const size_t per_b = (size_t)P.NS * P.K;
        for (int b0 = 0; b0 < P.nb;) {
            if (!used[b0]) {
                ++b0;
                continue;
            }
            int b1 = b0;
            while (b1 < P.nb && used[b1]) ++b1;
            const hipError_t e = hipMemcpyAsync(w.T + per_b * b0, Tp + per_b * b0, sizeof(double) * per_b * (b1 - b0),
                                                hipMemcpyDeviceToDevice, s);
            if (e != hipSuccess) return e;
            b0 = b1;
        }
        return hipSuccess;
    }

    // fill values only, for J <= kMaxJobs (b, bound) jobs staged in r, levels
    // 1..nlev, each job up to its own depth limit, from the starting stage
    // table in w.T
    void phase2_jobs(RelaxWs &r, int J, int nlev) {
        const int64_t jrows = (int64_t)kMaxJobs * (P.L + 1) * P.K;
        fill<double>(r.job_F, J, kInf, s);
        fill<int32_t>(r.row_cnt, (int64_t)P.nb * P.L, 0, s);
        with_kp([&](auto kp) {
            constexpr int KP = decltype(kp)::value;
            for (int d = 1; d <= nlev; ++d) {
                const dim3 grid((unsigned)(P.L - d + 1), (unsigned)J);
                const int sp = split_for<KP>((int)(grid.x * grid.y));
                const double *Gp = r.job_G + ((d - 1) & 1) * jrows;
                double *Gn = r.job_G + (d & 1) * jrows;
                auto go = [&](auto spc) {
                    constexpr int SP = decltype(spc)::value;
                    level_fill<KP, SP, true><<<grid, dim3(SP * KP), tri_lds, s>>>(
                        P, d, w.rowev, w.ev_cell, w.ev_val, w.T, w.T1, Gp, Gn, w.EoT, w.EiT, nullptr, r.job_b,
                        r.job_tau, r.jobs_of_b, r.row_cnt, nullptr, nullptr, r.job_F, r.job_dlim, nullptr, nullptr);
                };
                if (sp == 4)
                    go(std::integral_constant<int, 4>{});
                else if (sp == 3)
                    go(std::integral_constant<int, 3>{});
                else
                    go(std::integral_constant<int, 2>{});
            }
        });
    }

    // the plan into w.res and, when given, into res_host (device view of
    // pinned host memory)
    void finish(const double *bound, ComposeResult *res_host = nullptr) {
        finish_kernel<<<dim3(1), dim3(kFinishThreads), 0, s>>>(P, w.gcnt, w.ent_c, w.ent_d, w.ent_i, w.order, w.EoT,
                                                                 bound, w.rootF, w.root_o, w.root_d, w.argF, w.argG,
                                                                 w.res, res_host);
    }
};

hipError_t launch_compose(const DevProblem &P, const int64_t *surv, int64_t n_surv, const double *cost,
                          const uint8_t *dmax, const int32_t *order_dev, void *ws, hipStream_t s,
                          ComposeResult **result_dev, const ComposeHost *host) {
    (void)order_dev;
    Driver dr(P, n_surv, ws, s);
    *result_dev = dr.w.res;
    dr.setup(surv, n_surv, cost, dmax);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // the overlapped read-back pays at any depth past the lead: the GPU keeps
    // busy while the host waits
    const bool overlap = dr.D > kLeadLevels && host && host->dlim && host->ev;
    dr.phase1(overlap ? host->dlim_dev : nullptr);
    if (overlap) {
        e = dr.phase2_read_back(host->dlim, host->ev);
        if (e != hipSuccess) return e;
    } else {
        int nlev = 0;
        e = dr.fill_levels(&nlev);
        if (e != hipSuccess) return e;
        dr.phase2(dr.w.Pst, dr.w.dlim, nlev);
    }
    dr.finish(dr.w.Pst, host ? host->res_dev : nullptr);
    return hipGetLastError();
}

// The relaxation of step (4), per b: the bound is raised over the stage and
// link costs above P* while T = (m-1) * bound + F(bound) can still improve,
// where F(bound) is the least fill with every stage and link within the
// bound.  F never increases with the bound, so over an interval of bounds
// (u, v] the iteration time is at least (m-1) * (its first bound) + F(v): the
// search evaluates F at up to kSplitWays points per open interval per round
// (all jobs of a round in one batched run), drops an interval when that lower
// bound cannot beat the best (T, b, bound) found over every b (ties go to the
// smaller b, then the smaller bound) or when F is equal at both ends, and
// splits the rest.  Only b* needs its exact optimum: any other b is dropped
// once it cannot beat the incumbent.  The result is the least (T, b, bound),
// as a plain ascending sweep of every b would find.
constexpr int kSplitWays = 8;

struct BSearch {
    bool active = false;
    double Pst = 0, F0 = 0, mm1 = 0;
    std::vector<double> th;  // distinct bounds above P*, ascending
    std::vector<double> F;   // F at th[k], NaN if unknown
    std::vector<std::pair<int, int>> iv;  // open intervals (a, c]: F(a) known (a = -1 is P*)
    double Fat(int k) const { return k < 0 ? F0 : F[k]; }
    double tat(int k) const { return k < 0 ? Pst : th[k]; }
};

// The incumbent over every b: least T, ties to the least b, then the least
// bound.
struct Incumbent {
    double T = kInf;
    int b = INT_MAX;
    double tau = kInf;
    bool beaten_by(double T2, int b2, double tau2) const {
        return T2 < T || (T2 == T && (b2 < b || (b2 == b && tau2 < tau)));
    }
    void offer(double T2, int b2, double tau2) {
        if (beaten_by(T2, b2, tau2)) {
            T = T2;
            b = b2;
            tau = tau2;
        }
    }
};

hipError_t launch_compose_relaxed(const DevProblem &P, const RelaxHost &H, const int32_t *order_host,
                                  const int64_t *surv, int64_t n_surv, const double *cost, const uint8_t *dmax,
                                  void *ws, hipStream_t s, ComposeResult **result_dev,
                                  const ComposeResult **result_host, int *rounds_out) {
    Driver dr(P, n_surv, ws, s);
    RelaxWs r = carve_relax(P, n_surv, (char *)ws + compose_ws_bytes(P, n_surv));
    const RelaxXfer X = xfer_layout(P);
    *result_dev = dr.w.res;
    if (rounds_out) *rounds_out = 0;
    if (!H.stage || !H.stage->ptr || H.stage->bytes < X.host) return hipErrorInvalidValue;
    char *hs = (char *)H.stage->ptr;  // pinned: the copies below do not stall the host
    char *hd = hs, *hu = hs + X.h_up;
    // the finish kernel stores the result into the stage too (every success below finishes)
    ComposeResult *res_hd = (ComposeResult *)((char *)H.stage->dev + X.h_res);
    *result_host = (const ComposeResult *)(hs + X.h_res);
    double *h_jf = (double *)(hs + X.h_jf), *h_mm1 = (double *)(hs + X.h_mm1);
    const int nb = P.nb, D = dr.D;
    for (int bi = 0; bi < nb; ++bi) h_mm1[bi] = (double)(H.B / H.bvals[bi] - 1);
    hipError_t e = hipMemcpyAsync(r.mm1, h_mm1, sizeof(double) * nb, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return e;
    dr.setup(surv, n_surv, cost, dmax);
    e = hipGetLastError();
    if (e == hipSuccess)
        e = hipMemcpyAsync(r.Tp, dr.w.T0, sizeof(double) * n_groups(P), hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
    const bool overlap = D > kLeadLevels && H.ev;
    dr.phase1(overlap ? (int32_t *)H.stage->dev : nullptr);  // into hd, the host view of the same words
    if (overlap) {
        e = dr.phase2_read_back((const int32_t *)hd, H.ev);  // hd is written again only by the copy below
        if (e != hipSuccess) return e;
    } else {
        int nlev = 0;
        e = dr.fill_levels(&nlev);
        if (e != hipSuccess) return e;
        dr.phase2(dr.w.Pst, dr.w.dlim, nlev);
    }
    // the starting incumbent and the stage costs worth collecting, on the
    // device; one packed read-back brings the phase results, the collected
    // count and the first kSpecBounds collected bounds
    relax_init<<<dim3(1), dim3(kInitThreads), 0, s>>>(P, dr.w.Pst, dr.w.rootF, r.mm1, r.lo, r.hi);
    fill<int32_t>(r.th_cnt, 1, 0, s);
    {
        int64_t blocks = (n_surv + 256 * kBoundRecs - 1) / (256 * kBoundRecs);
        if (blocks < 1) blocks = 1;
        collect_bounds<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, dr.w.rec_g, dr.w.rec_c, n_surv, r.lo, r.hi,
                                                                   r.mm1, r.th_val, r.th_b, r.th_cnt,
                                                                   (int32_t)std::min<int64_t>(n_surv, INT32_MAX));
    }
    const int64_t spec = std::min<int64_t>(n_surv, kSpecBounds);
    {
        const int64_t most = std::max<int64_t>((int64_t)D * nb, spec);
        const unsigned blocks = (unsigned)std::min<int64_t>(std::max<int64_t>((most + 255) / 256, 1), 64);
        pack_readback<<<dim3(blocks), dim3(256), 0, s>>>(nb, D, dr.w.Pst, dr.w.rootF, dr.w.Rv, dr.w.res, r.th_cnt,
                                                         r.th_val, r.th_b, spec, r.down, X);
    }
    e = hipMemcpyAsync(hd, r.down, X.down, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
    const double *Pst = (const double *)(hd + X.pst), *F0 = (const double *)(hd + X.f0);
    const double *Rv = (const double *)(hd + X.rv);
    if (*(const int32_t *)(hd + X.err)) {  // invalid list: the finish kernel reports it
        dr.finish(dr.w.Pst, res_hd);
        return hipGetLastError();
    }
    // the fill at bound tau has no whole plan deeper than the deepest level
    // whose least whole-plan bottleneck (phase 1) is within tau: its levels
    // stop there
    auto dlim_of = [&](int bi, double tau) {
        int top = 0;
        for (int d = 1; d <= D; ++d)
            if (Rv[(size_t)(d - 1) * nb + bi] <= tau) top = d;
        return top;
    };
    std::vector<BSearch> bs(nb);
    Incumbent inc;
    for (int bi = 0; bi < nb; ++bi) {
        BSearch &q = bs[bi];
        q.mm1 = h_mm1[bi];
        if (!(Pst[bi] < kInf) || !(F0[bi] < kInf)) continue;
        q.active = true;
        q.Pst = Pst[bi];
        q.F0 = F0[bi];
        inc.offer((q.mm1 * q.Pst) + q.F0, bi, q.Pst);
    }
    // a bound tau of b gives T >= (m-1) tau (the fill is non-negative): b
    // takes part only while (m-1) P*_b can still reach the incumbent (the
    // rule relax_init applied on the device)
    bool any = false;
    for (int bi = 0; bi < nb; ++bi) {
        BSearch &q = bs[bi];
        if (q.active && !((q.mm1 * q.Pst) <= inc.T)) q.active = false;
        any = any || q.active;
    }
    if (any) {
        // candidate bounds: stage costs (collected on the device) and link
        // times (host); the rest of the collected list when it outgrew the
        // packed read-back
        const int32_t cnt = (int32_t)std::min<int64_t>(*(const int32_t *)(hd + X.cnt), n_surv);
        const double *tv = (const double *)(hd + X.thv);
        const int32_t *tb = (const int32_t *)(hd + X.thb);
        for (int32_t t = 0; t < cnt && t < spec; ++t) bs[tb[t]].th.push_back(tv[t]);
        if (cnt > spec) {
            std::vector<double> tv2(cnt - spec);
            std::vector<int32_t> tb2(cnt - spec);
            e = hipMemcpyAsync(tv2.data(), r.th_val + spec, sizeof(double) * (cnt - spec), hipMemcpyDeviceToHost, s);
            if (e == hipSuccess)
                e = hipMemcpyAsync(tb2.data(), r.th_b + spec, sizeof(int32_t) * (cnt - spec), hipMemcpyDeviceToHost,
                                   s);
            if (e == hipSuccess) e = hipStreamSynchronize(s);
            if (e != hipSuccess) return e;
            for (int64_t t = 0; t < cnt - spec; ++t) bs[tb2[t]].th.push_back(tv2[t]);
        }
        // link times x = (2 b * OA[j-1]) / E over links between positions
        // o < o2 of the order; x grows with OA, so each distinct E gives one
        // run of distinct OA values inside the window
        const int K = P.K, L = P.L;
        std::vector<double> Es;
        for (int o = 0; o < K; ++o)
            for (int o2 = o + 1; o2 < K; ++o2) {
                const double E = H.E[(int64_t)order_host[o] * K + order_host[o2]];
                if (E > 0.0) Es.push_back(E);
            }
        std::sort(Es.begin(), Es.end());
        Es.erase(std::unique(Es.begin(), Es.end()), Es.end());
        std::vector<int64_t> oa(H.outact, H.outact + (L > 1 ? L - 1 : 0));
        std::sort(oa.begin(), oa.end());
        oa.erase(std::unique(oa.begin(), oa.end()), oa.end());
        for (int bi = 0; bi < nb; ++bi) {
            BSearch &q = bs[bi];
            if (!q.active) continue;
            const double two_b = 2.0 * (double)H.bvals[bi];
            for (double E : Es) {
                auto x_of = [&](int64_t a) { return (two_b * (double)a) / E; };
                auto it = std::partition_point(oa.begin(), oa.end(), [&](int64_t a) { return !(x_of(a) > q.Pst); });
                for (; it != oa.end(); ++it) {
                    const double x = x_of(*it);
                    if (!(x < kInf) || !((q.mm1 * x) <= inc.T)) break;
                    q.th.push_back(x);
                }
            }
            std::sort(q.th.begin(), q.th.end());
            q.th.erase(std::unique(q.th.begin(), q.th.end()), q.th.end());
            q.F.assign(q.th.size(), std::nan(""));
            if (!q.th.empty()) q.iv.push_back({-1, (int)q.th.size() - 1});
        }
        // branch and bound over the bounds, one batched fill run per round
        double *h_tau = (double *)(hu + X.tau);
        int32_t *h_jb = (int32_t *)(hu + X.jb), *h_jd = (int32_t *)(hu + X.jd);
        int32_t *h_nj = (int32_t *)(hu + X.njob);
        for (int round = 0;; ++round) {
            std::vector<std::pair<int, int>> req;  // (b, index)
            for (int bi = 0; bi < nb; ++bi) {
                BSearch &q = bs[bi];
                for (auto &ab : q.iv) {
                    const int a = ab.first, c = ab.second;
                    const int u = c - a;  // bounds a+1 .. c
                    const int ways = std::min(kSplitWays, u);
                    for (int t = 1; t <= ways; ++t) {
                        const int k = a + (int)(((int64_t)u * t) / ways);
                        if (std::isnan(q.F[k])) {
                            q.F[k] = -1.0;  // requested
                            req.push_back({bi, k});
                        }
                    }
                }
            }
            if (req.empty()) break;
            if (rounds_out) *rounds_out = round + 1;
            for (size_t c0 = 0; c0 < req.size(); c0 += kMaxJobs) {
                const int J = (int)std::min<size_t>(kMaxJobs, req.size() - c0);
                int nlev_j = 0;
                std::vector<char> used(nb, 0);
                for (int t = 0; t < J; ++t) {
                    h_jb[t] = req[c0 + t].first;
                    h_tau[t] = bs[h_jb[t]].th[req[c0 + t].second];
                    h_jd[t] = dlim_of(h_jb[t], h_tau[t]);
                    nlev_j = std::max(nlev_j, (int)h_jd[t]);
                    used[h_jb[t]] = 1;
                }
                std::fill(h_nj, h_nj + (size_t)D * nb, 0);
                for (int t = 0; t < J; ++t)
                    for (int d = 1; d <= h_jd[t]; ++d) ++h_nj[(size_t)(d - 1) * nb + h_jb[t]];
                e = hipMemcpyAsync(r.up, hu, X.up, hipMemcpyHostToDevice, s);
                if (e == hipSuccess) e = dr.restore_tables(r.Tp, used);
                if (e != hipSuccess) return e;
                dr.phase2_jobs(r, J, nlev_j);
                e = hipMemcpyAsync(h_jf, r.job_F, sizeof(double) * J, hipMemcpyDeviceToHost, s);
                if (e == hipSuccess) e = hipStreamSynchronize(s);  // also frees the upload buffer for reuse
                if (e != hipSuccess) return e;
                for (int t = 0; t < J; ++t) {
                    BSearch &q = bs[h_jb[t]];
                    const int k = req[c0 + t].second;
                    q.F[k] = h_jf[t];
                    inc.offer((q.mm1 * q.th[k]) + h_jf[t], h_jb[t], q.th[k]);
                }
            }
            for (int bi = 0; bi < nb; ++bi) {
                BSearch &q = bs[bi];
                std::vector<std::pair<int, int>> next;
                for (auto &ab : q.iv) {
                    // the evaluated points split (a, c] into runs between known F
                    int u = ab.first;
                    for (int k = ab.first + 1; k <= ab.second; ++k) {
                        if (std::isnan(q.F[k])) continue;
                        const int v = k;
                        if (v > u + 1 && q.Fat(u) != q.F[v]) {
                            const double lb = (q.mm1 * q.th[u + 1]) + q.F[v];
                            if (inc.beaten_by(lb, bi, q.th[u + 1])) next.push_back({u, v});
                        }
                        u = v;
                    }
                }
                q.iv.swap(next);
            }
        }
    }
    // the best b and its bound: reuse the phase-2 argmins when the bound is P*
    const int bstar = inc.T < kInf ? inc.b : -1;
    if (bstar < 0 || inc.tau == Pst[bstar]) {
        dr.finish(dr.w.Pst, res_hd);
        return hipGetLastError();
    }
    double *h_bound = (double *)(hu + X.bound);
    int32_t *h_fdl = (int32_t *)(hu + X.fdl);
    for (int bi = 0; bi < nb; ++bi) {
        h_bound[bi] = kInf;
        h_fdl[bi] = 0;
    }
    h_bound[bstar] = inc.tau;
    h_fdl[bstar] = dlim_of(bstar, inc.tau);
    const int last_lev = h_fdl[bstar];
    e = hipMemcpyAsync(r.up, hu, X.up, hipMemcpyHostToDevice, s);
    std::vector<char> used(nb, 0);
    used[bstar] = 1;
    if (e == hipSuccess) e = dr.restore_tables(r.Tp, used);
    if (e != hipSuccess) return e;
    dr.phase2(r.bound, r.fdl, last_lev, dr.w.T);  // the relaxed bound
    dr.finish(r.bound, res_hd);
    return hipGetLastError();
}

}  // namespace tg
