// compose_orders.hip -- pipeline composition over every island subset and
// order (Sec. 5.2 builds the pipeline from any islands, each used at most
// once; Sec. 6.2 shows that the order in which islands are stacked changes
// the plan), for K <= 16 islands.
//
// With U the set of islands from a stage to the pipeline end, the stage's
// depth is |U|, so no island order is needed.  Per micro-batch size b:
//   V_d(i, k, U)  least bottleneck covering [i, L) with the stages on the
//                 islands of U (|U| = d), the first on k in U;
//   W_d(j, k, U)  least bottleneck of a continuation on U \ {k} after a stage
//                 on k ends at j: min over k' in U \ {k} of
//                 max(X(j, k, k'), V_{d-1}(j, k', U \ {k}));
//   F_d, G_d      the same for the fill, with every stage and link within the
//                 least bottleneck P* (step (3)), ties to the least cut j and
//                 the least next island k'.
// The levels are the set sizes d = 1..min(K, L), one launch per level and
// phase.  The states of level d are the pairs (k, U), k in U, |U| = d,
// numbered r * d + t: r is the rank of U among the d-sets in ascending
// numeric order (the combinatorial number system), t the position of k among
// U's islands.  Every state (k, U) reads the rows V_{d-1}(., k', U \ {k}) of
// the same smaller set for each k' in it, so a block owns one (d-1)-set U'
// (and b) and runs the states (k, U' + {k}) for the islands k outside U' one
// after the other: the rows come from HBM once, into LDS where they fit
// (13 KB with the two continuation rows), else from the cache after that.
// Where a level has few sets, the islands outside U' are split over several
// blocks.  Per state the block writes its continuation row W_d(., k, U) to
// LDS, then one thread per first layer i scans the cuts j.  As in the
// fixed-order composition, T_d(i, j, k) never decreases with j, so a scan
// stops at the first stage cost that cannot improve the running best.
#include <algorithm>
#include <type_traits>
#include <vector>

#include "compose_util.h"

#pragma clang fp contract(off)

namespace tg {

constexpr int kMaxSetIslands = 16;
constexpr int kMaxLayers = 512;
constexpr size_t kLevelLds = 12 * 1024;  // LDS bytes per level block: staged rows and continuation rows
constexpr int kLevelThreads = 128;
constexpr int64_t kPruneCells = (int64_t)1 << 22;  // fill cells below which every b runs at once
constexpr int kOrderFinishThreads = 1024;
constexpr uint32_t kNoKey = 0xFFFFFFFFu;
constexpr int64_t kTargetBlocks = 8192;  // blocks per level launch worth splitting for
constexpr int kReduceChunks = 64;        // partials per b in the root reductions

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Level bookkeeping, passed by value.
struct SetLevels {
    int32_t D;                            // levels 1..D = min(K, L)
    int32_t moff[kMaxSetIslands + 2];     // masks of popcount d start at moff[d]
    int32_t n[kMaxSetIslands + 2];        // states of level d: C(K, d) * d
    int64_t soff[kMaxSetIslands + 2];     // global number of level d's first state
    int64_t total;                        // states of all levels
    int32_t maxn;                         // largest level
};

static int64_t binom(int n, int k) {
    if (k < 0 || k > n) return 0;
    int64_t r = 1;
    for (int q = 1; q <= k; ++q) r = r * (n - k + q) / q;
    return r;
}

static SetLevels set_levels(const DevProblem &P) {
    SetLevels v{};
    v.D = std::min(P.K, P.L);
    int32_t mo = 0;
    int64_t so = 0;
    for (int d = 0; d <= P.K + 1 && d <= kMaxSetIslands + 1; ++d) {
        v.moff[d] = mo;
        v.soff[d] = so;
        const int64_t c = d <= P.K ? binom(P.K, d) : 0;
        v.n[d] = (d >= 1 && d <= v.D) ? (int32_t)(c * d) : 0;
        mo += (int32_t)c;
        so += v.n[d];
        v.maxn = std::max(v.maxn, v.n[d]);
    }
    v.total = v.soff[v.D + 1];
    return v;
}

struct OrdersWs {
    ComposeResult *res;
    int32_t *pos;       // [K] identity: groups are numbered by island id
    Groups g;
    int32_t *masks;     // [2^K] the d-sets of each level, ascending
    uint16_t *rank;     // [2^K] rank of a set among the sets of its size
    double *T;          // [D][nb][K][L][L] least cost of group ((i, j), k, b) fitting at depth d,
                        // by diagonal: [j - i - 1][i], so threads i read along a row
    double *X;          // [nb][K][K][L+1] link time after layer j-1 from island k to k'
    double *Vb[2];      // [nb][maxn][L+1] level values, double-buffered
    double *root;       // [nb][total] value at i = 0 of every state
    uint16_t *argF;     // [nb][total][L] least cut j of F
    uint8_t *argG;      // [nb][total][L+1] least next island of G (255: none)
    double *Pst;        // [nb]
    double *rootF;      // [nb]
    uint32_t *rootKey;  // [nb] (k << 24 | d << 16 | U) of the chosen root
    double *part_v;     // [nb][kReduceChunks] partial reductions
    uint32_t *part_k;   // [nb][kReduceChunks]
    int32_t *blist;     // [nb] the b of each grid row in a fill run
    size_t bytes;
};

static OrdersWs carve_orders(const DevProblem &P, int64_t n, void *base) {
    OrdersWs w{};
    char *p = (char *)base;
    size_t off = 0;
    auto take = [&](size_t bytes) -> void * {
        void *r = base ? (void *)(p + off) : nullptr;
        off += align256(bytes > 0 ? bytes : 1);
        return r;
    };
    const SetLevels lv = set_levels(P);
    const int64_t G = (int64_t)P.nb * P.NS * P.K, nb = P.nb, L = P.L, K = P.K;
    w.res = (ComposeResult *)take(sizeof(ComposeResult));
    w.pos = (int32_t *)take(sizeof(int32_t) * K);
    w.g.rec_g = (int32_t *)take(sizeof(int32_t) * n);
    w.g.rec_c = (double *)take(sizeof(double) * n);
    w.g.rec_d = (uint8_t *)take(n);
    w.g.gcnt = (int32_t *)take(sizeof(int32_t) * G);
    w.g.ent_c = (double *)take(sizeof(double) * n);
    w.g.ent_d = (uint8_t *)take(n);
    w.g.ent_i = (int64_t *)take(sizeof(int64_t) * n);
    w.g.tmp = (int64_t *)take(sizeof(int64_t) * group_scan_tiles(G));
    w.masks = (int32_t *)take(sizeof(int32_t) << K);
    w.rank = (uint16_t *)take(sizeof(uint16_t) << K);
    w.T = (double *)take(sizeof(double) * lv.D * nb * K * L * L);
    w.X = (double *)take(sizeof(double) * nb * K * K * (L + 1));
    w.Vb[0] = (double *)take(sizeof(double) * nb * lv.maxn * (L + 1));
    w.Vb[1] = (double *)take(sizeof(double) * nb * lv.maxn * (L + 1));
    w.root = (double *)take(sizeof(double) * nb * lv.total);
    w.argF = (uint16_t *)take(sizeof(uint16_t) * nb * lv.total * L);
    w.argG = (uint8_t *)take(sizeof(uint8_t) * nb * lv.total * (L + 1));
    w.Pst = (double *)take(sizeof(double) * nb);
    w.rootF = (double *)take(sizeof(double) * nb);
    w.rootKey = (uint32_t *)take(sizeof(uint32_t) * nb);
    w.blist = (int32_t *)take(sizeof(int32_t) * nb);
    w.part_v = (double *)take(sizeof(double) * nb * kReduceChunks);
    w.part_k = (uint32_t *)take(sizeof(uint32_t) * nb * kReduceChunks);
    w.bytes = off;
    return w;
}

size_t compose_orders_ws_bytes(const DevProblem &P, int64_t n_surv) { return carve_orders(P, n_surv, nullptr).bytes; }

// ---------------------------------------------------------------------------
// setup
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void orders_init(int K, int32_t *pos, ComposeResult *res) {
    const int t = threadIdx.x;
    if (t < K) pos[t] = t;
    if (t == 0) {
        res->err = 0;
        res->status = TG_ENOPLAN;
    }
}

// C(n, k) for the small arguments of the set numbering.
__device__ inline int32_t dbinom(int n, int k) {
    if (k < 0 || k > n) return 0;
    int32_t r = 1;
    for (int q = 1; q <= k; ++q) r = r * (n - k + q) / q;
    return r;
}

// Every nonempty set U of islands: its rank among the sets of its size (sum
// over its islands c_1 < c_2 < ... of C(c_t, t), ascending numeric order) and
// its slot in the level's list.
__global__ __launch_bounds__(256) void orders_masks(int K, SetLevels lv, int32_t *masks, uint16_t *rank) {
    const uint32_t U = blockIdx.x * blockDim.x + threadIdx.x;
    if (U == 0 || U >= (1u << K)) return;
    int r = 0, t = 0;
    for (uint32_t u = U; u; u &= u - 1) r += dbinom(__builtin_ctz(u), ++t);
    masks[lv.moff[t] + r] = (int32_t)U;
    rank[U] = (uint16_t)r;
}

// Stage tables: one thread per cell (diagonal j - i - 1, first layer i) of
// (island k, b) writes the least cost of group ((i, j), k, b)'s entries
// fitting at each depth d (+inf off the triangle).
__global__ __launch_bounds__(256) void orders_stage_table(DevProblem P, int D, const int32_t *__restrict__ gcnt,
                                                          const double *__restrict__ ent_c,
                                                          const uint8_t *__restrict__ ent_d, double *T) {
    const int64_t L = P.L;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t per_b = (int64_t)P.K * L * L;
    if (e >= (int64_t)P.nb * per_b) return;
    const int64_t bb = e / per_b, r = e - bb * per_b;
    const int64_t k = r / (L * L), c = r - k * L * L;
    const int64_t len = c / L + 1, i = c - (len - 1) * L;
    int32_t st = 0, en = 0;
    if (i + len <= L) {
        const int64_t G = group_id(P, k, bb, slice_of(L, i, i + len));
        st = G ? gcnt[G - 1] : 0;
        en = gcnt[G];
    }
    for (int d = 1; d <= D; ++d) {
        double v = kInf;
        for (int32_t a = st; a < en; ++a)
            if (ent_d[a] >= d && ent_c[a] < v) v = ent_c[a];
        T[(int64_t)(d - 1) * P.nb * per_b + e] = v;
    }
}

// Link times X[b][k][k'][j]: activations forward and gradients backward of one
// micro-batch across the boundary after layer j-1; no link (E = 0) is +inf.
__global__ __launch_bounds__(256) void orders_links(DevProblem P, double *X) {
    const int L = P.L, K = P.K;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t n = (int64_t)P.nb * K * K * (L + 1);
    if (e >= n) return;
    const int64_t j = e % (L + 1), q = e / (L + 1);
    const int64_t k2 = q % K, k = (q / K) % K, bb = q / ((int64_t)K * K);
    double x = kInf;
    if (j >= 1 && j < L) {
        const double E = P.E[k * K + k2];
        x = E == 0.0 ? kInf : ((2.0 * (double)P.bvals[bb]) * (double)P.outact[j - 1]) / E;
    }
    X[e] = x;
}

// ---------------------------------------------------------------------------
// levels
// ---------------------------------------------------------------------------
// Level 1: one stage on island k covering [i, L).
template <bool kFill>
__global__ __launch_bounds__(256) void orders_level1(DevProblem P, SetLevels lv, const double *__restrict__ T,
                                                     const double *__restrict__ Pst, double *cur, double *root,
                                                     const int32_t *__restrict__ blist) {
    const int L = P.L, K = P.K, bb = blist ? blist[blockIdx.y] : blockIdx.y;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= (int64_t)K * (L + 1)) return;
    const int k = (int)(e / (L + 1)), i = (int)(e - (int64_t)k * (L + 1));
    double v = kInf;
    if (i < L) {
        v = T[((int64_t)bb * K + k) * L * L + (int64_t)(L - i - 1) * L + i];
        if (kFill && !(v <= Pst[bb])) v = kInf;
    }
    cur[((int64_t)bb * lv.n[1] + k) * (L + 1) + i] = v;
    if (i == 0) root[(int64_t)bb * lv.total + lv.soff[1] + k] = v;
}

// Level d >= 2, block (part of the islands outside a (d-1)-set U', b).  kFill:
// the fill phase at bound P*, with argmins; otherwise the bottleneck phase.
// The block's states (k, U' + {k}) go in chunks of C: first every
// continuation row of the chunk into LDS (thread per (state, cut)), then every
// stage scan (thread per (state, first layer)), two barriers per chunk and
// every lane busy whatever L is.  kStage: the previous level's rows of U',
// read by every state, are staged in LDS first.
template <int NT, bool kFill, bool kStage>
__global__ __launch_bounds__(NT) void orders_level(DevProblem P, SetLevels lv, int d, int nsplit, int C,
                                                   const int32_t *__restrict__ masks,
                                                   const uint16_t *__restrict__ rank, const double *__restrict__ T,
                                                   const double *__restrict__ X, const double *__restrict__ prev,
                                                   double *cur, double *root, const double *__restrict__ Pst,
                                                   uint16_t *argF, uint8_t *argG, const int32_t *__restrict__ blist) {
    // LDS: (kStage) the set's previous-level rows, then C continuation rows
    extern __shared__ double lds_rows[];
    __shared__ int16_t s_k[kMaxSetIslands];
    __shared__ int32_t s_st[kMaxSetIslands];
    // per state: the first and last cut with a finite continuation (a scan
    // skips the cuts outside, where every candidate is +inf)
    __shared__ int32_t s_jlo[kMaxSetIslands], s_jhi[kMaxSetIslands];
    const int L = P.L, K = P.K, R = L + 1;
    const int rp = blockIdx.x / nsplit, part = blockIdx.x - rp * nsplit;
    const int bb = blist ? blist[blockIdx.y] : blockIdx.y;  // a fill run covers a list of b
    const uint32_t Up = (uint32_t)masks[lv.moff[d - 1] + rp];
    const int nk = K - (d - 1);
    const int per = (nk + nsplit - 1) / nsplit;
    const int q0 = part * per, q1 = min(nk, q0 + per);
    const int nu = d - 1;
    const int jmax = L - d + 1;
    const double bound = kFill ? Pst[bb] : 0.0;
    const double *Vp = prev + ((int64_t)bb * lv.n[d - 1] + (int64_t)rp * nu) * R;
    // (offsets from the LDS array itself keep these accesses LDS instructions)
    const double *Vs = lds_rows;
    double *Wl = lds_rows + (kStage ? nu * R : 0);
    // the islands of U' in ascending order (the same for every thread), and
    // each one's row offset in an X block
    int ks[kMaxSetIslands], koff[kMaxSetIslands];
    {
        uint32_t r2 = Up;
#pragma unroll
        for (int q = 0; q < kMaxSetIslands; ++q) {
            ks[q] = r2 ? __builtin_ctz(r2) : 0;
            koff[q] = ks[q] * R;
            r2 &= r2 - 1;
        }
    }
    constexpr int kIsl = kStage ? 8 : 4;  // islands' link loads in flight
    // the block's states: island k (the q-th outside U', from q0 on) and the
    // state number of (k, U' + {k})
    if ((int)threadIdx.x < q1 - q0) {
        uint32_t r2 = ((1u << K) - 1u) & ~Up;
        for (int t = 0; t < q0 + (int)threadIdx.x; ++t) r2 &= r2 - 1;
        const int k = __builtin_ctz(r2);
        const uint32_t U = Up | (1u << k);
        s_k[threadIdx.x] = (int16_t)k;
        s_st[threadIdx.x] = (int)rank[U] * d + __builtin_popcount(U & ((1u << k) - 1u));
        s_jlo[threadIdx.x] = INT_MAX;
        s_jhi[threadIdx.x] = -1;
    }
    if (kStage)
        for (int t = threadIdx.x; t < nu * R; t += NT) lds_rows[t] = Vp[t];
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1);
    for (int c0 = 0; c0 < q1 - q0; c0 += C) {
        const int nst = min(C, q1 - q0 - c0);
        // continuation rows W(j, k, U') of the chunk's states
        const int nwork = nst * jmax;
        for (int p0 = 0; p0 < nwork; p0 += NT) {
            const int p = p0 + (int)threadIdx.x;
            const bool act = p < nwork;
            const int s = act ? p / jmax : nst;  // lanes past the end: a state of their own
            const int j = act ? p - s * jmax + 1 : 0;
            int jf = INT_MAX;  // j if W is finite
            if (act) {
                const int qs = c0 + s;
                const int k = s_k[qs];
                const double *Xr = X + ((int64_t)bb * K + k) * K * R;
                double w = kInf;
                int arg = 255;
                for (int t0 = 0; t0 < nu; t0 += kIsl) {
                    // a link only matters next to a finite continuation: its
                    // load is skipped where V is +inf
                    double x[kIsl], vv[kIsl];
#pragma unroll
                    for (int u = 0; u < kIsl; ++u) {
                        const int t = min(t0 + u, nu - 1);
                        vv[u] = kStage ? Vs[t * R + j] : Vp[(int64_t)t * R + j];
                    }
#pragma unroll
                    for (int u = 0; u < kIsl; ++u) {
                        const int t = min(t0 + u, nu - 1);
                        x[u] = vv[u] < kInf ? Xr[koff[t] + j] : kInf;
                    }
#pragma unroll
                    for (int u = 0; u < kIsl; ++u) {
                        const int t = t0 + u;
                        const double v = vv[u];
                        if (t >= nu) {
                        } else if (kFill) {
                            if (x[u] <= bound) {
                                const double y = x[u] + v;
                                if (y < w) {
                                    w = y;
                                    arg = ks[t];
                                }
                            }
                        } else {
                            const double y = x[u] > v ? x[u] : v;
                            if (y < w) w = y;
                        }
                    }
                }
                Wl[s * R + j] = w;
                if (kFill) {
                    const int64_t gst = (int64_t)bb * lv.total + lv.soff[d] + s_st[qs];
                    argG[gst * R + j] = (uint8_t)arg;
                }
                if (w < kInf) jf = j;
            }
            // per state the least and greatest finite cut: a wave's lanes hold
            // runs of consecutive (state, cut) pairs, so a segmented reduction
            // over same-state lanes leaves each run's totals at its first lane
            int lo = jf, hi = jf == INT_MAX ? -1 : jf;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                const int lo2 = __shfl_down(lo, off), hi2 = __shfl_down(hi, off), s2 = __shfl_down(s, off);
                if (lane + off < kWave && s2 == s) {
                    lo = min(lo, lo2);
                    hi = max(hi, hi2);
                }
            }
            const int sprev = __shfl_up(s, 1);
            if (act && (lane == 0 || sprev != s) && hi >= 0) {
                atomicMin(&s_jlo[c0 + s], lo);
                atomicMax(&s_jhi[c0 + s], hi);
            }
        }
        __syncthreads();
        // the stage scans: one thread per (state, first layer i) walks the cuts j
        const int nrow = nst * R;
        for (int p = threadIdx.x; p < nrow; p += NT) {
            const int s = p / R, i = p - s * R;
            const int qs = c0 + s;
            const int k = s_k[qs];
            const int st = s_st[qs];
            const int64_t gst = (int64_t)bb * lv.total + lv.soff[d] + st;
            const double *Wrow = Wl + s * R;
            double best = kInf;
            int bj = 0;
            if (i <= L - d) {
                const int jend = min(jmax, s_jhi[qs]);
                // T_d(i, j, k) = Tr[(j - i - 1) * L + i]: the threads of a wave
                // read consecutive first layers
                const double *Ti = T + (((int64_t)(d - 1) * P.nb + bb) * K + k) * L * L + i;
                bool go = true;
                // with imbalance pruning the scan starts at the first balanced
                // cut; it starts no earlier than the first finite continuation
                const int js = max(P.jlo ? max(i + 1, P.jlo[k * L + i]) : i + 1, s_jlo[qs]);
                // four cuts' stage costs and continuation values read at a
                // time (clamped to the row), then taken in order without
                // branches: the scan stops at the first cost that cannot
                // improve the running best
                for (int j0 = js; go && j0 <= jend; j0 += 4) {
                    double tv[4], wv[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int jc = min(j0 + u, jend);
                        tv[u] = Ti[__umul24(jc - i - 1, L)];  // < L^2 <= 2^18
                        wv[u] = Wrow[jc];
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int j = j0 + u;
                        const bool live = go && j <= jend;
                        if (kFill) {
                            const bool stop = live && (tv[u] > bound || tv[u] >= best);
                            const double y = tv[u] + wv[u];
                            const bool take = live && !stop && y < best;
                            best = take ? y : best;
                            bj = take ? j : bj;
                            go = go && !stop;
                        } else {
                            const bool stop = live && tv[u] >= best;
                            const double y = tv[u] > wv[u] ? tv[u] : wv[u];
                            const bool take = live && !stop && y < best;
                            best = take ? y : best;
                            go = go && !stop;
                        }
                    }
                }
            }
            cur[((int64_t)bb * lv.n[d] + st) * R + i] = best;
            if (kFill && i < L) argF[gst * L + i] = (uint16_t)bj;
            if (i == 0) root[gst] = best;
        }
        __syncthreads();  // the chunk's rows are read; the next chunk rewrites them
    }
}

// ---------------------------------------------------------------------------
// roots and the plan
// ---------------------------------------------------------------------------
// Decodes global state number q of b's states into (k, d, U).
__device__ inline void state_of(const SetLevels &lv, const int32_t *masks, int64_t q, int *k, int *d, uint32_t *U) {
    int dd = 1;
    while (dd < lv.D && q >= lv.soff[dd + 1]) ++dd;
    const int64_t st = q - lv.soff[dd];
    const int r = (int)(st / dd), t = (int)(st - (int64_t)r * dd);
    uint32_t u = (uint32_t)masks[lv.moff[dd] + r];
    *U = u;
    for (int a = 0; a < t; ++a) u &= u - 1;
    *k = __builtin_ctz(u);
    *d = dd;
}

// Per b: P* = least root bottleneck (kRoot = false), or the root of the fill:
// least F, ties to the least first island k, then fewer stages d, then the
// least set U (kRoot = true).  Two passes: block (chunk, b) reduces a chunk of
// b's states to a partial, then block b reduces its partials.

__device__ inline bool key_less(double v1, uint32_t k1, double v2, uint32_t k2) {
    return v1 < v2 || (v1 == v2 && k1 < k2);
}

// Reduces (sv, sk) over the block (256 threads) into entry 0.
__device__ inline void block_argmin(double *sv, uint32_t *sk) {
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if (threadIdx.x < h && key_less(sv[threadIdx.x + h], sk[threadIdx.x + h], sv[threadIdx.x], sk[threadIdx.x])) {
            sv[threadIdx.x] = sv[threadIdx.x + h];
            sk[threadIdx.x] = sk[threadIdx.x + h];
        }
        __syncthreads();
    }
}

template <bool kRoot>
__global__ __launch_bounds__(256) void orders_reduce_part(SetLevels lv, const int32_t *__restrict__ masks,
                                                          const double *__restrict__ root, double *part_v,
                                                          uint32_t *part_k, const int32_t *__restrict__ blist) {
    __shared__ double sv[256];
    __shared__ uint32_t sk[256];
    const int c = blockIdx.x, bb = blist ? blist[blockIdx.y] : blockIdx.y;
    const int64_t per = (lv.total + kReduceChunks - 1) / kReduceChunks;
    const int64_t q0 = (int64_t)c * per, q1 = min(lv.total, q0 + per);
    const double *rv = root + (int64_t)bb * lv.total;
    double bv = kInf;
    uint32_t bk = kNoKey;
    for (int64_t q = q0 + threadIdx.x; q < q1; q += blockDim.x) {
        const double v = rv[q];
        if (!kRoot) {
            if (v < bv) bv = v;
            continue;
        }
        if (!(v < kInf) || v > bv) continue;
        int k, d;
        uint32_t U;
        state_of(lv, masks, q, &k, &d, &U);
        const uint32_t key = ((uint32_t)k << 24) | ((uint32_t)d << 16) | U;
        if (key_less(v, key, bv, bk)) {
            bv = v;
            bk = key;
        }
    }
    sv[threadIdx.x] = bv;
    sk[threadIdx.x] = bk;
    block_argmin(sv, sk);
    if (threadIdx.x == 0) {
        part_v[(int64_t)bb * kReduceChunks + c] = sv[0];
        part_k[(int64_t)bb * kReduceChunks + c] = sk[0];
    }
}

// No fill root yet for any b (a b whose fill does not run keeps none).
__global__ __launch_bounds__(256) void orders_clear_roots(int nb, double *rootF, uint32_t *rootKey) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t < nb) {
        rootF[t] = kInf;
        rootKey[t] = kNoKey;
    }
}

__global__ __launch_bounds__(256) void orders_reduce_final(const double *__restrict__ part_v,
                                                           const uint32_t *__restrict__ part_k, double *out_v,
                                                           uint32_t *out_key, const int32_t *__restrict__ blist) {
    __shared__ double sv[256];
    __shared__ uint32_t sk[256];
    const int bb = blist ? blist[blockIdx.x] : blockIdx.x;
    const bool in = threadIdx.x < kReduceChunks;
    sv[threadIdx.x] = in ? part_v[(int64_t)bb * kReduceChunks + threadIdx.x] : kInf;
    sk[threadIdx.x] = in ? part_k[(int64_t)bb * kReduceChunks + threadIdx.x] : kNoKey;
    block_argmin(sv, sk);
    if (threadIdx.x == 0) {
        out_v[bb] = sv[0];
        if (out_key) out_key[bb] = sk[0];
    }
}

// Choose b, walk the argmins from the root (one thread), then one wave per
// stage resolves its candidate.
__global__ __launch_bounds__(kOrderFinishThreads) void orders_finish(
    DevProblem P, SetLevels lv, const int32_t *__restrict__ masks, const uint16_t *__restrict__ rank,
    const int32_t *gcnt, const double *ent_c, const uint8_t *ent_d, const int64_t *ent_i, const double *X,
    const double *Pst, const double *rootF, const uint32_t *rootKey, const uint16_t *argF, const uint8_t *argG,
    ComposeResult *res) {
    __shared__ int32_t st_i[kMaxSetIslands], st_j[kMaxSetIslands], st_k[kMaxSetIslands], st_kn[kMaxSetIslands];
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
                if (!(Pst[bi] < kInf) || rootKey[bi] == kNoKey) continue;
                const int64_t m = P.B / P.bvals[bi];
                const double T = ((double)(m - 1) * Pst[bi]) + rootF[bi];
                if (T < bestT) {
                    bestT = T;
                    bb = bi;
                }
            }
        if (bb >= 0) {
            const int64_t b = P.bvals[bb];
            const uint32_t key = rootKey[bb];
            int k = (int)(key >> 24);
            const int S = (int)((key >> 16) & 0xFF);
            uint32_t U = key & 0xFFFFu;
            plan.b = (int32_t)b;
            plan.m = (int32_t)(P.B / b);
            plan.S = S;
            plan.P = Pst[bb];
            plan.F = rootF[bb];
            plan.T = bestT;
            res->status = TG_OK;
            int i = 0;
            bool ok = S >= 1 && S <= lv.D && (U >> k & 1u);
            for (int t = 0; ok && t < S; ++t) {
                const int d = S - t;
                int j = L, kn = -1;
                if (d > 1) {
                    const int tk = __builtin_popcount(U & ((1u << k) - 1u));
                    const int64_t gst = (int64_t)bb * lv.total + lv.soff[d] + (int64_t)rank[U] * d + tk;
                    j = argF[gst * L + i];
                    // an argmin on the optimal path is always set
                    ok = j > i && j <= L - d + 1;
                    if (ok) {
                        kn = argG[gst * (L + 1) + j];
                        ok = kn < K && kn != k && (U >> kn & 1u);
                    }
                }
                st_i[t] = i;
                st_j[t] = j;
                st_k[t] = k;
                st_kn[t] = kn;
                U &= ~(1u << k);
                i = j;
                k = kn;
            }
            if (ok) {
                sh_S = S;
                sh_bb = bb;
            } else {
                res->err = 4;
                res->status = TG_ENOPLAN;
            }
        }
    }
    __syncthreads();
    const int S = sh_S;
    if (S == 0) return;
    const int bb = sh_bb;
    const int wv = threadIdx.x / kWave;
    for (int t = wv; t < S; t += kOrderFinishThreads / kWave) {
        const int d = S - t, i = st_i[t], j = st_j[t], k = st_k[t], kn = st_kn[t];
        const double link = d > 1 ? X[(((int64_t)bb * K + k) * K + kn) * (L + 1) + j] : 0.0;
        resolve_stage(P, gcnt, ent_c, ent_d, ent_i, group_id(P, k, bb, slice_of(P.L, i, j)), i, j, k, d, link,
                      plan.stage[t], res);
    }
}

// ---------------------------------------------------------------------------
// host-side sequencing
// ---------------------------------------------------------------------------
// One phase's levels for nrow b: the b of grid row y is blist[y] (all b in
// order without a list).
template <bool kFill>
static void run_levels(const DevProblem &P, const SetLevels &lv, const OrdersWs &w, hipStream_t s, int nrow,
                       const int32_t *blist) {
    const int L = P.L;
    const dim3 g1((unsigned)(((int64_t)P.K * (L + 1) + 255) / 256), (unsigned)nrow);
    orders_level1<kFill><<<g1, dim3(256), 0, s>>>(P, lv, w.T, w.Pst, w.Vb[1], w.root, blist);
    for (int d = 2; d <= lv.D; ++d) {
        // blocks: the (d-1)-sets times b, each split over the islands outside
        // the set until there are enough blocks to fill the device
        const int64_t sets = binom(P.K, d - 1) * nrow;
        const int nk = P.K - (d - 1);
        const int nsplit = (int)std::max<int64_t>(1, std::min<int64_t>(nk, (kTargetBlocks + sets - 1) / sets));
        const dim3 grid((unsigned)(binom(P.K, d - 1) * nsplit), (unsigned)nrow);
        const double *prev = w.Vb[(d - 1) & 1];
        double *cur = w.Vb[d & 1];
        // LDS per block: the set's previous-level rows (when they fit) and a
        // chunk of continuation rows, within kLevelLds
        const size_t rowb = (size_t)(L + 1) * sizeof(double);
        const int fit = (int)std::max<size_t>(1, kLevelLds / rowb);  // rows within the budget
        const bool stage = d < fit;                                   // nu = d - 1 rows and one more
        const int C = std::max(1, std::min(std::min(nk, kMaxSetIslands), fit - (stage ? d - 1 : 0)));
        const size_t lds = ((stage ? (size_t)(d - 1) : 0) + (size_t)C) * rowb;
        auto go = [&](auto nt, auto st) {
            constexpr int NT = decltype(nt)::value;
            orders_level<NT, kFill, decltype(st)::value><<<grid, dim3(NT), lds, s>>>(
                P, lv, d, nsplit, C, w.masks, w.rank, w.T, w.X, prev, cur, w.root, w.Pst, w.argF, w.argG, blist);
        };
        auto pick = [&](auto nt) {
            if (stage)
                go(nt, std::true_type{});
            else
                go(nt, std::false_type{});
        };
        pick(std::integral_constant<int, kLevelThreads>{});
    }
}

hipError_t launch_compose_orders(const DevProblem &P, const int64_t *bvals_host, const int64_t *surv, int64_t n_surv,
                                 const double *cost, const uint8_t *dmax, void *ws, hipStream_t s,
                                 ComposeResult **result_dev) {
    if (P.K > kMaxSetIslands || P.L > kMaxLayers || P.nb > 65535) return hipErrorInvalidValue;
    const SetLevels lv = set_levels(P);
    const OrdersWs w = carve_orders(P, n_surv, ws);
    *result_dev = w.res;
    orders_init<<<dim3(1), dim3(64), 0, s>>>(P.K, w.pos, w.res);
    orders_masks<<<dim3((unsigned)(((1u << P.K) + 255) / 256)), dim3(256), 0, s>>>(P.K, lv, w.masks, w.rank);
    launch_grouping(P, surv, n_surv, cost, dmax, w.pos, w.g, w.res, s);
    const int64_t ncells = (int64_t)P.nb * P.K * P.L * P.L;
    orders_stage_table<<<dim3((unsigned)((ncells + 255) / 256)), dim3(256), 0, s>>>(P, lv.D, w.g.gcnt, w.g.ent_c,
                                                                                   w.g.ent_d, w.T);
    const int64_t nx = (int64_t)P.nb * P.K * P.K * (P.L + 1);
    orders_links<<<dim3((unsigned)((nx + 255) / 256)), dim3(256), 0, s>>>(P, w.X);
    // phase 1 for every b: the least bottleneck P*_b
    const int nb = P.nb;
    run_levels<false>(P, lv, w, s, nb, nullptr);
    orders_reduce_part<false><<<dim3(kReduceChunks, (unsigned)nb), dim3(256), 0, s>>>(lv, w.masks, w.root, w.part_v,
                                                                                     w.part_k, nullptr);
    orders_reduce_final<<<dim3((unsigned)nb), dim3(256), 0, s>>>(w.part_v, w.part_k, w.Pst, nullptr, nullptr);
    // phase 2 only where a b can still win: its fill is at least P*_b (every
    // stage and link adds a non-negative time and one of them is at least
    // P*_b), so T_b >= (m - 1) P*_b + P*_b.  The most promising b runs first;
    // then every b whose bound beats its T (ties to the smaller b).
    orders_clear_roots<<<dim3((unsigned)((nb + 255) / 256)), dim3(256), 0, s>>>(nb, w.rootF, w.rootKey);
    std::vector<int32_t> rows;
    if ((int64_t)nb * lv.total * (P.L + 1) < kPruneCells) {
        // a small search: every b in one run beats two host round trips
        for (int bi = 0; bi < nb; ++bi) rows.push_back(bi);
        hipError_t e = hipMemcpyAsync(w.blist, rows.data(), sizeof(int32_t) * nb, hipMemcpyHostToDevice, s);
        if (e != hipSuccess) return e;
        run_levels<true>(P, lv, w, s, nb, w.blist);
        orders_reduce_part<true><<<dim3(kReduceChunks, (unsigned)nb), dim3(256), 0, s>>>(lv, w.masks, w.root,
                                                                                        w.part_v, w.part_k, w.blist);
        orders_reduce_final<<<dim3((unsigned)nb), dim3(256), 0, s>>>(w.part_v, w.part_k, w.rootF, w.rootKey,
                                                                    w.blist);
        orders_finish<<<dim3(1), dim3(kOrderFinishThreads), 0, s>>>(P, lv, w.masks, w.rank, w.g.gcnt, w.g.ent_c,
                                                                    w.g.ent_d, w.g.ent_i, w.X, w.Pst, w.rootF,
                                                                    w.rootKey, w.argF, w.argG, w.res);
        e = hipGetLastError();
        if (e == hipSuccess) e = hipStreamSynchronize(s);  // the b list above must outlive its copy
        return e;
    }
    std::vector<double> pst(nb);
    hipError_t e = hipMemcpyAsync(pst.data(), w.Pst, sizeof(double) * nb, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
    std::vector<double> lb(nb, kInf), mm1(nb);
    int b0 = -1;
    for (int bi = 0; bi < nb; ++bi) {
        mm1[bi] = (double)(P.B / bvals_host[bi] - 1);
        if (!(pst[bi] < kInf)) continue;
        lb[bi] = (mm1[bi] * pst[bi]) + pst[bi];
        if (b0 < 0 || lb[bi] < lb[b0]) b0 = bi;
    }
    auto fill_run = [&](const std::vector<int32_t> &bl) -> hipError_t {
        hipError_t e2 = hipMemcpyAsync(w.blist, bl.data(), sizeof(int32_t) * bl.size(), hipMemcpyHostToDevice, s);
        if (e2 != hipSuccess) return e2;
        const int n = (int)bl.size();
        run_levels<true>(P, lv, w, s, n, w.blist);
        orders_reduce_part<true><<<dim3(kReduceChunks, (unsigned)n), dim3(256), 0, s>>>(lv, w.masks, w.root,
                                                                                       w.part_v, w.part_k, w.blist);
        orders_reduce_final<<<dim3((unsigned)n), dim3(256), 0, s>>>(w.part_v, w.part_k, w.rootF, w.rootKey,
                                                                   w.blist);
        return hipGetLastError();
    };
    if (b0 >= 0) {
        rows.assign(1, b0);
        e = fill_run(rows);
        double f0 = kInf;
        if (e == hipSuccess) e = hipMemcpyAsync(&f0, w.rootF + b0, sizeof(double), hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return e;
        const double t0 = (mm1[b0] * pst[b0]) + f0;
        std::vector<int32_t> rest;
        for (int bi = 0; bi < nb; ++bi)
            if (bi != b0 && lb[bi] < kInf && (lb[bi] < t0 || (lb[bi] == t0 && bi < b0))) rest.push_back(bi);
        if (!rest.empty()) {
            rows = rest;
            e = fill_run(rows);
            if (e != hipSuccess) return e;
        }
    }
    orders_finish<<<dim3(1), dim3(kOrderFinishThreads), 0, s>>>(P, lv, w.masks, w.rank, w.g.gcnt, w.g.ent_c,
                                                                w.g.ent_d, w.g.ent_i, w.X, w.Pst, w.rootF,
                                                                w.rootKey, w.argF, w.argG, w.res);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(s);  // the b list above must outlive its copy
    return e;
}

}  // namespace tg
