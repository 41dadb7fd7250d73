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

#include "tg_device.h"

#pragma clang fp contract(off)

namespace tg {

constexpr int kScanThreads = 256;
constexpr int kScanPerThread = 8;
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

__global__ __launch_bounds__(kScanThreads) void scan_reduce_i32(const int32_t *a, int64_t n, int64_t *tile_sum) {
    __shared__ int64_t lds[kScanThreads / kWave + 1];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPerThread;
    int64_t c = 0;
    for (int t = 0; t < kScanPerThread; ++t)
        if (base + t < n) c += a[base + t];
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
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPerThread;
    int32_t v[kScanPerThread];
    int64_t c = 0;
    for (int t = 0; t < kScanPerThread; ++t) {
        v[t] = (base + t < n) ? a[base + t] : 0;
        c += v[t];
    }
    int64_t total;
    int64_t run = tile_off[blockIdx.x] + block_excl_scan<int64_t>(c, lds, &total);
    for (int t = 0; t < kScanPerThread; ++t) {
        if (base + t < n) a[base + t] = (int32_t)run;
        run += v[t];
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
    int32_t *gcnt;     // [n_groups] counts -> offsets -> ends
    double *ent_c;     // [n] grouped entries: cost
    uint8_t *ent_d;    // [n] d_max
    int64_t *ent_i;    // [n] candidate index
    int32_t *bcnt;     // [n_buckets + 1] event counts -> bucket starts (last = total)
    int32_t *ev_cell;  // [2n]
    double *ev_val;    // [2n]
    double *T;         // [n_groups] current stage table, layout [b][s][o]
    double *Wb[2];     // [nb][L+1][K] continuation rows, double-buffered by level
    uint16_t *argF;    // [D][nb][L][K]
    uint8_t *argG;     // [D][nb][L+1][K]
    double *Pst;       // [nb]
    double *rootF;     // [nb]
    int32_t *root_o;   // [nb]
    int32_t *root_d;   // [nb]
    int64_t *tmp;      // scan tiles
    size_t bytes;
};

static int64_t n_groups(const DevProblem &P) { return (int64_t)P.nb * P.NS * P.K; }
static int levels(const DevProblem &P) { return P.K < P.L ? P.K : P.L; }
static int64_t n_buckets(const DevProblem &P) { return (int64_t)levels(P) * P.nb * P.L; }

static Ws carve(const DevProblem &P, int64_t n, void *base) {
    Ws w{};
    char *p = (char *)base;
    size_t off = 0;
    auto take = [&](size_t bytes) -> void * {
        void *r = base ? (void *)(p + off) : nullptr;
        off += align256(bytes > 0 ? bytes : 1);
        return r;
    };
    const int64_t G = n_groups(P), D = levels(P), nbk = n_buckets(P);
    const int64_t rows = (int64_t)P.nb * (P.L + 1) * P.K;
    const int64_t tiles = (std::max(G, nbk) + kScanTile - 1) / kScanTile + 1;
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
    w.bcnt = (int32_t *)take(sizeof(int32_t) * (nbk + 1));
    w.ev_cell = (int32_t *)take(sizeof(int32_t) * 2 * n);
    w.ev_val = (double *)take(sizeof(double) * 2 * n);
    w.T = (double *)take(sizeof(double) * G);
    w.Wb[0] = (double *)take(sizeof(double) * rows);
    w.Wb[1] = (double *)take(sizeof(double) * rows);
    w.argF = (uint16_t *)take(sizeof(uint16_t) * D * P.nb * P.L * P.K);
    w.argG = (uint8_t *)take(sizeof(uint8_t) * D * rows);
    w.Pst = (double *)take(sizeof(double) * P.nb);
    w.rootF = (double *)take(sizeof(double) * P.nb);
    w.root_o = (int32_t *)take(sizeof(int32_t) * P.nb);
    w.root_d = (int32_t *)take(sizeof(int32_t) * P.nb);
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

// Groups (slice, island position, b) are numbered position-major, then b,
// then slice: the candidate list runs through each config's slices in
// ascending order, so building the groups touches consecutive counters.  The
// stage table keeps the DP's layout [b][slice][position].
__host__ __device__ inline int64_t group_id(const DevProblem &P, int64_t o, int64_t bi, int64_t s) {
    return (o * P.nb + bi) * P.NS + s;
}
__host__ __device__ inline int64_t cell_id(const DevProblem &P, int64_t bi, int64_t s, int64_t o) {
    return (bi * P.NS + s) * P.K + o;
}

// Index of the pair of positions (o, o2), o < o2, in a packed triangle.
__host__ __device__ inline int tri(int o, int o2) { return o2 * (o2 - 1) / 2 + o; }

__global__ void prep_kernel(DevProblem P, const int32_t *order, int32_t *pos, double *EoT, uint8_t *EiT,
                            ComposeResult *res) {
    const int K = P.K;
    for (int t = threadIdx.x; t < K; t += blockDim.x) pos[order[t]] = t;
    for (int t = threadIdx.x; t < K * K; t += blockDim.x) {
        const int o2 = t / K, o = t - o2 * K;
        const int64_t e = (int64_t)order[o] * K + order[o2];
        EoT[t] = P.E[e];
        if (o < o2) EiT[tri(o, o2)] = P.n_ev ? (uint8_t)P.Eidx[e] : 0;
    }
    if (threadIdx.x == 0) {
        res->err = 0;
        res->status = TG_ENOPLAN;
    }
}

// ---------------------------------------------------------------------------
// grouping: candidate list -> per-group entry records -> per-level events
// ---------------------------------------------------------------------------
// Reads each listed candidate's score once (the list is ascending, so the
// reads walk the score arrays forward) and counts the group sizes.
__global__ __launch_bounds__(256) void gather_kernel(DevProblem P, const int64_t *surv, int64_t n,
                                                     const double *cost, const uint8_t *dmax, const int32_t *pos,
                                                     int32_t *rec_g, double *rec_c, uint8_t *rec_d, int32_t *gcnt,
                                                     ComposeResult *res) {
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x) {
        int32_t G = -1;
        const int64_t idx = surv[r];
        if (idx < 0 || idx >= P.N || (r > 0 && surv[r - 1] >= idx)) {
            atomicOr(&res->err, 1);
        } else {
            const int64_t g = idx / P.NS, s = idx - g * P.NS;
            const Coef &c = P.coef[g];
            if (c.b_idx < 0) {
                atomicOr(&res->err, 2);
            } else {
                const uint8_t d = dmax[idx];
                if (d > 0) {
                    G = (int32_t)group_id(P, pos[c.k], c.b_idx, s);
                    rec_c[r] = cost[idx];
                    rec_d[r] = d;
                    atomicAdd(&gcnt[G], 1);
                }
            }
        }
        rec_g[r] = G;
    }
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

// Stage table at depth 1: the least cost of each group.  A block transposes a
// tile of 64 slices x 32 positions of one b through LDS, so it reads the group
// offsets along slices and writes the table along positions.
constexpr int kTileS = 64, kTileO = 32;

__global__ __launch_bounds__(256) void table_init(DevProblem P, const int32_t *__restrict__ gcnt,
                                                  const double *__restrict__ ent_c, double *__restrict__ T) {
    __shared__ double tile[kTileO][kTileS + 1];
    const int64_t s0 = (int64_t)blockIdx.x * kTileS;
    const int o0 = blockIdx.y * kTileO, bi = blockIdx.z;
    for (int t = threadIdx.x; t < kTileS * kTileO; t += blockDim.x) {
        const int sl = t % kTileS, ol = t / kTileS;
        const int64_t s = s0 + sl;
        const int o = o0 + ol;
        double v = kInf;
        if (s < P.NS && o < P.K) {
            const int64_t G = group_id(P, o, bi, s);
            const int32_t st = G ? gcnt[G - 1] : 0, en = gcnt[G];
            for (int32_t e = st; e < en; ++e) v = fmin(v, ent_c[e]);
        }
        tile[ol][sl] = v;
    }
    __syncthreads();
    for (int t = threadIdx.x; t < kTileS * kTileO; t += blockDim.x) {
        const int ol = t % kTileO, sl = t / kTileO;
        const int64_t s = s0 + sl;
        const int o = o0 + ol;
        if (s < P.NS && o < P.K) T[cell_id(P, bi, s, o)] = tile[ol][sl];
    }
}

// Per group: entry e is the least fitting candidate at depths (D_e, d_e],
// D_e = the largest d_max among entries with a smaller key; it sets T at
// level D_e + 1 (level 1 is written by table_init).  After the group's
// largest d_max M nothing fits: T = +inf from level M + 1.  At most one event
// per (group, level).  Block (i, b) owns the groups of the slices starting at
// layer i, and with them every bucket (level, b, i): counts and slots come
// from LDS, with no global atomics.
constexpr int kGroupRegs = 8;

template <bool kEmit>
__global__ __launch_bounds__(256) void group_events(DevProblem P, const int32_t *__restrict__ gcnt,
                                                    const double *__restrict__ ent_c,
                                                    const uint8_t *__restrict__ ent_d,
                                                    const int64_t *__restrict__ ent_i, int32_t *bcnt,
                                                    int32_t *__restrict__ ev_cell, double *__restrict__ ev_val) {
    __shared__ int32_t hist[256];
    const int i = blockIdx.x, bi = blockIdx.y;
    const int L = P.L, K = P.K;
    const int D = K < L ? K : L;
    for (int lev = threadIdx.x; lev < D; lev += blockDim.x)
        hist[lev] = kEmit ? bcnt[((int64_t)lev * P.nb + bi) * L + i] : 0;
    __syncthreads();
    const int64_t s0 = slice_of(L, i, i + 1);
    const int64_t n_sl = L - i;
    const int64_t ncell = n_sl * K;
    for (int64_t t = threadIdx.x; t < ncell; t += blockDim.x) {
        const int64_t o = t / n_sl, s = s0 + (t - o * n_sl);
        const int64_t G = group_id(P, o, bi, s);
        const int32_t st = G ? gcnt[G - 1] : 0, en = gcnt[G];
        if (st == en) continue;
        const int64_t cell = cell_id(P, bi, s, o);
        auto emit = [&](int level, double v) {
            if (kEmit) {
                const int32_t slot = atomicAdd(&hist[level - 1], 1);
                ev_cell[slot] = (int32_t)cell;
                ev_val[slot] = v;
            } else {
                atomicAdd(&hist[level - 1], 1);
            }
        };
        int M = 0;
        if (en - st <= kGroupRegs) {
            // small group (the usual staircase): entries in registers, compared there
            double c[kGroupRegs];
            int d[kGroupRegs];
            int64_t id[kGroupRegs];
            const int n = en - st;
#pragma unroll
            for (int e = 0; e < kGroupRegs; ++e) {
                c[e] = e < n ? ent_c[st + e] : kInf;
                d[e] = e < n ? (int)ent_d[st + e] : 0;
                id[e] = e < n ? ent_i[st + e] : 0;
            }
#pragma unroll
            for (int e = 0; e < kGroupRegs; ++e) {
                if (e >= n) break;
                M = max(M, d[e]);
                int De = 0;
#pragma unroll
                for (int q = 0; q < kGroupRegs; ++q) {
                    const bool less = q < n && (c[q] < c[e] || (c[q] == c[e] && (d[q] > d[e] || (d[q] == d[e] && id[q] < id[e]))));
                    if (less) De = max(De, d[q]);
                }
                if (De >= 1 && De < d[e] && De + 1 <= D) emit(De + 1, c[e]);
            }
        } else {
            for (int32_t e = st; e < en; ++e) {
                const double ce = ent_c[e];
                const int de = ent_d[e];
                const int64_t ie = ent_i[e];
                M = max(M, de);
                int De = 0;
                for (int32_t q = st; q < en; ++q) {
                    const double cq = ent_c[q];
                    const int dq = ent_d[q];
                    const bool less = cq < ce || (cq == ce && (dq > de || (dq == de && ent_i[q] < ie)));
                    if (less) De = max(De, dq);
                }
                if (De >= 1 && De < de && De + 1 <= D) emit(De + 1, ce);
            }
        }
        if (M + 1 <= D) emit(M + 1, kInf);
    }
    if (!kEmit) {
        __syncthreads();
        for (int lev = threadIdx.x; lev < D; lev += blockDim.x) bcnt[((int64_t)lev * P.nb + bi) * L + i] = hist[lev];
    }
}

// ---------------------------------------------------------------------------
// dynamic program, one launch per level
// ---------------------------------------------------------------------------
__device__ inline void apply_events(const int32_t *__restrict__ bcnt, const int32_t *__restrict__ ev_cell,
                                    const double *__restrict__ ev_val, double *__restrict__ T, int64_t bucket) {
    const int32_t st = bcnt[bucket], en = bcnt[bucket + 1];
    const int step = blockDim.x;
    for (int32_t base = st + threadIdx.x; base < en; base += 4 * step) {
        int32_t c[4];
        double v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int32_t e = base + k * step;
            c[k] = e < en ? ev_cell[e] : -1;
            v[k] = e < en ? ev_val[e] : 0.0;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (c[k] >= 0) T[c[k]] = v[k];
    }
}

// Link times of the boundary after layer i-1 for this block's b.  With few
// distinct bandwidths (the usual case) the block divides once per distinct
// value and keeps the per-pair index triangle in LDS; otherwise it divides
// per pair.
struct Links {
    const double *xs;      // LDS [n_ev]
    const uint8_t *tri_s;  // LDS triangle of indices
    const double *EoT;     // global, used without a table
    double num;
    bool table;
    __device__ inline double operator()(int o, int o2, int K) const {
        if (table) return xs[tri_s[tri(o, o2)]];
        const double E = EoT[(int64_t)o2 * K + o];
        return E == 0.0 ? kInf : num / E;
    }
};

// Fills the block's LDS link tables for positions o < o2 <= top.
__device__ inline Links stage_links(const DevProblem &P, int i, int bi, int top, const uint8_t *EiT,
                                    const double *EoT, double *xs, uint8_t *tri_s) {
    Links X{xs, tri_s, EoT, 0.0, P.n_ev > 0};
    if (i == 0) return X;
    X.num = (2.0 * (double)P.bvals[bi]) * (double)P.outact[i - 1];
    if (X.table) {
        for (int u = threadIdx.x; u < P.n_ev; u += blockDim.x) {
            const double E = P.Ev[u];
            xs[u] = E == 0.0 ? kInf : X.num / E;
        }
        const int nbytes = top * (top + 1) / 2;  // rows o2 <= top
        const int nwords = (nbytes + 3) / 4;
        const uint32_t *src = (const uint32_t *)EiT;
        uint32_t *dst = (uint32_t *)tri_s;
        for (int t = threadIdx.x; t < nwords; t += blockDim.x) dst[t] = src[t];
    }
    return X;
}

// Each cell (i, o) is served by kSplit threads: sub-thread k scans
// j = i+1+k, i+1+k+kSplit, ... and o2 = o+1+k, o+1+k+kSplit, ..., and LDS
// combines them.  A sub-thread may stop at its own first T not below its own
// running best: everything it skips is no smaller than that best, which it
// reached at a smaller j, so neither the minimum nor the least j attaining it
// can be among the skipped ones.
constexpr int kSplit = 4;

__device__ inline int cell_pad(int K) { return K <= 64 ? 64 : (K <= 128 ? 128 : (K <= 192 ? 192 : 256)); }

// Phase 1: bottleneck values.  Block (i, b), thread (sub, o).
__global__ __launch_bounds__(1024) void level_bottleneck(DevProblem P, int d, const int32_t *bcnt,
                                                         const int32_t *ev_cell, const double *ev_val, double *T,
                                                         const double *Wprev, double *Wnext, const double *EoT,
                                                         const uint8_t *EiT, double *Pst) {
    extern __shared__ uint32_t tri_w[];
    uint8_t *tri_s = (uint8_t *)tri_w;
    __shared__ double part[kSplit][256];
    __shared__ double Vs[256];
    __shared__ double xs[kMaxDistinctE];
    const int i = blockIdx.x, bi = blockIdx.y;
    const int L = P.L, K = P.K, KP = cell_pad(K);
    const int o = threadIdx.x % KP, sub = threadIdx.x / KP;
    apply_events(bcnt, ev_cell, ev_val, T, ((int64_t)(d - 1) * P.nb + bi) * L + i);
    const Links X = stage_links(P, i, bi, K - d, EiT, EoT, xs, tri_s);
    __syncthreads();
    const int64_t srow = (int64_t)bi * P.NS + slice_of(L, i, i + 1);  // slice (i, j) is srow + j-i-1
    double v = kInf;
    if (o < K && o <= K - d) {
        if (d == 1) {
            if (sub == 0) v = T[(srow + (L - i - 1)) * K + o];
        } else {
            const double *Wp = Wprev + (int64_t)bi * (L + 1) * K + o;
            const double *Tp = T + srow * K + o;
            const int jmax = L - d + 1;
            for (int j0 = i + 1 + sub; j0 <= jmax; j0 += 2 * kSplit) {
                const int j1 = j0 + kSplit;
                const double t0 = Tp[(int64_t)(j0 - i - 1) * K], w0 = Wp[(int64_t)j0 * K];
                const double t1 = j1 <= jmax ? Tp[(int64_t)(j1 - i - 1) * K] : kInf;
                const double w1 = j1 <= jmax ? Wp[(int64_t)j1 * K] : kInf;
                if (!(t0 < v)) break;  // T never decreases in j
                v = fmin(v, fmax(t0, w0));
                if (!(t1 < v)) break;
                v = fmin(v, fmax(t1, w1));
            }
        }
    }
    part[sub][o] = v;
    __syncthreads();
    if (sub == 0) {
        double m = part[0][o];
#pragma unroll
        for (int k = 1; k < kSplit; ++k) m = fmin(m, part[k][o]);
        Vs[o] = m;
    }
    __syncthreads();
    if (i == 0) {
        if (threadIdx.x == 0) {
            double m = kInf;
            for (int t = 0; t < K; ++t) m = fmin(m, Vs[t]);
            Pst[bi] = fmin(Pst[bi], m);
        }
        return;
    }
    double w = kInf;
    if (o < K)
        for (int o2 = o + 1 + sub; o2 <= K - d; o2 += kSplit) w = fmin(w, fmax(X(o, o2, K), Vs[o2]));
    part[sub][o] = w;
    __syncthreads();
    if (sub == 0 && o < K) {
        double m = part[0][o];
#pragma unroll
        for (int k = 1; k < kSplit; ++k) m = fmin(m, part[k][o]);
        Wnext[((int64_t)bi * (L + 1) + i) * K + o] = m;
    }
}

// (value, index) pairs: the smaller value, ties to the smaller index.
__device__ inline bool lex_less(double v1, int a1, double v2, int a2) {
    return v1 < v2 || (v1 == v2 && a1 < a2);
}

// Phase 2: fill values and argmins at the bottleneck P*.
__global__ __launch_bounds__(1024) void level_fill(DevProblem P, int d, const int32_t *bcnt, const int32_t *ev_cell,
                                                   const double *ev_val, double *T, const double *Gprev,
                                                   double *Gnext, const double *EoT, const uint8_t *EiT,
                                                   const double *Pst, uint16_t *argF, uint8_t *argG,
                                                   double *rootF, int32_t *root_o, int32_t *root_d) {
    extern __shared__ uint32_t tri_w[];
    uint8_t *tri_s = (uint8_t *)tri_w;
    __shared__ double part[kSplit][256];
    __shared__ int32_t parg[kSplit][256];
    __shared__ double Fs[256];
    __shared__ double xs[kMaxDistinctE];
    const int i = blockIdx.x, bi = blockIdx.y;
    const int L = P.L, K = P.K, KP = cell_pad(K);
    const int o = threadIdx.x % KP, sub = threadIdx.x / KP;
    const double Ps = Pst[bi];
    if (!(Ps < kInf)) return;
    apply_events(bcnt, ev_cell, ev_val, T, ((int64_t)(d - 1) * P.nb + bi) * L + i);
    const Links X = stage_links(P, i, bi, K - d, EiT, EoT, xs, tri_s);
    __syncthreads();
    const int64_t srow = (int64_t)bi * P.NS + slice_of(L, i, i + 1);
    double v = kInf;
    int arg = 0xFFFF;
    if (o < K && o <= K - d) {
        if (d == 1) {
            if (sub == 0) {
                const double t = T[(srow + (L - i - 1)) * K + o];
                if (t <= Ps) {
                    v = t;
                    arg = L;
                }
            }
        } else {
            const double *Gp = Gprev + (int64_t)bi * (L + 1) * K + o;
            const double *Tp = T + srow * K + o;
            const int jmax = L - d + 1;
            for (int j0 = i + 1 + sub; j0 <= jmax; j0 += 2 * kSplit) {
                const int j1 = j0 + kSplit;
                const double t0 = Tp[(int64_t)(j0 - i - 1) * K], g0 = Gp[(int64_t)j0 * K];
                const double t1 = j1 <= jmax ? Tp[(int64_t)(j1 - i - 1) * K] : kInf;
                const double g1 = j1 <= jmax ? Gp[(int64_t)j1 * K] : kInf;
                if (!(t0 <= Ps) || !(t0 < v)) break;  // T never decreases in j
                const double c0 = t0 + g0;
                if (c0 < v) {
                    v = c0;
                    arg = j0;
                }
                if (!(t1 <= Ps) || !(t1 < v)) break;
                const double c1 = t1 + g1;
                if (c1 < v) {
                    v = c1;
                    arg = j1;
                }
            }
        }
    }
    part[sub][o] = v;
    parg[sub][o] = arg;
    __syncthreads();
    if (sub == 0) {
        double m = part[0][o];
        int a = parg[0][o];
#pragma unroll
        for (int k = 1; k < kSplit; ++k)
            if (lex_less(part[k][o], parg[k][o], m, a)) {
                m = part[k][o];
                a = parg[k][o];
            }
        Fs[o] = m;
        if (o < K) argF[(((int64_t)(d - 1) * P.nb + bi) * L + i) * K + o] = (uint16_t)(m < kInf ? a : 0xFFFF);
    }
    __syncthreads();
    if (i == 0) {
        if (threadIdx.x == 0) {
            double m = kInf;
            int mo = -1;
            for (int t = 0; t < K; ++t)
                if (Fs[t] < m) {
                    m = Fs[t];
                    mo = t;
                }
            // lexicographic (fill, position, depth); depths arrive in ascending order
            if (mo >= 0 && (m < rootF[bi] || (m == rootF[bi] && mo < root_o[bi]))) {
                rootF[bi] = m;
                root_o[bi] = mo;
                root_d[bi] = d;
            }
        }
        return;
    }
    double w = kInf;
    int a = 0xFF;
    if (o < K)
        for (int o2 = o + 1 + sub; o2 <= K - d; o2 += kSplit) {
            const double x = X(o, o2, K);
            if (!(x <= Ps)) continue;
            const double c = x + Fs[o2];
            if (c < w) {
                w = c;
                a = o2;
            }
        }
    part[sub][o] = w;
    parg[sub][o] = a;
    __syncthreads();
    if (sub == 0 && o < K) {
        double m = part[0][o];
        int aa = parg[0][o];
#pragma unroll
        for (int k = 1; k < kSplit; ++k)
            if (lex_less(part[k][o], parg[k][o], m, aa)) {
                m = part[k][o];
                aa = parg[k][o];
            }
        Gnext[((int64_t)bi * (L + 1) + i) * K + o] = m;
        argG[(((int64_t)(d - 1) * P.nb + bi) * (L + 1) + i) * K + o] = (uint8_t)(m < kInf ? aa : 0xFF);
    }
}

// ---------------------------------------------------------------------------
// choose b, walk the argmins, resolve each stage's candidate
// ---------------------------------------------------------------------------
__global__ void finish_kernel(DevProblem P, const int32_t *gcnt, const double *ent_c, const uint8_t *ent_d,
                              const int64_t *ent_i, const int32_t *order, const double *EoT, const double *Pst,
                              const double *rootF, const int32_t *root_o, const int32_t *root_d,
                              const uint16_t *argF, const uint8_t *argG, ComposeResult *res) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const int L = P.L, K = P.K;
    tg_plan &plan = res->plan;
    plan.b = 0;
    plan.m = 0;
    plan.S = 0;
    plan.reserved = 0;
    plan.P = kInf;
    plan.F = kInf;
    plan.T = kInf;
    if (res->err) return;
    double bestT = kInf;
    int bb = -1;
    for (int bi = 0; bi < P.nb; ++bi) {
        if (!(Pst[bi] < kInf) || root_o[bi] < 0) continue;
        const int64_t m = P.B / P.bvals[bi];
        const double T = ((double)(m - 1) * Pst[bi]) + rootF[bi];
        if (T < bestT) {
            bestT = T;
            bb = bi;
        }
    }
    if (bb < 0) return;
    const int64_t b = P.bvals[bb];
    plan.b = (int32_t)b;
    plan.m = (int32_t)(P.B / b);
    plan.S = root_d[bb];
    plan.P = Pst[bb];
    plan.F = rootF[bb];
    plan.T = bestT;
    res->status = TG_OK;
    int i = 0, o = root_o[bb];
    const int S = root_d[bb];
    for (int t = 0; t < S; ++t) {
        const int d = S - t;
        int j = L, o_next = -1;
        if (d > 1) {
            j = argF[(((int64_t)(d - 1) * P.nb + bb) * L + i) * K + o];
            if (j <= i || j > L - d + 1) {  // an argmin on the optimal path is always set
                res->err = 4;
                res->status = TG_ENOPLAN;
                return;
            }
            o_next = argG[(((int64_t)(d - 2) * P.nb + bb) * (L + 1) + j) * K + o];
            if (o_next <= o || o_next >= K) {
                res->err = 4;
                res->status = TG_ENOPLAN;
                return;
            }
        }
        const int64_t s = slice_of(L, i, j);
        const int64_t G = group_id(P, o, bb, s);
        const int32_t st = G ? gcnt[G - 1] : 0, en = gcnt[G];
        int64_t best = -1;
        double bc = kInf;
        int bd = 0;
        for (int32_t e = st; e < en; ++e) {
            const int64_t ie = ent_i[e];
            const double c = ent_c[e];
            const int dd = ent_d[e];
            if (dd < d) continue;
            if (best < 0 || c < bc || (c == bc && (dd > bd || (dd == bd && ie < best)))) {
                best = ie;
                bc = c;
                bd = dd;
            }
        }
        if (best < 0) {  // the stage table said a candidate fits here
            res->err = 4;
            res->status = TG_ENOPLAN;
            return;
        }
        const int64_t g = best / P.NS;
        const Coef &c = P.coef[g];
        const int64_t Lp = L + 1;
        const double Pd = (double)(P.pre[Lp + j] - P.pre[Lp + i]);
        const double Pe = (double)(P.pre[2 * Lp + j] - P.pre[2 * Lp + i]);
        const double Act = (double)(P.pre[3 * Lp + j] - P.pre[3 * Lp + i]);
        const double state = (c.mud * Pd) + (c.mue * Pe);
        const double A1 = c.rho * Act;
        tg_stage &sg = plan.stage[t];
        sg.island = order[o];
        sg.first_layer = i;
        sg.end_layer = j;
        sg.tp = c.tp;
        sg.dp = c.dp;
        sg.ep = c.ep;
        sg.zero = c.z;
        sg.mb = c.mb;
        sg.depth = d;
        sg.reserved = 0;
        sg.pair_index = best;
        sg.cost = bc;
        sg.mem_bytes = state + (fmin((double)d, c.m_real) * A1);
        if (d > 1) {
            const double E = EoT[(int64_t)o_next * K + o];
            sg.link_out = E == 0.0 ? kInf : ((2.0 * (double)b) * (double)P.outact[j - 1]) / E;
        } else {
            sg.link_out = 0.0;
        }
        i = j;
        o = o_next;
    }
}

hipError_t launch_compose(const DevProblem &P, const int64_t *surv, int64_t n_surv, const double *cost,
                          const uint8_t *dmax, const int32_t *order_dev, void *ws, hipStream_t s,
                          ComposeResult **result_dev) {
    (void)order_dev;
    Ws w = carve(P, n_surv, ws);
    *result_dev = w.res;
    const int64_t G = n_groups(P), nbk = n_buckets(P);
    const int D = levels(P);
    const int64_t rows = (int64_t)P.nb * (P.L + 1) * P.K;
    prep_kernel<<<dim3(1), dim3(256), 0, s>>>(P, w.order, w.pos, w.EoT, w.EiT, w.res);
    fill<int32_t>(w.gcnt, G, 0, s);
    fill<int32_t>(w.bcnt, nbk + 1, 0, s);
    fill<double>(w.Pst, P.nb, kInf, s);
    fill<double>(w.rootF, P.nb, kInf, s);
    fill<int32_t>(w.root_o, P.nb, -1, s);
    fill<int32_t>(w.root_d, P.nb, -1, s);
    if (n_surv > 0) {
        int64_t blocks = (n_surv + 255) / 256;
        if (blocks > 65536) blocks = 65536;
        gather_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, surv, n_surv, cost, dmax, w.pos, w.rec_g,
                                                                    w.rec_c, w.rec_d, w.gcnt, w.res);
        scan_i32(w.gcnt, G, w.tmp, s);
        scatter_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(surv, n_surv, w.rec_g, w.rec_c, w.rec_d,
                                                                     w.gcnt, w.ent_c, w.ent_d, w.ent_i);
        const dim3 egrid((unsigned)P.L, (unsigned)P.nb);
        group_events<false><<<egrid, dim3(256), 0, s>>>(P, w.gcnt, w.ent_c, w.ent_d, w.ent_i, w.bcnt, w.ev_cell,
                                                       w.ev_val);
        scan_i32(w.bcnt, nbk + 1, w.tmp, s);
        group_events<true><<<egrid, dim3(256), 0, s>>>(P, w.gcnt, w.ent_c, w.ent_d, w.ent_i, w.bcnt, w.ev_cell,
                                                      w.ev_val);
    } else {
        scan_i32(w.gcnt, G, w.tmp, s);  // all zeros: offsets stay zero
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int threads = kSplit * (P.K <= 64 ? 64 : (P.K <= 128 ? 128 : (P.K <= 192 ? 192 : 256)));
    const size_t tri_lds = P.n_ev ? (size_t)(P.K * (P.K - 1) / 2 + 4) : 0;
    const dim3 tgrid((unsigned)((P.NS + kTileS - 1) / kTileS), (unsigned)((P.K + kTileO - 1) / kTileO),
                     (unsigned)P.nb);
    // phase 1: least bottleneck per b
    table_init<<<tgrid, dim3(256), 0, s>>>(P, w.gcnt, w.ent_c, w.T);
    fill<double>(w.Wb[0], rows, kInf, s);
    fill<double>(w.Wb[1], rows, kInf, s);
    for (int d = 1; d <= D; ++d)
        level_bottleneck<<<dim3((unsigned)(P.L - d + 1), (unsigned)P.nb), dim3(threads), tri_lds, s>>>(
            P, d, w.bcnt, w.ev_cell, w.ev_val, w.T, w.Wb[(d - 1) & 1], w.Wb[d & 1], w.EoT, w.EiT, w.Pst);
    // phase 2: least fill at that bottleneck
    table_init<<<tgrid, dim3(256), 0, s>>>(P, w.gcnt, w.ent_c, w.T);
    fill<double>(w.Wb[0], rows, kInf, s);
    fill<double>(w.Wb[1], rows, kInf, s);
    for (int d = 1; d <= D; ++d)
        level_fill<<<dim3((unsigned)(P.L - d + 1), (unsigned)P.nb), dim3(threads), tri_lds, s>>>(
            P, d, w.bcnt, w.ev_cell, w.ev_val, w.T, w.Wb[(d - 1) & 1], w.Wb[d & 1], w.EoT, w.EiT, w.Pst, w.argF,
            w.argG, w.rootF, w.root_o, w.root_d);
    finish_kernel<<<dim3(1), dim3(64), 0, s>>>(P, w.gcnt, w.ent_c, w.ent_d, w.ent_i, w.order, w.EoT, w.Pst, w.rootF,
                                                w.root_o, w.root_d, w.argF, w.argG, w.res);
    return hipGetLastError();
}

}  // namespace tg
