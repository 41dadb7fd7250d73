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

__global__ __launch_bounds__(1024) void scan_tiles_i64(int64_t *a, int64_t n, int64_t *total) {
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
    if (threadIdx.x == 0 && total) *total = carry;
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

// In-place exclusive scan of an int32 array; tmp holds >= tiles + 1 int64.
static void scan_i32(int32_t *a, int64_t n, int64_t *tmp, hipStream_t s) {
    if (n <= 0) return;
    const int64_t tiles = (n + kScanTile - 1) / kScanTile;
    scan_reduce_i32<<<dim3((unsigned)tiles), dim3(kScanThreads), 0, s>>>(a, n, tmp);
    scan_tiles_i64<<<dim3(1), dim3(1024), 0, s>>>(tmp, tiles, nullptr);
    scan_apply_i32<<<dim3((unsigned)tiles), dim3(kScanThreads), 0, s>>>(a, n, tmp);
}

// ---------------------------------------------------------------------------
// grouping: candidate list -> per-group entry lists -> per-level events
// ---------------------------------------------------------------------------
struct Ws {
    int32_t *pos;     // [K] island -> position
    double *EoT;      // [K*K] EoT[o2*K + o] = E[order[o]][order[o2]]
    int32_t *gcnt;    // [n_groups] counts -> offsets -> ends
    int32_t *entries; // [n_surv] survivor positions grouped
    int32_t *bcnt;    // [n_buckets] event counts -> offsets -> ends
    int32_t *ev_cell; // [2 n_surv]
    double *ev_val;   // [2 n_surv]
    double *T;        // [n_groups] current stage table, layout [b][s][o]
    double *Wb[2];    // [nb][L+1][K] continuation rows, double-buffered by level
    uint16_t *argF;   // [D][nb][L][K]
    uint8_t *argG;    // [D][nb][L+1][K]
    double *Pst;      // [nb]
    double *rootF;    // [nb]
    int32_t *root_o;  // [nb]
    int32_t *root_d;  // [nb]
    int64_t *tmp;     // scan tiles
    ComposeResult *res;
    int32_t *order;   // [K] copy of the caller's order
    size_t bytes;
};

static int64_t n_groups(const DevProblem &P) { return (int64_t)P.nb * P.NS * P.K; }
static int levels(const DevProblem &P) { return P.K < P.L ? P.K : P.L; }
static int64_t n_buckets(const DevProblem &P) { return (int64_t)levels(P) * P.nb * P.L; }

static Ws carve(const DevProblem &P, int64_t n_surv, void *base) {
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
    w.res = (ComposeResult *)take(sizeof(ComposeResult));
    w.order = (int32_t *)take(sizeof(int32_t) * P.K);
    w.pos = (int32_t *)take(sizeof(int32_t) * P.K);
    w.EoT = (double *)take(sizeof(double) * P.K * P.K);
    w.gcnt = (int32_t *)take(sizeof(int32_t) * G);
    w.entries = (int32_t *)take(sizeof(int32_t) * n_surv);
    w.bcnt = (int32_t *)take(sizeof(int32_t) * nbk);
    w.ev_cell = (int32_t *)take(sizeof(int32_t) * 2 * n_surv);
    w.ev_val = (double *)take(sizeof(double) * 2 * n_surv);
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
    (void)n_surv;
    return align256(sizeof(ComposeResult));
}

__global__ void prep_kernel(DevProblem P, const int32_t *order, int32_t *pos, double *EoT, ComposeResult *res) {
    const int K = P.K;
    for (int t = threadIdx.x; t < K; t += blockDim.x) pos[order[t]] = t;
    for (int t = threadIdx.x; t < K * K; t += blockDim.x) {
        const int o2 = t / K, o = t - o2 * K;
        EoT[t] = P.E[(int64_t)order[o] * K + order[o2]];
    }
    if (threadIdx.x == 0) {
        res->err = 0;
        res->status = TG_ENOPLAN;
    }
}

// Validates entry r and returns its group (or -1 when it has d_max 0).
__device__ inline int64_t group_of(const DevProblem &P, const int64_t *surv, int64_t r, const uint8_t *dmax,
                                   const int32_t *pos, ComposeResult *res) {
    const int64_t idx = surv[r];
    if (idx < 0 || idx >= P.N || (r > 0 && surv[r - 1] >= idx)) {
        atomicOr(&res->err, 1);
        return -1;
    }
    const int64_t g = idx / P.NS, s = idx - g * P.NS;
    const Coef &c = P.coef[g];
    if (c.b_idx < 0) {
        atomicOr(&res->err, 2);
        return -1;
    }
    if (dmax[idx] == 0) return -1;
    return ((int64_t)c.b_idx * P.NS + s) * P.K + pos[c.k];
}

__global__ __launch_bounds__(256) void count_groups(DevProblem P, const int64_t *surv, int64_t n, const uint8_t *dmax,
                                                    const int32_t *pos, int32_t *gcnt, ComposeResult *res) {
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x) {
        const int64_t G = group_of(P, surv, r, dmax, pos, res);
        if (G >= 0) atomicAdd(&gcnt[G], 1);
    }
}

__global__ __launch_bounds__(256) void scatter_groups(DevProblem P, const int64_t *surv, int64_t n,
                                                      const uint8_t *dmax, const int32_t *pos, int32_t *gcnt,
                                                      int32_t *entries, ComposeResult *res) {
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x) {
        const int64_t G = group_of(P, surv, r, dmax, pos, res);
        if (G >= 0) entries[atomicAdd(&gcnt[G], 1)] = (int32_t)r;
    }
}

// Per group: entry e is the least fitting candidate at depths (D_e, d_e],
// D_e = the largest d_max among entries with a smaller key; it sets T at
// level D_e + 1.  After the group's largest d_max M nothing fits: T = +inf
// from level M + 1.  At most one event per (group, level).
template <bool kEmit>
__global__ __launch_bounds__(256) void group_events(DevProblem P, const int64_t *surv, const double *cost,
                                                    const uint8_t *dmax, const int32_t *gcnt,
                                                    const int32_t *entries, int32_t *bcnt, int32_t *ev_cell,
                                                    double *ev_val) {
    const int64_t NG = (int64_t)P.nb * P.NS * P.K;
    const int D = P.K < P.L ? P.K : P.L;
    for (int64_t G = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; G < NG; G += (int64_t)gridDim.x * blockDim.x) {
        const int32_t st = G ? gcnt[G - 1] : 0, en = gcnt[G];
        if (st == en) continue;
        const int64_t bs = G / P.K;
        const int64_t bi = bs / P.NS, s = bs - bi * P.NS;
        const int i = (int)(P.sij[s] & 0xFFFFu);
        auto emit = [&](int level, double v) {
            const int64_t bucket = ((int64_t)(level - 1) * P.nb + bi) * P.L + i;
            if (kEmit) {
                const int32_t slot = atomicAdd(&bcnt[bucket], 1);
                ev_cell[slot] = (int32_t)G;
                ev_val[slot] = v;
            } else {
                atomicAdd(&bcnt[bucket], 1);
            }
        };
        int M = 0;
        for (int32_t e = st; e < en; ++e) {
            const int64_t ie = surv[entries[e]];
            const double ce = cost[ie];
            const int de = dmax[ie];
            M = max(M, de);
            int De = 0;
            for (int32_t q = st; q < en; ++q) {
                const int64_t iq = surv[entries[q]];
                const double cq = cost[iq];
                const int dq = dmax[iq];
                const bool less = cq < ce || (cq == ce && (dq > de || (dq == de && iq < ie)));
                if (less) De = max(De, dq);
            }
            if (De < de && De + 1 <= D) emit(De + 1, ce);
        }
        if (M + 1 <= D) emit(M + 1, kInf);
    }
}

// ---------------------------------------------------------------------------
// dynamic program, one launch per level
// ---------------------------------------------------------------------------
__device__ inline void apply_events(const int32_t *bcnt, const int32_t *ev_cell, const double *ev_val, double *T,
                                    int64_t bucket) {
    const int32_t st = bucket ? bcnt[bucket - 1] : 0, en = bcnt[bucket];
    for (int32_t e = st + threadIdx.x; e < en; e += blockDim.x) T[ev_cell[e]] = ev_val[e];
}

// Phase 1: bottleneck values.
__global__ __launch_bounds__(256) void level_bottleneck(DevProblem P, int d, const int32_t *bcnt,
                                                        const int32_t *ev_cell, const double *ev_val, double *T,
                                                        const double *Wprev, double *Wnext, const double *EoT,
                                                        double *Pst) {
    __shared__ double Vs[256];
    const int i = blockIdx.x, bi = blockIdx.y, o = threadIdx.x;
    const int L = P.L, K = P.K;
    if (i > L - d) return;
    apply_events(bcnt, ev_cell, ev_val, T, ((int64_t)(d - 1) * P.nb + bi) * L + i);
    __syncthreads();
    const int64_t srow = (int64_t)bi * P.NS + slice_of(L, i, i + 1);  // slice (i, i+1); (i, j) is + j-i-1
    double v = kInf;
    if (o < K && o <= K - d) {
        if (d == 1) {
            v = T[(srow + (L - i - 1)) * K + o];
        } else {
            const double *Wp = Wprev + (int64_t)bi * (L + 1) * K + o;
            for (int j = i + 1; j <= L - d + 1; ++j) {
                const double t = T[(srow + (j - i - 1)) * K + o];
                const double w = Wp[(int64_t)j * K];
                v = fmin(v, fmax(t, w));
            }
        }
    }
    Vs[o] = v;
    __syncthreads();
    if (i == 0) {
        if (o == 0) {
            double m = kInf;
            for (int t = 0; t < K; ++t) m = fmin(m, Vs[t]);
            Pst[bi] = fmin(Pst[bi], m);
        }
        return;
    }
    if (o < K) {
        double w = kInf;
        const double num = (2.0 * (double)P.bvals[bi]) * (double)P.outact[i - 1];
        for (int o2 = o + 1; o2 <= K - d; ++o2) {
            const double E = EoT[(int64_t)o2 * K + o];
            const double x = E == 0.0 ? kInf : num / E;
            w = fmin(w, fmax(x, Vs[o2]));
        }
        Wnext[((int64_t)bi * (L + 1) + i) * K + o] = w;
    }
}

// Phase 2: fill values and argmins at the bottleneck P*.
__global__ __launch_bounds__(256) void level_fill(DevProblem P, int d, const int32_t *bcnt, const int32_t *ev_cell,
                                                  const double *ev_val, double *T, const double *Gprev,
                                                  double *Gnext, const double *EoT, const double *Pst,
                                                  uint16_t *argF, uint8_t *argG, double *rootF, int32_t *root_o,
                                                  int32_t *root_d) {
    __shared__ double Fs[256];
    const int i = blockIdx.x, bi = blockIdx.y, o = threadIdx.x;
    const int L = P.L, K = P.K;
    const double Ps = Pst[bi];
    if (!(Ps < kInf) || i > L - d) return;
    apply_events(bcnt, ev_cell, ev_val, T, ((int64_t)(d - 1) * P.nb + bi) * L + i);
    __syncthreads();
    const int64_t srow = (int64_t)bi * P.NS + slice_of(L, i, i + 1);
    double v = kInf;
    int arg = 0xFFFF;
    if (o < K && o <= K - d) {
        if (d == 1) {
            const double t = T[(srow + (L - i - 1)) * K + o];
            if (t <= Ps) {
                v = t;
                arg = L;
            }
        } else {
            const double *Gp = Gprev + (int64_t)bi * (L + 1) * K + o;
            for (int j = i + 1; j <= L - d + 1; ++j) {
                const double t = T[(srow + (j - i - 1)) * K + o];
                if (!(t <= Ps)) continue;
                const double c = t + Gp[(int64_t)j * K];
                if (c < v) {
                    v = c;
                    arg = j;
                }
            }
        }
    }
    if (o < K) argF[(((int64_t)(d - 1) * P.nb + bi) * L + i) * K + o] = (uint16_t)arg;
    Fs[o] = v;
    __syncthreads();
    if (i == 0) {
        if (o == 0) {
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
    if (o < K) {
        double w = kInf;
        int a = 0xFF;
        const double num = (2.0 * (double)P.bvals[bi]) * (double)P.outact[i - 1];
        for (int o2 = o + 1; o2 <= K - d; ++o2) {
            const double E = EoT[(int64_t)o2 * K + o];
            const double x = E == 0.0 ? kInf : num / E;
            if (!(x <= Ps)) continue;
            const double c = x + Fs[o2];
            if (c < w) {
                w = c;
                a = o2;
            }
        }
        Gnext[((int64_t)bi * (L + 1) + i) * K + o] = w;
        argG[(((int64_t)(d - 1) * P.nb + bi) * (L + 1) + i) * K + o] = (uint8_t)a;
    }
}

// ---------------------------------------------------------------------------
// choose b, walk the argmins, resolve each stage's candidate
// ---------------------------------------------------------------------------
__global__ void finish_kernel(DevProblem P, const int64_t *surv, const double *cost, const uint8_t *dmax,
                              const int32_t *gcnt, const int32_t *entries, const int32_t *order,
                              const double *EoT, const double *Pst, const double *rootF, const int32_t *root_o,
                              const int32_t *root_d, const uint16_t *argF, const uint8_t *argG,
                              ComposeResult *res) {
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
        const int64_t G = ((int64_t)bb * P.NS + s) * K + o;
        const int32_t st = G ? gcnt[G - 1] : 0, en = gcnt[G];
        int64_t best = -1;
        double bc = kInf;
        int bd = 0;
        for (int32_t e = st; e < en; ++e) {
            const int64_t ie = surv[entries[e]];
            const double c = cost[ie];
            const int dd = dmax[ie];
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
    Ws w = carve(P, n_surv, ws);
    *result_dev = w.res;
    const int64_t G = n_groups(P), nbk = n_buckets(P);
    const int D = levels(P);
    const int64_t rows = (int64_t)P.nb * (P.L + 1) * P.K;
    (void)order_dev;
    prep_kernel<<<dim3(1), dim3(256), 0, s>>>(P, w.order, w.pos, w.EoT, w.res);
    fill<int32_t>(w.gcnt, G, 0, s);
    fill<int32_t>(w.bcnt, nbk, 0, s);
    fill<double>(w.Pst, P.nb, kInf, s);
    fill<double>(w.rootF, P.nb, kInf, s);
    fill<int32_t>(w.root_o, P.nb, -1, s);
    fill<int32_t>(w.root_d, P.nb, -1, s);
    fill<double>(w.Wb[0], rows, kInf, s);
    fill<double>(w.Wb[1], rows, kInf, s);
    if (n_surv > 0) {
        int64_t blocks = (n_surv + 255) / 256;
        if (blocks > 65536) blocks = 65536;
        count_groups<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, surv, n_surv, dmax, w.pos, w.gcnt, w.res);
        scan_i32(w.gcnt, G, w.tmp, s);
        scatter_groups<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, surv, n_surv, dmax, w.pos, w.gcnt,
                                                                     w.entries, w.res);
        int64_t gblocks = (G + 255) / 256;
        if (gblocks > 65536) gblocks = 65536;
        group_events<false><<<dim3((unsigned)gblocks), dim3(256), 0, s>>>(P, surv, cost, dmax, w.gcnt, w.entries,
                                                                          w.bcnt, w.ev_cell, w.ev_val);
        scan_i32(w.bcnt, nbk, w.tmp, s);
        group_events<true><<<dim3((unsigned)gblocks), dim3(256), 0, s>>>(P, surv, cost, dmax, w.gcnt, w.entries,
                                                                         w.bcnt, w.ev_cell, w.ev_val);
    } else {
        scan_i32(w.gcnt, G, w.tmp, s);  // all zeros: offsets stay zero
        scan_i32(w.bcnt, nbk, w.tmp, s);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int threads = P.K <= 64 ? 64 : (P.K <= 128 ? 128 : (P.K <= 192 ? 192 : 256));
    const dim3 grid((unsigned)P.L, (unsigned)P.nb);
    // phase 1: least bottleneck per b
    fill<double>(w.T, G, kInf, s);
    for (int d = 1; d <= D; ++d)
        level_bottleneck<<<grid, dim3(threads), 0, s>>>(P, d, w.bcnt, w.ev_cell, w.ev_val, w.T, w.Wb[(d - 1) & 1],
                                                        w.Wb[d & 1], w.EoT, w.Pst);
    // phase 2: least fill at that bottleneck
    fill<double>(w.T, G, kInf, s);
    fill<double>(w.Wb[0], rows, kInf, s);
    fill<double>(w.Wb[1], rows, kInf, s);
    for (int d = 1; d <= D; ++d)
        level_fill<<<grid, dim3(threads), 0, s>>>(P, d, w.bcnt, w.ev_cell, w.ev_val, w.T, w.Wb[(d - 1) & 1],
                                                  w.Wb[d & 1], w.EoT, w.Pst, w.argF, w.argG, w.rootF, w.root_o,
                                                  w.root_d);
    finish_kernel<<<dim3(1), dim3(64), 0, s>>>(P, surv, cost, dmax, w.gcnt, w.entries, w.order, w.EoT, w.Pst,
                                                w.rootF, w.root_o, w.root_d, w.argF, w.argG, w.res);
    return hipGetLastError();
}

}  // namespace tg
