// islands.hip -- GPU island construction from nodes (Sec. 4.1).
//
// An island holds nodes with the same GPU count whose compute, memory
// (Eq. 1) and intra-node bandwidth (Eq. 2) differ by at most a factor 1 + eps
// pairwise, and every member's links inside the island are at least as fast
// as its links leaving it (Eq. 3).  Steps (1)-(2): one block splits the nodes
// by GPU count, compute, memory and intra-node bandwidth, each split a block
// bitonic sort by (group, value, node) followed by a sweep that opens a new
// group at the first value above the group's smallest times (1 + eps).  Step
// (3): one block per group runs agglomerative clustering: the pair of
// clusters with the highest complete linkage (the least bandwidth between
// their nodes, a node pair counted by its slower direction; ties to the
// least node ids) is merged if the union satisfies Eq. 3 against every node
// outside it, else marked; the group is done when every pair of its clusters
// is marked.  Each row keeps its best partner so a step scans rows, not
// pairs, a wave per row that must be scanned again.  The Eq. 3 test gives
// one wave to each member of the union: its slowest link inside from the
// member list, its fastest link leaving from its bandwidth row sorted once
// per cluster (the first entry outside the union).  A finish pass numbers islands by their
// smallest node and reduces the island attributes and island-to-island
// bandwidths (least over node pairs).
#include <stdint.h>

#include <vector>

#include "tg_device.h"

#pragma clang fp contract(off)

namespace tg {

constexpr int kMaxNodes = 4096;
constexpr int kGroupThreads = 1024;
constexpr int kMergeThreads = 256;
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
    double *link;       // [n][n] complete linkage between cluster representatives (-inf: no pair)
    uint8_t *marked;    // [n][n] pairs whose union breaks Eq. 3
    int32_t *cl;        // [n] cluster (its smallest node) of each node
    double *rbest;      // [n] best linkage of each representative's row
    int32_t *rarg;      // [n] its partner
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
    w.link = (double *)take(8 * n * n);
    w.marked = (uint8_t *)take(n * n);
    w.cl = (int32_t *)take(4 * n);
    w.rbest = (double *)take(8 * n);
    w.rarg = (int32_t *)take(4 * n);
    w.island_of = (int32_t *)take(4 * n);
    w.out_k = (int32_t *)take(4);
    w.isl_gpus = (int32_t *)take(4 * n);
    w.isl_val = (double *)take(8 * 4 * n);
    w.isl_e = (double *)take(8 * n * n);
    w.bytes = off;
    return w;
}

size_t islands_ws_bytes(int n) { return carve_islands(n, nullptr).bytes; }

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
                                                                int32_t *gstart, int32_t *gnodes, int32_t *ngroups) {
    __shared__ int32_t ord[kMaxNodes];
    __shared__ int32_t g[kMaxNodes];
    __shared__ double x[kMaxNodes];
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
        if (threadIdx.x == 0) {  // the sweep: dense new groups in sorted order
            int cur = -1, prev = -1;
            double v0 = 0.0;
            for (int t = 0; t < n; ++t) {
                const int u = ord[t];
                if (t == 0 || g[u] != prev || !(x[u] <= v0 * (1.0 + eps))) {
                    ++cur;
                    v0 = x[u];
                }
                prev = g[u];
                gnodes[t] = cur;  // new group of the t-th node, kept until all are read
            }
            for (int t = 0; t < n; ++t) g[ord[t]] = gnodes[t];
            // after the last split: group starts and member lists in sorted order
            if (f == 3) {
                for (int t = 0; t < n; ++t) {
                    const int gg = g[ord[t]];
                    if (t == 0 || gg != g[ord[t - 1]]) gstart[gg] = t;
                }
                gstart[cur + 1] = n;
                *ngroups = cur + 1;
            }
        }
        __syncthreads();
    }
    for (int t = threadIdx.x; t < n; t += blockDim.x) {
        gnodes[t] = ord[t];
        grp[ord[t]] = g[ord[t]];
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

// Linkage of node pairs in one group (the slower direction), everything else
// no pair; every node its own cluster.
__global__ __launch_bounds__(256) void islands_link_init(int n, const double *__restrict__ e,
                                                         const int32_t *__restrict__ grp, double *link,
                                                         uint8_t *marked, int32_t *cl) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n * n) return;
    const int u = (int)(t / n), v = (int)(t - (int64_t)u * n);
    double l = kNoPair;
    if (u != v && grp[u] == grp[v]) {
        const double a = e[t], b = e[(int64_t)v * n + u];
        l = a < b ? a : b;
    }
    link[t] = l;
    marked[t] = 0;
    if (v == 0) cl[u] = u;
}

// ---------------------------------------------------------------------------
// step (3): agglomerative clustering, one block per group
// ---------------------------------------------------------------------------
// Best partner of representative u among the group's representatives, by one
// wave: highest linkage of an unmarked pair, ties to the least partner.
__device__ inline void row_best(int u, int n, const int32_t *mem, int nm, const int32_t *cl, const double *link,
                                const uint8_t *marked, double *rbest, int32_t *rarg, int lane) {
    double b = kNoPair;
    int a = -1;
    for (int q = lane; q < nm; q += kWave) {
        const int v = mem[q];
        if (v == u || cl[v] != v || marked[(int64_t)u * n + v]) continue;
        const double l = link[(int64_t)u * n + v];
        if (l == kNoPair) continue;
        if (a < 0 || l > b || (l == b && v < a)) {
            b = l;
            a = v;
        }
    }
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double b2 = __shfl_xor(b, off);
        const int a2 = __shfl_xor(a, off);
        if (a2 >= 0 && (a < 0 || b2 > b || (b2 == b && a2 < a))) {
            b = b2;
            a = a2;
        }
    }
    if (lane == 0) {
        rbest[u] = b;
        rarg[u] = a;
    }
}

// The group members u with keep(u) into out (LDS, in no particular order;
// every use is order-free); the count, the same for every thread.
template <typename Keep>
__device__ inline int collect(const int32_t *mem, int nm, Keep keep, int32_t *out, int32_t *cnt) {
    if (threadIdx.x == 0) *cnt = 0;
    __syncthreads();
    for (int q = threadIdx.x; q < nm; q += blockDim.x) {
        const int u = mem[q];
        if (keep(u)) out[atomicAdd(cnt, 1)] = u;
    }
    __syncthreads();
    const int c = *cnt;
    __syncthreads();  // the counter is free again
    return c;
}

__global__ __launch_bounds__(kMergeThreads) void islands_merge(int n, const double *__restrict__ e,
                                                               const int32_t *__restrict__ srt,
                                                               const int32_t *__restrict__ gstart,
                                                               const int32_t *__restrict__ gnodes,
                                                               const int32_t *__restrict__ ngroups, double *link,
                                                               uint8_t *marked, int32_t *cl, double *rbest,
                                                               int32_t *rarg) {
    __shared__ double sv[kMergeThreads / kWave];
    __shared__ int32_t su[kMergeThreads / kWave];
    __shared__ int32_t s_cnt;
    __shared__ int32_t ulist[kMaxNodes];  // members of the candidate union
    __shared__ int32_t rlist[kMaxNodes];  // rows whose best partner must be found again
    __shared__ int32_t s_a, s_b, s_ok;
    const int g = blockIdx.x;
    if (g >= *ngroups) return;
    const int32_t *mem = gnodes + gstart[g];
    const int nm = gstart[g + 1] - gstart[g];
    if (nm < 2) return;
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave, nw = kMergeThreads / kWave;
    for (int q = wv; q < nm; q += nw) row_best(mem[q], n, mem, nm, cl, link, marked, rbest, rarg, lane);
    __syncthreads();
    // every pass merges two clusters or marks a pair: it ends
    for (;;) {
        // the best pair: highest row best, ties to the least row
        double bv = kNoPair;
        int bu = -1;
        for (int q = threadIdx.x; q < nm; q += blockDim.x) {
            const int u = mem[q];
            if (cl[u] != u || rarg[u] < 0) continue;
            const double r = rbest[u];
            if (bu < 0 || r > bv || (r == bv && u < bu)) {
                bv = r;
                bu = u;
            }
        }
        for (int off = kWave / 2; off > 0; off >>= 1) {
            const double v2 = __shfl_xor(bv, off);
            const int u2 = __shfl_xor(bu, off);
            if (u2 >= 0 && (bu < 0 || v2 > bv || (v2 == bv && u2 < bu))) {
                bv = v2;
                bu = u2;
            }
        }
        if (lane == 0) {
            sv[wv] = bv;
            su[wv] = bu;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            for (int w = 1; w < nw; ++w)
                if (su[w] >= 0 && (bu < 0 || sv[w] > bv || (sv[w] == bv && su[w] < bu))) {
                    bv = sv[w];
                    bu = su[w];
                }
            s_a = bu;
            s_b = bu >= 0 ? rarg[bu] : -1;
            s_ok = 1;
        }
        __syncthreads();
        const int a0 = s_a, b0 = s_b;
        if (a0 < 0) break;  // every pair is marked
        const int a = a0 < b0 ? a0 : b0, b = a0 < b0 ? b0 : a0;
        const int s = collect(mem, nm, [&](int u) { return cl[u] == a || cl[u] == b; }, ulist, &s_cnt);
        // Eq. 3 for the union, one wave per member: its slowest link inside
        // against its fastest link to a node outside (the first entry of its
        // sorted row that is not in the union; none if every node is in it)
        for (int t = wv; t < s; t += nw) {
            const int u = ulist[t];
            const double *row = e + (int64_t)u * n;
            double in = __builtin_huge_val(), out = kNoPair;
            for (int k = lane; k < s; k += kWave) {
                const int v = ulist[k];
                if (v != u && row[v] < in) in = row[v];
            }
            const int32_t *order = srt + (int64_t)u * n;
            for (int base = 0; base < n - 1; base += kWave) {
                const int k = base + lane;
                const int w = k < n - 1 ? order[k] : -1;
                const bool outside = w >= 0 && cl[w] != a && cl[w] != b;
                const uint64_t hit = __ballot(outside);
                if (hit) {
                    const int first = __builtin_ctzll(hit);
                    out = row[__shfl(w, first)];
                    break;
                }
            }
            for (int off = kWave / 2; off > 0; off >>= 1) in = fmin(in, __shfl_xor(in, off));
            if (lane == 0 && !(in >= out)) s_ok = 0;
        }
        __syncthreads();
        if (s_ok) {
            // merge b into a: complete linkage is the lesser of the two rows
            for (int q = threadIdx.x; q < nm; q += blockDim.x) {
                const int v = mem[q];
                if (v == a || v == b) continue;
                const double la = link[(int64_t)a * n + v], lb = link[(int64_t)b * n + v];
                const double l = la < lb ? la : lb;
                link[(int64_t)a * n + v] = l;
                link[(int64_t)v * n + a] = l;
                // pairs with the grown cluster are new pairs
                marked[(int64_t)a * n + v] = 0;
                marked[(int64_t)v * n + a] = 0;
            }
            for (int q = threadIdx.x; q < nm; q += blockDim.x)
                if (cl[mem[q]] == b) cl[mem[q]] = a;
            __syncthreads();
            // rows whose best partner was a or b, and a itself, start over;
            // the others may now prefer the grown cluster
            auto again = [&](int u) { return cl[u] == u && (u == a || rarg[u] == a || rarg[u] == b); };
            const int r = collect(mem, nm, again, rlist, &s_cnt);
            for (int q = threadIdx.x; q < nm; q += blockDim.x) {
                const int u = mem[q];
                if (cl[u] != u || again(u)) continue;
                const double l = link[(int64_t)u * n + a];
                if (l != kNoPair && (l > rbest[u] || (l == rbest[u] && a < rarg[u]))) {
                    rbest[u] = l;
                    rarg[u] = a;
                }
            }
            __syncthreads();  // the test above reads rarg of the listed rows too
            for (int t = wv; t < r; t += nw) row_best(rlist[t], n, mem, nm, cl, link, marked, rbest, rarg, lane);
        } else {
            if (threadIdx.x == 0) {
                marked[(int64_t)a * n + b] = 1;
                marked[(int64_t)b * n + a] = 1;
            }
            __syncthreads();
            if (wv == 0) row_best(a, n, mem, nm, cl, link, marked, rbest, rarg, lane);
            if (wv == 1) row_best(b, n, mem, nm, cl, link, marked, rbest, rarg, lane);
        }
        __syncthreads();
    }
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
    for (int u = threadIdx.x; u < n; u += blockDim.x) island_of[u] = id[cl[u]];
    if (threadIdx.x == 0) {
        *out_k = K;
        // sums and least values in node order (a few thousand nodes)
        for (int u = 0; u < n; ++u) {
            const int k = id[cl[u]];
            isl_gpus[k] += gpus[u];
            for (int f = 0; f < 4; ++f) {
                const double v = val[(int64_t)f * n + u];
                if (v < isl_val[(int64_t)f * n + k]) isl_val[(int64_t)f * n + k] = v;
            }
        }
    }
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
                                tg_island *islands, double *inter_bw, int32_t *n_islands) {
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
    if (e == hipSuccess) e = hipStreamSynchronize(s);  // the host staging arrays go away
    if (e != hipSuccess) return e;
    islands_groups<<<dim3(1), dim3(kGroupThreads), 0, s>>>(n, w.gpus, w.val, eps_c, eps_m, eps_i, w.grp, w.gstart,
                                                           w.gnodes, w.ngroups);
    const int64_t nn = (int64_t)n * n;
    islands_link_init<<<dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, s>>>(n, w.e, w.grp, w.link, w.marked,
                                                                               w.cl);
    islands_sort_rows<<<dim3((unsigned)n), dim3(1024), 0, s>>>(n, w.e, w.srt);
    islands_merge<<<dim3((unsigned)n), dim3(kMergeThreads), 0, s>>>(n, w.e, w.srt, w.gstart, w.gnodes, w.ngroups,
                                                                     w.link, w.marked, w.cl, w.rbest, w.rarg);
    islands_number<<<dim3(1), dim3(1024), 0, s>>>(n, w.cl, w.gpus, w.val, w.island_of, w.out_k, w.isl_gpus,
                                                  w.isl_val);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    int32_t K = 0;
    e = hipMemcpyAsync(&K, w.out_k, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
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
