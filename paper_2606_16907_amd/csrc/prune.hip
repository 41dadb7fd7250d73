// prune.hip -- the surviving set: incompatibility, infeasibility and
// dominance pruning (Sec. 5.1), as a frontier pass plus a stream compaction.
//
// Group G = (slice s, island k, micro-batch b).  A member p survives iff b
// divides the global batch, (s, k) passes imbalance pruning when it is on,
// d_max_p >= 1 and p has the least key
// (cost, -d_max, idx) among members whose d_max reaches d_max_p.  Equivalently
// the survivors are rep(G, d) for d = 1..K, the least-key member fitting at
// depth d.  The frontier pass finds those reps depth band by depth band: pass t
// takes the least-key member whose d_max exceeds the previous rep's d_max.
//
// Frontier: a wave owns 64 consecutive slices of one (island, b) group list;
// every lane walks the same members (a scalar loop), reading one coalesced
// 512-byte row of costs and 64 bytes of depths per member, eight members in
// flight.  The first pass also finds the group's largest d_max, so a lane
// stops as soon as its rep reaches it instead of spending a pass to find
// nothing deeper.  Survivors are
// recorded in an LDS bit mask per member (lane bit = slice) and written as
// whole 64-bit words of a bitmap with one row per compatible config.
// Compaction: popcount per tile, scan of tile counts, then each thread writes
// the candidate indices of its words' set bits in ascending order.
#include <algorithm>

#include "tg_device.h"

namespace tg {

constexpr int kFrontWaves = 4;
constexpr int kCountThreads = 256;
constexpr int kWordsPerThread = 4;
constexpr int kTileWords = kCountThreads * kWordsPerThread;

__global__ __launch_bounds__(256) void frontier_kernel(DevProblem P, const double *__restrict__ cost,
                                                       const uint8_t *__restrict__ dmax, uint64_t *bitmap,
                                                       int64_t n_tiles) {
    extern __shared__ uint64_t smask[];
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t tile = (int64_t)blockIdx.x * kFrontWaves + wv;
    uint64_t *mask = smask + (int64_t)wv * P.max_members;
    const bool tv = tile < n_tiles;
    int q = 0, m0 = 0, nm = 0;
    int64_t sc = 0;
    if (tv) {
        q = (int)(tile / P.words);
        sc = tile - (int64_t)q * P.words;
        m0 = P.kb_off[q];
        nm = P.kb_off[q + 1] - m0;
    }
    for (int m = lane; m < nm; m += kWave) mask[m] = 0;
    __syncthreads();
    if (tv) {
        const int64_t s = sc * kWave + lane;
        const int64_t NS = P.NS;
        const int K = P.K;
        bool live = s < NS;
        if (live && P.imb) {  // an unbalanced (slice, island) group has no survivors
            const uint32_t ij = P.sij[s];
            live = slice_balanced(P, P.pre, (int)(ij & 0xFFFFu), (int)(ij >> 16), P.kb_island[q]);
        }
        int prev = 0;   // d_max of the previous rep of this lane's group
        int top = -1;   // the group's largest d_max, known after the first pass
        while (__ballot(live) != 0) {
            double bc = kInf;
            int bd = 0, bm = -1, mx = 0;
            // members in batches of eight loads in flight; they come in ascending
            // idx, so equal (cost, d_max) keeps the earlier one.  Depths are
            // read first and a cost only where the member reaches past the
            // previous rep: after the first pass most members do not, so the
            // later passes move about one byte per member instead of nine.
            for (int mb = 0; mb < nm; mb += 8) {
                double c[8];
                int d[8];
                int64_t idx[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    d[u] = 0;
                    idx[u] = (int64_t)P.kb_members[m0 + min(mb + u, nm - 1)] * NS + s;
                    if (mb + u < nm && live) d[u] = dmax[idx[u]];
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    c[u] = kInf;
                    if (d[u] > prev) c[u] = cost[idx[u]];
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    mx = max(mx, d[u]);
                    if (d[u] > prev && (c[u] < bc || (c[u] == bc && d[u] > bd))) {
                        bc = c[u];
                        bd = d[u];
                        bm = mb + u;
                    }
                }
            }
            if (top < 0) top = mx;
            if (live) {
                if (bm >= 0) {
                    atomicOr((unsigned long long *)&mask[bm], 1ull << lane);
                    prev = bd;
                    // nothing reaches deeper than the group's largest d_max
                    if (prev >= K || prev >= top) live = false;
                } else {
                    live = false;
                }
            }
        }
    }
    __syncthreads();
    if (tv)
        for (int m = lane; m < nm; m += kWave) {
            const int32_t row = P.coef[P.kb_members[m0 + m]].row;
            bitmap[(int64_t)row * P.words + sc] = mask[m];
        }
}

__global__ __launch_bounds__(kCountThreads) void count_kernel(const uint64_t *__restrict__ bitmap, int64_t n_words,
                                                              int64_t *tile_cnt) {
    __shared__ int64_t lds[kCountThreads / kWave + 1];
    const int64_t base = (int64_t)blockIdx.x * kTileWords + (int64_t)threadIdx.x * kWordsPerThread;
    int64_t c = 0;
#pragma unroll
    for (int w = 0; w < kWordsPerThread; ++w)
        if (base + w < n_words) c += __popcll(bitmap[base + w]);
    int64_t total;
    block_excl_scan<int64_t>(c, lds, &total);
    if (threadIdx.x == 0) tile_cnt[blockIdx.x] = total;
}

// Exclusive scan of n int64 values in place by one block; writes the sum to *total.
__global__ __launch_bounds__(1024) void scan_small_i64(int64_t *a, int64_t n, int64_t *total) {
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
    if (threadIdx.x == 0) *total = carry;
}

__global__ __launch_bounds__(kCountThreads) void emit_kernel(DevProblem P, const uint64_t *__restrict__ bitmap,
                                                             int64_t n_words, const int64_t *tile_off,
                                                             int64_t *out, int64_t capacity) {
    __shared__ int64_t lds[kCountThreads / kWave + 1];
    const int64_t base = (int64_t)blockIdx.x * kTileWords + (int64_t)threadIdx.x * kWordsPerThread;
    uint64_t w[kWordsPerThread];
    int64_t c = 0;
#pragma unroll
    for (int t = 0; t < kWordsPerThread; ++t) {
        w[t] = (base + t < n_words) ? bitmap[base + t] : 0ull;
        c += __popcll(w[t]);
    }
    int64_t total;
    int64_t pos = tile_off[blockIdx.x] + block_excl_scan<int64_t>(c, lds, &total);
#pragma unroll
    for (int t = 0; t < kWordsPerThread; ++t) {
        uint64_t bits = w[t];
        if (!bits) continue;
        const int64_t wi = base + t;
        const int64_t row = wi / P.words;
        const int64_t s0 = (wi - row * P.words) * kWave;
        const int64_t g = P.row_cfg[row];
        while (bits) {
            const int bit = __ffsll((unsigned long long)bits) - 1;
            bits &= bits - 1;
            if (pos < capacity) out[pos] = g * P.NS + s0 + bit;
            ++pos;
        }
    }
}

// Redundancy pruning: bit s of a row of the slice bitmap is bit cls[s] of
// the same row of the class bitmap (a class's staircase holds on every slice
// of the class).  A wave builds kExpandWords consecutive 64-bit words, lane b
// testing slice 64 w + b of each, the loads of all its words in flight.
constexpr int kExpandWords = 8;

__global__ __launch_bounds__(256) void expand_kernel(DevProblem P, const uint64_t *__restrict__ cbits,
                                                     int32_t cwords, uint64_t *bits, int64_t n_words) {
    const int64_t w0 = ((int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave) * kExpandWords;
    if (w0 >= n_words) return;  // whole waves leave together
    const int lane = threadIdx.x & (kWave - 1);
    uint32_t c[kExpandWords];
    int64_t row[kExpandWords];
#pragma unroll
    for (int t = 0; t < kExpandWords; ++t) {
        const int64_t w = min(w0 + t, n_words - 1);
        row[t] = w / P.words;
        const int64_t s = (w - row[t] * P.words) * kWave + lane;
        c[t] = s < P.NS ? P.cls[s] : 0xFFFFFFFFu;
    }
    uint64_t x[kExpandWords];
#pragma unroll
    for (int t = 0; t < kExpandWords; ++t)
        x[t] = c[t] != 0xFFFFFFFFu ? cbits[row[t] * cwords + (c[t] >> 6)] : 0ull;
#pragma unroll
    for (int t = 0; t < kExpandWords; ++t) {
        const uint64_t word = __ballot(c[t] != 0xFFFFFFFFu && ((x[t] >> (c[t] & 63)) & 1ull));
        if (lane == 0 && w0 + t < n_words) bits[w0 + t] = word;
    }
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static int64_t bitmap_words(const DevProblem &P) { return (int64_t)P.n_rows * P.words; }

size_t prune_ws_bytes(const DevProblem &P) {
    const int64_t nw = bitmap_words(P);
    const int64_t nt = (nw + kTileWords - 1) / kTileWords;
    return align256(sizeof(uint64_t) * (size_t)(nw > 0 ? nw : 1)) + align256(sizeof(int64_t) * (size_t)(nt + 1)) +
           align256(sizeof(int64_t));
}

static hipError_t launch_frontier(const DevProblem &P, const double *cost, const uint8_t *dmax, uint64_t *bitmap,
                                  hipStream_t s) {
    const int64_t n_front = (int64_t)P.n_kb * P.words;
    if (n_front > 0) {
        const int64_t blocks = (n_front + kFrontWaves - 1) / kFrontWaves;
        const size_t lds = sizeof(uint64_t) * (size_t)kFrontWaves * (size_t)P.max_members;
        frontier_kernel<<<dim3((unsigned)blocks), dim3(kFrontWaves * kWave), lds, s>>>(P, cost, dmax, bitmap,
                                                                                       n_front);
    }
    return hipGetLastError();
}

// Survivor bitmap (at the start of ws) -> ascending candidate indices.
static hipError_t launch_compact(const DevProblem &P, int64_t *surv, int64_t capacity, void *ws, hipStream_t s,
                                 int64_t **d_total_out) {
    const int64_t nw = bitmap_words(P);
    const int64_t nt = (nw + kTileWords - 1) / kTileWords;
    char *p = (char *)ws;
    uint64_t *bitmap = (uint64_t *)p;
    p += align256(sizeof(uint64_t) * (size_t)(nw > 0 ? nw : 1));
    int64_t *tiles = (int64_t *)p;
    p += align256(sizeof(int64_t) * (size_t)(nt + 1));
    int64_t *total = (int64_t *)p;
    *d_total_out = total;
    if (nt > 0) count_kernel<<<dim3((unsigned)nt), dim3(kCountThreads), 0, s>>>(bitmap, nw, tiles);
    scan_small_i64<<<dim3(1), dim3(1024), 0, s>>>(tiles, nt, total);
    if (nt > 0)
        emit_kernel<<<dim3((unsigned)nt), dim3(kCountThreads), 0, s>>>(P, bitmap, nw, tiles, surv, capacity);
    return hipGetLastError();
}

hipError_t launch_prune(const DevProblem &P, const double *cost, const uint8_t *dmax, int64_t *surv,
                        int64_t capacity, void *ws, hipStream_t s, int64_t **d_total_out) {
    hipError_t e = launch_frontier(P, cost, dmax, (uint64_t *)ws, s);
    if (e != hipSuccess) return e;
    return launch_compact(P, surv, capacity, ws, s, d_total_out);
}

// Class bitmap after the slice-level workspace of launch_prune.
size_t prune_classes_ws_bytes(const DevProblem &P) {
    const DevProblem C = class_view(P);
    return prune_ws_bytes(P) + align256(sizeof(uint64_t) * (size_t)std::max<int64_t>(1, bitmap_words(C)));
}

hipError_t launch_prune_classes(const DevProblem &P, const double *cost, const uint8_t *dmax, int64_t *surv,
                                int64_t capacity, void *ws, hipStream_t s, int64_t **d_total_out) {
    const DevProblem C = class_view(P);
    uint64_t *cbits = (uint64_t *)((char *)ws + prune_ws_bytes(P));
    hipError_t e = launch_frontier(C, cost, dmax, cbits, s);
    if (e != hipSuccess) return e;
    const int64_t nw = bitmap_words(P);
    if (nw > 0)
        expand_kernel<<<dim3((unsigned)((nw + 4 * kExpandWords - 1) / (4 * kExpandWords))), dim3(256), 0, s>>>(
            P, cbits, C.words, (uint64_t *)ws, nw);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_compact(P, surv, capacity, ws, s, d_total_out);
}

}  // namespace tg
