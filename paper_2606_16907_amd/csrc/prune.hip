// prune.hip -- the surviving set: incompatibility, infeasibility and
// dominance pruning (Sec. 5.1), as a frontier pass plus a stream compaction.
//
// Group G = (slice s, island k, micro-batch b).  A member p survives iff b
// divides the global batch, (s, k) passes imbalance pruning when it is on,
// d_max_p >= 1 and p has the least key
// (cost, -d_max, idx) among members whose d_max reaches d_max_p.  Equivalently
// the survivors are rep(G, d) for d = 1..K, the least-key member fitting at
// depth d: a member survives iff no other member at least as deep has a
// smaller key.
//
// Frontier: a wave owns 64 consecutive slices of one (island, b) group list;
// every lane walks the same members (a scalar loop) in ascending idx, reading
// one coalesced 64-byte row of depths per member and, where the depth can
// still matter, one 512-byte row of costs, eight members in flight.  Each
// lane keeps the staircase of its group in registers (up to kStair entries of
// strictly increasing depth and key): a member is dropped when an entry at
// least as deep costs no more; otherwise it removes the entries it beats and
// takes a slot.  When the slots are full the shallowest of them and the
// newcomer leaves and the pass ignores every member at or above its depth
// from then on: survival of a member depends only on members at least as
// deep, so the entries kept are exactly the survivors deeper than that depth.
// A further pass (rare: more than kStair survivors in one group) settles the
// shallower ones, with the least kept entry as a cost cap.  Each pass
// records its entries in an LDS bit mask per member (lane bit = slice), 512
// members at a time, written as whole 64-bit words of a bitmap with one row
// per compatible config (a later pass ORs into the words it wrote).
// Compaction: popcount per tile, scan of tile counts, then each thread writes
// the candidate indices of its words' set bits in ascending order.
#include <algorithm>
#include <mutex>

#include "tg_device.h"

namespace tg {

constexpr int kFrontWaves = 4;
// Staircase entries a lane keeps per pass: 4 for groups of up to 64 members
// (60 VGPRs, 8 waves per SIMD), 8 above (82 VGPRs, 5 waves per SIMD), where
// staircases grow longer and a second pass would cost more than occupancy.
constexpr int kSmallGroup = 64;
constexpr int kMaskChunk = 512;   // members per LDS mask round when a pass is recorded
constexpr int kMemberBits = 23;   // an entry packs depth << kMemberBits | member
constexpr uint32_t kMemberMask = (1u << kMemberBits) - 1u;
constexpr int kCountThreads = 256;
constexpr int kWordsPerThread = 4;
constexpr int kTileWords = kCountThreads * kWordsPerThread;

// Offer member m (cost c, depth d >= 1, later in idx than every entry) to a
// lane's staircase.  Entry e beats m when d_e >= d and c_e <= c (equal cost:
// the deeper key is smaller, and equal depth: the earlier idx).
template <int R>
__device__ inline void stair_offer(double (&cv)[R], uint32_t (&pk)[R], double c, int d, int m, int &floor) {
    const uint32_t dk = (uint32_t)d << kMemberBits;
    bool beaten = false;
#pragma unroll
    for (int r = 0; r < R; ++r) beaten = beaten || (pk[r] >= dk && cv[r] <= c);  // empty slots hold 0
    if (beaten) return;
    const uint32_t dk1 = (uint32_t)(d + 1) << kMemberBits;
    const uint32_t x = dk | (uint32_t)m;
#pragma unroll
    for (int r = 0; r < R; ++r)
        if (pk[r] < dk1 && cv[r] >= c) pk[r] = 0u;  // entries m beats
    bool placed = false;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool t = !placed && pk[r] == 0u;
        if (t) {
            pk[r] = x;
            cv[r] = c;
        }
        placed = placed || t;
    }
    if (placed) return;
    // full: the shallowest of the entries and m leaves, and its depth becomes the floor
    uint32_t lo = x;
#pragma unroll
    for (int r = 0; r < R; ++r) lo = min(lo, pk[r]);
    floor = (int)(lo >> kMemberBits);
    if (lo == x) return;
#pragma unroll
    for (int r = 0; r < R; ++r)
        if (pk[r] == lo) {
            pk[r] = x;
            cv[r] = c;
        }
}

__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Writes the bitmap words of every member of the wave's group for its slice
// chunk: the lanes' entries set their bits in an LDS mask, kMaskChunk members
// at a time.  After the first pass a word also keeps the bits it already
// has.
template <int kStair>
__device__ inline void record_pass(const DevProblem &P, uint64_t *mask, const uint32_t (&pk)[kStair], bool mine,
                                   int lane, int m0, int nm, int64_t sc, bool merge, uint64_t *bitmap) {
    for (int base = 0; base < nm; base += kMaskChunk) {
        const int n = min(kMaskChunk, nm - base);
        for (int m = lane; m < n; m += kWave) mask[m] = 0;
        wave_sync();
        if (mine) {
#pragma unroll
            for (int r = 0; r < kStair; ++r) {
                const int m = (int)(pk[r] & kMemberMask) - base;
                if (pk[r] != 0u && m >= 0 && m < n) atomicOr((unsigned long long *)&mask[m], 1ull << lane);
            }
        }
        wave_sync();
        for (int m = lane; m < n; m += kWave) {
            uint64_t *at = bitmap + (int64_t)P.coef[P.kb_members[m0 + base + m]].row * P.words + sc;
            *at = merge ? (*at | mask[m]) : mask[m];
        }
        wave_sync();
    }
}

template <int kStair>
__global__ __launch_bounds__(256) void frontier_kernel(DevProblem P, const double *__restrict__ cost,
                                                       const uint8_t *__restrict__ dmax, uint64_t *bitmap,
                                                       int64_t n_tiles) {
    __shared__ uint64_t smask[kFrontWaves][kMaskChunk];
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t tile = (int64_t)blockIdx.x * kFrontWaves + wv;
    if (tile >= n_tiles) return;  // whole waves leave; nothing below synchronises the block
    const int q = (int)(tile / P.words);
    const int64_t sc = tile - (int64_t)q * P.words;
    const int m0 = P.kb_off[q];
    const int nm = P.kb_off[q + 1] - m0;
    const int64_t s = sc * kWave + lane;
    const int64_t NS = P.NS;
    bool need = s < NS;
    if (need && P.imb) {  // an unbalanced (slice, island) group has no survivors
        const uint32_t ij = P.sij[s];
        need = slice_balanced(P, P.pre, (int)(ij & 0xFFFFu), (int)(ij >> 16), P.kb_island[q]);
    }
    int hi = 1 << 30;  // members deeper than hi are settled (by an earlier pass)
    double cap = 0.0;  // least cost among the settled members, once there are any
    bool capped = false;
    bool merge = false;
    do {  // every wave records at least one pass: it writes all of its words
        double cv[kStair];
        uint32_t pk[kStair];
#pragma unroll
        for (int r = 0; r < kStair; ++r) {
            cv[r] = 0.0;
            pk[r] = 0u;
        }
        int floor = 0;  // members at or above this depth no longer matter in this pass
        for (int mb = 0; mb < nm; mb += 8) {
            int d[8];
            double c[8];
            const double *crow[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int64_t row = (int64_t)P.kb_members[m0 + min(mb + u, nm - 1)] * NS;
                crow[u] = cost + row;
                d[u] = (mb + u < nm && need) ? (int)dmax[row + s] : 0;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) c[u] = (d[u] > floor && d[u] <= hi) ? crow[u][s] : 0.0;
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (d[u] > floor && d[u] <= hi && !(capped && cap <= c[u]))
                    stair_offer<kStair>(cv, pk, c[u], d[u], mb + u, floor);
        }
        record_pass<kStair>(P, smask[wv], pk, need, lane, m0, nm, sc, merge, bitmap);
        merge = true;
        if (need) {
            if (floor == 0) {
                need = false;
            } else {  // the survivors at or above the floor are still to be found
                uint32_t lo = 0xFFFFFFFFu;
#pragma unroll
                for (int r = 0; r < kStair; ++r)
                    if (pk[r] != 0u && pk[r] < lo) {
                        lo = pk[r];
                        cap = cv[r];
                    }
                hi = floor;
                capped = true;
            }
        }
        // a further pass reads back the words this wave wrote (each lane the
        // same words, so program order already holds; the fence makes it plain)
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    } while (__ballot(need) != 0);
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

// Exclusive scan of n int64 values in place by one block; writes the sum to
// *total and, when given, to *total_host.
__global__ __launch_bounds__(1024) void scan_small_i64(int64_t *a, int64_t n, int64_t *total, int64_t *total_host) {
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
    if (threadIdx.x == 0) {
        *total = carry;
        if (total_host) *total_host = carry;
    }
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
        if (P.max_members <= kSmallGroup)
            frontier_kernel<4><<<dim3((unsigned)blocks), dim3(kFrontWaves * kWave), 0, s>>>(P, cost, dmax, bitmap,
                                                                                            n_front);
        else
            frontier_kernel<8><<<dim3((unsigned)blocks), dim3(kFrontWaves * kWave), 0, s>>>(P, cost, dmax, bitmap,
                                                                                            n_front);
    }
    return hipGetLastError();
}

// Survivor bitmap (at the start of ws) -> ascending candidate indices.
static hipError_t launch_compact(const DevProblem &P, int64_t *surv, int64_t capacity, void *ws, hipStream_t s,
                                 int64_t **d_total_out, int64_t *total_host = nullptr) {
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
    scan_small_i64<<<dim3(1), dim3(1024), 0, s>>>(tiles, nt, total, total_host);
    if (nt > 0)
        emit_kernel<<<dim3((unsigned)nt), dim3(kCountThreads), 0, s>>>(P, bitmap, nw, tiles, surv, capacity);
    return hipGetLastError();
}

hipError_t launch_prune(const DevProblem &P, const double *cost, const uint8_t *dmax, int64_t *surv,
                        int64_t capacity, void *ws, hipStream_t s, int64_t **d_total_out, int64_t *total_host) {
    hipError_t e = launch_frontier(P, cost, dmax, (uint64_t *)ws, s);
    if (e != hipSuccess) return e;
    return launch_compact(P, surv, capacity, ws, s, d_total_out, total_host);
}

// Scratch of the prune variant that allocates nothing: a device array the
// code object carries, one copy per GPU, held until the process ends.  Host
// code never names it in a kernel argument or a copy (the name is a host-side
// stand-in there); it reaches the array through the device address that
// hipGetSymbolAddress returns for the current GPU, resolved once per GPU.
// Every call rewrites all the workspace it reads (each bitmap word, tile
// count and the total), so nothing needs clearing between calls.
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

hipError_t static_scratch(int device, void **out) {
    static std::mutex mu;
    static void *addr[kMaxScratchDevices] = {};
    if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[device]) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress((void **)&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[device] = ptr;
    }
    *out = addr[device];
    return hipSuccess;
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
