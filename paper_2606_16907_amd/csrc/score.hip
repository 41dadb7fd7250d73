// score.hip -- per-config coefficients, candidate scoring and decoding.
//
// Scoring is the analytic stand-in for the per-pair parallelizer query of
// Tab. 2 (profile() + parallelize()): a step-time cost per micro-batch and the
// deepest 1F1B position the pair fits at (Sec. 5.2).  Candidates are
// idx = g * NS + s (g: global config, s: slice).  A wave owns 64 consecutive
// slices and walks a run of 16 configs: the slice sums live in VGPRs for the
// whole run, the run's coefficients are staged once in LDS, and every
// config writes one coalesced 512-byte row of costs and 64 bytes of depths,
// the costs with streaming (nontemporal) stores, the depths too when their
// runs are 64-byte aligned.  The kernel is bound by HBM writes (9 bytes per
// candidate).
#include <type_traits>

#include "tg_device.h"

#pragma clang fp contract(off)

namespace tg {

// ---------------------------------------------------------------------------
// coefficients of one config (exact operation order of the stated model)
// ---------------------------------------------------------------------------
__device__ inline double ring_share(int64_t D) { return (double)(D - 1) / (double)D; }

// bf16 bytes per parameter moved for data-parallel sync, per micro-batch
__device__ inline double sync_per_microbatch(int z, int64_t D) {
    if (z <= 1) return 0.0;
    if (z == 2) return 2.0 * ring_share(D);
    return 6.0 * ring_share(D);
}

// bf16 bytes per parameter moved for data-parallel sync, per iteration
__device__ inline double sync_per_iteration(int z, int64_t D) {
    if (z <= 1) return 4.0 * ring_share(D);
    if (z == 2) return 2.0 * ring_share(D);
    return 0.0;
}

// model-state bytes per parameter (bf16 weight + bf16 grad + fp32 master, m, v)
__device__ inline double state_per_param(int z, int64_t D) {
    if (z == 0) return 16.0;
    if (z == 1) return 4.0 + 12.0 / (double)D;
    if (z == 2) return 2.0 + 14.0 / (double)D;
    return 16.0 / (double)D;
}

// q = tp * cp GPUs share a micro-batch's tokens; the data-parallel group
// (gradient sync, ZeRO sharding) is dp * cp; recomputation runs the forward
// pass twice (compute passes nc = 4, forward-collective passes nt = 3).
__global__ __launch_bounds__(256) void coef_kernel(DevProblem P, Coef *coef) {
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= P.ncfg) return;
    Coef c = coef[g];
    const double F = P.peak[c.k], W = P.intra[c.k], M = P.hbm[c.k], Hb = P.host[c.k];
    const int64_t b = (int64_t)c.dp * c.mb;
    const int64_t Dd = (int64_t)c.dp * c.cp, De = (int64_t)(c.dp / c.ep) * c.cp;
    const double qd = (double)c.tp, qe = (double)((int64_t)c.tp * c.ep);
    const int64_t q = (int64_t)c.tp * c.cp;
    const double nc = c.rc ? 4.0 : 3.0;
    const int nt = c.rc ? 3 : 2;
    c.m_real = (double)P.B / (double)b;
    c.alpha = (nc * (double)c.mb) / (((double)q * F) * P.eta);
    c.beta = c.tp > 1 ? (((double)(2 * nt) * (double)c.mb) * (double)(c.tp - 1)) / ((double)q * W) : 0.0;
    c.gamma = c.ep > 1 ? (((double)nt * (double)c.mb) * (double)(c.ep - 1)) / (((double)c.ep * (double)q) * W)
                       : 0.0;
    c.kappa = c.cp > 1 ? (((double)(nt + 1) * (double)c.mb) * (double)(c.cp - 1)) /
                             (((double)c.cp * (double)c.tp) * W)
                       : 0.0;
    c.dd = ((sync_per_microbatch(c.z, Dd) / qd) / W) + (((sync_per_iteration(c.z, Dd) / qd) / W) / c.m_real);
    c.de = ((sync_per_microbatch(c.z, De) / qe) / W) + (((sync_per_iteration(c.z, De) / qe) / W) / c.m_real);
    c.mud = state_per_param(c.z, Dd) / qd;
    c.mue = state_per_param(c.z, De) / qe;
    c.rho = (double)c.mb / (double)q;
    c.omega = c.of ? (2.0 * (double)c.mb) / ((double)q * Hb) : 0.0;
    c.H = M * P.mem_frac;
    c.inv_rho = (double)q / (double)c.mb;
    coef[g] = c;
}

hipError_t launch_coef(const DevProblem &P, Coef *coef, hipStream_t s) {
    const int64_t blocks = (P.ncfg + 255) / 256;
    coef_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, coef);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// scoring
// ---------------------------------------------------------------------------
constexpr int kScoreWaves = 4;     // waves per block
// Configs per wave tile: 16 where a wave's depth rows are line-aligned and go
// out as streaming stores (more rows a tile scatter those stores: the
// 128-layer instance took 1.74 -> 1.91 ms at 32), 32 elsewhere, where a
// tile's slice sums and coefficient staging then serve more configs (MoE
// 110 -> 105 µs, 70B 122 -> 114 µs).
constexpr int score_configs(bool nt_depth) { return nt_depth ? 16 : 32; }

// Largest d in 1..K with state + min(d, m) * A1 <= H, or 0.  fits() is
// monotone in d, so a first guess d0 from (H - state) / A1 (K once the
// stash saturates at m micro-batches) is the answer exactly when d0 fits and
// d0 + 1 does not; otherwise a short walk from d0 finds it.  Every decision
// is an exact evaluation of fits(); the guess only picks where to look.  The
// guess and both checks run on every lane without branches (in doubles: the
// guess is a small integer, so min(d0, m) and min(d0 + 1, m) are the values
// fits() takes); the wave walks only when a lane that scores a candidate
// (`live`) has a wrong guess, and the walk returns d0 to a lane whose guess
// is right.
__device__ inline int max_depth(double state, double A1, double H, double m_real, double guess_scale, int K,
                                bool live) {
    auto fits = [&](int d) -> bool {
        const double inflight = fmin((double)d, m_real);
        return state + inflight * A1 <= H;
    };
    const double Kd = (double)K;
    const double q = (H - state) * guess_scale;
    // floor(q) within [0, K] (NaN: 0)
    const double g = q >= m_real ? Kd : floor(fmin(fmax(q, 0.0), Kd));
    const bool lo_ok = g == 0.0 || state + fmin(g, m_real) * A1 <= H;
    const bool hi_ok = g == Kd || !(state + fmin(g + 1.0, m_real) * A1 <= H);
    const int d0 = (int)g;
    if (__builtin_expect(__ballot(live && !(lo_ok && hi_ok)) == 0, 1)) return d0;
    int d = d0 > K - 1 ? K - 1 : d0;
#pragma nounroll
    while (live && d > 0 && !fits(d)) --d;
#pragma nounroll
    while (live && d < K && fits(d + 1)) ++d;
    return d;
}

// Blocks are dispatched round-robin over the 8 XCDs.  Renumbering them so
// that consecutive tiles run on the same XCD keeps every cache line of the
// output (depth rows are not line-aligned) inside one L2, which merges the
// partial lines before they reach HBM.
constexpr int kXcds = 8;

// The coefficients a wave needs for its run of configs, staged in LDS: one
// coalesced load per lane at the start of the tile instead of scalar loads in
// every iteration (the coefficient table falls out of L2 under the streaming
// writes, and scalar misses would stall each iteration).
struct StagedCoef {
    double alpha, beta, gamma, dd, de, mud, mue, rho, H, m_real, inv_rho, kappa, omega;
    int32_t rc, of;
};

// kExt: the space has context parallelism, recomputation or offloading
// (two more slice sums, two more cost terms, the stash and depth rules).
// kNtDepth: a wave's 64 depths of a row start on a 64-byte boundary (NS a
// multiple of 64) and go out with streaming stores like the costs; otherwise
// the run straddles segments that the neighbouring waves also write, and
// ordinary stores let L2 merge them.
template <bool kDense, bool kExt, bool kNtDepth>
__global__ __launch_bounds__(256) void score_kernel(DevProblem P, int64_t first, int64_t last, int64_t g_lo,
                                                    int64_t g_hi, int64_t n_stiles, int64_t n_tiles,
                                                    double *__restrict__ cost, uint8_t *__restrict__ dmax) {
    constexpr int kCfg = score_configs(kNtDepth);
    __shared__ StagedCoef cs[kScoreWaves][kCfg];
    const int64_t per_xcd = gridDim.x / kXcds;
    const int64_t blk = (int64_t)(blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t tile = blk * kScoreWaves + wv;
    if (tile >= n_tiles) return;
    const int64_t gt = tile / n_stiles;
    const int64_t st = tile - gt * n_stiles;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t s = st * kWave + lane;
    const bool sv = s < P.NS;
    const int64_t g_beg = g_lo + gt * kCfg;
    const int ng = (int)(min(g_beg + kCfg, g_hi + 1) - g_beg);
    if (lane < ng) {
        const Coef &c = P.coef[g_beg + lane];
        StagedCoef x;
        x.alpha = c.alpha;
        x.beta = c.beta;
        x.gamma = c.gamma;
        x.dd = c.dd;
        x.de = c.de;
        x.mud = c.mud;
        x.mue = c.mue;
        x.rho = c.rho;
        x.H = c.H;
        x.m_real = c.m_real;
        x.inv_rho = c.inv_rho;
        if (kExt) {  // read only by the extended variant
            x.kappa = c.kappa;
            x.omega = c.omega;
            x.rc = c.rc;
            x.of = c.of;
        }
        cs[wv][lane] = x;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // slice sums: exact int64 prefix differences, then one rounding to binary64
    double Fl = 0.0, Pd = 0.0, Pe = 0.0, Act = 0.0, Tb = 0.0, Ab = 0.0, inv_act = 0.0;
    double Oa = 0.0, Cb = 0.0, inv_oa = 0.0;
    if (sv) {
        const uint32_t ij = P.sij[s];
        const int i = (int)(ij & 0xFFFFu), j = (int)(ij >> 16);
        const int64_t *pre = P.pre;
        const int64_t Lp = P.L + 1;
        Fl = (double)(pre[j] - pre[i]);
        Pd = (double)(pre[Lp + j] - pre[Lp + i]);
        Act = (double)(pre[3 * Lp + j] - pre[3 * Lp + i]);
        Tb = (double)(pre[4 * Lp + j] - pre[4 * Lp + i]);
        if (!kDense) {
            Pe = (double)(pre[2 * Lp + j] - pre[2 * Lp + i]);
            Ab = (double)(pre[5 * Lp + j] - pre[5 * Lp + i]);
        }
        inv_act = 1.0 / Act;
        if (kExt) {
            Oa = (double)(pre[6 * Lp + j] - pre[6 * Lp + i]);
            Cb = (double)(pre[7 * Lp + j] - pre[7 * Lp + i]);
            inv_oa = 1.0 / Oa;
        }
    }
    const int K = P.K;
    const int64_t NS = P.NS;
    // a tile wholly inside [first, last) with a slice for every lane stores
    // without per-candidate checks, from a per-row base
    const int64_t t0 = g_beg * NS + st * kWave;
    const bool whole = (st + 1) * kWave <= NS && t0 >= first && t0 + (int64_t)(ng - 1) * NS + (kWave - 1) < last;
    for (int t = 0; t < ng; ++t) {
        const StagedCoef &c = cs[wv][t];
        // with recomputation only the layer boundaries (outputs) are stashed
        const double S = (kExt && c.rc) ? Oa : Act;
        double v = c.alpha * Fl;
        v = v + c.beta * Tb;
        if (!kDense) v = v + c.gamma * Ab;
        v = v + c.dd * Pd;
        if (!kDense) v = v + c.de * Pe;
        if (kExt) {
            v = v + c.kappa * Cb;
            v = v + c.omega * S;
        }
        double state = c.mud * Pd;
        if (!kDense) state = state + c.mue * Pe;
        const double A1 = c.rho * S;
        int dm;
        if (kExt && c.of) {
            // offloaded: one micro-batch on the device at every depth
            dm = (state + (fmin(1.0, c.m_real) * A1)) <= c.H ? K : 0;
        } else {
            dm = max_depth(state, A1, c.H, c.m_real, c.inv_rho * ((kExt && c.rc) ? inv_oa : inv_act), K, sv);
        }
        if (whole) {
            const int64_t row = t0 + (int64_t)t * NS - first;
            __builtin_nontemporal_store(v, cost + row + lane);
            if (kNtDepth)
                __builtin_nontemporal_store((uint8_t)dm, dmax + row + lane);
            else
                dmax[row + lane] = (uint8_t)dm;
            continue;
        }
        const int64_t idx = (g_beg + t) * NS + s;
        if (sv && idx >= first && idx < last) {
            // streaming stores: the arrays are far larger than the caches
            __builtin_nontemporal_store(v, cost + (idx - first));
            if (kNtDepth)
                __builtin_nontemporal_store((uint8_t)dm, dmax + (idx - first));
            else
                dmax[idx - first] = (uint8_t)dm;
        }
    }
}

hipError_t launch_score(const DevProblem &P, int64_t first, int64_t count, double *cost, uint8_t *dmax,
                        hipStream_t s) {
    if (count <= 0) return hipSuccess;
    const int64_t last = first + count;
    const int64_t g_lo = first / P.NS, g_hi = (last - 1) / P.NS;
    const bool nt_depth = (P.NS & 63) == 0;
    const int cfg = score_configs(nt_depth);
    const int64_t n_gtiles = (g_hi - g_lo + cfg) / cfg;
    const int64_t n_stiles = (P.NS + kWave - 1) / kWave;
    const int64_t n_tiles = n_gtiles * n_stiles;
    int64_t blocks = (n_tiles + kScoreWaves - 1) / kScoreWaves;
    blocks = (blocks + kXcds - 1) / kXcds * kXcds;  // whole rounds over the XCDs
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    auto go = [&](auto dense, auto ext) {
        constexpr bool D = decltype(dense)::value, X = decltype(ext)::value;
        if (nt_depth)
            score_kernel<D, X, true><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, first, last, g_lo, g_hi,
                                                                                   n_stiles, n_tiles, cost, dmax);
        else
            score_kernel<D, X, false><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, first, last, g_lo, g_hi,
                                                                                    n_stiles, n_tiles, cost, dmax);
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    if (P.dense && !P.ext)
        go(T_{}, F_{});
    else if (!P.dense && !P.ext)
        go(F_{}, F_{});
    else if (P.dense)
        go(T_{}, T_{});
    else
        go(F_{}, T_{});
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// decoding
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void enumerate_kernel(DevProblem P, int64_t first, int64_t count, tg_pair *out) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= count) return;
    const int64_t idx = first + t;
    const int64_t g = idx / P.NS, s = idx - g * P.NS;
    const uint32_t ij = P.sij[s];
    const Coef &c = P.coef[g];
    tg_pair p;
    p.i = (int32_t)(ij & 0xFFFFu);
    p.j = (int32_t)(ij >> 16);
    p.island = c.k;
    p.tp = c.tp;
    p.cp = c.cp;
    p.dp = c.dp;
    p.ep = c.ep;
    p.zero = c.z;
    p.recompute = c.rc;
    p.offload = c.of;
    p.mb = c.mb;
    p.reserved = 0;
    out[t] = p;
}

hipError_t launch_enumerate(const DevProblem &P, int64_t first, int64_t count, tg_pair *out, hipStream_t s) {
    if (count <= 0) return hipSuccess;
    const int64_t blocks = (count + 255) / 256;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    enumerate_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(P, first, count, out);
    return hipGetLastError();
}

}  // namespace tg
