// tg_device.h -- device-side problem tables and helpers shared by the HIP
// kernels of the plan-search library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/tangram.h"

#pragma clang fp contract(off)

namespace tg {

constexpr int kWave = 64;
constexpr double kInf = __builtin_huge_val();

// Per-config coefficients of the step-time and memory model, one row per
// config.
struct alignas(64) Coef {
    double alpha, beta, gamma, dd, de;  // cost = alpha Fl + beta Tb + gamma Ab + dd Pd + de Pe
    double mud, mue;                    // state = mud Pd + mue Pe
    double rho;                         // A1 = rho S (stash of one micro-batch)
    double H;                           // usable bytes per GPU
    double m_real;                      // B / b
    double inv_rho;                     // 1 / rho, only for the d_max first guess
    double kappa, omega;                // + kappa Cb + omega S (ring attention, offload traffic)
    int32_t k, tp, cp, dp, ep, z, rc, of, mb;  // the config tuple
    int32_t b_idx;                      // index of b in the compatible list, -1 if B mod b != 0
    int32_t row;                        // bitmap row of a compatible config, -1 otherwise
};
static_assert(sizeof(Coef) == 192, "Coef row must be 192 bytes");

// All device tables of one problem.  Passed to kernels by value.
struct DevProblem {
    int32_t L, K, nb, dense;
    int32_t ext;          // some config has cp > 1, recomputation or offloading
    int32_t pad0_;
    int64_t NS, ncfg, N, B;
    int32_t n_kb;         // (island, b) groups with at least one compatible config
    int32_t max_members;  // largest group
    int32_t n_rows;       // compatible configs = bitmap rows
    int32_t words;        // 64-bit bitmap words per row = ceil(NS / 64)
    const int64_t *pre;   // [8][L+1] prefix sums: flops, dparam, eparam, act, tpcomm, a2a, outact, cpcomm
    const int64_t *outact;  // [L]
    const double *E;        // [K*K] inter-island bytes/s
    const uint32_t *sij;    // [NS] slice -> i | j << 16
    const Coef *coef;       // [ncfg]
    const int64_t *bvals;   // [nb]
    const int32_t *kb_off;  // [n_kb+1] offsets into kb_members
    const int32_t *kb_members;  // config ids of each (island, b) group, ascending
    const int32_t *kb_island;   // [n_kb]
    const int32_t *kb_bidx;     // [n_kb]
    const int32_t *row_cfg;     // [n_rows] config id of each bitmap row
    const double *peak, *hbm, *intra, *host;  // [K] island rates
    double eta, mem_frac;
    int32_t n_ev;            // distinct inter-island bandwidth values (<= kMaxDistinctE), else 0
    int32_t imb;             // imbalance pruning on
    const double *Ev;        // [n_ev] the distinct values, ascending
    const uint16_t *Eidx;    // [K*K] index of E[a][b] in Ev
    double imb_r;            // 1 + eps
    int64_t total_flops;     // forward FLOPs of the whole model
    const double *cap;       // [K] island's share of the cluster's compute
    const int32_t *jlo;      // [K][L] first balanced cut j of slices starting at i (L + 1: none)
    const int32_t *jlo_pos;  // the same by island position of one composition call, or null
    int64_t NC;              // slice classes (equal per-slice sums)
    const uint32_t *cls;     // [NS] class of each slice
    const uint32_t *cls_ij;  // [NC] first slice of each class, i | j << 16
    int32_t class_scores;    // composition reads scores by class candidate (g * NC + cls[s])
    int32_t pad2_;
};

// The problem seen through its slice classes: class c stands for its first
// slice, so the score and frontier kernels run unchanged on NC "slices".
inline DevProblem class_view(const DevProblem &P) {
    DevProblem C = P;
    C.NS = P.NC;
    C.sij = P.cls_ij;
    C.N = P.ncfg * P.NC;
    C.words = (int32_t)((P.NC + 63) / 64);
    return C;
}

// Imbalance pruning: the slice's share of the model's FLOPs against the
// island's share of the cluster's compute, within a factor imb_r either way.
__host__ __device__ inline bool slice_balanced(const DevProblem &P, const int64_t *pre, int i, int j, int k) {
    if (!P.imb) return true;
    const double q = (double)(pre[j] - pre[i]) / (double)P.total_flops;
    const double c = P.cap[k];
    return q <= c * P.imb_r && q * P.imb_r >= c;
}

// Link times use one division per distinct bandwidth when there are few.
constexpr int kMaxDistinctE = 256;

// Slice index of [i, j): slices with first layer < i, then the offset of j.
__host__ __device__ inline int64_t slice_of(int64_t L, int64_t i, int64_t j) {
    return i * L - (i * (i - 1)) / 2 + (j - i - 1);
}

__device__ inline int wave_lane() { return threadIdx.x & (kWave - 1); }

// Inclusive prefix sum across a wave.
template <typename T>
__device__ inline T wave_incl_scan(T v) {
    const int lane = wave_lane();
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        T t = __shfl_up(v, off, kWave);
        if (lane >= off) v += t;
    }
    return v;
}

// Exclusive prefix sum over a block of blockDim.x (multiple of 64) threads.
// `lds` holds at least blockDim.x / 64 + 1 entries.  Returns the thread's
// exclusive prefix and writes the block total to *total.
template <typename T>
__device__ inline T block_excl_scan(T v, T *lds, T *total) {
    const int lane = wave_lane(), wave = threadIdx.x / kWave, nw = blockDim.x / kWave;
    T inc = wave_incl_scan(v);
    if (lane == kWave - 1) lds[wave] = inc;
    __syncthreads();
    if (threadIdx.x == 0) {
        T acc = 0;
        for (int w = 0; w < nw; w++) {
            T t = lds[w];
            lds[w] = acc;
            acc += t;
        }
        lds[nw] = acc;
    }
    __syncthreads();
    T out = inc - v + lds[wave];
    *total = lds[nw];
    __syncthreads();
    return out;
}

}  // namespace tg

// Host-side launchers (defined in the .hip files), all asynchronous on `s`.
namespace tg {
hipError_t launch_coef(const DevProblem &P, Coef *coef_inout, hipStream_t s);
hipError_t launch_score(const DevProblem &P, int64_t first, int64_t count, double *cost, uint8_t *dmax,
                        hipStream_t s);
hipError_t launch_enumerate(const DevProblem &P, int64_t first, int64_t count, tg_pair *out, hipStream_t s);

size_t prune_ws_bytes(const DevProblem &P);
size_t prune_classes_ws_bytes(const DevProblem &P);
hipError_t launch_prune_classes(const DevProblem &P, const double *cost, const uint8_t *dmax, int64_t *surv,
                                int64_t capacity, void *ws, hipStream_t s, int64_t **d_total_out);
// total_host: the device view of a pinned host word the count is also stored
// to, or null
hipError_t launch_prune(const DevProblem &P, const double *cost, const uint8_t *dmax, int64_t *surv,
                        int64_t capacity, void *ws, hipStream_t s, int64_t **d_total_out,
                        int64_t *total_host = nullptr);
// The static scratch of the prune variant that allocates nothing: its size,
// and its device address on `device` (which must be current), resolved once
// per GPU.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
constexpr int kMaxScratchDevices = 64;
hipError_t static_scratch(int device, void **out);

size_t compose_ws_bytes(const DevProblem &P, int64_t n_surv);
// Runs composition; on return (after the stream is synchronised by the
// caller) the result block at *result_dev holds the plan and status.
struct ComposeResult {
    int32_t err;     // non-zero: the candidate list was invalid
    int32_t status;  // TG_OK or TG_ENOPLAN
    int32_t pad[2];
    tg_plan plan;
};
// Pinned host memory, each block seen from the host and from the device (the
// address kernels store to).  The kernels store the fill depth limits (at
// least nb int32) and the result straight into it, and the host waits on the
// event `ev` (on the current device) for the limits while the first fill
// levels run.  Without it (null) the limits are copied back by a stream
// synchronisation and the result stays on the device alone.
struct ComposeHost {
    int32_t *dlim, *dlim_dev;
    ComposeResult *res, *res_dev;
    hipEvent_t ev;
};
hipError_t launch_compose(const DevProblem &P, const int64_t *surv, int64_t n_surv, const double *cost,
                          const uint8_t *dmax, const int32_t *order_dev, void *ws, hipStream_t s,
                          ComposeResult **result_dev, const ComposeHost *host = nullptr);
size_t compose_order_offset(const DevProblem &P, int64_t n_surv);  // where the order table lives in ws

// Host tables the relaxed search reads (link times are enumerated on the host).
// Pinned host memory owned by a caller and reused across calls (small
// transfers that the host waits for).
// `dev` is the same memory's device address (kernels store to it; the host
// reads what they stored once it has waited for them).
struct HostStage {
    void *ptr = nullptr, *dev = nullptr;
    size_t bytes = 0;
    hipError_t reserve(size_t n, unsigned flags = hipHostMallocPortable) {  // contents are not kept
        if (n <= bytes) return hipSuccess;
        release();
        hipError_t e = hipHostMalloc(&ptr, n, flags);
        if (e == hipSuccess) e = hipHostGetDevicePointer(&dev, ptr, 0);
        if (e != hipSuccess) {
            release();
            return e;
        }
        bytes = n;
        return e;
    }
    void release() {
        if (ptr) (void)hipHostFree(ptr);
        ptr = dev = nullptr;
        bytes = 0;
    }
};
size_t compose_relaxed_stage_bytes(const DevProblem &P);
struct RelaxHost {
    const int64_t *outact;  // [L] output activation bytes per layer
    const double *E;        // [K*K] inter-island bandwidth, island ids, row-major
    const int64_t *bvals;   // [nb] compatible micro-batch sizes, ascending
    int64_t B;              // global batch
    HostStage *stage;       // at least compose_relaxed_stage_bytes(P) bytes of pinned memory
    hipEvent_t ev;          // an event on the current device, or null (then the fill depth
                            // limits are read back by a stream synchronisation)
};
size_t compose_relaxed_ws_bytes(const DevProblem &P, int64_t n_surv);
// Island construction from nodes (n <= 4096); synchronises the stream.
size_t islands_ws_bytes(int n);
// *bad_bw: the first node_bw entry that is negative or not finite (checked on
// the device after the upload; nothing else runs then), else -1.
hipError_t launch_build_islands(int n, const tg_island *nodes_host, const double *e_host, double eps_c,
                                double eps_m, double eps_i, void *ws, hipStream_t s, int32_t *island_of,
                                tg_island *islands, double *inter_bw, int32_t *n_islands, int64_t *bad_bw);
// Composition over every island subset and order (K <= 16).
size_t compose_orders_ws_bytes(const DevProblem &P, int64_t n_surv);
hipError_t launch_compose_orders(const DevProblem &P, const int64_t *bvals_host, const int64_t *surv, int64_t n_surv,
                                 const double *cost, const uint8_t *dmax, void *ws, hipStream_t s,
                                 ComposeResult **result_dev);
// Synchronises the stream several times (once per search round).  On
// success the result is also stored into the stage at *result_host (host
// view), read once the stream is synchronised.
hipError_t launch_compose_relaxed(const DevProblem &P, const RelaxHost &H, const int32_t *order_host,
                                  const int64_t *surv, int64_t n_surv, const double *cost, const uint8_t *dmax,
                                  void *ws, hipStream_t s, ComposeResult **result_dev,
                                  const ComposeResult **result_host, int *rounds_out);
}  // namespace tg
