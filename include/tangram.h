/*
 * tangram.h -- C ABI of the MI355X (gfx950) plan-search library.
 *
 * The library computes the search at the core of Tangram's heterogeneous
 * planner (arXiv 2606.16907): every model slice (a contiguous layer range,
 * Sec. 4.2) is paired with every GPU island (Sec. 4.1) and every intra-island
 * parallel configuration (tensor, context, data and expert parallelism, ZeRO,
 * activation recomputation and offloading, micro-batch size; Sec. 2.1); each
 * pair gets an analytic step-time cost and the
 * deepest 1F1B pipeline position it fits at (Sec. 5.2); incompatible,
 * infeasible and dominated pairs are pruned (Sec. 5.1); the survivors are
 * composed into a work-balanced pipeline across islands, lowest bottleneck
 * first, then lowest fill (Sec. 5.2, composition steps (1)-(3)).
 *
 * Conventions shared by every entry point:
 *   - Units: FLOPs, parameters and bytes are per sample (one sequence), for
 *     the forward pass of one layer; FLOP/s, bytes and bytes/s are per GPU.
 *   - Device buffers ("d_" prefix) are allocated and owned by the caller and
 *     must live on the device that was current at tg_problem_create, and
 *     that device must be current at every call that takes the problem
 *     (TG_EINVAL otherwise); host
 *     pointers are plain host memory.  The library allocates device memory
 *     only inside tg_problem_create (small input tables) and frees it in
 *     tg_problem_destroy.
 *   - Alignment: score cost arrays and survivor lists 8 bytes, candidate
 *     pair buffers 4 bytes, workspaces 256 bytes (they are carved at 256-byte
 *     offsets and hold atomic counters); a misaligned buffer is TG_EINVAL.
 *     hipMalloc'd memory meets all of these.
 *   - `stream` is a hipStream_t (NULL: the default stream).  Calls are
 *     asynchronous on it except where a host result is returned; those calls
 *     synchronise the stream once.
 *   - Concurrency: a problem is read-only after create, so calls on
 *     different streams or host threads may share it.  A workspace belongs
 *     to one call at a time: calls whose workspaces overlap must be ordered
 *     on one stream (or by events), or they race on its counters and tables.
 *     tg_problem_destroy must not overlap a call that uses the problem.
 *   - Errors are returned as tg_status; no call throws.  tg_last_error()
 *     returns a message for the calling thread's most recent failure.
 *   - Results are a pure function of the inputs, independent of launch
 *     configuration and repeatable bit for bit.
 *   - Floating point is IEEE binary64 with one rounding per operation in a
 *     fixed order; no operation is fused or reassociated.
 */
#ifndef TANGRAM_H
#define TANGRAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *tg_stream; /* a hipStream_t */

typedef enum {
    TG_OK = 0,
    TG_EINVAL = -1,    /* invalid argument or input table */
    TG_ENOMEM = -2,    /* device allocation failed, or workspace too small */
    TG_EDEVICE = -3,   /* a HIP runtime call or kernel launch failed */
    TG_ECAPACITY = -4, /* output buffer too small; the required count is returned */
    TG_ENOPLAN = -5    /* no pipeline fits the cluster */
} tg_status;

/* One model atom (a layer), Sec. 4.2 / Tab. 2 slice_model().  All values are
   integers >= 0 and every whole-model sum must stay below 2^62. */
typedef struct {
    int64_t fwd_flops;       /* forward FLOPs per sample */
    int64_t dense_params;    /* parameters replicated across expert-parallel ranks */
    int64_t expert_params;   /* expert parameters, sharded by expert parallelism */
    int64_t act_stash_bytes; /* activation bytes kept per sample for the backward pass */
    int64_t tp_comm_bytes;   /* bytes per sample in the layer's tensor-parallel collectives, one pass */
    int64_t a2a_bytes;       /* bytes per sample moved by the layer's all-to-alls, one pass */
    int64_t out_act_bytes;   /* bytes per sample of the layer's output activation */
    int64_t cp_comm_bytes;   /* key and value bytes per sample of the layer's attention (whole
                                sequence), circulated by ring attention under context parallelism */
} tg_layer;

/* One GPU island (Sec. 4.1): nodes of identical GPUs.  n_gpus in [1, 2^28]
   (every island tg_build_islands returns is accepted);
   peak_flops, hbm_bytes and intra_bw are finite and > 0; host_bw is finite
   and >= 0 (0: no host link, activation offloading is not admitted). */
typedef struct {
    int32_t n_gpus;
    int32_t reserved; /* must be 0 */
    double peak_flops; /* FLOP/s per GPU */
    double hbm_bytes;  /* memory per GPU */
    double intra_bw;   /* bytes/s per GPU for intra-island collectives */
    double host_bw;    /* bytes/s per GPU to host memory (activation offloading) */
} tg_island;

/* The intra-island configuration space.  Each set holds 1..8 strictly
   ascending entries >= 1 (cp may be empty: n_cp = 0 means {1}).  zero_mask:
   bit z set admits ZeRO stage z (0..3); it must be non-zero.  recompute_mask
   and offload_mask: bit 0 admits "off", bit 1 "on" (0 means {off}).
   n_experts = 0 describes a dense model (then only ep = 1 is admitted);
   otherwise ep must divide n_experts.  eta scales peak FLOP/s (efficiency),
   mem_frac scales usable memory; both finite and > 0.  A zero-filled tail
   (n_cp, masks, imbalance_eps) keeps the space without context parallelism,
   recomputation, offloading and imbalance pruning.

   imbalance_eps (Sec. 5.1 (ii), imbalance pruning; finite, >= 0, 0 = off):
   with q = Fl(i, j) / Fl(0, L) the slice's share of the model's forward FLOPs
   and c_k = (n_k F_k) / sum_k' (n_k' F_k') the island's share of the
   cluster's compute (the sum taken in island order), the pair (slice, island)
   is kept iff q <= c_k (1 + eps) and q (1 + eps) >= c_k, each operation one
   binary64 rounding in that order.  Unbalanced pairs are scored but never
   survive, and the compositions reject them.  A model with no FLOPs is never
   pruned. */
typedef struct {
    int64_t global_batch; /* samples per iteration, >= 1; every compatible b and B / b below 2^31 */
    int32_t n_experts;
    int32_t n_tp;
    int32_t tp[8];
    int32_t n_ep;
    int32_t ep[8];
    int32_t n_mb;
    int32_t mb[8];
    uint32_t zero_mask;
    int32_t reserved; /* must be 0 */
    double eta;
    double mem_frac;
    int32_t n_cp;
    int32_t cp[8];           /* context-parallel degrees */
    uint32_t recompute_mask; /* activation recomputation (Sec. 2.1 RC) */
    uint32_t offload_mask;   /* activation offloading to host memory (Sec. 2.1 OF) */
    int32_t reserved2;       /* must be 0 */
    double imbalance_eps;    /* imbalance-pruning tolerance, 0 = off */
} tg_space;

/* A decoded candidate: layers [i, j) on island `island` with the given
   degrees (tensor, context, data, expert), ZeRO stage, recomputation and
   offloading flags (0/1) and micro-batch size (samples per DP rank). */
typedef struct {
    int32_t i, j, island, tp, cp, dp, ep, zero, recompute, offload, mb, reserved;
} tg_pair;

/* One pipeline stage of a plan; stage 0 is the pipeline front. */
typedef struct {
    int32_t island, first_layer, end_layer, tp, cp, dp, ep, zero, recompute, offload, mb;
    int32_t depth; /* stages from this one to the pipeline end, inclusive */
    int64_t pair_index; /* candidate index of the chosen pair */
    double cost;        /* seconds per micro-batch (step-time cost of the pair) */
    double mem_bytes;   /* per-GPU memory at this depth */
    double link_out;    /* seconds per micro-batch on the link to the next stage (0 for the last) */
} tg_stage;

/* A composed plan.  b = samples per pipeline micro-batch (dp * mb, the same
   for every stage), m = global_batch / b micro-batches, S stages,
   P = bottleneck, F = pipeline fill, T = (m - 1) * P + F. */
typedef struct {
    int32_t b, m, S, reserved;
    double P, F, T;
    tg_stage stage[255];
} tg_plan;

/* Problem sizes after create. */
typedef struct {
    int32_t L, K;
    int32_t n_b;        /* distinct compatible b values (B mod b == 0) */
    int32_t dense;      /* 1 when no layer has expert parameters or all-to-all bytes */
    int64_t NS;         /* slices = L (L + 1) / 2 */
    int64_t n_configs;  /* intra-island configs summed over islands */
    int64_t N;          /* candidates = NS * n_configs */
    int64_t n_compatible_configs;
    int64_t n_slice_classes; /* NC: classes of slices with equal per-slice sums (redundancy pruning) */
} tg_info;

typedef struct tg_problem tg_problem;

/*
 * Validates and copies one planning instance to the current device: the
 * model's layers (the atoms slices are cut from, Sec. 4.2), the GPU islands
 * and their links (Sec. 4.1) and the intra-island configuration space
 * (Sec. 2.1).
 *   layers[L], L in [1, 512]; islands[K], K in [1, 255];
 *   inter_bw: K*K row-major bytes/s from island a to island b (>= 0 or +inf;
 *             0 means no link; the diagonal is ignored);
 *   space: the configuration space.
 * Candidate order (the linear index used by every other call):
 *   idx = (cfg_off[k] + c) * NS + s, where s enumerates slices 0 <= i < j <= L
 *   lexicographically (i, then j), c enumerates island k's configs
 *   lexicographically over (tp, dp, ep, zero, mb) with tp in space.tp,
 *   tp <= n_gpus, dp in 1..floor(n_gpus / tp), ep admitted and dividing dp,
 *   zero in zero_mask, mb in space.mb; cfg_off is the running count over
 *   islands in input order.  With context parallelism, recomputation or
 *   offloading the order is lexicographic over (tp, cp, dp, ep, zero,
 *   recompute, offload, mb), tp * cp * dp <= n_gpus, and offloading needs
 *   host_bw > 0; with their defaults it is the order above.
 * At most 2^23 - 1 configs in all (the pruning pass packs a config's index
 * within its group into 23 bits); a larger space is refused with TG_EINVAL
 * after a counting pass, before any of its tables is allocated.
 * Returns TG_EINVAL on any invalid value, TG_ENOMEM on a failed host or
 * device allocation, TG_EDEVICE on other device failures; *out is NULL on
 * failure.
 */
tg_status tg_problem_create(const tg_layer *layers, int32_t L, const tg_island *islands, int32_t K,
                            const double *inter_bw, const tg_space *space, tg_problem **out);
/* Frees the problem's device tables (NULL is ignored).  Must not overlap a
   call that uses the problem. */
void tg_problem_destroy(tg_problem *p);
/* Fills *out with the problem's sizes; TG_EINVAL if p or out is NULL. */
tg_status tg_problem_info(const tg_problem *p, tg_info *out);
/* Writes the n_b distinct compatible micro-batch sizes b (the composition
   of Sec. 5.2 runs once per b), ascending, into out (capacity entries).
   Returns TG_ECAPACITY if capacity < n_b, TG_EINVAL if out is NULL and
   n_b > 0. */
tg_status tg_problem_bvalues(const tg_problem *p, int64_t *out, int32_t capacity);

/*
 * Enumeration of the model-slice/island/config candidates (Sec. 5.1):
 * *n_candidates = N.  When d_out is not NULL, decodes candidates
 * [first, first + count) into d_out[0 .. count) on the device.
 * TG_EINVAL if the range leaves [0, N).
 */
tg_status tg_enumerate_pairs(const tg_problem *p, int64_t *n_candidates, int64_t first, int64_t count,
                             tg_pair *d_out, tg_stream stream);

/*
 * Scoring (the per-pair profile()/parallelize() query of Tab. 2, made
 * analytic): for every candidate in [first, first + count) writes
 *   d_cost[idx - first]: seconds per micro-batch, including data-parallel
 *                        synchronisation amortised over the iteration;
 *   d_dmax[idx - first]: the largest pipeline depth d in 1..K at which the
 *                        pair fits in memory when min(d, m) micro-batches of
 *                        activations are in flight (1F1B, Sec. 5.2), or 0.
 * With b = dp*mb, m = B/b, r(D) = (D-1)/D, q = tp*cp, Dd = dp*cp (the
 * data-parallel group), De = (dp/ep)*cp, W the island's intra bandwidth, F
 * its peak, Hb its host bandwidth, nc = 3 (4 with recomputation: the forward
 * pass runs twice), nt = 2 (3 with recomputation: forward collectives run
 * twice), and slice sums Fl, Tb, Ab, Pd, Pe, Act, Oa, Cb of the tg_layer
 * fields fwd_flops, tp_comm, a2a, dense_params, expert_params, act_stash,
 * out_act and cp_comm over [i, j); S = Oa with recomputation (only layer
 * boundaries are stashed), else Act:
 *   cost  = alpha*Fl + beta*Tb + gamma*Ab + dd*Pd + de*Pe + kappa*Cb + omega*S
 *           (summed left to right)
 *   alpha = nc mb / (q F eta)                    compute over tp*cp GPUs
 *   beta  = 2 nt mb (tp-1) / (q W)               TP collectives, nt passes x 2r
 *   gamma = nt mb (ep-1) / (ep q W)              all-to-all, nt passes
 *   kappa = (nt+1) mb (cp-1) / (cp tp W)         ring attention: keys/values once
 *                                                forward, twice backward
 *   omega = 2 mb / (q Hb) with offloading, else 0   stash to host and back
 *   dd/de = (zm/qd)/W + ((zi/qd)/W)/m with qd = tp (dense) or tp*ep (expert),
 *           D = Dd (dense) or De (expert), and per-parameter bf16 traffic
 *           zm = {0, 0, 2r, 6r} per micro-batch, zi = {4r, 4r, 2r, 0} per
 *           iteration for ZeRO stage 0..3
 *   state = (w(Dd)/tp)*Pd + (w(De)/(tp ep))*Pe, w(D) = {16, 4+12/D, 2+14/D, 16/D}
 *   fits(d) <=> state + n(d) * (mb/q) * S <= hbm * mem_frac, n(d) = min(d, m),
 *           or min(1, m) at every depth with offloading
 * cp = 1, no recomputation and no offloading reduce this exactly to the
 * model without them (the added terms are +0).
 * Asynchronous.  TG_EINVAL if the range leaves [0, N).
 */
tg_status tg_score_pairs(const tg_problem *p, int64_t first, int64_t count, double *d_cost,
                         uint8_t *d_dmax, tg_stream stream);

/*
 * Pruning (Sec. 5.1 infeasibility and incompatibility pruning, plus
 * dominance): from the full score arrays (d_cost, d_dmax over all N
 * candidates) writes the ascending list of survivors to d_survivors.  A
 * candidate survives iff its micro-batch b divides the global batch, its
 * d_max >= 1, and it has the least key (cost, -d_max, idx) among the members
 * of its group (same slice, island and b) whose d_max reaches its own d_max.
 * *n_survivors (host) receives the count; if it exceeds `capacity`, nothing
 * past capacity is written and TG_ECAPACITY is returned.  d_ws: caller
 * workspace of at least tg_prune_workspace_bytes(p) bytes (TG_ENOMEM if
 * smaller).  Synchronises the stream once to read the count, which the
 * kernels also store into about 20 KB of pinned host memory that the handle
 * owns (its read-back words: allocated at the first prune or composition
 * call, freed by tg_problem_destroy); a call that finds them in use by
 * another call on the same handle copies the count back instead.
 */
size_t tg_prune_workspace_bytes(const tg_problem *p);
tg_status tg_prune(const tg_problem *p, const double *d_cost, const uint8_t *d_dmax, int64_t *d_survivors,
                   int64_t capacity, int64_t *n_survivors, void *d_ws, size_t ws_bytes, tg_stream stream);

/*
 * tg_prune without a workspace, for callers that cannot allocate device
 * memory: code being captured into a HIP graph, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, result and errors as
 * tg_prune; the workspace is instead a static device array of 64 MiB that
 * the library holds on each GPU it runs on until the process ends (enough for
 * every problem whose tg_prune_workspace_bytes is at most 64 MiB, e.g. 128
 * layers x 33,536 compatible configs).  A larger problem is refused with
 * TG_ENOMEM before any work is queued.  The call allocates nothing (no
 * hipMalloc, no host or device allocation by the library).  Every call on one
 * GPU uses that GPU's array: calls that overlap on one GPU (other streams or
 * threads) race and must be serialised by the caller.  Each call rewrites all
 * the scratch it reads, so earlier calls leave nothing behind that matters.
 */
tg_status tg_prune_no_alloc(const tg_problem *p, const double *d_cost, const uint8_t *d_dmax,
                            int64_t *d_survivors, int64_t capacity, int64_t *n_survivors, tg_stream stream);

/*
 * Redundancy pruning (Sec. 5.1 (i): slices of the same composition are one
 * query).  Two slices are equivalent when all eight of their per-slice sums
 * (the tg_layer fields summed over the slice) are equal; every config scores
 * them alike.  Classes c = 0..NC-1 are numbered by their first slice (the
 * slice order of tg_score_pairs).  A class candidate is idx_c = (cfg_off[k] +
 * c_cfg) * NC + c, config-major like the candidate index.
 *   tg_score_classes: as tg_score_pairs over class candidates [first, first +
 * count) of [0, n_configs * NC): the score of each class's first slice.
 *   tg_prune_classes: the surviving set from class scores (d_cost, d_dmax over
 * all n_configs * NC class candidates), found once per (island, b, class) and
 * copied to the class's slices: writes exactly tg_prune's survivor list (full
 * candidate indices, ascending) under tg_prune's capacity rules.  d_ws: at
 * least tg_prune_classes_workspace_bytes(p) bytes.  Synchronises once.
 *   tg_compose_pipeline_classes: tg_compose_pipeline with class scores: the
 * list is tg_prune_classes' (or tg_prune's) output, d_cost / d_dmax are
 * tg_score_classes' arrays; same plan, workspace and errors.
 */
tg_status tg_score_classes(const tg_problem *p, int64_t first, int64_t count, double *d_cost, uint8_t *d_dmax,
                           tg_stream stream);
size_t tg_prune_classes_workspace_bytes(const tg_problem *p);
tg_status tg_prune_classes(const tg_problem *p, const double *d_cost, const uint8_t *d_dmax, int64_t *d_survivors,
                           int64_t capacity, int64_t *n_survivors, void *d_ws, size_t ws_bytes, tg_stream stream);
tg_status tg_compose_pipeline_classes(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                                      const double *d_cost, const uint8_t *d_dmax, const int32_t *island_order,
                                      tg_plan *out, void *d_ws, size_t ws_bytes, tg_stream stream);

/*
 * Composition (Sec. 5.2): builds the pipeline from the candidates listed in
 * d_survivors, scored by d_cost / d_dmax over all N.  The list holds strictly
 * ascending indices of compatible candidates (anything else is TG_EINVAL;
 * entries with d_max 0 are ignored) and must contain the whole surviving set:
 * tg_prune's output, or any superset of it drawn from the compatible
 * candidates, which composes to the same plan.  island_order (host, a permutation of 0..K-1) fixes the
 * order in which islands may appear from pipeline front to back; islands may
 * be skipped.  For each b the plan minimises the bottleneck P = max of stage
 * costs and link times, then the fill F = f1 + (x1 + (f2 + ... + fS)) among
 * plans with that bottleneck; across b it minimises T = (m - 1) P + F, ties
 * to the smaller b.  Ties inside a b go to the earliest first island, then
 * fewer stages, then the earliest cut, then the earliest next island.
 * Writes *out (stages past out->S zero); TG_ENOPLAN (out->S = 0, out->T =
 * +inf) if nothing fits.  d_ws: at least tg_compose_workspace_bytes(p,
 * n_survivors) bytes.  Synchronises the stream at its end.  The kernels
 * store the fill depth limits and the result into the handle's read-back
 * words (those of tg_prune); with more than 8 levels (min(K, L)) the host
 * also waits once part-way, for the depth limits, while the first fill
 * levels run.  A call that finds the words in use by another call on the
 * same handle copies the result back instead, and reads the depth limits by
 * a stream synchronisation when there are 64 levels or more, otherwise
 * launching every fill level.
 */
size_t tg_compose_workspace_bytes(const tg_problem *p, int64_t n_survivors);
tg_status tg_compose_pipeline(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                              const double *d_cost, const uint8_t *d_dmax, const int32_t *island_order,
                              tg_plan *out, void *d_ws, size_t ws_bytes, tg_stream stream);

/*
 * Composition with the relaxation of step (4) of Sec. 5.2: after the least
 * bottleneck P* and the least fill at it, the bound on every stage and link
 * is raised over the stage and link costs above P* while the iteration time
 * can still improve.  Per b the plan minimises T = (m - 1) * tau + F(tau)
 * over bounds tau >= P*, where F(tau) is the least fill among plans whose
 * every stage cost and link time is <= tau; ties go to the smallest tau, and
 * the plan is the one tg_compose_pipeline's rules pick at that bound (least
 * fill, then earliest first island, fewer stages, earliest cut, earliest next
 * island).  This is the least T over every plan of that b.  Across b: least
 * T, ties to the smaller b.  out->P is the chosen bound (the plan's
 * bottleneck), out->F its fill, out->T = (m - 1) * P + F.  Arguments, list
 * requirements and errors as for tg_compose_pipeline; d_ws: at least
 * tg_compose_relaxed_workspace_bytes(p, n_survivors) bytes.  Synchronises the
 * stream after the bottleneck and fill phases and once per search round (a
 * few rounds; each evaluates F at a batch of bounds on the device), and with
 * more than 8 levels waits once more part-way, for the fill depth limits,
 * while the first fill levels run.  The host side of the search reads back
 * and uploads through a small pinned host buffer that the handle owns
 * (allocated at the first call, freed by tg_problem_destroy), into which the
 * kernels also store the depth limits and the result; relaxed calls on one
 * handle from several threads take turns.  Stages past out->S are zero.
 */
size_t tg_compose_relaxed_workspace_bytes(const tg_problem *p, int64_t n_survivors);
tg_status tg_compose_pipeline_relaxed(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                                      const double *d_cost, const uint8_t *d_dmax, const int32_t *island_order,
                                      tg_plan *out, void *d_ws, size_t ws_bytes, tg_stream stream);

/*
 * Composition over every island subset and order (Sec. 5.2 builds the
 * pipeline from any islands, each used at most once; Sec. 6.2 shows that the
 * order in which islands are stacked changes the plan): the island order is
 * searched instead of given.  For each b the plan minimises the bottleneck P,
 * then the fill F at it, over all plans on any ordered subset of islands;
 * across b it minimises T = (m - 1) P + F, ties to the smaller b.  Ties inside
 * a b go to the least first island id, then fewer stages, then the least set
 * of islands (as a bit mask, island k = bit k), then the earliest cut, then
 * the least next island id, stage by stage.  The set dynamic program has
 * K 2^(K-1) states per first layer and b, so K <= 16 (TG_EINVAL otherwise,
 * and the workspace query returns 0); at most 65535 distinct b.  List
 * requirements, scores and errors as for tg_compose_pipeline (no island
 * order).  d_ws: at least tg_compose_all_orders_workspace_bytes(p,
 * n_survivors) bytes, about nb K 2^(K-1) (3L + 8) bytes for the argmin and
 * root tables plus two level buffers.  Synchronises the stream once.
 */
size_t tg_compose_all_orders_workspace_bytes(const tg_problem *p, int64_t n_survivors);
tg_status tg_compose_pipeline_all_orders(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                                         const double *d_cost, const uint8_t *d_dmax, tg_plan *out, void *d_ws,
                                         size_t ws_bytes, tg_stream stream);

/*
 * Island construction (Sec. 4.1): groups the nodes of a cluster into GPU
 * islands that a homogeneous parallelizer accepts, the input of
 * tg_problem_create.  nodes (host, n_nodes entries in [1, 4096]): one
 * tg_island per node, its n_gpus the GPUs of the node and the other fields
 * per GPU as for islands.  node_bw (host, n_nodes x n_nodes, row = source
 * node, finite and >= 0; the diagonal is ignored): bytes/s between nodes.
 * eps_compute, eps_memory, eps_intra (finite, >= 0): the tolerances of Eq. 1
 * (compute, memory) and Eq. 2 (intra-node bandwidth).
 *   An island holds nodes with the same GPU count whose compute, memory and
 * intra-node bandwidth differ pairwise by at most a factor 1 + eps, and every
 * member's links to the other members are at least as fast as its links to
 * any node outside (Eq. 3).  Steps (1)-(2) split the nodes by GPU count, then
 * compute, memory and intra-node bandwidth, each split a sweep over ascending
 * values (ties by node index) that opens a new group at the first value
 * above the group's smallest times (1 + eps), each operation one binary64
 * rounding.  Step (3) runs agglomerative clustering inside each group: take
 * the pair of clusters with the highest complete linkage (least bandwidth
 * over their node pairs, each pair counted by its slower direction), ties to
 * the least pair of smallest node indices; merge it if the union satisfies
 * Eq. 3 against every node outside it, else set the pair aside until one of
 * its clusters grows; stop when no pair is left.
 *   Outputs (host): island_of[n_nodes] the island of each node, islands
 * numbered by their smallest node index; islands[K] (capacity n_nodes) with
 * n_gpus the sum over members and the other fields the least over members;
 * inter_bw[K * K] (capacity n_nodes^2, row-major) the least node-to-node
 * bandwidth from island a to island b, 0 on the diagonal; *n_islands = K.
 * d_ws: at least tg_build_islands_workspace_bytes(n_nodes) device bytes
 * (about 29 n_nodes^2).  Synchronises the stream.
 */
size_t tg_build_islands_workspace_bytes(int32_t n_nodes);
tg_status tg_build_islands(const tg_island *nodes, int32_t n_nodes, const double *node_bw, double eps_compute,
                           double eps_memory, double eps_intra, int32_t *island_of, tg_island *islands,
                           double *inter_bw, int32_t *n_islands, void *d_ws, size_t ws_bytes, tg_stream stream);

/* Message of the calling thread's last failed call ("" if none). */
const char *tg_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* TANGRAM_H */
