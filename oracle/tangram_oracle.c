/*
 * tangram_oracle.c -- plain, slow, single-threaded CPU oracle for the
 * model-slice / GPU-island plan search of Tangram (arXiv 2606.16907).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this file's library.  It shares no code,
 * header, table or constant generator with the HIP library; the two are
 * written separately from the same definitions.
 *
 * What it computes (every quantity is a plain definition written out):
 *   1. the candidate space: every contiguous layer range [i, j) ("model slice",
 *      Sec. 4.2) times every island (Sec. 4.1) times every intra-island config
 *      (tp, context-parallel degree cp, dp, ep, zero stage, activation
 *      recomputation, activation offloading, micro-batch) -- the
 *      model-slice/island pairs that Sec. 5.1 enumerates and hands to a
 *      homogeneous parallelizer, with the parallelisms and memory-saving
 *      techniques of Sec. 2.1;
 *   2. per candidate an analytic step-time cost and the deepest 1F1B pipeline
 *      position it fits at (Sec. 5.2: memory depends on the stage's position,
 *      a plan is reused "until it is no longer feasible");
 *   3. pruning (Sec. 5.1 infeasibility pruning, the incompatibility pruning of
 *      the contributions and of the Fig. 12 ablation, and dominance): the
 *      surviving set;
 *   4. pipeline composition (Sec. 5.2, steps (1)-(3) of the composition
 *      algorithm): lowest bottleneck first, then lowest fill at that bottleneck,
 *      islands used at most once and possibly eliminated.
 * The paper delegates the cost model to the parallelizer's profile() and
 * parallelize() (Tab. 2); the analytic model below is this project's stated
 * reading of it.  Floating point is IEEE binary64, each operation rounded once
 * in the parenthesised order written here; build with -ffp-contract=off.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define TGO_OK 0
#define TGO_EINVAL (-1)
#define TGO_ENOMEM (-2)
#define TGO_ECAPACITY (-4)
#define TGO_ENOPLAN (-5)

#define NF 8 /* per-layer fields */
enum { F_FLOPS = 0, F_DPARAM, F_EPARAM, F_ACT, F_TPCOMM, F_A2A, F_OUTACT, F_CPCOMM };
#define NSUM 8 /* slice sums: flops, dparam, eparam, act, tpcomm, a2a, outact, cpcomm */

typedef struct {
    int32_t island, first_layer, end_layer, tp, cp, dp, ep, zero, recompute, offload, mb, depth;
    int64_t pair_index;
    double cost, mem_bytes, link_out;
} tgo_stage;

typedef struct {
    int32_t status, b, m, S;
    double P, F, T;
    tgo_stage stage[255];
} tgo_plan;

typedef struct {
    int k, tp, cp, dp, ep, z, rc, of, mb;
    int64_t b;
} ocfg;

typedef struct {
    int L, K;
    int64_t *layer[NF]; /* [f][L] */
    int32_t *n_gpus;
    double *peak, *hbm, *intra, *host, *inter; /* inter: K*K row-major */
    int64_t B;
    int n_experts;
    int ntp, tp[8], ncp, cp[8], nep, ep[8], nmb, mb[8], nz, zs[4], nrc, rcs[2], nof, ofs[2];
    double eta, mem_frac;
    double imb_eps; /* imbalance-pruning tolerance, 0 = off */
    /* derived */
    int64_t NS, ncfg, N;
    int64_t *cfg_off; /* K+1 */
    ocfg *cfg;        /* ncfg */
    int64_t *slice_sum; /* NS x 6: flops, dparam, eparam, act, tpcomm, a2a */
    int nb;
    int64_t *bvals; /* distinct compatible b, ascending */
    double *cap_share; /* [K] island's share of the cluster's compute */
} oprob;

/* ------------------------------------------------------------------------ */
/* slices: s enumerates 0 <= i < j <= L lexicographically (i, then j)       */
/* ------------------------------------------------------------------------ */
static int64_t slice_index(int L, int i, int j) {
    /* number of slices with first layer < i, plus the offset of j */
    int64_t before = 0;
    for (int a = 0; a < i; a++) before += (int64_t)(L - a);
    return before + (int64_t)(j - i - 1);
}

static void slice_ij(int L, int64_t s, int *pi, int *pj) {
    int i = 0;
    while (s >= (int64_t)(L - i)) { s -= (int64_t)(L - i); i++; }
    *pi = i;
    *pj = i + 1 + (int)s;
}

/* ------------------------------------------------------------------------ */
/* configs of one island: lexicographic (tp, cp, dp, ep, z, rc, of, mb)      */
/* ------------------------------------------------------------------------ */
static int ep_admissible(const oprob *p, int ep, int dp) {
    if (dp % ep != 0) return 0;
    if (p->n_experts == 0) return ep == 1;
    return p->n_experts % ep == 0;
}

/* A config uses tp * cp * dp <= n GPUs of the island; offloading needs a
   host link (host bandwidth > 0). */
static int64_t island_configs(const oprob *p, int k, ocfg *out) {
    int64_t c = 0;
    int n = p->n_gpus[k];
    for (int a = 0; a < p->ntp; a++) {
        int tp = p->tp[a];
        if (tp > n) continue;
        for (int ci = 0; ci < p->ncp; ci++) {
            int cp = p->cp[ci];
            if ((int64_t)tp * cp > n) continue;
            int q = tp * cp;
            for (int dp = 1; dp <= n / q; dp++)
                for (int e = 0; e < p->nep; e++) {
                    if (!ep_admissible(p, p->ep[e], dp)) continue;
                    for (int zi = 0; zi < p->nz; zi++)
                        for (int ri = 0; ri < p->nrc; ri++)
                            for (int oi = 0; oi < p->nof; oi++) {
                                if (p->ofs[oi] && !(p->host[k] > 0.0)) continue;
                                for (int mi = 0; mi < p->nmb; mi++) {
                                    if (out) {
                                        ocfg *g = &out[c];
                                        g->k = k; g->tp = tp; g->cp = cp; g->dp = dp; g->ep = p->ep[e];
                                        g->z = p->zs[zi]; g->rc = p->rcs[ri]; g->of = p->ofs[oi];
                                        g->mb = p->mb[mi];
                                        g->b = (int64_t)dp * (int64_t)p->mb[mi];
                                    }
                                    c++;
                                }
                            }
                }
        }
    }
    return c;
}

static int strictly_ascending_pos(const int32_t *v, int n) {
    if (n < 1 || n > 8) return 0;
    for (int a = 0; a < n; a++) {
        if (v[a] < 1) return 0;
        if (a > 0 && v[a] <= v[a - 1]) return 0;
    }
    return 1;
}

static int cmp_i64(const void *a, const void *b) {
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return (x > y) - (x < y);
}

void tgo_destroy(void *h) {
    oprob *p = (oprob *)h;
    if (!p) return;
    for (int f = 0; f < NF; f++) free(p->layer[f]);
    free(p->n_gpus); free(p->peak); free(p->hbm); free(p->intra); free(p->host); free(p->inter);
    free(p->cfg_off); free(p->cfg); free(p->slice_sum); free(p->bvals); free(p->cap_share);
    free(p);
}

/* layers: NF*L int64, field-major (all fwd_flops, then dense_params, ...).
   cp: context-parallel degrees (ncp = 0 means {1}); rc_mask / of_mask: bit r
   admits recomputation / offloading option r (0 means {off}).  imb_eps: the
   imbalance-pruning tolerance (0 = off; otherwise finite and > 0). */
int tgo_create(const int64_t *layers, int L, const int32_t *n_gpus, const double *peak,
               const double *hbm, const double *intra, const double *host_bw, int K, const double *inter,
               int64_t global_batch, int n_experts, const int32_t *tp, int ntp,
               const int32_t *cp, int ncp, const int32_t *ep, int nep, const int32_t *mb, int nmb,
               uint32_t zero_mask, uint32_t rc_mask, uint32_t of_mask, double eta, double mem_frac,
               double imb_eps, void **out) {
    *out = NULL;
    if (L < 1 || L > 512 || K < 1 || K > 255) return TGO_EINVAL;
    if (global_batch < 1 || n_experts < 0) return TGO_EINVAL;
    if (!strictly_ascending_pos(tp, ntp) || !strictly_ascending_pos(ep, nep) ||
        !strictly_ascending_pos(mb, nmb) || (ncp != 0 && !strictly_ascending_pos(cp, ncp)))
        return TGO_EINVAL;
    if (zero_mask == 0 || (zero_mask & ~0xFu)) return TGO_EINVAL;
    if ((rc_mask & ~0x3u) || (of_mask & ~0x3u)) return TGO_EINVAL;
    if (!(eta > 0.0) || !isfinite(eta) || !(mem_frac > 0.0) || !isfinite(mem_frac))
        return TGO_EINVAL;
    if (!(imb_eps >= 0.0) || !isfinite(imb_eps)) return TGO_EINVAL;
    for (int k = 0; k < K; k++) {
        if (n_gpus[k] < 1 || n_gpus[k] > (1 << 28)) return TGO_EINVAL; /* any island built from nodes */
        if (!(peak[k] > 0.0) || !isfinite(peak[k])) return TGO_EINVAL;
        if (!(hbm[k] > 0.0) || !isfinite(hbm[k])) return TGO_EINVAL;
        if (!(intra[k] > 0.0) || !isfinite(intra[k])) return TGO_EINVAL;
        if (!(host_bw[k] >= 0.0) || !isfinite(host_bw[k])) return TGO_EINVAL;
    }
    for (int a = 0; a < K * K; a++)
        if (!(inter[a] >= 0.0)) return TGO_EINVAL; /* rejects NaN and negatives; +inf allowed */
    /* every layer value >= 0 and every whole-model sum < 2^62 */
    for (int f = 0; f < NF; f++) {
        int64_t acc = 0;
        for (int l = 0; l < L; l++) {
            int64_t v = layers[(int64_t)f * L + l];
            if (v < 0 || v >= ((int64_t)1 << 62) - acc) return TGO_EINVAL;
            acc += v;
        }
    }

    oprob *p = (oprob *)calloc(1, sizeof(oprob));
    if (!p) return TGO_ENOMEM;
    p->L = L; p->K = K;
    for (int f = 0; f < NF; f++) {
        p->layer[f] = (int64_t *)malloc(sizeof(int64_t) * L);
        memcpy(p->layer[f], layers + (int64_t)f * L, sizeof(int64_t) * L);
    }
    p->n_gpus = (int32_t *)malloc(sizeof(int32_t) * K);
    p->peak = (double *)malloc(sizeof(double) * K);
    p->hbm = (double *)malloc(sizeof(double) * K);
    p->intra = (double *)malloc(sizeof(double) * K);
    p->host = (double *)malloc(sizeof(double) * K);
    p->inter = (double *)malloc(sizeof(double) * K * K);
    memcpy(p->n_gpus, n_gpus, sizeof(int32_t) * K);
    memcpy(p->peak, peak, sizeof(double) * K);
    memcpy(p->hbm, hbm, sizeof(double) * K);
    memcpy(p->intra, intra, sizeof(double) * K);
    memcpy(p->host, host_bw, sizeof(double) * K);
    memcpy(p->inter, inter, sizeof(double) * K * K);
    p->B = global_batch;
    p->n_experts = n_experts;
    p->ntp = ntp; memcpy(p->tp, tp, sizeof(int32_t) * ntp);
    if (ncp == 0) { p->ncp = 1; p->cp[0] = 1; }
    else { p->ncp = ncp; memcpy(p->cp, cp, sizeof(int32_t) * ncp); }
    p->nep = nep; memcpy(p->ep, ep, sizeof(int32_t) * nep);
    p->nmb = nmb; memcpy(p->mb, mb, sizeof(int32_t) * nmb);
    p->nz = 0;
    for (int z = 0; z < 4; z++)
        if (zero_mask & (1u << z)) p->zs[p->nz++] = z;
    p->nrc = 0;
    for (int r = 0; r < 2; r++)
        if ((rc_mask ? rc_mask : 1u) & (1u << r)) p->rcs[p->nrc++] = r;
    p->nof = 0;
    for (int r = 0; r < 2; r++)
        if ((of_mask ? of_mask : 1u) & (1u << r)) p->ofs[p->nof++] = r;
    p->eta = eta;
    p->mem_frac = mem_frac;
    p->imb_eps = imb_eps;
    /* an island's compute capacity is n_k F_k; its share of the cluster's is
       the capacity over the sum of all islands' (summed in island order) */
    p->cap_share = (double *)malloc(sizeof(double) * K);
    double cap_sum = 0.0;
    for (int k = 0; k < K; k++) cap_sum = cap_sum + ((double)n_gpus[k] * peak[k]);
    for (int k = 0; k < K; k++) p->cap_share[k] = ((double)n_gpus[k] * peak[k]) / cap_sum;

    p->NS = (int64_t)L * (L + 1) / 2;
    p->cfg_off = (int64_t *)malloc(sizeof(int64_t) * (K + 1));
    p->cfg_off[0] = 0;
    for (int k = 0; k < K; k++) p->cfg_off[k + 1] = p->cfg_off[k] + island_configs(p, k, NULL);
    p->ncfg = p->cfg_off[K];
    p->N = p->ncfg * p->NS;
    p->cfg = (ocfg *)malloc(sizeof(ocfg) * (p->ncfg > 0 ? p->ncfg : 1));
    for (int k = 0; k < K; k++) island_configs(p, k, p->cfg + p->cfg_off[k]);

    /* Slice sums by running accumulation over the layers of [i, j) (the
       "concatenate" of Tab. 2 for integer per-layer quantities). */
    p->slice_sum = (int64_t *)malloc(sizeof(int64_t) * NSUM * p->NS);
    const int fmap[NSUM] = {F_FLOPS, F_DPARAM, F_EPARAM, F_ACT, F_TPCOMM, F_A2A, F_OUTACT, F_CPCOMM};
    int64_t s = 0;
    for (int i = 0; i < L; i++) {
        int64_t acc[NSUM] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int j = i + 1; j <= L; j++, s++)
            for (int q = 0; q < NSUM; q++) {
                acc[q] += p->layer[fmap[q]][j - 1];
                p->slice_sum[s * NSUM + q] = acc[q];
            }
    }

    /* distinct compatible micro-batch sizes b = dp * mb with B mod b == 0 */
    p->bvals = (int64_t *)malloc(sizeof(int64_t) * (p->ncfg > 0 ? p->ncfg : 1));
    int64_t nb = 0;
    for (int64_t g = 0; g < p->ncfg; g++) {
        int64_t b = p->cfg[g].b;
        if (p->B % b != 0) continue;
        int seen = 0;
        for (int64_t a = 0; a < nb; a++) if (p->bvals[a] == b) { seen = 1; break; }
        if (!seen) p->bvals[nb++] = b;
    }
    if (nb > 0) qsort(p->bvals, (size_t)nb, sizeof(int64_t), cmp_i64);
    p->nb = (int)nb;
    /* a plan reports b and m = B / b as 32-bit integers */
    if (nb > 0 && (p->bvals[nb - 1] > INT32_MAX || p->B / p->bvals[0] > INT32_MAX)) {
        tgo_destroy(p);
        return TGO_EINVAL;
    }
    *out = p;
    return TGO_OK;
}

int tgo_counts(void *h, int64_t *out) {
    oprob *p = (oprob *)h;
    out[0] = p->NS; out[1] = p->ncfg; out[2] = p->N; out[3] = p->nb;
    return TGO_OK;
}

int tgo_bvalues(void *h, int64_t *out) {
    oprob *p = (oprob *)h;
    for (int a = 0; a < p->nb; a++) out[a] = p->bvals[a];
    return p->nb;
}

/* idx = (cfg_off[k] + c) * NS + s  ->  (i, j, k, tp, cp, dp, ep, z, rc, of, mb) */
int tgo_decode(void *h, int64_t idx, int32_t *out) {
    oprob *p = (oprob *)h;
    if (idx < 0 || idx >= p->N) return TGO_EINVAL;
    int64_t g = idx / p->NS, s = idx % p->NS;
    int i, j;
    slice_ij(p->L, s, &i, &j);
    const ocfg *c = &p->cfg[g];
    out[0] = i; out[1] = j; out[2] = c->k; out[3] = c->tp; out[4] = c->cp; out[5] = c->dp;
    out[6] = c->ep; out[7] = c->z; out[8] = c->rc; out[9] = c->of; out[10] = c->mb;
    return TGO_OK;
}

/* ------------------------------------------------------------------------ */
/* cost model (stated reading of profile()/parallelize(), Tab. 2)            */
/* ------------------------------------------------------------------------ */
typedef struct {
    double alpha, beta, gamma, delta_d, delta_e, mu_d, mu_e, rho, H, m_real, kappa, omega;
    int rc, of;
} ocoef;

/* ring collectives over D GPUs move (D-1)/D of the data per phase */
static double ring_r(int64_t D) { return (double)(D - 1) / (double)D; }

/* bf16 bytes per parameter moved once per micro-batch for data-parallel sync */
static double zero_per_mb(int z, int64_t D) {
    if (z <= 1) return 0.0;            /* grads all-reduced once per iteration */
    if (z == 2) return 2.0 * ring_r(D); /* reduce-scatter of grads every micro-batch */
    return 6.0 * ring_r(D);             /* ZeRO-3: all-gather fwd + all-gather bwd + RS */
}

/* bf16 bytes per parameter moved once per iteration */
static double zero_per_iter(int z, int64_t D) {
    if (z <= 1) return 4.0 * ring_r(D); /* all-reduce (or RS + AG) of grads */
    if (z == 2) return 2.0 * ring_r(D); /* all-gather of updated params */
    return 0.0;
}

/* model-state bytes per parameter: bf16 param + bf16 grad + fp32 master/m/v */
static double state_bytes(int z, int64_t D) {
    if (z == 0) return 16.0;
    if (z == 1) return 4.0 + 12.0 / (double)D;
    if (z == 2) return 2.0 + 14.0 / (double)D;
    return 16.0 / (double)D;
}

static void config_coef(const oprob *p, const ocfg *c, ocoef *o) {
    double Fk = p->peak[c->k], Wk = p->intra[c->k], Mk = p->hbm[c->k], Hk = p->host[c->k];
    /* the data-parallel group (gradient sync, ZeRO sharding) spans the dp
       replicas and the cp ranks of each, which hold the same parameters */
    int64_t Dd = (int64_t)c->dp * c->cp, De = (int64_t)(c->dp / c->ep) * c->cp;
    double qd = (double)c->tp, qe = (double)((int64_t)c->tp * c->ep);
    int64_t q = (int64_t)c->tp * c->cp; /* GPUs sharing one micro-batch's tokens */
    /* forward passes over the data: forward, recomputed forward, backward
       (= 2 forwards) for compute; forward, recompute, backward for the
       collectives issued in the forward pass */
    double nc = c->rc ? 4.0 : 3.0;
    int nt = c->rc ? 3 : 2;
    o->rc = c->rc;
    o->of = c->of;
    o->m_real = (double)p->B / (double)c->b;
    /* compute, split over the tp * cp GPUs of a replica */
    o->alpha = (nc * (double)c->mb) / (((double)q * Fk) * p->eta);
    /* ring all-reduce-equivalent TP collectives, 2(t-1)/t per pass, tokens
       split by cp */
    o->beta = c->tp > 1 ? (((double)(2 * nt) * (double)c->mb) * (double)(c->tp - 1)) / ((double)q * Wk) : 0.0;
    /* all-to-all per pass, (e-1)/e leaves the GPU, tokens split by tp and cp */
    o->gamma = c->ep > 1
                   ? (((double)nt * (double)c->mb) * (double)(c->ep - 1)) / (((double)c->ep * (double)q) * Wk)
                   : 0.0;
    /* ring attention over cp ranks: each receives the other (cp-1)/cp of the
       keys and values (heads split by tp), once forward and twice backward
       (keys/values and their gradients), plus once more when recomputing */
    o->kappa = c->cp > 1
                   ? (((double)(nt + 1) * (double)c->mb) * (double)(c->cp - 1)) / (((double)c->cp * (double)c->tp) * Wk)
                   : 0.0;
    o->delta_d = ((zero_per_mb(c->z, Dd) / qd) / Wk) + (((zero_per_iter(c->z, Dd) / qd) / Wk) / o->m_real);
    o->delta_e = ((zero_per_mb(c->z, De) / qe) / Wk) + (((zero_per_iter(c->z, De) / qe) / Wk) / o->m_real);
    o->mu_d = state_bytes(c->z, Dd) / qd;
    o->mu_e = state_bytes(c->z, De) / qe;
    /* stashed activations per GPU: sequence split by tp (sequence
       parallelism) and cp */
    o->rho = (double)c->mb / (double)q;
    /* offloading: the stash goes to host memory after the forward pass and
       comes back before the backward pass */
    o->omega = c->of ? (2.0 * (double)c->mb) / ((double)q * Hk) : 0.0;
    o->H = Mk * p->mem_frac;
}

/* 1F1B: a stage with d stages at or after it holds min(d, m) micro-batches of
   stashed activations (Sec. 5.2: memory depends on the pipeline position).
   With offloading only the micro-batch being computed stays on the device,
   at every depth. */
static int fits(double state, double A1, double H, double m_real, int d, int of) {
    double dd = of ? 1.0 : (double)d;
    double inflight = dd < m_real ? dd : m_real;
    return (state + (inflight * A1)) <= H;
}

static void score_candidate(const oprob *p, const ocoef *o, const int64_t *sum, double *cost,
                            int *dmax, double *state_out, double *A1_out) {
    double Fl = (double)sum[0], Pd = (double)sum[1], Pe = (double)sum[2];
    double Act = (double)sum[3], Tb = (double)sum[4], Ab = (double)sum[5];
    double Oa = (double)sum[6], Cb = (double)sum[7];
    /* with recomputation only each layer's boundary activation (its output)
       is stashed; the rest is recomputed in the backward pass */
    double S = o->rc ? Oa : Act;
    double c = o->alpha * Fl;
    c = c + (o->beta * Tb);
    c = c + (o->gamma * Ab);
    c = c + (o->delta_d * Pd);
    c = c + (o->delta_e * Pe);
    c = c + (o->kappa * Cb);
    c = c + (o->omega * S);
    double state = (o->mu_d * Pd) + (o->mu_e * Pe);
    double A1 = o->rho * S;
    /* d_max = largest d in 1..K that fits, 0 if none.  fits() is monotone in d
       (min(d, m) and each rounded operation are non-decreasing), so a binary
       search over d finds exactly the largest fitting depth. */
    int lo = 0, hi = p->K; /* invariant: fits(lo) or lo == 0; !fits(hi+1) */
    while (lo < hi) {
        int mid = lo + (hi - lo + 1) / 2;
        if (fits(state, A1, o->H, o->m_real, mid, o->of)) lo = mid; else hi = mid - 1;
    }
    *cost = c;
    *dmax = lo;
    if (state_out) *state_out = state;
    if (A1_out) *A1_out = A1;
}

int tgo_coef(void *h, int64_t g, double *out /* 12 */) {
    oprob *p = (oprob *)h;
    if (g < 0 || g >= p->ncfg) return TGO_EINVAL;
    ocoef o;
    config_coef(p, &p->cfg[g], &o);
    out[0] = o.alpha; out[1] = o.beta; out[2] = o.gamma; out[3] = o.delta_d; out[4] = o.delta_e;
    out[5] = o.mu_d; out[6] = o.mu_e; out[7] = o.rho; out[8] = o.H; out[9] = o.m_real;
    out[10] = o.kappa; out[11] = o.omega;
    return TGO_OK;
}

int tgo_score(void *h, int64_t first, int64_t count, double *cost, uint8_t *dmax) {
    oprob *p = (oprob *)h;
    if (first < 0 || count < 0 || first > p->N || count > p->N - first) return TGO_EINVAL;
    int64_t prev_g = -1;
    ocoef o;
    for (int64_t t = 0; t < count; t++) {
        int64_t idx = first + t, g = idx / p->NS, s = idx % p->NS;
        if (g != prev_g) { config_coef(p, &p->cfg[g], &o); prev_g = g; }
        int dm;
        score_candidate(p, &o, &p->slice_sum[s * NSUM], &cost[t], &dm, NULL, NULL);
        dmax[t] = (uint8_t)dm;
    }
    return TGO_OK;
}

/* score an arbitrary list of candidate indices */
int tgo_score_list(void *h, const int64_t *idx, int64_t n, double *cost, uint8_t *dmax) {
    oprob *p = (oprob *)h;
    for (int64_t t = 0; t < n; t++) {
        if (idx[t] < 0 || idx[t] >= p->N) return TGO_EINVAL;
        int64_t g = idx[t] / p->NS, s = idx[t] % p->NS;
        ocoef o;
        config_coef(p, &p->cfg[g], &o);
        int dm;
        score_candidate(p, &o, &p->slice_sum[s * NSUM], &cost[t], &dm, NULL, NULL);
        dmax[t] = (uint8_t)dm;
    }
    return TGO_OK;
}

/* ------------------------------------------------------------------------ */
/* imbalance pruning (Sec. 5.1 (ii))                                         */
/* ------------------------------------------------------------------------ */
/* A slice demands its share q of the model's forward FLOPs; an island offers
   its share c of the cluster's compute.  With tolerance eps the pair is kept
   iff q <= c (1 + eps) (the island does not stall) and q (1 + eps) >= c (it is
   not left underused).  Off when eps = 0 or the model has no FLOPs. */
static int balanced(const oprob *p, int64_t s, int k) {
    if (p->imb_eps == 0.0) return 1;
    int64_t total = p->slice_sum[slice_index(p->L, 0, p->L) * NSUM + 0];
    if (total == 0) return 1;
    double q = (double)p->slice_sum[s * NSUM + 0] / (double)total;
    double r = 1.0 + p->imb_eps;
    double c = p->cap_share[k];
    return q <= c * r && q * r >= c;
}

int tgo_balanced(void *h, int64_t s, int k) {
    oprob *p = (oprob *)h;
    if (s < 0 || s >= p->NS || k < 0 || k >= p->K) return -1;
    return balanced(p, s, k);
}

/* ------------------------------------------------------------------------ */
/* pruning: the surviving set                                                */
/* ------------------------------------------------------------------------ */
/* A group is (slice, island, b).  Preference key (cost, -d_max, idx) ascending.
   rep(G, d) = min-key member with d_max >= d; the surviving set is the union of
   rep(G, d) over d = 1..K.  Equivalently p survives iff p is compatible,
   d_max_p >= 1 and no member q has key_q < key_p with d_max_q >= d_max_p, i.e.
   d_max_p exceeds the largest d_max among all members preceding p in key
   order.  Sorting by key and sweeping a running maximum evaluates exactly that.
   With imbalance pruning on, groups of unbalanced (slice, island) pairs have
   no survivors. */
typedef struct {
    double cost;
    int dmax;
    int64_t idx;
} omember;

static int cmp_key(const void *a, const void *b) {
    const omember *x = (const omember *)a, *y = (const omember *)b;
    if (x->cost < y->cost) return -1;
    if (x->cost > y->cost) return 1;
    if (x->dmax > y->dmax) return -1;
    if (x->dmax < y->dmax) return 1;
    return (x->idx > y->idx) - (x->idx < y->idx);
}

typedef struct {
    int64_t *v;
    int64_t n, cap;
} ivec;

static int ivec_push(ivec *a, int64_t x) {
    if (a->n == a->cap) {
        int64_t nc = a->cap ? a->cap * 2 : 1024;
        int64_t *nv = (int64_t *)realloc(a->v, sizeof(int64_t) * nc);
        if (!nv) return TGO_ENOMEM;
        a->v = nv; a->cap = nc;
    }
    a->v[a->n++] = x;
    return TGO_OK;
}

int tgo_prune(void *h, int64_t *out, int64_t cap, int64_t *n_out) {
    oprob *p = (oprob *)h;
    ivec surv = {0, 0, 0};
    int64_t maxc = 0;
    for (int k = 0; k < p->K; k++)
        if (p->cfg_off[k + 1] - p->cfg_off[k] > maxc) maxc = p->cfg_off[k + 1] - p->cfg_off[k];
    omember *mem = (omember *)malloc(sizeof(omember) * (maxc > 0 ? maxc : 1));
    ocoef *coef = (ocoef *)malloc(sizeof(ocoef) * (maxc > 0 ? maxc : 1));
    int64_t *members = (int64_t *)malloc(sizeof(int64_t) * (maxc > 0 ? maxc : 1));
    for (int k = 0; k < p->K; k++) {
        int64_t c0 = p->cfg_off[k], nc = p->cfg_off[k + 1] - c0;
        for (int64_t c = 0; c < nc; c++) config_coef(p, &p->cfg[c0 + c], &coef[c]);
        for (int bi = 0; bi < p->nb; bi++) {
            int64_t b = p->bvals[bi];
            /* the group's members: configs of island k with this b */
            int64_t nm = 0;
            for (int64_t c = 0; c < nc; c++)
                if (p->cfg[c0 + c].b == b) members[nm++] = c;
            if (nm == 0) continue;
            for (int64_t s = 0; s < p->NS; s++) {
                if (!balanced(p, s, k)) continue;
                int64_t n = 0;
                for (int64_t a = 0; a < nm; a++) {
                    int64_t c = members[a];
                    omember *m = &mem[n++];
                    score_candidate(p, &coef[c], &p->slice_sum[s * NSUM], &m->cost, &m->dmax, NULL, NULL);
                    m->idx = (c0 + c) * p->NS + s;
                }
                qsort(mem, (size_t)n, sizeof(omember), cmp_key);
                int run = 0;
                for (int64_t a = 0; a < n; a++)
                    if (mem[a].dmax > run) {
                        if (ivec_push(&surv, mem[a].idx) != TGO_OK) {
                            free(mem); free(coef); free(members); free(surv.v);
                            return TGO_ENOMEM;
                        }
                        run = mem[a].dmax;
                    }
            }
        }
    }
    free(mem);
    free(coef);
    free(members);
    if (surv.n > 0) qsort(surv.v, (size_t)surv.n, sizeof(int64_t), cmp_i64); /* no set: no array */
    *n_out = surv.n;
    int rc = TGO_OK;
    if (surv.n > cap) rc = TGO_ECAPACITY;
    else if (out && surv.n > 0) memcpy(out, surv.v, sizeof(int64_t) * surv.n);
    free(surv.v);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* redundancy pruning (Sec. 5.1 (i))                                         */
/* ------------------------------------------------------------------------ */
/* Slices with the same composition are the same work: here two slices are
   equivalent when all eight of their per-slice sums are equal, so every
   config scores them alike (the score reads nothing else of the slice).
   Classes are numbered in the order of their first slice. */
static const int64_t *cls_sums = NULL;

static int cmp_slice_sums(const void *a, const void *b) {
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    for (int q = 0; q < NSUM; q++) {
        int64_t u = cls_sums[x * NSUM + q], v = cls_sums[y * NSUM + q];
        if (u != v) return u < v ? -1 : 1;
    }
    return (x > y) - (x < y);
}

int tgo_slice_classes(void *h, int32_t *cls, int64_t *n_classes) {
    oprob *p = (oprob *)h;
    const int64_t NS = p->NS;
    int64_t *ord = (int64_t *)malloc(sizeof(int64_t) * NS);
    int64_t *first = (int64_t *)malloc(sizeof(int64_t) * NS);
    for (int64_t s = 0; s < NS; s++) ord[s] = s;
    cls_sums = p->slice_sum;
    qsort(ord, (size_t)NS, sizeof(int64_t), cmp_slice_sums);
    /* first[s] = the smallest slice with the same sums as s (runs of equal
       sums are sorted by slice index, so a run's head is its smallest) */
    int64_t head = 0;
    for (int64_t t = 0; t < NS; t++) {
        if (t == 0 ||
            memcmp(&p->slice_sum[ord[t - 1] * NSUM], &p->slice_sum[ord[t] * NSUM], sizeof(int64_t) * NSUM) != 0)
            head = ord[t];
        first[ord[t]] = head;
    }
    int64_t nc = 0;
    for (int64_t s = 0; s < NS; s++) {
        if (first[s] == s) cls[s] = (int32_t)nc++;
        else cls[s] = cls[first[s]];
    }
    *n_classes = nc;
    free(ord);
    free(first);
    return TGO_OK;
}

/* The surviving set with redundancy pruning: each group's staircase is found
   once per (island, b, slice class) at the class's first slice, scoring only
   that slice, and copied to the other slices of the class.  Equal to
   tgo_prune's set: a group's members score alike on equivalent slices and
   their candidate indices keep the same order. */
int tgo_prune_classes(void *h, int64_t *out, int64_t cap, int64_t *n_out) {
    oprob *p = (oprob *)h;
    const int64_t NS = p->NS;
    int32_t *cls = (int32_t *)malloc(sizeof(int32_t) * NS);
    int64_t nc = 0;
    tgo_slice_classes(h, cls, &nc);
    int64_t *rep = (int64_t *)malloc(sizeof(int64_t) * (nc > 0 ? nc : 1));
    for (int64_t s = NS - 1; s >= 0; s--) rep[cls[s]] = s; /* first slice of each class */
    ivec surv = {0, 0, 0};
    int64_t maxc = 0;
    for (int k = 0; k < p->K; k++)
        if (p->cfg_off[k + 1] - p->cfg_off[k] > maxc) maxc = p->cfg_off[k + 1] - p->cfg_off[k];
    omember *mem = (omember *)malloc(sizeof(omember) * (maxc > 0 ? maxc : 1));
    ocoef *coef = (ocoef *)malloc(sizeof(ocoef) * (maxc > 0 ? maxc : 1));
    int64_t *members = (int64_t *)malloc(sizeof(int64_t) * (maxc > 0 ? maxc : 1));
    /* kept[c * maxc + a] = member a survives on class c */
    unsigned char *kept = (unsigned char *)malloc((size_t)(nc > 0 ? nc : 1) * (size_t)(maxc > 0 ? maxc : 1));
    for (int k = 0; k < p->K; k++) {
        int64_t c0 = p->cfg_off[k], nc0 = p->cfg_off[k + 1] - c0;
        for (int64_t c = 0; c < nc0; c++) config_coef(p, &p->cfg[c0 + c], &coef[c]);
        for (int bi = 0; bi < p->nb; bi++) {
            int64_t b = p->bvals[bi];
            int64_t nm = 0;
            for (int64_t c = 0; c < nc0; c++)
                if (p->cfg[c0 + c].b == b) members[nm++] = c;
            if (nm == 0) continue;
            for (int64_t q = 0; q < nc; q++) {
                int64_t s = rep[q];
                for (int64_t a = 0; a < nm; a++) kept[q * maxc + a] = 0;
                if (!balanced(p, s, k)) continue;
                for (int64_t a = 0; a < nm; a++) {
                    omember *m = &mem[a];
                    score_candidate(p, &coef[members[a]], &p->slice_sum[s * NSUM], &m->cost, &m->dmax, NULL, NULL);
                    m->idx = a; /* member order = candidate index order on every slice */
                }
                qsort(mem, (size_t)nm, sizeof(omember), cmp_key);
                int run = 0;
                for (int64_t a = 0; a < nm; a++)
                    if (mem[a].dmax > run) { kept[q * maxc + mem[a].idx] = 1; run = mem[a].dmax; }
            }
            for (int64_t s = 0; s < NS; s++)
                for (int64_t a = 0; a < nm; a++)
                    if (kept[(int64_t)cls[s] * maxc + a] &&
                        ivec_push(&surv, (c0 + members[a]) * NS + s) != TGO_OK) {
                        free(mem); free(coef); free(members); free(kept); free(cls); free(rep); free(surv.v);
                        return TGO_ENOMEM;
                    }
        }
    }
    free(mem); free(coef); free(members); free(kept); free(cls); free(rep);
    if (surv.n > 0) qsort(surv.v, (size_t)surv.n, sizeof(int64_t), cmp_i64); /* no set: no array */
    *n_out = surv.n;
    int rc = TGO_OK;
    if (surv.n > cap) rc = TGO_ECAPACITY;
    else if (out && surv.n > 0) memcpy(out, surv.v, sizeof(int64_t) * surv.n);
    free(surv.v);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* composition (Sec. 5.2)                                                    */
/* ------------------------------------------------------------------------ */
/* An entry is one usable candidate of the list handed to composition. */
typedef struct {
    int64_t gkey; /* (b_index * NS + s) * K + position of the island */
    double cost;
    int dmax;
    int64_t idx;
} oentry;

static int cmp_entry(const void *a, const void *b) {
    const oentry *x = (const oentry *)a, *y = (const oentry *)b;
    if (x->gkey != y->gkey) return (x->gkey > y->gkey) - (x->gkey < y->gkey);
    if (x->cost < y->cost) return -1;
    if (x->cost > y->cost) return 1;
    if (x->dmax > y->dmax) return -1;
    if (x->dmax < y->dmax) return 1;
    return (x->idx > y->idx) - (x->idx < y->idx);
}

static double maxd(double a, double b) { return a > b ? a : b; }

/* Activation transfer across boundary j (after layer j-1) from island ka to
   island kb: forward activations and backward gradients of one micro-batch of
   b samples, over the inter-island link (Sec. 5.2: PP only moves stage
   inputs and outputs).  No link (bandwidth 0) is unusable. */
static double transfer(const oprob *p, int64_t b, int j, int ka, int kb) {
    double E = p->inter[(int64_t)ka * p->K + kb];
    if (E == 0.0) return INFINITY;
    return ((2.0 * (double)b) * (double)p->layer[F_OUTACT][j - 1]) / E;
}

/* Working tables of one b during composition. */
typedef struct {
    const oprob *p;
    const int32_t *order;
    int L, K, D;
    int64_t NS;
    const oentry *ent;
    int64_t *gstart, *gend; /* [NS*K] entry range of each (slice, position) group */
    double *V, *Wt;         /* [D+1][L+1][K]: V/W in step (1)-(2), F/G in step (3) */
    double *Td;             /* [D+1][NS][K] stage table by depth */
    double *X;              /* [L+1][K][K] link times */
    int64_t b, m;
} octx;

#define AT(A, d, i, o) A[((int64_t)(d) * (c->L + 1) + (i)) * c->K + (o)]
#define TD(d, s, o) c->Td[((int64_t)(d) * c->NS + (s)) * c->K + (o)]
#define XA(j, o, o2) c->X[((int64_t)(j) * c->K + (o)) * c->K + (o2)]

/* Stage table Td(d, s, o) = least cost of the group's entries that fit at
   depth d (entries are key-sorted, so the first fitting one), and the link
   table X(j, o, o') for micro-batch b. */
static void build_tables(octx *c, int64_t e0, int64_t e1, int bi) {
    const int L = c->L, K = c->K;
    const int64_t NS = c->NS;
    for (int64_t a = 0; a < NS * K; a++) { c->gstart[a] = 0; c->gend[a] = 0; }
    for (int64_t a = e0; a < e1; a++) {
        int64_t gk = c->ent[a].gkey % (NS * K);
        if (c->gend[gk] == 0) c->gstart[gk] = a;
        c->gend[gk] = a + 1;
    }
    (void)bi;
    for (int d = 1; d <= c->D; d++)
        for (int64_t s = 0; s < NS; s++)
            for (int o = 0; o < K; o++) {
                double v = INFINITY;
                int64_t gk = s * K + o;
                for (int64_t a = c->gstart[gk]; a < c->gend[gk]; a++)
                    if (c->ent[a].dmax >= d) { v = c->ent[a].cost; break; }
                TD(d, s, o) = v;
            }
    for (int j = 1; j < L; j++)
        for (int o = 0; o < K; o++)
            for (int o2 = 0; o2 < K; o2++)
                XA(j, o, o2) = transfer(c->p, c->b, j, c->order[o], c->order[o2]);
}

/* Steps (1)-(2): least achievable bottleneck.
   V(d,i,o): best bottleneck covering layers [i, L) with d stages, the first on
   island position o and the rest on later positions.
   W(d,j,o): best continuation after a stage on position o ends at j. */
static double least_bottleneck(octx *c) {
    const int L = c->L, K = c->K, D = c->D;
    for (int d = 1; d <= D; d++) {
        for (int i = 0; i < L; i++)
            for (int o = 0; o < K; o++) {
                double v = INFINITY;
                if (d == 1) v = TD(1, slice_index(L, i, L), o);
                else
                    for (int j = i + 1; j <= L - d + 1; j++) {
                        double x = maxd(TD(d, slice_index(L, i, j), o), AT(c->Wt, d - 1, j, o));
                        if (x < v) v = x;
                    }
                AT(c->V, d, i, o) = v;
            }
        for (int j = 1; j < L; j++)
            for (int o = 0; o < K; o++) {
                double w = INFINITY;
                for (int o2 = o + 1; o2 < K; o2++) {
                    double x = maxd(XA(j, o, o2), AT(c->V, d, j, o2));
                    if (x < w) w = x;
                }
                AT(c->Wt, d, j, o) = w;
            }
    }
    double Pst = INFINITY;
    for (int d = 1; d <= D; d++)
        for (int o = 0; o < K; o++)
            if (AT(c->V, d, 0, o) < Pst) Pst = AT(c->V, d, 0, o);
    return Pst;
}

/* Step (3) at bound tau: least fill among plans whose every stage and link
   stays within tau.  Fill = f1 + (x1 + (f2 + ... + fS)), a right fold; F and G
   reuse the V and W arrays.  Returns the least root fill; *ro, *rS get its
   first position (ties to the earliest) and stage count (then fewer). */
static double least_fill(octx *c, double tau, int *ro, int *rS) {
    const int L = c->L, K = c->K, D = c->D;
    for (int d = 1; d <= D; d++) {
        for (int i = 0; i < L; i++)
            for (int o = 0; o < K; o++) {
                double v = INFINITY;
                if (d == 1) {
                    double t = TD(1, slice_index(L, i, L), o);
                    if (t <= tau) v = t;
                } else
                    for (int j = i + 1; j <= L - d + 1; j++) {
                        double t = TD(d, slice_index(L, i, j), o);
                        if (!(t <= tau)) continue;
                        double x = t + AT(c->Wt, d - 1, j, o);
                        if (x < v) v = x;
                    }
                AT(c->V, d, i, o) = v;
            }
        for (int j = 1; j < L; j++)
            for (int o = 0; o < K; o++) {
                double w = INFINITY;
                for (int o2 = o + 1; o2 < K; o2++) {
                    double x = XA(j, o, o2);
                    if (!(x <= tau)) continue;
                    double y = x + AT(c->V, d, j, o2);
                    if (y < w) w = y;
                }
                AT(c->Wt, d, j, o) = w;
            }
    }
    double Fst = INFINITY;
    *ro = -1;
    *rS = -1;
    for (int o = 0; o < K; o++)
        for (int d = 1; d <= D; d++)
            if (AT(c->V, d, 0, o) < Fst) { Fst = AT(c->V, d, 0, o); *ro = o; *rS = d; }
    return Fst;
}

/* Fill one plan stage: layers [i, j) on island position o at depth d; the
   candidate is the group's least-key entry fitting at d; `link` is the
   transfer to the next stage (0 for the last). */
static void emit_stage(octx *c, tgo_stage *st, int i, int j, int o, int d, double link) {
    const oprob *p = c->p;
    const int K = c->K;
    int64_t s = slice_index(c->L, i, j);
    int64_t gk = s * K + o;
    int64_t rep = -1;
    for (int64_t a = c->gstart[gk]; a < c->gend[gk]; a++)
        if (c->ent[a].dmax >= d) { rep = a; break; }
    const oentry *e = &c->ent[rep];
    int64_t g = e->idx / c->NS;
    const ocfg *cf = &p->cfg[g];
    ocoef co;
    config_coef(p, cf, &co);
    double cost, state, A1;
    int dm;
    score_candidate(p, &co, &p->slice_sum[s * NSUM], &cost, &dm, &state, &A1);
    double dd = cf->of ? 1.0 : (double)d;
    double inflight = dd < co.m_real ? dd : co.m_real;
    st->island = c->order[o]; st->first_layer = i; st->end_layer = j;
    st->tp = cf->tp; st->cp = cf->cp; st->dp = cf->dp; st->ep = cf->ep; st->zero = cf->z;
    st->recompute = cf->rc; st->offload = cf->of; st->mb = cf->mb;
    st->depth = d; st->pair_index = e->idx; st->cost = e->cost;
    st->mem_bytes = state + (inflight * A1);
    st->link_out = link;
}

/* Walk the argmins of the step-(3) tables at bound tau from root (ro, rS) and
   fill the plan's stages: smallest j attaining F, then smallest later
   position attaining G; each stage's candidate is its group's least-key entry
   fitting at the stage's depth. */
static void backtrack(octx *c, double tau, int ro, int rS, tgo_plan *plan) {
    const int L = c->L, K = c->K;
    int i = 0, o = ro;
    for (int t = 0; t < rS; t++) {
        int d = rS - t, j, o_next = -1;
        if (d == 1) j = L;
        else {
            for (j = i + 1; j <= L - d + 1; j++) {
                double tt = TD(d, slice_index(L, i, j), o);
                if (tt <= tau && tt + AT(c->Wt, d - 1, j, o) == AT(c->V, d, i, o)) break;
            }
            for (o_next = o + 1; o_next < K; o_next++) {
                double x = XA(j, o, o_next);
                if (x <= tau && x + AT(c->V, d - 1, j, o_next) == AT(c->Wt, d - 1, j, o)) break;
            }
        }
        emit_stage(c, &plan->stage[t], i, j, o, d, d > 1 ? XA(j, o, o_next) : 0.0);
        i = j;
        o = o_next;
    }
}

static int cmp_dbl(const void *a, const void *b) {
    double x = *(const double *)a, y = *(const double *)b;
    return (x > y) - (x < y);
}

/* Step (4): the stage and link costs above P* in ascending order are the
   relaxed bounds at which the least fill can drop.  Returns them (distinct,
   ascending) for the bounds whose iteration time could still beat `best`
   given that no plan fills less than Finf; *nt gets the count. */
static double *relaxed_bounds(octx *c, double Pst, double Finf, double best, int64_t *nt) {
    const int L = c->L, K = c->K, D = c->D;
    const int64_t cap = (int64_t)D * c->NS * K + (int64_t)L * K * K;
    double *th = (double *)malloc(sizeof(double) * (cap > 0 ? cap : 1));
    int64_t n = 0;
    const double mm1 = (double)(c->m - 1);
    for (int d = 1; d <= D; d++)
        for (int64_t s = 0; s < c->NS; s++)
            for (int o = 0; o < K; o++) {
                double v = TD(d, s, o);
                if (v > Pst && v < INFINITY && (mm1 * v) + Finf < best) th[n++] = v;
            }
    for (int j = 1; j < L; j++)
        for (int o = 0; o < K; o++)
            for (int o2 = o + 1; o2 < K; o2++) {
                double v = XA(j, o, o2);
                if (v > Pst && v < INFINITY && (mm1 * v) + Finf < best) th[n++] = v;
            }
    qsort(th, (size_t)n, sizeof(double), cmp_dbl);
    int64_t u = 0;
    for (int64_t a = 0; a < n; a++)
        if (u == 0 || th[a] != th[u - 1]) th[u++] = th[a];
    *nt = u;
    return th;
}

/* Composition.  relax = 0: steps (1)-(3) per b (least bottleneck, then least
   fill at it).  relax = 1: also step (4), relaxing the bound over the stage
   and link costs above P* in ascending order while the iteration time can
   still improve; per b the least T wins, ties to the smaller bound.
   per_b (may be NULL): relax = 0: nb x 3 (P*, F*, T); relax = 1: nb x 4
   (P*, chosen bound, F at it, T). */
static int compose_impl(void *h, const int64_t *cands, int64_t n, const int32_t *order, tgo_plan *plan,
                        double *per_b, int relax) {
    oprob *p = (oprob *)h;
    const int L = p->L, K = p->K;
    const int64_t NS = p->NS;
    const int ncol = relax ? 4 : 3;
    memset(plan, 0, sizeof(tgo_plan));
    plan->status = TGO_ENOPLAN;
    plan->T = INFINITY; plan->P = INFINITY; plan->F = INFINITY;

    int *pos = (int *)malloc(sizeof(int) * K);
    for (int k = 0; k < K; k++) pos[k] = -1;
    for (int o = 0; o < K; o++) {
        if (order[o] < 0 || order[o] >= K || pos[order[o]] != -1) { free(pos); return TGO_EINVAL; }
        pos[order[o]] = o;
    }
    /* entries: compatible candidates with d_max >= 1, strictly ascending idx */
    oentry *ent = (oentry *)malloc(sizeof(oentry) * (n > 0 ? n : 1));
    int64_t ne = 0;
    for (int64_t t = 0; t < n; t++) {
        int64_t idx = cands[t];
        if (idx < 0 || idx >= p->N || (t > 0 && idx <= cands[t - 1])) {
            free(pos); free(ent); return TGO_EINVAL;
        }
        int64_t g = idx / NS, s = idx % NS;
        const ocfg *cf = &p->cfg[g];
        if (p->B % cf->b != 0 || !balanced(p, s, cf->k)) { free(pos); free(ent); return TGO_EINVAL; }
        int bi = 0;
        while (p->bvals[bi] != cf->b) bi++;
        ocoef o;
        config_coef(p, cf, &o);
        oentry *e = &ent[ne];
        score_candidate(p, &o, &p->slice_sum[s * NSUM], &e->cost, &e->dmax, NULL, NULL);
        if (e->dmax < 1) continue;
        e->gkey = ((int64_t)bi * NS + s) * K + pos[cf->k];
        e->idx = idx;
        ne++;
    }
    qsort(ent, (size_t)ne, sizeof(oentry), cmp_entry);

    octx cx;
    octx *c = &cx;
    c->p = p; c->order = order; c->L = L; c->K = K; c->NS = NS; c->ent = ent;
    c->D = K < L ? K : L; /* a pipeline has at most min(K, L) stages */
    const int64_t cell = (int64_t)(L + 1) * K;
    c->V = (double *)malloc(sizeof(double) * (c->D + 1) * cell);
    c->Wt = (double *)malloc(sizeof(double) * (c->D + 1) * cell);
    c->Td = (double *)malloc(sizeof(double) * (c->D + 1) * NS * K);
    c->X = (double *)malloc(sizeof(double) * (L + 1) * K * K);
    c->gstart = (int64_t *)malloc(sizeof(int64_t) * NS * K);
    c->gend = (int64_t *)malloc(sizeof(int64_t) * NS * K);
    if (!c->V || !c->Wt || !c->Td || !c->X || !c->gstart || !c->gend) {
        free(pos); free(ent); free(c->V); free(c->Wt); free(c->Td); free(c->X); free(c->gstart); free(c->gend);
        return TGO_ENOMEM;
    }

    double bestT = INFINITY;
    int64_t e0 = 0;
    for (int bi = 0; bi < p->nb; bi++) {
        c->b = p->bvals[bi];
        c->m = p->B / c->b;
        if (per_b)
            for (int q = 0; q < ncol; q++) per_b[bi * ncol + q] = INFINITY;
        int64_t e1 = e0;
        while (e1 < ne && ent[e1].gkey / (NS * K) == bi) e1++;
        build_tables(c, e0, e1, bi);
        e0 = e1;
        double Pst = least_bottleneck(c);
        if (!(Pst < INFINITY)) continue;
        int ro, rS;
        double Fst = least_fill(c, Pst, &ro, &rS);
        if (ro < 0) continue;
        const double mm1 = (double)(c->m - 1);
        double tau = Pst;
        double Tb = (mm1 * Pst) + Fst;
        if (relax) {
            /* step (4): relax the bound while T can still improve */
            int ro2, rS2;
            double Finf = least_fill(c, INFINITY, &ro2, &rS2);
            int64_t nt = 0;
            double *th = relaxed_bounds(c, Pst, Finf, Tb, &nt);
            for (int64_t a = 0; a < nt; a++) {
                if ((mm1 * th[a]) + Finf >= Tb) break; /* no larger bound can improve */
                double F = least_fill(c, th[a], &ro2, &rS2);
                double Tt = (mm1 * th[a]) + F;
                if (Tt < Tb) { Tb = Tt; tau = th[a]; }
            }
            free(th);
            Fst = least_fill(c, tau, &ro, &rS); /* tables at the chosen bound */
        }
        if (per_b) {
            per_b[bi * ncol] = Pst;
            if (relax) {
                per_b[bi * ncol + 1] = tau; per_b[bi * ncol + 2] = Fst; per_b[bi * ncol + 3] = Tb;
            } else {
                per_b[bi * ncol + 1] = Fst; per_b[bi * ncol + 2] = Tb;
            }
        }
        if (Tb < bestT) {
            /* backtrack now, while this b's tables are live */
            bestT = Tb;
            plan->status = TGO_OK;
            plan->b = (int32_t)c->b; plan->m = (int32_t)c->m; plan->S = rS;
            plan->P = tau; plan->F = Fst; plan->T = Tb;
            backtrack(c, tau, ro, rS, plan);
        }
    }
    free(pos); free(ent); free(c->V); free(c->Wt); free(c->Td); free(c->X); free(c->gstart); free(c->gend);
    return plan->status;
}
/* ------------------------------------------------------------------------ */
/* composition over every island order: the subset dynamic program           */
/* ------------------------------------------------------------------------ */
/* A plan uses a set U of islands, each at most once, in any order (Sec. 5.2
   builds the pipeline from any islands; Sec. 6.2 shows that their order
   changes the plan).  With U the set of islands from a stage to the pipeline
   end, the stage's depth is |U|, so the island order needs no input:
     V(U,k,i)  least bottleneck covering [i, L) with the stages on the islands
               of U, the first on k (k in U);
     W(U',k,j) least bottleneck of a continuation on the islands of U' after a
               stage on k (k not in U') ends at j.
   Every proper subset of U is numerically smaller than U, so visiting the
   sets in ascending order computes each continuation before it is used.
   The arrays are indexed [U][k][i], (2^K x K x (L+1)), so K <= 16. */
#define SV(A, U, k, i) A[(((int64_t)(U) * c->K) + (k)) * (c->L + 1) + (i)]

static int popcount32(uint32_t x) {
    int n = 0;
    while (x) { n += (int)(x & 1u); x >>= 1; }
    return n;
}

static double least_bottleneck_sets(octx *c, double *V, double *W) {
    const int L = c->L, K = c->K, D = c->D;
    const uint32_t full = 1u << K;
    for (uint32_t U = 1; U < full; U++) {
        const int d = popcount32(U);
        for (int k = 0; k < K; k++) {
            if (!(U >> k & 1u)) continue;
            const uint32_t Up = U & ~(1u << k);
            for (int i = 0; i <= L; i++) {
                double v = INFINITY;
                if (d > D || i == L) v = INFINITY;
                else if (d == 1) v = TD(1, slice_index(L, i, L), k);
                else
                    for (int j = i + 1; j <= L - d + 1; j++) {
                        double x = maxd(TD(d, slice_index(L, i, j), k), SV(W, Up, k, j));
                        if (x < v) v = x;
                    }
                SV(V, U, k, i) = v;
            }
        }
        /* continuations on exactly the islands of U, after a stage on k0 */
        for (int k0 = 0; k0 < K; k0++) {
            if (U >> k0 & 1u) continue;
            for (int j = 0; j <= L; j++) {
                double w = INFINITY;
                if (j >= 1 && j < L)
                    for (int k = 0; k < K; k++) {
                        if (!(U >> k & 1u)) continue;
                        double x = maxd(XA(j, k0, k), SV(V, U, k, j));
                        if (x < w) w = x;
                    }
                SV(W, U, k0, j) = w;
            }
        }
    }
    double Pst = INFINITY;
    for (uint32_t U = 1; U < full; U++)
        for (int k = 0; k < K; k++)
            if ((U >> k & 1u) && SV(V, U, k, 0) < Pst) Pst = SV(V, U, k, 0);
    return Pst;
}

/* Step (3) over sets at bound tau: least fill with every stage and link
   within tau, ties to the least cut j and then the least next island.  The
   root is the least F(U, k, 0); ties go to the least first island k, then
   fewer stages |U|, then the numerically least set U. */
static double least_fill_sets(octx *c, double tau, double *F, double *G, int *rk, uint32_t *rU) {
    const int L = c->L, K = c->K, D = c->D;
    const uint32_t full = 1u << K;
    for (uint32_t U = 1; U < full; U++) {
        const int d = popcount32(U);
        for (int k = 0; k < K; k++) {
            if (!(U >> k & 1u)) continue;
            const uint32_t Up = U & ~(1u << k);
            for (int i = 0; i <= L; i++) {
                double v = INFINITY;
                if (d > D || i == L) v = INFINITY;
                else if (d == 1) {
                    double t = TD(1, slice_index(L, i, L), k);
                    if (t <= tau) v = t;
                } else
                    for (int j = i + 1; j <= L - d + 1; j++) {
                        double t = TD(d, slice_index(L, i, j), k);
                        if (!(t <= tau)) continue;
                        double x = t + SV(G, Up, k, j);
                        if (x < v) v = x;
                    }
                SV(F, U, k, i) = v;
            }
        }
        for (int k0 = 0; k0 < K; k0++) {
            if (U >> k0 & 1u) continue;
            for (int j = 0; j <= L; j++) {
                double g = INFINITY;
                if (j >= 1 && j < L)
                    for (int k = 0; k < K; k++) {
                        if (!(U >> k & 1u)) continue;
                        double x = XA(j, k0, k);
                        if (!(x <= tau)) continue;
                        double y = x + SV(F, U, k, j);
                        if (y < g) g = y;
                    }
                SV(G, U, k0, j) = g;
            }
        }
    }
    double Fst = INFINITY;
    *rk = -1;
    *rU = 0;
    for (int k = 0; k < K; k++)
        for (int d = 1; d <= D; d++)
            for (uint32_t U = 1; U < full; U++) {
                if (!(U >> k & 1u) || popcount32(U) != d) continue;
                if (SV(F, U, k, 0) < Fst) { Fst = SV(F, U, k, 0); *rk = k; *rU = U; }
            }
    return Fst;
}

/* Walk the step-(3) set tables from root (rk, rU): least j attaining F, then
   least next island attaining G. */
static void backtrack_sets(octx *c, double tau, const double *F, const double *G, int rk, uint32_t rU,
                           tgo_plan *plan) {
    const int L = c->L, K = c->K;
    const int S = popcount32(rU);
    int i = 0, k = rk;
    uint32_t U = rU;
    for (int t = 0; t < S; t++) {
        int d = S - t, j, k_next = -1;
        const uint32_t Up = U & ~(1u << k);
        if (d == 1) j = L;
        else {
            for (j = i + 1; j <= L - d + 1; j++) {
                double tt = TD(d, slice_index(L, i, j), k);
                if (tt <= tau && tt + SV(G, Up, k, j) == SV(F, U, k, i)) break;
            }
            for (k_next = 0; k_next < K; k_next++) {
                if (!(Up >> k_next & 1u)) continue;
                double x = XA(j, k, k_next);
                if (x <= tau && x + SV(F, Up, k_next, j) == SV(G, Up, k, j)) break;
            }
        }
        emit_stage(c, &plan->stage[t], i, j, k, d, d > 1 ? XA(j, k, k_next) : 0.0);
        i = j;
        k = k_next;
        U = Up;
    }
}
#undef SV

/* Composition over every island subset and order, steps (1)-(3) per b.
   per_b (may be NULL): nb x 3 (P*, F*, T).  K <= 16. */
int tgo_compose_all_orders(void *h, const int64_t *cands, int64_t n, tgo_plan *plan, double *per_b) {
    oprob *p = (oprob *)h;
    const int L = p->L, K = p->K;
    const int64_t NS = p->NS;
    memset(plan, 0, sizeof(tgo_plan));
    plan->status = TGO_ENOPLAN;
    plan->T = INFINITY; plan->P = INFINITY; plan->F = INFINITY;
    if (K > 16) return TGO_EINVAL;
    int32_t *ident = (int32_t *)malloc(sizeof(int32_t) * K);
    for (int k = 0; k < K; k++) ident[k] = k;
    oentry *ent = (oentry *)malloc(sizeof(oentry) * (n > 0 ? n : 1));
    int64_t ne = 0;
    for (int64_t t = 0; t < n; t++) {
        int64_t idx = cands[t];
        if (idx < 0 || idx >= p->N || (t > 0 && idx <= cands[t - 1])) {
            free(ident); free(ent); return TGO_EINVAL;
        }
        int64_t g = idx / NS, s = idx % NS;
        const ocfg *cf = &p->cfg[g];
        if (p->B % cf->b != 0 || !balanced(p, s, cf->k)) { free(ident); free(ent); return TGO_EINVAL; }
        int bi = 0;
        while (p->bvals[bi] != cf->b) bi++;
        ocoef o;
        config_coef(p, cf, &o);
        oentry *e = &ent[ne];
        score_candidate(p, &o, &p->slice_sum[s * NSUM], &e->cost, &e->dmax, NULL, NULL);
        if (e->dmax < 1) continue;
        e->gkey = ((int64_t)bi * NS + s) * K + cf->k;
        e->idx = idx;
        ne++;
    }
    qsort(ent, (size_t)ne, sizeof(oentry), cmp_entry);

    octx cx;
    octx *c = &cx;
    c->p = p; c->order = ident; c->L = L; c->K = K; c->NS = NS; c->ent = ent;
    c->D = K < L ? K : L;
    const int64_t sets = ((int64_t)1 << K) * K * (L + 1);
    double *V = (double *)malloc(sizeof(double) * sets);
    double *W = (double *)malloc(sizeof(double) * sets);
    c->V = NULL; c->Wt = NULL;
    c->Td = (double *)malloc(sizeof(double) * (c->D + 1) * NS * K);
    c->X = (double *)malloc(sizeof(double) * (L + 1) * K * K);
    c->gstart = (int64_t *)malloc(sizeof(int64_t) * NS * K);
    c->gend = (int64_t *)malloc(sizeof(int64_t) * NS * K);
    if (!V || !W || !c->Td || !c->X || !c->gstart || !c->gend) {
        free(ident); free(ent); free(V); free(W); free(c->Td); free(c->X); free(c->gstart); free(c->gend);
        return TGO_ENOMEM;
    }
    double bestT = INFINITY;
    int64_t e0 = 0;
    for (int bi = 0; bi < p->nb; bi++) {
        c->b = p->bvals[bi];
        c->m = p->B / c->b;
        if (per_b)
            for (int q = 0; q < 3; q++) per_b[bi * 3 + q] = INFINITY;
        int64_t e1 = e0;
        while (e1 < ne && ent[e1].gkey / (NS * K) == bi) e1++;
        build_tables(c, e0, e1, bi);
        e0 = e1;
        double Pst = least_bottleneck_sets(c, V, W);
        if (!(Pst < INFINITY)) continue;
        int rk;
        uint32_t rU;
        double Fst = least_fill_sets(c, Pst, V, W, &rk, &rU);
        if (rk < 0) continue;
        double Tb = ((double)(c->m - 1) * Pst) + Fst;
        if (per_b) { per_b[bi * 3] = Pst; per_b[bi * 3 + 1] = Fst; per_b[bi * 3 + 2] = Tb; }
        if (Tb < bestT) {
            bestT = Tb;
            plan->status = TGO_OK;
            plan->b = (int32_t)c->b; plan->m = (int32_t)c->m; plan->S = popcount32(rU);
            plan->P = Pst; plan->F = Fst; plan->T = Tb;
            backtrack_sets(c, Pst, V, W, rk, rU, plan);
        }
    }
    free(ident); free(ent); free(V); free(W); free(c->Td); free(c->X); free(c->gstart); free(c->gend);
    return plan->status;
}

#undef AT
#undef TD
#undef XA

int tgo_compose(void *h, const int64_t *cands, int64_t n, const int32_t *order, tgo_plan *plan,
                double *per_b /* nb x 3: P*, F*, T; may be NULL */) {
    return compose_impl(h, cands, n, order, plan, per_b, 0);
}

int tgo_compose_relaxed(void *h, const int64_t *cands, int64_t n, const int32_t *order, tgo_plan *plan,
                        double *per_b /* nb x 4: P*, bound, F, T; may be NULL */) {
    return compose_impl(h, cands, n, order, plan, per_b, 1);
}

/* ------------------------------------------------------------------------ */
/* island construction (Sec. 4.1)                                            */
/* ------------------------------------------------------------------------ */
/* Nodes: gpus[u] GPUs of compute c[u], memory m[u] and intra-node bandwidth
   bi[u] each (host[u]: host-link bandwidth); e[u*n + v] is the bandwidth from
   node u to node v.  An island I must hold nodes with the same GPU count and
   pairwise ratios max/min <= 1 + eps of compute and memory (Eq. 1) and of
   intra-node bandwidth (Eq. 2), and every member's links inside I must be at
   least as fast as its links leaving I (Eq. 3).  Steps (1)-(2): split the
   nodes by GPU count, then by compute, memory and intra-node bandwidth, each
   split a sweep over the values in ascending order that opens a new group at
   the first value above the group's smallest times (1 + eps).  Step (3):
   agglomerative clustering inside each group: repeatedly take the pair of
   clusters with the highest complete linkage (least bandwidth between their
   nodes, each node pair counted by its slower direction), ties to the least
   pair of smallest node ids; merge it if the union satisfies Eq. 3, else mark
   the pair and go on; stop when every remaining pair is marked.  Islands are
   numbered by smallest node id; an island has the sum of its members' GPUs,
   the least of their compute, memory, intra and host bandwidth, and the
   island-to-island bandwidth is the least over node pairs. */
static const double *node_cmp_val = NULL;
static const int64_t *node_cmp_grp = NULL;

static int cmp_nodes(const void *a, const void *b) {
    int x = *(const int *)a, y = *(const int *)b;
    if (node_cmp_grp[x] != node_cmp_grp[y]) return node_cmp_grp[x] < node_cmp_grp[y] ? -1 : 1;
    if (node_cmp_val[x] != node_cmp_val[y]) return node_cmp_val[x] < node_cmp_val[y] ? -1 : 1;
    return (x > y) - (x < y);
}

/* Refine groups grp[] by a sweep over val[] within each group (tolerance eps):
   new group numbers are dense, in (old group, value, node id) order. */
static void split_by(int n, int64_t *grp, const double *val, double eps, int *ord) {
    for (int u = 0; u < n; u++) ord[u] = u;
    node_cmp_val = val;
    node_cmp_grp = grp;
    qsort(ord, (size_t)n, sizeof(int), cmp_nodes);
    int64_t *ng = (int64_t *)malloc(sizeof(int64_t) * (n > 0 ? n : 1));
    int64_t g = -1;
    double v0 = 0.0;
    int64_t prev = -1;
    for (int t = 0; t < n; t++) {
        int u = ord[t];
        if (t == 0 || grp[u] != prev || !(val[u] <= v0 * (1.0 + eps))) {
            g++;
            v0 = val[u];
        }
        prev = grp[u];
        ng[u] = g;
    }
    for (int u = 0; u < n; u++) grp[u] = ng[u];
    free(ng);
}

/* Eq. 3 for the node set given by in_set[]: every member's least link to
   another member is at least its greatest link to a non-member. */
static int eq3_holds(int n, const double *e, const unsigned char *in_set) {
    for (int u = 0; u < n; u++) {
        if (!in_set[u]) continue;
        double in = INFINITY, out = -INFINITY;
        for (int w = 0; w < n; w++) {
            if (w == u) continue;
            double x = e[(int64_t)u * n + w];
            if (in_set[w]) { if (x < in) in = x; }
            else if (x > out) out = x;
        }
        if (!(in >= out)) return 0;
    }
    return 1;
}

int tgo_build_islands(const int32_t *gpus, const double *c, const double *m, const double *bi,
                      const double *host, int n, const double *e, double eps_c, double eps_m,
                      double eps_i, int32_t *island_of, int32_t *n_islands, int32_t *isl_gpus,
                      double *isl_peak, double *isl_hbm, double *isl_intra, double *isl_host,
                      double *isl_e /* n*n, K*K used */) {
    if (n < 1) return TGO_EINVAL;
    if (!(eps_c >= 0.0) || !(eps_m >= 0.0) || !(eps_i >= 0.0) || !isfinite(eps_c) || !isfinite(eps_m) ||
        !isfinite(eps_i))
        return TGO_EINVAL;
    for (int u = 0; u < n; u++) {
        if (gpus[u] < 1 || !(c[u] > 0.0) || !(m[u] > 0.0) || !(bi[u] > 0.0) || !(host[u] >= 0.0) ||
            !isfinite(c[u]) || !isfinite(m[u]) || !isfinite(bi[u]) || !isfinite(host[u]))
            return TGO_EINVAL;
        for (int v = 0; v < n; v++)
            if (!(e[(int64_t)u * n + v] >= 0.0) || !isfinite(e[(int64_t)u * n + v])) return TGO_EINVAL;
    }
    int64_t *grp = (int64_t *)malloc(sizeof(int64_t) * n);
    int *ord = (int *)malloc(sizeof(int) * n);
    double *gd = (double *)malloc(sizeof(double) * n);
    /* step (1): GPU count (exact), compute, memory; step (2): intra-node bandwidth */
    for (int u = 0; u < n; u++) { grp[u] = 0; gd[u] = (double)gpus[u]; }
    split_by(n, grp, gd, 0.0, ord);
    split_by(n, grp, c, eps_c, ord);
    split_by(n, grp, m, eps_m, ord);
    split_by(n, grp, bi, eps_i, ord);
    /* step (3): clusters start as single nodes; cl[u] = cluster (its smallest node) */
    int *cl = (int *)malloc(sizeof(int) * n);
    unsigned char *marked = (unsigned char *)calloc((size_t)n * n, 1); /* [a][b] by cluster ids */
    unsigned char *in_set = (unsigned char *)calloc((size_t)n, 1);
    for (int u = 0; u < n; u++) cl[u] = u;
    /* members of each cluster, listed by cluster id: start[a], then members */
    int *mstart = (int *)malloc(sizeof(int) * (n + 1));
    int *mlist = (int *)malloc(sizeof(int) * n);
    for (;;) {
        int pos = 0;
        for (int a = 0; a < n; a++) {
            mstart[a] = pos;
            for (int u = 0; u < n; u++) if (cl[u] == a) mlist[pos++] = u;
        }
        mstart[n] = pos;
        double best = -INFINITY;
        int ba = -1, bb = -1;
        for (int a = 0; a < n; a++) {
            if (cl[a] != a) continue; /* a is a cluster id */
            for (int b = a + 1; b < n; b++) {
                if (cl[b] != b || grp[a] != grp[b] || marked[(int64_t)a * n + b]) continue;
                double l = INFINITY;
                for (int p = mstart[a]; p < mstart[a + 1]; p++)
                    for (int q = mstart[b]; q < mstart[b + 1]; q++) {
                        int u = mlist[p], v = mlist[q];
                        double x = e[(int64_t)u * n + v], y = e[(int64_t)v * n + u];
                        double xy = x < y ? x : y;
                        if (xy < l) l = xy;
                    }
                if (l > best) { best = l; ba = a; bb = b; }
            }
        }
        if (ba < 0) break;
        for (int u = 0; u < n; u++) in_set[u] = (cl[u] == ba || cl[u] == bb);
        if (eq3_holds(n, e, in_set)) {
            for (int u = 0; u < n; u++) if (cl[u] == bb) cl[u] = ba;
            /* pairs involving the grown cluster are new pairs */
            for (int x = 0; x < n; x++) {
                marked[(int64_t)ba * n + x] = 0; marked[(int64_t)x * n + ba] = 0;
            }
        } else {
            marked[(int64_t)ba * n + bb] = 1;
        }
    }
    /* number islands by smallest node id (= cluster id) */
    int K = 0;
    int *isl_id = (int *)malloc(sizeof(int) * n);
    for (int u = 0; u < n; u++) isl_id[u] = -1;
    for (int u = 0; u < n; u++)
        if (cl[u] == u) isl_id[u] = K++;
    for (int u = 0; u < n; u++) island_of[u] = isl_id[cl[u]];
    *n_islands = K;
    for (int k = 0; k < K; k++) {
        isl_gpus[k] = 0; isl_peak[k] = INFINITY; isl_hbm[k] = INFINITY; isl_intra[k] = INFINITY;
        isl_host[k] = INFINITY;
    }
    for (int u = 0; u < n; u++) {
        int k = island_of[u];
        isl_gpus[k] += gpus[u];
        if (c[u] < isl_peak[k]) isl_peak[k] = c[u];
        if (m[u] < isl_hbm[k]) isl_hbm[k] = m[u];
        if (bi[u] < isl_intra[k]) isl_intra[k] = bi[u];
        if (host[u] < isl_host[k]) isl_host[k] = host[u];
    }
    for (int a = 0; a < K; a++)
        for (int b = 0; b < K; b++) isl_e[a * K + b] = a == b ? 0.0 : INFINITY;
    for (int u = 0; u < n; u++)
        for (int v = 0; v < n; v++) {
            int a = island_of[u], b = island_of[v];
            if (a == b) continue;
            double x = e[(int64_t)u * n + v];
            if (x < isl_e[a * K + b]) isl_e[a * K + b] = x;
        }
    free(grp); free(ord); free(gd); free(cl); free(marked); free(in_set); free(isl_id); free(mstart); free(mlist);
    return TGO_OK;
}
