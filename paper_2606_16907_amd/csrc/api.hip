// api.hip -- the C ABI declared in include/tangram.h: validation, the
// problem's device tables, and the entry points that launch the kernels.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstddef>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "tg_device.h"
#include "tg_problem.h"

namespace {

thread_local char g_err[512] = "";

tg_status fail(tg_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

tg_status hip_fail(hipError_t e, const char *what) {
    return fail(e == hipErrorOutOfMemory ? TG_ENOMEM : TG_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

bool ascending_set(const int32_t *v, int32_t n) {
    if (n < 1 || n > 8) return false;
    for (int a = 0; a < n; ++a) {
        if (v[a] < 1) return false;
        if (a > 0 && v[a] <= v[a - 1]) return false;
    }
    return true;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Kernels launch on the current device; the problem's tables live on the
// device that was current at create.
tg_status check_device(const tg_problem *p) {
    int cur = -1;
    const hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur != p->device)
        return fail(TG_EINVAL, "device %d is current; the problem lives on device %d", cur, p->device);
    return TG_OK;
}

bool aligned(const void *ptr, uintptr_t a) { return ((uintptr_t)ptr & (a - 1)) == 0; }

// Score arrays and survivor lists hold 8-byte values; workspaces are carved
// at 256-byte offsets from their base, and their counters take atomics.
tg_status check_alignment(const void *cost, const void *survivors, const void *ws) {
    if ((cost && !aligned(cost, 8)) || (survivors && !aligned(survivors, 8)) || (ws && !aligned(ws, 256)))
        return fail(TG_EINVAL, "misaligned buffer: cost and survivors need 8-byte, workspaces 256-byte alignment");
    return TG_OK;
}

// Configs per problem, at most: the frontier packs a member's index within
// its group into 23 bits.
constexpr int64_t kMaxConfigs = (int64_t)1 << 23;
// GPUs per island, at most: 4096 nodes of 65536 GPUs, the largest island
// tg_build_islands can return.
constexpr int32_t kMaxIslandGpus = 1 << 28;
constexpr int32_t kMaxNodeGpus = 1 << 16;

// Host containers may throw std::bad_alloc; no exception crosses the C ABI.
template <typename F>
tg_status no_throw(F f) {
    try {
        return f();
    } catch (const std::bad_alloc &) {
        return fail(TG_ENOMEM, "host allocation");
    }
}

}  // namespace


static tg_status problem_create(const tg_layer *layers, int32_t L, const tg_island *islands, int32_t K,
                                const double *inter_bw, const tg_space *space, tg_problem **out) {
    if (!layers || !islands || !inter_bw || !space) return fail(TG_EINVAL, "NULL input table");
    if (L < 1 || L > 512) return fail(TG_EINVAL, "L=%d outside [1, 512]", L);
    if (K < 1 || K > 255) return fail(TG_EINVAL, "K=%d outside [1, 255]", K);
    const tg_space &sp = *space;
    if (sp.global_batch < 1) return fail(TG_EINVAL, "global_batch < 1");
    if (sp.n_experts < 0) return fail(TG_EINVAL, "n_experts < 0");
    if (sp.reserved != 0) return fail(TG_EINVAL, "space reserved field not 0");
    if (!ascending_set(sp.tp, sp.n_tp)) return fail(TG_EINVAL, "tp set invalid");
    if (!ascending_set(sp.ep, sp.n_ep)) return fail(TG_EINVAL, "ep set invalid");
    if (!ascending_set(sp.mb, sp.n_mb)) return fail(TG_EINVAL, "mb set invalid");
    if (sp.zero_mask == 0 || (sp.zero_mask & ~0xFu)) return fail(TG_EINVAL, "zero_mask invalid");
    if (sp.n_cp != 0 && !ascending_set(sp.cp, sp.n_cp)) return fail(TG_EINVAL, "cp set invalid");
    if (sp.recompute_mask & ~0x3u) return fail(TG_EINVAL, "recompute_mask invalid");
    if (sp.offload_mask & ~0x3u) return fail(TG_EINVAL, "offload_mask invalid");
    if (sp.reserved2 != 0) return fail(TG_EINVAL, "space reserved2 field not 0");
    if (!(sp.eta > 0.0) || !std::isfinite(sp.eta)) return fail(TG_EINVAL, "eta invalid");
    if (!(sp.mem_frac > 0.0) || !std::isfinite(sp.mem_frac)) return fail(TG_EINVAL, "mem_frac invalid");
    if (!(sp.imbalance_eps >= 0.0) || !std::isfinite(sp.imbalance_eps))
        return fail(TG_EINVAL, "imbalance_eps invalid");
    for (int k = 0; k < K; ++k) {
        const tg_island &is = islands[k];
        if (is.n_gpus < 1 || is.n_gpus > kMaxIslandGpus) return fail(TG_EINVAL, "island %d: n_gpus", k);
        if (is.reserved != 0) return fail(TG_EINVAL, "island %d: reserved field not 0", k);
        if (!(is.peak_flops > 0.0) || !std::isfinite(is.peak_flops)) return fail(TG_EINVAL, "island %d: peak", k);
        if (!(is.hbm_bytes > 0.0) || !std::isfinite(is.hbm_bytes)) return fail(TG_EINVAL, "island %d: hbm", k);
        if (!(is.intra_bw > 0.0) || !std::isfinite(is.intra_bw)) return fail(TG_EINVAL, "island %d: intra", k);
        if (!(is.host_bw >= 0.0) || !std::isfinite(is.host_bw)) return fail(TG_EINVAL, "island %d: host_bw", k);
    }
    for (int a = 0; a < K * K; ++a)
        if (!(inter_bw[a] >= 0.0)) return fail(TG_EINVAL, "inter_bw[%d] negative or NaN", a);

    // prefix sums of the eight summed layer fields; every whole-model sum < 2^62
    const int64_t Lp = L + 1;
    std::vector<int64_t> pre(8 * Lp, 0), outact(L);
    const int64_t lim = (int64_t)1 << 62;
    for (int l = 0; l < L; ++l) {
        const tg_layer &y = layers[l];
        const int64_t f[8] = {y.fwd_flops,     y.dense_params, y.expert_params, y.act_stash_bytes,
                              y.tp_comm_bytes, y.a2a_bytes,    y.out_act_bytes, y.cp_comm_bytes};
        for (int q = 0; q < 8; ++q) {
            if (f[q] < 0 || f[q] >= lim - pre[q * Lp + l]) return fail(TG_EINVAL, "layer %d field %d", l, q);
            pre[q * Lp + l + 1] = pre[q * Lp + l] + f[q];
        }
        outact[l] = y.out_act_bytes;
    }
    const int dense = (pre[2 * Lp + L] == 0 && pre[5 * Lp + L] == 0) ? 1 : 0;

    // the config list of every island: lexicographic (tp, cp, dp, ep, z, rc,
    // of, mb) with tp * cp * dp <= n; offloading needs a host link.  The list
    // is counted before it is built, so an oversized space is refused before
    // any of it is allocated.
    std::vector<int> zs, cps, rcs, ofs;
    for (int z = 0; z < 4; ++z)
        if (sp.zero_mask & (1u << z)) zs.push_back(z);
    if (sp.n_cp == 0) cps.push_back(1);
    for (int a = 0; a < sp.n_cp; ++a) cps.push_back(sp.cp[a]);
    for (int r = 0; r < 2; ++r) {
        if ((sp.recompute_mask ? sp.recompute_mask : 1u) & (1u << r)) rcs.push_back(r);
        if ((sp.offload_mask ? sp.offload_mask : 1u) & (1u << r)) ofs.push_back(r);
    }
    auto visit = [&](auto &&emit) -> bool {  // false once emit asks to stop
        for (int k = 0; k < K; ++k) {
            const int n = islands[k].n_gpus;
            for (int a = 0; a < sp.n_tp; ++a) {
                const int tp = sp.tp[a];
                if (tp > n) continue;
                for (int cp : cps) {
                    if ((int64_t)tp * cp > n) continue;
                    const int q = tp * cp;
                    for (int dp = 1; dp <= n / q; ++dp)
                        for (int e = 0; e < sp.n_ep; ++e) {
                            const int ep = sp.ep[e];
                            if (dp % ep) continue;
                            if (sp.n_experts == 0 ? ep != 1 : (sp.n_experts % ep) != 0) continue;
                            for (int z : zs)
                                for (int rc : rcs)
                                    for (int of : ofs) {
                                        if (of && !(islands[k].host_bw > 0.0)) continue;
                                        for (int mi = 0; mi < sp.n_mb; ++mi)
                                            if (!emit(k, tp, cp, dp, ep, z, rc, of, sp.mb[mi])) return false;
                                    }
                        }
                }
            }
        }
        return true;
    };
    int64_t n_listed = 0;
    if (!visit([&](int, int, int, int, int, int, int, int, int) { return ++n_listed < kMaxConfigs; }))
        return fail(TG_EINVAL, "candidate space too large: %lld configs or more", (long long)kMaxConfigs);
    std::vector<tg::Coef> cfg;
    cfg.reserve((size_t)n_listed);
    int ext = 0;
    visit([&](int k, int tp, int cp, int dp, int ep, int z, int rc, int of, int mb) {
        tg::Coef c;
        std::memset(&c, 0, sizeof(c));
        c.k = k;
        c.tp = tp;
        c.cp = cp;
        c.dp = dp;
        c.ep = ep;
        c.z = z;
        c.rc = rc;
        c.of = of;
        c.mb = mb;
        if (cp > 1 || rc || of) ext = 1;
        cfg.push_back(c);
        return true;
    });
    const int64_t ncfg = (int64_t)cfg.size();
    const int64_t NS = (int64_t)L * (L + 1) / 2;
    if (ncfg > ((int64_t)1 << 31) - 1 || NS * ncfg >= ((int64_t)1 << 62))
        return fail(TG_EINVAL, "candidate space too large");

    // compatible b values, bitmap rows, (island, b) groups
    std::vector<int64_t> bv;
    for (auto &c : cfg) {
        const int64_t b = (int64_t)c.dp * c.mb;
        if (sp.global_batch % b == 0) bv.push_back(b);
    }
    std::sort(bv.begin(), bv.end());
    bv.erase(std::unique(bv.begin(), bv.end()), bv.end());
    const int nb = (int)bv.size();
    // a plan reports b and m = B / b as int32
    if (nb > 0 && (bv.back() > INT32_MAX || sp.global_batch / bv.front() > INT32_MAX))
        return fail(TG_EINVAL, "global_batch %lld: b or B / b exceeds 2^31 - 1", (long long)sp.global_batch);
    std::vector<int32_t> row_cfg;
    for (int64_t g = 0; g < ncfg; ++g) {
        const int64_t b = (int64_t)cfg[g].dp * cfg[g].mb;
        auto it = std::lower_bound(bv.begin(), bv.end(), b);
        if (it != bv.end() && *it == b) {
            cfg[g].b_idx = (int32_t)(it - bv.begin());
            cfg[g].row = (int32_t)row_cfg.size();
            row_cfg.push_back((int32_t)g);
        } else {
            cfg[g].b_idx = -1;
            cfg[g].row = -1;
        }
    }
    std::vector<int32_t> kb_off(1, 0), kb_members, kb_island, kb_bidx;
    int max_members = 0;
    {
        int64_t c0 = 0;
        for (int k = 0; k < K; ++k) {
            int64_t c1 = c0;
            while (c1 < ncfg && cfg[c1].k == k) ++c1;
            for (int bi = 0; bi < nb; ++bi) {
                int cnt = 0;
                for (int64_t g = c0; g < c1; ++g)
                    if (cfg[g].b_idx == bi) {
                        kb_members.push_back((int32_t)g);
                        ++cnt;
                    }
                if (cnt) {
                    kb_off.push_back((int32_t)kb_members.size());
                    kb_island.push_back(k);
                    kb_bidx.push_back(bi);
                    max_members = std::max(max_members, cnt);
                }
            }
            c0 = c1;
        }
    }
    // distinct inter-island bandwidths (link times need one division per value)
    std::vector<double> ev(inter_bw, inter_bw + (size_t)K * K);
    std::sort(ev.begin(), ev.end());
    ev.erase(std::unique(ev.begin(), ev.end()), ev.end());
    std::vector<uint16_t> eidx((size_t)K * K, 0);
    const bool e_table = ev.size() <= (size_t)tg::kMaxDistinctE;
    if (e_table)
        for (int a = 0; a < K * K; ++a)
            eidx[a] = (uint16_t)(std::lower_bound(ev.begin(), ev.end(), inter_bw[a]) - ev.begin());
    std::vector<uint32_t> sij(NS);
    {
        int64_t s = 0;
        for (int i = 0; i < L; ++i)
            for (int j = i + 1; j <= L; ++j) sij[s++] = (uint32_t)i | ((uint32_t)j << 16);
    }

    // imbalance pruning: each island's share of the cluster's compute (summed
    // in island order) and, per island and first layer, the first balanced cut
    // (a slice's FLOP share only grows with its end, so the balanced cuts of a
    // first layer are one interval)
    const int64_t total_flops = pre[L] - pre[0];
    const int imb = (sp.imbalance_eps > 0.0 && total_flops > 0) ? 1 : 0;
    const double imb_r = 1.0 + sp.imbalance_eps;
    std::vector<double> cap(K);
    {
        double cap_sum = 0.0;
        for (int k = 0; k < K; ++k) cap_sum = cap_sum + ((double)islands[k].n_gpus * islands[k].peak_flops);
        for (int k = 0; k < K; ++k) cap[k] = ((double)islands[k].n_gpus * islands[k].peak_flops) / cap_sum;
    }
    std::vector<int32_t> jlo(imb ? (size_t)K * L : 0);
    for (int k = 0; imb && k < K; ++k)
        for (int i = 0; i < L; ++i) {
            int j = i + 1;
            for (; j <= L; ++j) {
                const double q = (double)(pre[j] - pre[i]) / (double)total_flops;
                if (q <= cap[k] * imb_r && q * imb_r >= cap[k]) break;
            }
            jlo[(size_t)k * L + i] = j;
        }

    // redundancy pruning: slices with equal per-slice sums form a class,
    // classes numbered by their first slice
    std::vector<uint32_t> cls(NS), cls_ij;
    {
        auto sums = [&](int64_t s, int q) {
            const uint32_t ij = sij[s];
            return pre[(size_t)q * Lp + (ij >> 16)] - pre[(size_t)q * Lp + (ij & 0xFFFFu)];
        };
        std::vector<int64_t> ord(NS);
        for (int64_t s = 0; s < NS; ++s) ord[s] = s;
        std::sort(ord.begin(), ord.end(), [&](int64_t x, int64_t y) {
            for (int q = 0; q < 8; ++q) {
                const int64_t u = sums(x, q), v = sums(y, q);
                if (u != v) return u < v;
            }
            return x < y;
        });
        std::vector<int64_t> first(NS);
        int64_t head = 0;
        for (int64_t t = 0; t < NS; ++t) {
            bool same = t > 0;
            for (int q = 0; same && q < 8; ++q) same = sums(ord[t - 1], q) == sums(ord[t], q);
            if (!same) head = ord[t];
            first[ord[t]] = head;
        }
        for (int64_t s = 0; s < NS; ++s) {
            if (first[s] == s) {
                cls[s] = (uint32_t)cls_ij.size();
                cls_ij.push_back(sij[s]);
            } else {
                cls[s] = cls[first[s]];
            }
        }
    }

    // one device block for all tables
    struct Part {
        const void *src;
        size_t bytes;
        size_t off;
    };
    std::vector<double> peak(K), hbm(K), intra(K), host(K);
    for (int k = 0; k < K; ++k) {
        peak[k] = islands[k].peak_flops;
        hbm[k] = islands[k].hbm_bytes;
        intra[k] = islands[k].intra_bw;
        host[k] = islands[k].host_bw;
    }
    Part parts[] = {
        {pre.data(), pre.size() * 8, 0},
        {outact.data(), outact.size() * 8, 0},
        {inter_bw, (size_t)K * K * 8, 0},
        {sij.data(), sij.size() * 4, 0},
        {cfg.data(), cfg.size() * sizeof(tg::Coef), 0},
        {bv.data(), bv.size() * 8, 0},
        {kb_off.data(), kb_off.size() * 4, 0},
        {kb_members.data(), kb_members.size() * 4, 0},
        {kb_island.data(), kb_island.size() * 4, 0},
        {kb_bidx.data(), kb_bidx.size() * 4, 0},
        {row_cfg.data(), row_cfg.size() * 4, 0},
        {peak.data(), (size_t)K * 8, 0},
        {hbm.data(), (size_t)K * 8, 0},
        {intra.data(), (size_t)K * 8, 0},
        {ev.data(), ev.size() * 8, 0},
        {eidx.data(), eidx.size() * 2, 0},
        {host.data(), (size_t)K * 8, 0},
        {cap.data(), (size_t)K * 8, 0},
        {jlo.data(), jlo.size() * 4, 0},
        {cls.data(), cls.size() * 4, 0},
        {cls_ij.data(), cls_ij.size() * 4, 0},
    };
    size_t total = 0;
    for (auto &p : parts) {
        p.off = total;
        total += align256(p.bytes > 0 ? p.bytes : 1);
    }
    tg_problem *pr = new tg_problem();
    // host copies first: nothing below the device allocation throws
    pr->bvals = bv;
    pr->n_compat_cfg = (int64_t)row_cfg.size();
    pr->B = space->global_batch;
    pr->outact = outact;
    pr->E.assign(inter_bw, inter_bw + (size_t)K * K);
    hipError_t e = hipGetDevice(&pr->device);
    if (e != hipSuccess) {
        delete pr;
        return hip_fail(e, "hipGetDevice");
    }
    e = hipMalloc(&pr->dev_block, total);
    if (e != hipSuccess) {
        delete pr;
        return hip_fail(e, "hipMalloc");
    }
    char *base = (char *)pr->dev_block;
    for (auto &p : parts) {
        if (p.bytes == 0) continue;
        e = hipMemcpy(base + p.off, p.src, p.bytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(pr->dev_block);
            delete pr;
            return hip_fail(e, "hipMemcpy");
        }
    }
    tg::DevProblem &P = pr->P;
    P.L = L;
    P.K = K;
    P.nb = nb;
    P.dense = dense;
    P.ext = ext;
    P.NS = NS;
    P.ncfg = ncfg;
    P.N = NS * ncfg;
    P.B = sp.global_batch;
    P.n_kb = (int32_t)kb_island.size();
    P.max_members = max_members;
    P.n_rows = (int32_t)row_cfg.size();
    P.words = (int32_t)((NS + 63) / 64);
    P.pre = (const int64_t *)(base + parts[0].off);
    P.outact = (const int64_t *)(base + parts[1].off);
    P.E = (const double *)(base + parts[2].off);
    P.sij = (const uint32_t *)(base + parts[3].off);
    P.coef = (const tg::Coef *)(base + parts[4].off);
    P.bvals = (const int64_t *)(base + parts[5].off);
    P.kb_off = (const int32_t *)(base + parts[6].off);
    P.kb_members = (const int32_t *)(base + parts[7].off);
    P.kb_island = (const int32_t *)(base + parts[8].off);
    P.kb_bidx = (const int32_t *)(base + parts[9].off);
    P.row_cfg = (const int32_t *)(base + parts[10].off);
    P.peak = (const double *)(base + parts[11].off);
    P.hbm = (const double *)(base + parts[12].off);
    P.intra = (const double *)(base + parts[13].off);
    P.eta = sp.eta;
    P.mem_frac = sp.mem_frac;
    P.n_ev = e_table ? (int32_t)ev.size() : 0;
    P.Ev = (const double *)(base + parts[14].off);
    P.Eidx = (const uint16_t *)(base + parts[15].off);
    P.host = (const double *)(base + parts[16].off);
    P.imb = imb;
    P.imb_r = imb_r;
    P.total_flops = total_flops;
    P.cap = (const double *)(base + parts[17].off);
    P.jlo = imb ? (const int32_t *)(base + parts[18].off) : nullptr;
    P.jlo_pos = nullptr;
    P.NC = (int64_t)cls_ij.size();
    P.cls = (const uint32_t *)(base + parts[19].off);
    P.cls_ij = (const uint32_t *)(base + parts[20].off);
    P.class_scores = 0;
    // the per-config coefficients are computed on the device
    e = tg::launch_coef(P, (tg::Coef *)(base + parts[4].off), nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        (void)hipFree(pr->dev_block);
        delete pr;
        return hip_fail(e, "coefficient kernel");
    }
    *out = pr;
    return TG_OK;
}

extern "C" {

const char *tg_last_error(void) { return g_err; }

tg_status tg_problem_create(const tg_layer *layers, int32_t L, const tg_island *islands, int32_t K,
                            const double *inter_bw, const tg_space *space, tg_problem **out) {
    g_err[0] = 0;
    if (!out) return fail(TG_EINVAL, "out is NULL");
    *out = nullptr;
    return no_throw([&] { return problem_create(layers, L, islands, K, inter_bw, space, out); });
}

void tg_problem_destroy(tg_problem *p) {
    if (!p) return;
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(p->device);
    (void)hipFree(p->dev_block);
    p->relax_stage.release();
    p->readback_stage.release();
    if (p->compose_ev) (void)hipEventDestroy(p->compose_ev);
    if (p->relax_ev) (void)hipEventDestroy(p->relax_ev);
    (void)hipSetDevice(cur);
    delete p;
}

tg_status tg_problem_info(const tg_problem *p, tg_info *out) {
    if (!p || !out) return fail(TG_EINVAL, "NULL argument");
    out->L = p->P.L;
    out->K = p->P.K;
    out->n_b = p->P.nb;
    out->dense = p->P.dense;
    out->NS = p->P.NS;
    out->n_configs = p->P.ncfg;
    out->N = p->P.N;
    out->n_compatible_configs = p->n_compat_cfg;
    out->n_slice_classes = p->P.NC;
    return TG_OK;
}

tg_status tg_problem_bvalues(const tg_problem *p, int64_t *out, int32_t capacity) {
    if (!p) return fail(TG_EINVAL, "NULL problem");
    if (capacity < p->P.nb) return fail(TG_ECAPACITY, "capacity %d < n_b %d", capacity, p->P.nb);
    if (p->P.nb > 0 && !out) return fail(TG_EINVAL, "NULL output");
    for (int a = 0; a < p->P.nb; ++a) out[a] = p->bvals[a];
    return TG_OK;
}

tg_status tg_enumerate_pairs(const tg_problem *p, int64_t *n_candidates, int64_t first, int64_t count,
                             tg_pair *d_out, tg_stream stream) {
    if (!p) return fail(TG_EINVAL, "NULL problem");
    if (n_candidates) *n_candidates = p->P.N;
    if (!d_out) return TG_OK;
    if (first < 0 || count < 0 || first > p->P.N || count > p->P.N - first)
        return fail(TG_EINVAL, "range [%lld, +%lld) outside [0, %lld)", (long long)first, (long long)count,
                    (long long)p->P.N);
    if (!aligned(d_out, 4)) return fail(TG_EINVAL, "misaligned buffer: pairs need 4-byte alignment");
    if (tg_status st = check_device(p); st != TG_OK) return st;
    hipError_t e = tg::launch_enumerate(p->P, first, count, d_out, (hipStream_t)stream);
    return e == hipSuccess ? TG_OK : hip_fail(e, "enumerate kernel");
}

tg_status tg_score_pairs(const tg_problem *p, int64_t first, int64_t count, double *d_cost, uint8_t *d_dmax,
                         tg_stream stream) {
    if (!p) return fail(TG_EINVAL, "NULL problem");
    if (first < 0 || count < 0 || first > p->P.N || count > p->P.N - first)
        return fail(TG_EINVAL, "range [%lld, +%lld) outside [0, %lld)", (long long)first, (long long)count,
                    (long long)p->P.N);
    if (count > 0 && (!d_cost || !d_dmax)) return fail(TG_EINVAL, "NULL output");
    if (check_alignment(d_cost, nullptr, nullptr) != TG_OK) return TG_EINVAL;
    if (tg_status st = check_device(p); st != TG_OK) return st;
    hipError_t e = tg::launch_score(p->P, first, count, d_cost, d_dmax, (hipStream_t)stream);
    return e == hipSuccess ? TG_OK : hip_fail(e, "score kernel");
}

size_t tg_prune_workspace_bytes(const tg_problem *p) { return p ? tg::prune_ws_bytes(p->P) : 0; }

tg_status tg_score_classes(const tg_problem *p, int64_t first, int64_t count, double *d_cost, uint8_t *d_dmax,
                           tg_stream stream) {
    if (!p) return fail(TG_EINVAL, "NULL problem");
    const tg::DevProblem C = tg::class_view(p->P);
    if (first < 0 || count < 0 || first > C.N || count > C.N - first)
        return fail(TG_EINVAL, "range [%lld, +%lld) outside [0, %lld)", (long long)first, (long long)count,
                    (long long)C.N);
    if (count > 0 && (!d_cost || !d_dmax)) return fail(TG_EINVAL, "NULL output");
    if (check_alignment(d_cost, nullptr, nullptr) != TG_OK) return TG_EINVAL;
    if (tg_status st = check_device(p); st != TG_OK) return st;
    hipError_t e = tg::launch_score(C, first, count, d_cost, d_dmax, (hipStream_t)stream);
    return e == hipSuccess ? TG_OK : hip_fail(e, "score kernel");
}

size_t tg_prune_classes_workspace_bytes(const tg_problem *p) { return p ? tg::prune_classes_ws_bytes(p->P) : 0; }

}  // extern "C"

// The handle's pinned read-back words, which kernels store into: the
// composition's result block at 0 (the prune's count there too, in calls of
// its own), then the fill depth limits (nb int32).
static size_t readback_dlim_at() { return (sizeof(tg::ComposeResult) + 255) & ~(size_t)255; }
static size_t readback_bytes(const tg_problem *p) { return readback_dlim_at() + sizeof(int32_t) * (size_t)p->P.nb; }

// The read-back words (the first call allocates them) when no other call
// holds them: locks `lock` and returns them, else null (the caller reads back
// into pageable memory).
static const tg::HostStage *pinned_words(const tg_problem *p, std::unique_lock<std::mutex> &lock) {
    lock = std::unique_lock<std::mutex>(p->readback_mu, std::try_to_lock);
    if (!lock.owns_lock()) return nullptr;
    // coherent: the kernels' stores go straight to host memory
    if (p->readback_stage.reserve(readback_bytes(p), hipHostMallocPortable | hipHostMallocCoherent) != hipSuccess) {
        (void)hipGetLastError();  // a failed allocation only means the pageable read-back
        return nullptr;
    }
    return &p->readback_stage;
}

// The prune kernels on a checked workspace, then the survivor count (through
// the pinned words only when the call may allocate them).
static tg_status prune_run(const tg_problem *p, const double *d_cost, const uint8_t *d_dmax, int64_t *d_survivors,
                           int64_t capacity, int64_t *n_survivors, void *d_ws, tg_stream stream, bool may_alloc) {
    int64_t *d_total = nullptr;
    hipStream_t s = (hipStream_t)stream;
    std::unique_lock<std::mutex> lock;
    const tg::HostStage *pw = may_alloc ? pinned_words(p, lock) : nullptr;  // the count is stored there too
    hipError_t e = tg::launch_prune(p->P, d_cost, d_dmax, d_survivors, capacity, d_ws, s, &d_total,
                                    pw ? (int64_t *)pw->dev : nullptr);
    if (e != hipSuccess) {
        (void)hipStreamSynchronize(s);  // nothing queued may store into the words once they are let go
        return hip_fail(e, "prune kernels");
    }
    int64_t total = 0;
    e = pw ? hipSuccess : hipMemcpyAsync(&total, d_total, sizeof(total), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "prune count");
    if (pw) total = *(const int64_t *)pw->ptr;
    *n_survivors = total;
    if (total > capacity)
        return fail(TG_ECAPACITY, "%lld survivors exceed capacity %lld", (long long)total, (long long)capacity);
    return TG_OK;
}

static tg_status prune_args(const tg_problem *p, const double *d_cost, const uint8_t *d_dmax,
                            const int64_t *d_survivors, int64_t capacity, const int64_t *n_survivors) {
    if (!p || !n_survivors) return fail(TG_EINVAL, "NULL argument");
    if (!d_cost || !d_dmax) return fail(TG_EINVAL, "NULL score arrays");
    if (capacity < 0 || (capacity > 0 && !d_survivors)) return fail(TG_EINVAL, "bad survivor buffer");
    return TG_OK;
}

extern "C" {

tg_status tg_prune(const tg_problem *p, const double *d_cost, const uint8_t *d_dmax, int64_t *d_survivors,
                   int64_t capacity, int64_t *n_survivors, void *d_ws, size_t ws_bytes, tg_stream stream) {
    if (tg_status st = prune_args(p, d_cost, d_dmax, d_survivors, capacity, n_survivors); st != TG_OK) return st;
    if (!d_ws || ws_bytes < tg::prune_ws_bytes(p->P))
        return fail(TG_ENOMEM, "workspace %zu < %zu bytes", ws_bytes, tg::prune_ws_bytes(p->P));
    if (check_alignment(d_cost, d_survivors, d_ws) != TG_OK) return TG_EINVAL;
    if (tg_status st = check_device(p); st != TG_OK) return st;
    return prune_run(p, d_cost, d_dmax, d_survivors, capacity, n_survivors, d_ws, stream, true);
}

tg_status tg_prune_no_alloc(const tg_problem *p, const double *d_cost, const uint8_t *d_dmax, int64_t *d_survivors,
                            int64_t capacity, int64_t *n_survivors, tg_stream stream) {
    if (tg_status st = prune_args(p, d_cost, d_dmax, d_survivors, capacity, n_survivors); st != TG_OK) return st;
    const size_t need = tg::prune_ws_bytes(p->P);
    if (need > tg::kStaticScratchBytes)
        return fail(TG_ENOMEM, "the surviving set of this problem needs %zu bytes of scratch; the static scratch "
                               "holds %zu (use tg_prune with a workspace)", need, tg::kStaticScratchBytes);
    if (check_alignment(d_cost, d_survivors, nullptr) != TG_OK) return TG_EINVAL;
    if (tg_status st = check_device(p); st != TG_OK) return st;
    void *ws = nullptr;
    const hipError_t e = tg::static_scratch(p->device, &ws);
    if (e != hipSuccess) return hip_fail(e, "static scratch address");
    return prune_run(p, d_cost, d_dmax, d_survivors, capacity, n_survivors, ws, stream, false);
}

tg_status tg_prune_classes(const tg_problem *p, const double *d_cost, const uint8_t *d_dmax, int64_t *d_survivors,
                           int64_t capacity, int64_t *n_survivors, void *d_ws, size_t ws_bytes, tg_stream stream) {
    if (!p || !n_survivors) return fail(TG_EINVAL, "NULL argument");
    if (!d_cost || !d_dmax) return fail(TG_EINVAL, "NULL score arrays");
    if (capacity < 0 || (capacity > 0 && !d_survivors)) return fail(TG_EINVAL, "bad survivor buffer");
    const size_t need = tg::prune_classes_ws_bytes(p->P);
    if (!d_ws || ws_bytes < need) return fail(TG_ENOMEM, "workspace %zu < %zu bytes", ws_bytes, need);
    if (check_alignment(d_cost, d_survivors, d_ws) != TG_OK) return TG_EINVAL;
    if (tg_status st = check_device(p); st != TG_OK) return st;
    int64_t *d_total = nullptr;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = tg::launch_prune_classes(p->P, d_cost, d_dmax, d_survivors, capacity, d_ws, s, &d_total);
    if (e != hipSuccess) return hip_fail(e, "prune kernels");
    int64_t total = 0;
    e = hipMemcpyAsync(&total, d_total, sizeof(total), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "prune count");
    *n_survivors = total;
    if (total > capacity)
        return fail(TG_ECAPACITY, "%lld survivors exceed capacity %lld", (long long)total, (long long)capacity);
    return TG_OK;
}

size_t tg_compose_workspace_bytes(const tg_problem *p, int64_t n_survivors) {
    if (!p || n_survivors < 0) return 0;
    return tg::compose_ws_bytes(p->P, n_survivors);
}

size_t tg_compose_relaxed_workspace_bytes(const tg_problem *p, int64_t n_survivors) {
    if (!p || n_survivors < 0) return 0;
    return tg::compose_relaxed_ws_bytes(p->P, n_survivors);
}

size_t tg_compose_all_orders_workspace_bytes(const tg_problem *p, int64_t n_survivors) {
    if (!p || n_survivors < 0 || p->P.K > 16) return 0;
    return tg::compose_orders_ws_bytes(p->P, n_survivors);
}

}  // extern "C"

// Argument checks shared by both compositions; uploads the island order.
static tg_status compose_begin(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                               const double *d_cost, const uint8_t *d_dmax, const int32_t *island_order,
                               tg_plan *out, void *d_ws, size_t ws_bytes, size_t need, hipStream_t s) {
    if (!p || !out) return fail(TG_EINVAL, "NULL argument");
    std::memset(out, 0, sizeof(*out));
    out->P = out->F = out->T = HUGE_VAL;
    const int K = p->P.K;
    bool seen[256] = {};  // K <= 255
    for (int o = 0; island_order && o < K; ++o) {
        const int k = island_order[o];
        if (k < 0 || k >= K || seen[k]) return fail(TG_EINVAL, "island_order is not a permutation");
        seen[k] = true;
    }
    if (n_survivors < 0 || n_survivors > ((int64_t)1 << 30) || (n_survivors > 0 && !d_survivors))
        return fail(TG_EINVAL, "bad survivor list");
    if (n_survivors > 0 && (!d_cost || !d_dmax)) return fail(TG_EINVAL, "NULL score arrays");
    if ((int64_t)p->P.nb * p->P.NS * K >= ((int64_t)1 << 31)) return fail(TG_EINVAL, "stage table too large");
    if (p->P.nb > 65535) return fail(TG_EINVAL, "more than 65535 micro-batch sizes");
    if (!d_ws || ws_bytes < need) return fail(TG_ENOMEM, "workspace %zu < %zu bytes", ws_bytes, need);
    if (check_alignment(n_survivors > 0 ? d_cost : nullptr, d_survivors, d_ws) != TG_OK) return TG_EINVAL;
    if (tg_status st = check_device(p); st != TG_OK) return st;
    if (p->P.nb == 0) return fail(TG_ENOPLAN, "no micro-batch size divides the global batch");
    if (!island_order) return TG_OK;
    hipError_t e = hipMemcpyAsync((char *)d_ws + tg::compose_order_offset(p->P, n_survivors), island_order,
                                  sizeof(int32_t) * K, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "order upload");
    return TG_OK;
}

// Reads the device result after the composition kernels.
// stored: the pinned host copy the kernels stored the result into (header
// and the plan's stages), or null (then it is copied from res_dev)
static tg_status compose_end(tg::ComposeResult *res_dev, tg_plan *out, hipStream_t s,
                             const tg::ComposeResult *stored = nullptr) {
    tg::ComposeResult *owned = stored ? nullptr : new (std::nothrow) tg::ComposeResult;
    const tg::ComposeResult *res = stored ? stored : owned;
    if (!res) return fail(TG_ENOMEM, "host allocation");
    hipError_t e = stored ? hipSuccess : hipMemcpyAsync(owned, res_dev, sizeof(*owned), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        delete owned;
        return hip_fail(e, "compose result");
    }
    tg_status st = TG_OK;
    if (res->err & 3) {
        st = fail(TG_EINVAL, "candidate list invalid (code %d): not strictly ascending, out of range, or "
                             "incompatible", res->err);
    } else if (res->err) {
        st = fail(TG_EDEVICE, "internal consistency check failed during backtracking (code %d)", res->err);
    } else if (res->status != TG_OK) {
        st = fail(TG_ENOPLAN, "no pipeline fits");
    } else {  // the header and the S stages; the stages past S are zero
        const int S = std::min(std::max(res->plan.S, 0), 255);
        std::memcpy(out, &res->plan, offsetof(tg_plan, stage) + sizeof(tg_stage) * S);
        std::memset(out->stage + S, 0, sizeof(tg_stage) * (255 - S));
    }
    delete owned;
    return st;
}

extern "C" {

tg_status tg_compose_pipeline(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                              const double *d_cost, const uint8_t *d_dmax, const int32_t *island_order,
                              tg_plan *out, void *d_ws, size_t ws_bytes, tg_stream stream) {
    hipStream_t s = (hipStream_t)stream;
    if (!island_order) return fail(TG_EINVAL, "NULL argument");
    const size_t need = p && n_survivors >= 0 ? tg::compose_ws_bytes(p->P, n_survivors) : 0;
    tg_status st = compose_begin(p, d_survivors, n_survivors, d_cost, d_dmax, island_order, out, d_ws, ws_bytes,
                                 need, s);
    if (st != TG_OK) return st;
    tg::ComposeResult *res_dev = nullptr;
    // the handle's pinned read-back words, when no other call holds them: the
    // kernels store the depth limits and the result there
    std::unique_lock<std::mutex> lock;
    const tg::HostStage *pw = pinned_words(p, lock);
    if (pw && !p->compose_ev && hipEventCreateWithFlags(&p->compose_ev, hipEventDisableTiming) != hipSuccess) {
        p->compose_ev = nullptr;  // then the depth limits are read back by a stream synchronisation
        (void)hipGetLastError();
    }
    tg::ComposeHost host{};
    if (pw) {
        const size_t at = readback_dlim_at();
        host = tg::ComposeHost{(int32_t *)((char *)pw->ptr + at), (int32_t *)((char *)pw->dev + at),
                               (tg::ComposeResult *)pw->ptr, (tg::ComposeResult *)pw->dev, p->compose_ev};
        if (!host.ev) host.dlim = host.dlim_dev = nullptr;
    }
    hipError_t e = tg::launch_compose(p->P, d_survivors, n_survivors, d_cost, d_dmax, nullptr, d_ws, s, &res_dev,
                                      pw ? &host : nullptr);
    if (e != hipSuccess) {
        (void)hipStreamSynchronize(s);  // nothing queued may store into the words once they are let go
        return hip_fail(e, "compose kernels");
    }
    return compose_end(res_dev, out, s, host.res);
}

tg_status tg_compose_pipeline_classes(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                                      const double *d_cost, const uint8_t *d_dmax, const int32_t *island_order,
                                      tg_plan *out, void *d_ws, size_t ws_bytes, tg_stream stream) {
    hipStream_t s = (hipStream_t)stream;
    if (!island_order) return fail(TG_EINVAL, "NULL argument");
    const size_t need = p && n_survivors >= 0 ? tg::compose_ws_bytes(p->P, n_survivors) : 0;
    tg_status st = compose_begin(p, d_survivors, n_survivors, d_cost, d_dmax, island_order, out, d_ws, ws_bytes,
                                 need, s);
    if (st != TG_OK) return st;
    tg::DevProblem P = p->P;
    P.class_scores = 1;
    tg::ComposeResult *res_dev = nullptr;
    hipError_t e = tg::launch_compose(P, d_survivors, n_survivors, d_cost, d_dmax, nullptr, d_ws, s, &res_dev);
    if (e != hipSuccess) return hip_fail(e, "compose kernels");
    return compose_end(res_dev, out, s);
}

tg_status tg_compose_pipeline_relaxed(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                                      const double *d_cost, const uint8_t *d_dmax, const int32_t *island_order,
                                      tg_plan *out, void *d_ws, size_t ws_bytes, tg_stream stream) {
    hipStream_t s = (hipStream_t)stream;
    if (!island_order) return fail(TG_EINVAL, "NULL argument");
    const size_t need = p && n_survivors >= 0 ? tg::compose_relaxed_ws_bytes(p->P, n_survivors) : 0;
    tg_status st = compose_begin(p, d_survivors, n_survivors, d_cost, d_dmax, island_order, out, d_ws, ws_bytes,
                                 need, s);
    if (st != TG_OK) return st;
    return no_throw([&] {
        std::lock_guard<std::mutex> lock(p->relax_mu);  // one relaxed call at a time uses the handle's staging
        // coherent: kernels store the depth limits and the result straight to host memory
        const hipError_t es = p->relax_stage.reserve(tg::compose_relaxed_stage_bytes(p->P),
                                                     hipHostMallocPortable | hipHostMallocCoherent);
        if (es != hipSuccess) return hip_fail(es, "pinned host staging");
        if (!p->relax_ev && hipEventCreateWithFlags(&p->relax_ev, hipEventDisableTiming) != hipSuccess) {
            p->relax_ev = nullptr;  // the depth limits are then read back by a stream synchronisation
            (void)hipGetLastError();
        }
        const tg::RelaxHost H{p->outact.data(), p->E.data(), p->bvals.data(), p->B, &p->relax_stage, p->relax_ev};
        tg::ComposeResult *res_dev = nullptr;
        const tg::ComposeResult *res_host = nullptr;
        int rounds = 0;
        hipError_t e = tg::launch_compose_relaxed(p->P, H, island_order, d_survivors, n_survivors, d_cost, d_dmax,
                                                  d_ws, s, &res_dev, &res_host, &rounds);
        if (e != hipSuccess) {
            (void)hipStreamSynchronize(s);  // nothing queued may use the staging once it is let go
            return hip_fail(e, "relaxed compose kernels");
        }
        return compose_end(res_dev, out, s, res_host);
    });
}

size_t tg_build_islands_workspace_bytes(int32_t n_nodes) {
    if (n_nodes < 1 || n_nodes > 4096) return 0;
    return tg::islands_ws_bytes(n_nodes);
}

tg_status tg_build_islands(const tg_island *nodes, int32_t n_nodes, const double *node_bw, double eps_compute,
                           double eps_memory, double eps_intra, int32_t *island_of, tg_island *islands,
                           double *inter_bw, int32_t *n_islands, void *d_ws, size_t ws_bytes, tg_stream stream) {
    if (!nodes || !node_bw || !island_of || !islands || !inter_bw || !n_islands)
        return fail(TG_EINVAL, "NULL argument");
    if (n_nodes < 1 || n_nodes > 4096) return fail(TG_EINVAL, "n_nodes %d outside [1, 4096]", n_nodes);
    for (double x : {eps_compute, eps_memory, eps_intra})
        if (!(x >= 0.0) || !std::isfinite(x)) return fail(TG_EINVAL, "tolerance invalid");
    for (int u = 0; u < n_nodes; ++u) {
        const tg_island &v = nodes[u];
        if (v.n_gpus < 1 || v.n_gpus > kMaxNodeGpus || v.reserved != 0) return fail(TG_EINVAL, "node %d GPU count", u);
        if (!(v.peak_flops > 0.0) || !std::isfinite(v.peak_flops) || !(v.hbm_bytes > 0.0) ||
            !std::isfinite(v.hbm_bytes) || !(v.intra_bw > 0.0) || !std::isfinite(v.intra_bw) ||
            !(v.host_bw >= 0.0) || !std::isfinite(v.host_bw))
            return fail(TG_EINVAL, "node %d specs", u);
    }
    const size_t need = tg::islands_ws_bytes(n_nodes);
    if (!d_ws || ws_bytes < need) return fail(TG_ENOMEM, "workspace %zu < %zu bytes", ws_bytes, need);
    if (check_alignment(nullptr, nullptr, d_ws) != TG_OK) return TG_EINVAL;
    return no_throw([&] {
        int64_t bad = -1;  // node_bw is checked on the device, right after its upload
        hipError_t e = tg::launch_build_islands(n_nodes, nodes, node_bw, eps_compute, eps_memory, eps_intra, d_ws,
                                                (hipStream_t)stream, island_of, islands, inter_bw, n_islands, &bad);
        if (e != hipSuccess) return hip_fail(e, "island construction kernels");
        if (bad >= 0) return fail(TG_EINVAL, "node_bw[%lld]", (long long)bad);
        return TG_OK;
    });
}

tg_status tg_compose_pipeline_all_orders(const tg_problem *p, const int64_t *d_survivors, int64_t n_survivors,
                                         const double *d_cost, const uint8_t *d_dmax, tg_plan *out, void *d_ws,
                                         size_t ws_bytes, tg_stream stream) {
    hipStream_t s = (hipStream_t)stream;
    if (p && p->P.K > 16) return fail(TG_EINVAL, "composition over all island orders takes at most 16 islands");
    if (p && p->P.nb > 65535) return fail(TG_EINVAL, "more than 65535 micro-batch sizes");
    const size_t need = p && n_survivors >= 0 ? tg::compose_orders_ws_bytes(p->P, n_survivors) : 0;
    tg_status st = compose_begin(p, d_survivors, n_survivors, d_cost, d_dmax, nullptr, out, d_ws, ws_bytes, need, s);
    if (st != TG_OK) return st;
    tg::ComposeResult *res_dev = nullptr;
    hipError_t e = tg::launch_compose_orders(p->P, p->bvals.data(), d_survivors, n_survivors, d_cost, d_dmax, d_ws, s,
                                             &res_dev);
    if (e != hipSuccess) return hip_fail(e, "all-orders compose kernels");
    return compose_end(res_dev, out, s);
}

}  // extern "C"
