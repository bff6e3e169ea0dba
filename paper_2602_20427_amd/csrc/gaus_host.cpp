// Host side of libgaus: problem validation and preprocessing, device buffers,
// launch configuration and the extern "C" entry points declared in gaus.h.
#include "../../include/gaus.h"
#include "gaus_internal.h"

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

using namespace gaus;

namespace {

thread_local std::string g_init_error = "no error";


}  // namespace

struct gaus_ctx {
    Graph g{};
    Work w{};
    HP hp{};
    LaunchCfg lc{};
    hipStream_t stream = nullptr;
    int device = 0;
    void *scratch = nullptr;            // this device's copy of the library's scratch array
    std::vector<void *> allocs;
    std::vector<int> asap, alap;
    std::string err = "no error";
    // bound optimizer state (caller-owned device memory)
    float *mu = nullptr, *sigma = nullptr, *m = nullptr, *v = nullptr, *lambda = nullptr;
    int *adam_t = nullptr;
    bool bound = false;
    PolyArgs pa{};
    int poly_slots = 0;                 // per-work-group output slots of the polynomial kernels
    // kernel timing (gaus_kernel_timing): per sampled iteration two pairs of
    // events, [4k, 4k+1] around the op kernel and [4k+2, 4k+3] around the
    // polynomial kernel; every timing_every-th iteration is sampled
    bool timing = false;
    int timing_every = 1;
    long long timing_iter = 0;          // iterations enqueued since timing was enabled
    std::vector<hipEvent_t> ev_pool;
    size_t ev_used = 0;                 // iterations recorded since the last read
};

constexpr int kPolySplitMax = 4;   // polynomial work-groups per op group, at most
constexpr int kPackOpsPerWave = 8; // packed grids: ops per wave, at most (when the split allows)
constexpr int kPackSplitMax = 16;  // packed grids: work-groups per op group, at most

namespace {

gaus_status fail(gaus_ctx *c, gaus_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (c) c->err = buf;
    else g_init_error = buf;
    return s;
}

gaus_status hip_fail(gaus_ctx *c, hipError_t e, const char *what) {
    return fail(c, GAUS_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

void free_all(gaus_ctx *c) {
    for (void *p : c->allocs) (void)hipFree(p);
    c->allocs.clear();
    for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
    c->ev_pool.clear();
    c->ev_used = 0;
}

// Timing events of the next iteration (nulls when timing is off).
hipError_t next_events(gaus_ctx *c, IterArgs &a) {
    a.ops_begin = a.ops_end = a.poly_begin = a.poly_end = nullptr;
    if (!c->timing || c->timing_iter++ % c->timing_every != 0) return hipSuccess;
    while (4 * c->ev_used + 4 > c->ev_pool.size()) {
        hipEvent_t ev;
        hipError_t r = hipEventCreate(&ev);
        if (r != hipSuccess) return r;
        c->ev_pool.push_back(ev);
    }
    hipEvent_t *e = &c->ev_pool[4 * c->ev_used];
    a.ops_begin = e[0]; a.ops_end = e[1];
    if (c->pa.enabled) { a.poly_begin = e[2]; a.poly_end = e[3]; }
    c->ev_used++;
    return hipSuccess;
}

// Truncation bound of an op's chunk series at degree d and rho = lam/sigma:
// the error of the density series (degree d-1) over the chunk, relative to
// the family's peak density.
//   Gaussian: Taylor remainder with Cramer's bound |He_n(x)| e^(-x^2/4) <=
//     1.09 sqrt(n!): 1.09 rho^d / sqrt(d!);
//   logistic: the density 1/(4 cosh^2(u/2)) has double poles at u = +-i pi,
//     so its n-th coefficient is at most 2 (n+1)/pi^(n+2); with x = rho/sqrt(3)
//     (rho in u units over pi): 8 (d+1)/pi^2 x^d/(1 - x);
//   Cauchy: the coefficients of 1/(1 + u^2) are at most 1 in modulus (poles
//     at +-i), x = rho/sqrt(2 ln 2): x^d/(1 - x).
double poly_bound(int fam, int d, double rho) {
    auto fact = [](int n) { double f = 1.0; for (int q = 2; q <= n; ++q) f *= q; return f; };
    if (fam == 1) {
        const double x = rho / std::sqrt(3.0);
        return 8.0 * (d + 1) / (M_PI * M_PI) * std::pow(x, d) / (1.0 - x);
    }
    if (fam == 3) {
        const double x = rho / std::sqrt(2.0 * std::log(2.0));
        return std::pow(x, d) / (1.0 - x);
    }
    return 1.09 * std::pow(rho, d) / std::sqrt(fact(d));
}

// Tier bounds and moment table of a grid with chunk width W: each tier's rho
// bound gives the family's truncation bound the value of the Gaussian
// degree-8 bound at rho = kRhoMax (the Gaussian in closed form,
// rho_d = (kRhoMax^8 sqrt(d!) / sqrt(8!))^(1/d); the other families by
// bisection of their increasing bounds).
void setup_grid(int D, int W, int nc, int fam, GridArgs &gr) {
    gr = GridArgs{};
    gr.on = 1;
    gr.W = W; gr.nc = nc;
    gr.L0 = D - 2 - nc * W;
    gr.SP = gr.L0 + 2;
    const double lam = (W - 1) / 2.0;
    gr.lam = (float)lam;
    auto fact = [](int n) { double f = 1.0; for (int q = 2; q <= n; ++q) f *= q; return f; };
    const double target = poly_bound(0, kDeg, kRhoMax);
    for (int t = 1; t <= kTiers; ++t) {
        const int d = kTierDeg[t];
        double rho;
        if (fam == 0) {
            rho = std::pow(std::pow((double)kRhoMax, kDeg) * std::sqrt(fact(d) / fact(kDeg)), 1.0 / d);
        } else {
            double lo = 0.0, hi = kRhoMax;
            for (int it = 0; it < 200; ++it) {
                const double m = 0.5 * (lo + hi);
                (poly_bound(fam, d, m) <= target ? lo : hi) = m;
            }
            rho = lo;
        }
        gr.sig_thr[t] = (float)(lam / rho);
    }
    gr.sig_thr[0] = gr.sig_thr[1];
    for (int k = 0; k <= kDeg; ++k) {
        double acc = 0.0;
        for (int i = 0; i < W; ++i) acc += std::pow(i - lam, 2 * k);
        gr.H[k] = (float)acc;   // symmetric points: odd moments vanish
    }
}

// Chunk grids, strips, tier bounds and constant tables of the polynomial
// path (families with an analytic CDF: Gaussian, logistic, Cauchy).
// requested: grid-0 chunk width (0 = chosen here, < 0 = path off);
// pack: packed grids (0 = when the width is chosen here, > 0 = on, < 0 = off),
// used only for grids whose restart pack fits B; storage: the storage term
// is on (a chosen width stays >= kMinChunkStorage).
void setup_poly(int D, int requested, int pack, int fam, int B, bool storage, PolyArgs &pa) {
    pa = PolyArgs{};
    if (requested < 0 || !(fam == 0 || fam == 1 || fam == 3)) return;
    // Grid 0: chunks tile [L0, D-2) with nc <= 64 chunks (one per lane); the
    // strip [0, L0) u {D-2, D-1} is evaluated step by step in passes of 64
    // lanes.  Take the fewest strip passes, then the smallest W (the lowest
    // sigma threshold 2(W-1) for the polynomial path).
    int W = 0, nc = 0, best_passes = 1 << 30;
    const int w0 = requested > 0 ? kMinChunk : storage ? kMinChunkStorage : kMinChunk;
    for (int w = w0; w <= kMaxChunk; ++w) {
        if (requested > 0 && w != requested) continue;
        const int n = std::min(kMaxChunks, (D - 2 - kSmax) / w);
        if (n < 4) continue;
        const int sp = D - 2 - n * w + 2;
        if (sp > kStripMax) continue;
        const int passes = (sp + 63) / 64;
        if (passes < best_passes) { best_passes = passes; W = w; nc = n; }
    }
    if (W == 0) return;
    pa.enabled = 1;
    pa.fam = fam;
    setup_grid(D, W, nc, fam, pa.gr[0]);
    pa.W = W; pa.nc = nc; pa.L0 = pa.gr[0].L0; pa.SP = pa.gr[0].SP; pa.lam = pa.gr[0].lam;
    for (int t = 0; t <= kTiers; ++t) pa.sig_thr[t] = pa.gr[0].sig_thr[t];
    for (int k = 0; k <= kDeg; ++k) pa.H[k] = pa.gr[0].H[k];
    // storage holders: the Gaussian's 1/4, scaled for the other families as
    // their degree-8 rho is to the Gaussian's (the rho at which the family's
    // truncation bound equals the Gaussian one)
    pa.mem_rho = fam == 0 ? kMemRhoMax : (float)(kMemRhoMax / kRhoMax * pa.lam / pa.sig_thr[1]);
    // Packed grids: 64/P lanes per restart, at most that many chunks and a
    // strip of at most that many positions (one pass); the smallest such W
    // (W <= 256 keeps the degree-16 moments within fp32 range).
    const bool packing = pack > 0 || (pack == 0 && requested == 0);
    for (int g = 1; g < kGrids && packing; ++g) {
        const int P = kGridP[g], L = 64 / P;
        if (B < P) continue;
        for (int w = kMinChunkStorage; w <= kMaxChunk; ++w) {
            const int n = std::min(L, (D - 2 - kSmax) / w);
            if (n < 4) continue;
            if (D - 2 - n * w + 2 > L) continue;
            setup_grid(D, w, n, fam, pa.gr[g]);
            break;
        }
    }
}

template <class T>
gaus_status dalloc(gaus_ctx *c, T **out, size_t count) {
    void *p = nullptr;
    const size_t bytes = std::max<size_t>(count, 1) * sizeof(T);
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) return fail(nullptr, GAUS_E_NOMEM, "hipMalloc(%zu bytes): %s", bytes, hipGetErrorString(e));
    c->allocs.push_back(p);
    *out = static_cast<T *>(p);
    return GAUS_OK;
}

template <class T>
gaus_status dupload(gaus_ctx *c, const T **out, const std::vector<T> &h) {
    T *d = nullptr;
    gaus_status s = dalloc(c, &d, h.size());
    if (s != GAUS_OK) return s;
    if (!h.empty()) {
        hipError_t e = hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice);
        if (e != hipSuccess) return fail(nullptr, GAUS_E_DEVICE, "hipMemcpy: %s", hipGetErrorString(e));
    }
    *out = d;
    return GAUS_OK;
}

// Preprocessed host copy of a validated problem.
struct HostGraph {
    int N = 0, E = 0, K = 0, D = 0, II = 0, nb = 0;
    std::vector<int> row_ptr, col, delay, rtype, bsrc, bdst, bdist;
    std::vector<int> esrc;                   // producer of each CSR edge
    std::vector<float> cap, bmem;
    std::vector<int> pred_ptr, pred_eid, pred_src;
    std::vector<int> bin_ptr, bin, bout_ptr, bout;
    std::vector<int> level, lvl_ptr, lvl_ops;
    std::vector<int> leg_items, leg_over;   // legalization items in level order (see Graph::leg_items)
    int leg_nover = 0;                       // predecessors in leg_over (before padding)
    std::vector<int> leg_batch;              // ring batches (see Graph::leg_batch)
    std::vector<int> asap, alap;
    std::vector<int> perm, grp_start, type_grp, grp_of;
    std::vector<int> big_ops, big_of;
};

gaus_status validate(const gaus_problem *p, int32_t B) {
    if (!p) return fail(nullptr, GAUS_E_INVALID_ARG, "problem is NULL");
    if (p->n_ops < 1) return fail(nullptr, GAUS_E_INVALID_ARG, "n_ops must be >= 1 (got %d)", p->n_ops);
    if (p->n_edges < 0) return fail(nullptr, GAUS_E_INVALID_ARG, "n_edges must be >= 0");
    if (p->n_types < 1) return fail(nullptr, GAUS_E_INVALID_ARG, "n_types must be >= 1");
    if (p->D < 1 || p->D > (1 << 22)) return fail(nullptr, GAUS_E_INVALID_ARG, "D must be in [1, 2^22] (got %d)", p->D);
    if (p->II < 0) return fail(nullptr, GAUS_E_INVALID_ARG, "II must be >= 0");
    if (p->n_back < 0) return fail(nullptr, GAUS_E_INVALID_ARG, "n_back must be >= 0");
    if (p->n_back > 0 && p->II == 0) return fail(nullptr, GAUS_E_INVALID_ARG, "back edges require II > 0");
    if (B < 1 || B > 65535) return fail(nullptr, GAUS_E_INVALID_ARG, "B must be in [1, 65535] (got %d)", B);
    if (!p->row_ptr || !p->delay || !p->rtype || !p->capacity || (p->n_edges > 0 && !p->col_idx) ||
        (p->n_back > 0 && (!p->back_src || !p->back_dst || !p->back_dist)))
        return fail(nullptr, GAUS_E_INVALID_ARG, "null array pointer in problem");
    const int N = p->n_ops;
    if (p->row_ptr[0] != 0 || p->row_ptr[N] != p->n_edges)
        return fail(nullptr, GAUS_E_INVALID_ARG, "row_ptr must start at 0 and end at n_edges");
    for (int i = 0; i < N; ++i)
        if (p->row_ptr[i + 1] < p->row_ptr[i]) return fail(nullptr, GAUS_E_INVALID_ARG, "row_ptr decreases at %d", i);
    for (int e = 0; e < p->n_edges; ++e)
        if (p->col_idx[e] < 0 || p->col_idx[e] >= N) return fail(nullptr, GAUS_E_INVALID_ARG, "col_idx[%d] out of range", e);
    {
        std::vector<int> row;
        for (int i = 0; i < N; ++i) {
            row.assign(p->col_idx + p->row_ptr[i], p->col_idx + p->row_ptr[i + 1]);
            std::sort(row.begin(), row.end());
            if (std::adjacent_find(row.begin(), row.end()) != row.end())
                return fail(nullptr, GAUS_E_INVALID_ARG, "duplicate edge from op %d", i);
        }
    }
    if (p->mem_units)
        for (int i = 0; i < N; ++i)
            if (!std::isfinite(p->mem_units[i]) || p->mem_units[i] < 0.0f)
                return fail(nullptr, GAUS_E_INVALID_ARG, "mem_units[%d] must be finite and >= 0", i);
    for (int i = 0; i < N; ++i) {
        if (p->delay[i] < 0 || p->delay[i] > (1 << 20)) return fail(nullptr, GAUS_E_INVALID_ARG, "delay[%d] out of [0, 2^20]", i);
        if (p->rtype[i] < 0 || p->rtype[i] >= p->n_types) return fail(nullptr, GAUS_E_INVALID_ARG, "rtype[%d] out of range", i);
    }
    for (int k = 0; k < p->n_types; ++k)
        if (!std::isfinite(p->capacity[k]) || p->capacity[k] < 0.0f)
            return fail(nullptr, GAUS_E_INVALID_ARG, "capacity[%d] must be finite and >= 0", k);
    for (int e = 0; e < p->n_back; ++e) {
        const int j = p->back_src[e], i = p->back_dst[e], k = p->back_dist[e];
        if (j < 0 || j >= N || i < 0 || i >= N) return fail(nullptr, GAUS_E_INVALID_ARG, "back edge %d: op out of range", e);
        if (i == j) return fail(nullptr, GAUS_E_INVALID_ARG, "back edge %d is a self loop (Lat <= k*II is a static check)", e);
        if (k < 1 || (long long)k * p->II > (1LL << 30)) return fail(nullptr, GAUS_E_INVALID_ARG, "back edge %d: need 1 <= k, k*II <= 2^30", e);
    }
    return GAUS_OK;
}

gaus_status preprocess(const gaus_problem *p, HostGraph &h) {
    const int N = p->n_ops, E = p->n_edges;
    h.N = N; h.E = E; h.K = p->n_types; h.D = p->D; h.II = p->II; h.nb = p->n_back;
    h.row_ptr.assign(p->row_ptr, p->row_ptr + N + 1);
    h.col.assign(p->col_idx, p->col_idx + E);
    h.delay.assign(p->delay, p->delay + N);
    h.rtype.assign(p->rtype, p->rtype + N);
    h.cap.assign(p->capacity, p->capacity + h.K);
    if (p->mem_units) h.bmem.assign(p->mem_units, p->mem_units + N);
    else h.bmem.assign(N, 1.0f);
    h.bsrc.assign(p->back_src, p->back_src + h.nb);
    h.bdst.assign(p->back_dst, p->back_dst + h.nb);
    h.bdist.assign(p->back_dist, p->back_dist + h.nb);

    // CSC (predecessors in producer-id order, with the CSR edge id)
    h.pred_ptr.assign(N + 1, 0);
    for (int e = 0; e < E; ++e) h.pred_ptr[h.col[e] + 1]++;
    for (int i = 0; i < N; ++i) h.pred_ptr[i + 1] += h.pred_ptr[i];
    h.pred_eid.assign(E, 0); h.pred_src.assign(E, 0);
    {
        std::vector<int> fill(N, 0);
        for (int i = 0; i < N; ++i)
            for (int e = h.row_ptr[i]; e < h.row_ptr[i + 1]; ++e) {
                const int j = h.col[e];
                const int q = h.pred_ptr[j] + fill[j]++;
                h.pred_eid[q] = e; h.pred_src[q] = i;
            }
    }

    // back edges by consumer and by producer
    h.bin_ptr.assign(N + 1, 0); h.bout_ptr.assign(N + 1, 0);
    for (int e = 0; e < h.nb; ++e) { h.bin_ptr[h.bdst[e] + 1]++; h.bout_ptr[h.bsrc[e] + 1]++; }
    for (int i = 0; i < N; ++i) { h.bin_ptr[i + 1] += h.bin_ptr[i]; h.bout_ptr[i + 1] += h.bout_ptr[i]; }
    h.bin.assign(h.nb, 0); h.bout.assign(h.nb, 0);
    {
        std::vector<int> f1(N, 0), f2(N, 0);
        for (int e = 0; e < h.nb; ++e) {
            h.bin[h.bin_ptr[h.bdst[e]] + f1[h.bdst[e]]++] = e;
            h.bout[h.bout_ptr[h.bsrc[e]] + f2[h.bsrc[e]]++] = e;
        }
    }
    // Kahn levels; ops by (level, id)
    h.level.assign(N, 0);
    {
        std::vector<int> indeg(N), queue;
        queue.reserve(N);
        for (int i = 0; i < N; ++i) indeg[i] = h.pred_ptr[i + 1] - h.pred_ptr[i];
        for (int i = 0; i < N; ++i) if (indeg[i] == 0) queue.push_back(i);
        for (size_t qh = 0; qh < queue.size(); ++qh) {
            const int u = queue[qh];
            for (int e = h.row_ptr[u]; e < h.row_ptr[u + 1]; ++e) {
                const int v = h.col[e];
                h.level[v] = std::max(h.level[v], h.level[u] + 1);
                if (--indeg[v] == 0) queue.push_back(v);
            }
        }
        if ((int)queue.size() != N) return fail(nullptr, GAUS_E_CYCLE, "forward edges contain a cycle");
        const int L = 1 + *std::max_element(h.level.begin(), h.level.end());
        h.lvl_ptr.assign(L + 1, 0);
        for (int i = 0; i < N; ++i) h.lvl_ptr[h.level[i] + 1]++;
        for (int l = 0; l < L; ++l) h.lvl_ptr[l + 1] += h.lvl_ptr[l];
        h.lvl_ops.assign(N, 0);
        std::vector<int> fill(L, 0);
        for (int i = 0; i < N; ++i) h.lvl_ops[h.lvl_ptr[h.level[i]] + fill[h.level[i]]++] = i;
    }
    // ASAP / ALAP with delays; sinks' ALAP = D-1
    {
        std::vector<long long> as(N, 0), al(N, 0);
        for (int q = 0; q < N; ++q) {
            const int u = h.lvl_ops[q];
            for (int e = h.row_ptr[u]; e < h.row_ptr[u + 1]; ++e) {
                const int v = h.col[e];
                as[v] = std::max(as[v], as[u] + h.delay[u]);
            }
        }
        for (int q = N - 1; q >= 0; --q) {
            const int v = h.lvl_ops[q];
            long long best = (long long)h.D - 1;
            for (int e = h.row_ptr[v]; e < h.row_ptr[v + 1]; ++e) best = std::min(best, al[h.col[e]] - h.delay[v]);
            al[v] = best;
        }
        for (int i = 0; i < N; ++i)
            if (as[i] > al[i])
                return fail(nullptr, GAUS_E_HORIZON, "critical path does not fit the horizon: ASAP[%d]=%lld > ALAP=%lld (D=%d)",
                            i, as[i], al[i], h.D);
        h.asap.assign(as.begin(), as.end());
        h.alap.assign(al.begin(), al.end());
    }
    return GAUS_OK;
}

// Launch shape of the op kernel and op grouping.
void choose_config(HostGraph &h, int B, LaunchCfg &lc, int &tile, int &ntiles) {
    if (h.D <= 64) { lc.bs = 64; lc.spt = 1; }
    else if (h.D <= 512) { lc.bs = 256; lc.spt = 1; }
    else { lc.bs = 256; lc.spt = 4; }
    tile = lc.bs * lc.spt;
    ntiles = (h.D + tile - 1) / tile;
    // group size: enough work-groups to fill 256 CUs several times over
    const long long target = 2048;
    long long per = (long long)h.N * B * ntiles / target;
    // at most one op per thread of the op kernel's work-group (it flags the group's ops in parallel)
    int G = (int)std::min<long long>(lc.bs, std::max<long long>(4, per));
    // ops sorted by (type, id), cut into type-pure groups of <= G ops
    h.perm.resize(h.N);
    for (int i = 0; i < h.N; ++i) h.perm[i] = i;
    std::stable_sort(h.perm.begin(), h.perm.end(), [&](int a, int b) { return h.rtype[a] < h.rtype[b]; });
    h.grp_start.clear();
    h.type_grp.assign(h.K + 1, 0);
    int q = 0;
    for (int k = 0; k < h.K; ++k) {
        h.type_grp[k] = (int)h.grp_start.size();
        int cnt = 0;
        while (q + cnt < h.N && h.rtype[h.perm[q + cnt]] == k) ++cnt;
        for (int s = 0; s < cnt; s += G) h.grp_start.push_back(q + s);
        q += cnt;
    }
    h.type_grp[h.K] = (int)h.grp_start.size();
    h.grp_start.push_back(h.N);
    h.big_of.assign(h.N, -1);
    for (int i = 0; i < h.N; ++i)
        if (h.pred_ptr[i + 1] - h.pred_ptr[i] > kBigIn) {
            h.big_of[i] = (int)h.big_ops.size();
            h.big_ops.push_back(i);
        }
    h.grp_of.assign(h.N, 0);
    for (size_t gi = 0; gi + 1 < h.grp_start.size(); ++gi)
        for (int q = h.grp_start[gi]; q < h.grp_start[gi + 1]; ++q) h.grp_of[h.perm[q]] = (int)gi;
}

}  // namespace

extern "C" {

void gaus_default_hparams(gaus_hparams *hp) {
    if (!hp) return;
    hp->lr = 1e-2f;
    hp->beta1 = 0.9f;
    hp->beta2 = 0.999f;
    hp->eps = 1e-8f;
    hp->rho = 1e-4f;
    hp->lambda0 = 1e-6f;
    hp->alpha_com = 0.01f;
    hp->sigma_min = 0.05f;
    hp->kappa = 1.0f / 6.0f;
    hp->poly_chunk = 0;
    hp->beta_res = 0.0f;
    hp->tau = 1e-2f;
    hp->gamma_mem = 0.0f;
    hp->family = 0;
    hp->poly_pack = 0;
}

const char *gaus_status_string(gaus_status s) {
    switch (s) {
        case GAUS_OK: return "GAUS_OK";
        case GAUS_E_INVALID_ARG: return "GAUS_E_INVALID_ARG";
        case GAUS_E_CYCLE: return "GAUS_E_CYCLE";
        case GAUS_E_HORIZON: return "GAUS_E_HORIZON";
        case GAUS_E_NOT_CONVERGED: return "GAUS_E_NOT_CONVERGED";
        case GAUS_E_OVERFLOW: return "GAUS_E_OVERFLOW";
        case GAUS_E_DEVICE: return "GAUS_E_DEVICE";
        case GAUS_E_NOMEM: return "GAUS_E_NOMEM";
    }
    return "GAUS_E_UNKNOWN";
}

const char *gaus_last_error(const gaus_ctx *ctx) {
    return ctx ? ctx->err.c_str() : g_init_error.c_str();
}

gaus_status gaus_init(const gaus_problem *prob, const gaus_hparams *hp_in, int32_t B, void *hip_stream,
                      gaus_ctx **out) {
    if (!out) return fail(nullptr, GAUS_E_INVALID_ARG, "out is NULL");
    *out = nullptr;
    gaus_status s = validate(prob, B);
    if (s != GAUS_OK) return s;
    gaus_hparams hp;
    if (hp_in) hp = *hp_in; else gaus_default_hparams(&hp);
    if (hp.poly_chunk > 0 && (hp.poly_chunk < kMinChunk || hp.poly_chunk > kMaxChunk))
        return fail(nullptr, GAUS_E_INVALID_ARG, "poly_chunk must be 0 (auto), negative (off) or in [%d, %d]", kMinChunk,
                    kMaxChunk);
    if (!(hp.beta_res >= 0.0f) || !std::isfinite(hp.beta_res) || !(hp.tau > 0.0f) || !std::isfinite(hp.tau) ||
        !(hp.gamma_mem >= 0.0f) || !std::isfinite(hp.gamma_mem))
        return fail(nullptr, GAUS_E_INVALID_ARG, "beta_res and gamma_mem must be finite and >= 0, tau finite and > 0");
    if (hp.family < 0 || hp.family > 3)
        return fail(nullptr, GAUS_E_INVALID_ARG, "family must be 0 (Gaussian), 1 (logistic), 2 (Laplace) or 3 (Cauchy)");
    HostGraph h;
    s = preprocess(prob, h);
    if (s != GAUS_OK) return s;

    gaus_ctx *c = new (std::nothrow) gaus_ctx();
    if (!c) return fail(nullptr, GAUS_E_NOMEM, "host allocation failed");
    c->hp = HP{hp.lr,        hp.beta1,     hp.beta2,     hp.eps,      hp.rho, hp.lambda0,
               hp.alpha_com, hp.sigma_min, hp.kappa,     hp.beta_res, hp.tau, hp.gamma_mem,
               hp.family};
    c->stream = static_cast<hipStream_t>(hip_stream);
    (void)hipGetDevice(&c->device);
    {
        // address of the scratch array on this device (the allocation-free
        // entry point's workspace), taken once per device with it current
        const hipError_t e = scratch_address(c->device, &c->scratch);
        if (e != hipSuccess) {
            delete c;
            return fail(nullptr, GAUS_E_DEVICE, "scratch address: %s", hipGetErrorString(e));
        }
    }
    int tile = 0, ntiles = 0;
    choose_config(h, B, c->lc, tile, ntiles);
    c->lc.fam = hp.family;
    // the chunk polynomials take the Gaussian, logistic and Cauchy laws; the
    // Laplace CDF has a kink at the median (no series over a chunk there)
    setup_poly(h.D, hp.poly_chunk, hp.poly_pack, hp.family, B, hp.gamma_mem > 0.0f, c->pa);

    Graph &g = c->g;
    g.N = h.N; g.E = h.E; g.K = h.K; g.D = h.D; g.II = h.II; g.T = h.II > 0 ? h.II : h.D;
    g.nb = h.nb; g.B = B; g.tile = tile; g.ntiles = ntiles;
    g.ngroups = (int)h.grp_start.size() - 1;
    // the narrow kernel pays off where the op kernel would visit each op in
    // several tiles; its usage row must fit LDS
    // Laplace start times: the forward edges in closed form (the op kernel
    // keeps the usage), so the narrow kernel has nothing to take
    g.lap_on = hp.family == 2 ? 1 : 0;
    g.nar_on = (ntiles > 1 && h.D <= kNarMaxD && !g.lap_on) ? 1 : 0;
    {
        // a small op-kernel grid (few tiles) over many ops leaves the last round
        // of work-groups mostly idle: split each (group, tile) over 2
        // work-groups (small problems keep one: their op kernel is short).
        // Each part writes a usage row of its own, which k_usage reads: 4
        // parts cost more there than they saved in the op kernel.
        const long long wgs = (long long)g.ngroups * ntiles * B;
        g.parts = (wgs >= 4096 || (long long)h.N * B < (1 << 18))
                      ? 1 : (int)std::min<long long>(2, (8192 + wgs - 1) / wgs);
    }
    if (c->pa.enabled) {
        // polynomial work-groups per op group: at most 16 ops per wave, so that
        // every SIMD receives many short waves and the last ones end together
        int gmax = 1;
        for (int q = 0; q < g.ngroups; ++q) gmax = std::max(gmax, h.grp_start[q + 1] - h.grp_start[q]);
        c->pa.split = std::max(1, std::min(kPolySplitMax, (gmax + 63) / 64));
        c->pa.gr[0].split = c->pa.split;
        // packed grids: at most kPackOpsPerWave ops per wave (each wave-op
        // carries P restarts, so fewer ops per wave keep the last waves short)
        int base = 0;
        for (int gi = 0; gi < kGrids; ++gi) {
            GridArgs &gr = c->pa.gr[gi];
            if (gi > 0)
                gr.split = std::max(1, std::min(kPackSplitMax, (gmax + 4 * kPackOpsPerWave - 1) / (4 * kPackOpsPerWave)));
            // the packed kernels load each wave's ops on 64/P >= 16 lanes per restart
            if (gi > 0 && (gmax + gr.split - 1) / gr.split > 64) gr.on = 0;
            gr.slot_base = base;
            if (gr.on) base += B * g.ngroups * gr.split;
        }
        c->poly_slots = base;
    }
    g.nlevels = (int)h.lvl_ptr.size() - 1;
    {
        // one 32-byte item per op in level order: op, delay, predecessor
        // count, start of the ones past kLegPre in leg_over, first kLegPre
        h.leg_items.assign((size_t)8 * std::max(h.N, 1), 0);
        h.leg_over.clear();
        for (int q = 0; q < h.N; ++q) {
            const int v = h.lvl_ops[q], p0 = h.pred_ptr[v], n = h.pred_ptr[v + 1] - p0;
            int *it = &h.leg_items[(size_t)8 * q];
            it[0] = v; it[1] = h.delay[v]; it[2] = n; it[3] = (int)h.leg_over.size();
            for (int k = 0; k < n; ++k) {
                if (k < kLegPre) it[4 + k] = h.pred_src[p0 + k];
                else h.leg_over.push_back(h.pred_src[p0 + k]);
            }
        }
        h.leg_nover = (int)h.leg_over.size();
        if (h.leg_over.empty()) h.leg_over.push_back(0);
    }
    {
        // legalization schedule in LDS when it fits: 16-bit ready times for
        // II = 0 (every s stays in [ASAP, ALAP] within [0, D-1]); 32-bit ones
        // and their pass snapshot for II > 0 while D + dmax + N^2 dmax (a
        // bound on what N passes can reach) stays below 2^31
        int lds = 0;
        if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, c->device) != hipSuccess)
            lds = 65536;
        const long long budget = std::min(lds, 160 * 1024) - 2048;
        long long dmax = 0;
        for (int d : h.delay) dmax = std::max<long long>(dmax, d);
        const long long N = h.N;
        const long long room = budget - 4LL * ((g.nlevels + 1 + 3) & ~3);   // after the level bounds
        g.leg_mode = 0;
        if (h.II == 0 && (long long)h.D + dmax < 32767 && 2 * N <= room) g.leg_mode = 1;
        else if (h.II == 0 && (long long)h.D + dmax < (1LL << 31) - 1 && 4 * N <= room) g.leg_mode = 2;
        else if (h.II > 0 && (long long)h.D + dmax + N * N * (dmax + 1) < (1LL << 31) - 1 && 8 * N <= room)
            g.leg_mode = 2;
        // II = 0 with the schedule in LDS: the level items through a double
        // ring in the LDS left over (two halves of RI items of 32 bytes and
        // RO = RI overflow predecessors), unless one op's predecessors exceed
        // a half
        g.leg_ring = 0;
        if (h.II == 0 && (g.leg_mode == 1 || g.leg_mode == 2) && g.nlevels > 1) {
            const long long rdb = (long long)(g.leg_mode == 1 ? 2 : 4) * N;
            const long long left = room - ((rdb + 15) & ~15LL);
            // ring halves of RI items; the batch table needs 12 bytes per
            // batch (at most N / RI + 2 batches unless one op's predecessors
            // fill a half) and is checked after the cut
            long long ri = std::min<long long>({left / 2 / 36, kLegRingItemsMax, kLegRingOverMax});
            for (; ri >= 64 && !g.leg_ring; ri = ri * 7 / 8) {
                const int RI = (int)ri, RO = (int)ri;
                // batches: contiguous item ranges from the first item of level 1
                // (a wide level spans several), each within RI items and RO
                // overflow predecessors; row = (level of the first item, first
                // item, first overflow predecessor)
                auto over_at = [&](int q) { return q < h.N ? h.leg_items[(size_t)8 * q + 3] : h.leg_nover; };
                std::vector<int> bt;
                bool fits = true;
                int q = h.lvl_ptr[1], l = 1;
                while (q < h.N && fits) {
                    while (h.lvl_ptr[l + 1] <= q) ++l;
                    const int o0 = over_at(q);
                    int q1 = std::min(h.N, q + RI);
                    while (q1 > q && over_at(q1) - o0 > RO) --q1;
                    if (q1 == q) fits = false;   // one item's predecessors exceed a half
                    bt.insert(bt.end(), {l, q, o0});
                    q = q1;
                }
                if (!fits) break;
                bt.insert(bt.end(), {g.nlevels, h.N, over_at(h.N)});
                const long long nbatch = (long long)bt.size() / 3 - 1;
                const long long need = ((rdb + 15) & ~15LL) + 4LL * ((3 * (nbatch + 1) + 3) & ~3LL) +
                                       2LL * 16 * (2 * RI + (RO + 3) / 4);
                if (need > room) continue;   // smaller halves, more batches
                h.leg_batch = bt;
                g.leg_nbatch = (int)nbatch;
                g.leg_ring_items = RI;
                g.leg_ring_over = RO;
                g.leg_ring = 1;
            }
        }
        if (h.leg_batch.empty()) h.leg_batch.assign(3, 0);
    }
    std::vector<float> cap(h.cap);
    const size_t BN = (size_t)B * h.N;
#define UP(field, vec) do { s = dupload(c, &g.field, vec); if (s != GAUS_OK) goto fail_alloc; } while (0)
    h.esrc.assign(std::max(h.E, 1), 0);
    for (int i = 0; i < h.N; ++i)
        for (int e = h.row_ptr[i]; e < h.row_ptr[i + 1]; ++e) h.esrc[e] = i;
    UP(esrc, h.esrc);
    UP(row_ptr, h.row_ptr); UP(col, h.col); UP(pred_ptr, h.pred_ptr); UP(pred_eid, h.pred_eid);
    UP(pred_src, h.pred_src); UP(delay, h.delay); UP(rtype, h.rtype); UP(cap, cap);
    UP(bsrc, h.bsrc); UP(bdst, h.bdst); UP(bdist, h.bdist); UP(bin_ptr, h.bin_ptr); UP(bin, h.bin);
    UP(bout_ptr, h.bout_ptr); UP(bout, h.bout); UP(perm, h.perm); UP(grp_start, h.grp_start);
    UP(type_grp, h.type_grp); UP(lvl_ptr, h.lvl_ptr); UP(lvl_ops, h.lvl_ops); UP(asap, h.asap);
    UP(leg_items, h.leg_items); UP(leg_over, h.leg_over); UP(leg_batch, h.leg_batch);
    UP(grp_of, h.grp_of);
    UP(bmem, h.bmem);
    UP(big_ops, h.big_ops);
    UP(big_of, h.big_of);
    g.nbig = (int)h.big_ops.size();
    UP(alap, h.alap);
#undef UP
#define AL(field, n) do { s = dalloc(c, &c->w.field, (n)); if (s != GAUS_OK) goto fail_alloc; } while (0)
    AL(Upart, (size_t)B * g.ngroups * g.parts * h.D);
    AL(ppart, BN * ntiles * kPP);
    AL(cpart, (size_t)B * h.E * ntiles * kCP);
    AL(bpart, (size_t)B * h.nb * ntiles * kBP);
    AL(U, (size_t)B * h.K * g.T);
    AL(trans, (size_t)B * h.K * h.D);
    AL(ntrans, (size_t)B * h.K);
    AL(terms, (size_t)B * kTerms);
    AL(lres_part, (size_t)B * h.K);
    AL(soft, (size_t)B * h.K * g.T);
    AL(lmom, (size_t)B * h.K * kMaxChunks * kNC);
    AL(lstrip, (size_t)B * h.K * kStripMax);
    AL(lpart, BN * ntiles * 2);
    AL(lpoly, BN * 2);
    AL(Mpart, (size_t)B * g.ngroups * h.D);
    AL(mpoly, BN);
    {
        const size_t slots = (size_t)B * g.ngroups * std::max(1, c->pa.split);
        AL(mcoef, slots * kMaxChunks * kNC);
        AL(mstrip, slots * kStripMax);
        AL(mcoef_r, (size_t)B * (kMaxChunks * kNC + kStripMax));
        AL(mmom, (size_t)B * kMaxChunks * kNC);
        AL(mopoly, BN * 2);
        AL(mspoly, (size_t)B * h.E * 2);
    }
    AL(mreg, (size_t)B * g.T);
    AL(mregd, (size_t)B * g.T);
    AL(msoft, (size_t)B * g.T);
    AL(lmem, (size_t)B);
    AL(mown, BN * ntiles * 2);
    AL(msucc, (size_t)B * h.E * ntiles * 2);
    AL(bigsum, (size_t)B * std::max<size_t>(h.big_ops.size(), 1) * 6);
    AL(cand, BN);
    AL(cand_cost, (size_t)B * kCost);
    AL(hist, (size_t)B * h.K * g.T);
    AL(mdiff, (size_t)B * (h.D + 1));
    AL(mprof, (size_t)B * g.T);
    AL(lcom_acc, (size_t)B);
    AL(illegal, (size_t)B);
    AL(round_bad, (size_t)B);
    AL(mode, (size_t)B);
    AL(n_reinit, (size_t)B);
    AL(n_improve, (size_t)B);
    AL(wts, (size_t)B * 4);
    AL(adamf, (size_t)B * 2);
    AL(cls, BN);
    AL(rsig, BN);
    AL(dflag, BN);
    AL(gbits, (size_t)B * g.ngroups);
    AL(gnar, (size_t)B * g.ngroups);
    AL(Unar, g.nar_on ? (size_t)B * g.ngroups * h.D : 1);
    AL(gsum_nar, (size_t)B * g.ngroups * 2);
    AL(gsum_lap, g.lap_on ? (size_t)B * lap_blocks(g) * 2 : 1);
    AL(pedge, g.lap_on ? (size_t)B * std::max(h.E, 1) * 4 : 1);
    AL(gsum_ops, (size_t)B * g.ngroups * g.parts * ntiles * 2);
    AL(gsum_poly, (size_t)std::max(c->poly_slots, 1) * 2);
    AL(gsel, BN);
    AL(gtier, BN);
    AL(vres_part, (size_t)B * h.K);
    AL(Ucoef_k, (size_t)B * h.K * kGrids * (kMaxChunks * kNC + kStripMax));
    AL(ppoly, BN * kPP);
    AL(cpoly, (size_t)B * h.E * kCP);
    AL(Ucoef, (size_t)std::max(c->poly_slots, 1) * kMaxChunks * kNC);
    AL(Ustrip, (size_t)std::max(c->poly_slots, 1) * kStripMax);
    AL(s64, BN);
    AL(s64b, BN);
    AL(status, (size_t)B);
#undef AL
    {
        hipError_t e = hipMemset(c->w.U, 0, sizeof(float) * (size_t)B * h.K * g.T);
        if (e == hipSuccess) e = hipMemset(c->w.ppoly, 0, sizeof(float) * BN * kPP);
        if (e == hipSuccess) e = hipMemset(c->w.cls, 0, BN);
        if (e == hipSuccess) e = hipMemset(c->w.gsum_poly, 0, sizeof(float) * (size_t)std::max(c->poly_slots, 1) * 2);
        if (e == hipSuccess) e = hipMemset(c->w.gsel, kNoGrid, BN);
        if (e == hipSuccess) e = hipMemset(c->w.gbits, 0, sizeof(unsigned) * (size_t)B * g.ngroups);
        if (e == hipSuccess) e = hipDeviceSynchronize();
        if (e != hipSuccess) { s = fail(nullptr, GAUS_E_DEVICE, "init: %s", hipGetErrorString(e)); goto fail_alloc; }
    }
    c->asap = h.asap;
    c->alap = h.alap;
    *out = c;
    return GAUS_OK;
fail_alloc:
    free_all(c);
    delete c;
    return s;
}

void gaus_destroy(gaus_ctx *ctx) {
    if (!ctx) return;
    (void)hipStreamSynchronize(ctx->stream);
    free_all(ctx);
    delete ctx;
}

gaus_status gaus_bind_state(gaus_ctx *ctx, float *mu, float *sigma, float *adam_m, float *adam_v,
                            float *lambda, int32_t *adam_t) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!mu || !sigma || !adam_m || !adam_v || !lambda || !adam_t)
        return fail(ctx, GAUS_E_INVALID_ARG, "bind_state: null pointer");
    ctx->mu = mu; ctx->sigma = sigma; ctx->m = adam_m; ctx->v = adam_v; ctx->lambda = lambda;
    ctx->adam_t = adam_t;
    ctx->bound = true;
    return GAUS_OK;
}

gaus_status gaus_loss_grad(gaus_ctx *ctx, const float *mu, const float *sigma, const float *lambda,
                           float *terms, float *grad_mu, float *grad_sigma) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!mu || !sigma || !lambda || !terms || !grad_mu || !grad_sigma)
        return fail(ctx, GAUS_E_INVALID_ARG, "loss_grad: null pointer");
    IterArgs a{};
    a.mu = mu; a.sigma = sigma; a.lambda_in = lambda; a.terms_out = terms;
    a.gmu = grad_mu; a.gsig = grad_sigma; a.mode = 0;
    hipError_t e = next_events(ctx, a);
    if (e != hipSuccess) return hip_fail(ctx, e, "timing events");
    e = enqueue_iteration(ctx->g, ctx->w, ctx->hp, ctx->lc, ctx->pa, a, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "loss_grad launch");
    return GAUS_OK;
}

gaus_status gaus_step(gaus_ctx *ctx, int32_t n_iters, float *terms_last) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!ctx->bound) return fail(ctx, GAUS_E_INVALID_ARG, "step: state not bound");
    if (n_iters < 0) return fail(ctx, GAUS_E_INVALID_ARG, "step: n_iters < 0");
    for (int it = 0; it < n_iters; ++it) {
        IterArgs a{};
        a.mu = ctx->mu; a.sigma = ctx->sigma; a.lambda_in = ctx->lambda; a.lambda_out = ctx->lambda;
        a.adam_t = ctx->adam_t; a.terms_out = (it == n_iters - 1) ? terms_last : nullptr;
        a.mu_io = ctx->mu; a.sig_io = ctx->sigma; a.m = ctx->m; a.v = ctx->v; a.mode = 1;
        hipError_t e = next_events(ctx, a);
        if (e != hipSuccess) return hip_fail(ctx, e, "timing events");
        e = enqueue_iteration(ctx->g, ctx->w, ctx->hp, ctx->lc, ctx->pa, a, ctx->stream);
        if (e != hipSuccess) return hip_fail(ctx, e, "step launch");
    }
    return GAUS_OK;
}

gaus_status gaus_adam_from_grad(gaus_ctx *ctx, const float *g_mu, const float *g_sigma, const float *terms) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!ctx->bound) return fail(ctx, GAUS_E_INVALID_ARG, "adam_from_grad: state not bound");
    if (!g_mu || !g_sigma || !terms) return fail(ctx, GAUS_E_INVALID_ARG, "adam_from_grad: null pointer");
    hipError_t e = enqueue_adam_from_grad(ctx->g, ctx->w, ctx->hp, g_mu, g_sigma, terms, ctx->mu, ctx->sigma,
                                          ctx->m, ctx->v, ctx->lambda, ctx->adam_t, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "adam_from_grad launch");
    return GAUS_OK;
}

gaus_status gaus_legalize(gaus_ctx *ctx, const float *mu, int32_t *sched, int32_t *status) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!mu || !sched || !status) return fail(ctx, GAUS_E_INVALID_ARG, "legalize: null pointer");
    hipError_t e = enqueue_legalize(ctx->g, ctx->w, mu, sched, ctx->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(status, ctx->w.status, sizeof(int) * ctx->g.B, hipMemcpyDeviceToHost, ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "legalize");
    return GAUS_OK;
}

gaus_status gaus_schedule_cost(gaus_ctx *ctx, const int32_t *sched, double *cost) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!sched || !cost) return fail(ctx, GAUS_E_INVALID_ARG, "schedule_cost: null pointer");
    hipError_t e = enqueue_schedule_cost(ctx->g, ctx->w, ctx->hp, sched, cost, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "schedule_cost launch");
    return GAUS_OK;
}

gaus_status gaus_schedule_cost_noalloc(gaus_ctx *ctx, const int32_t *sched, double *cost) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!sched || !cost) return fail(ctx, GAUS_E_INVALID_ARG, "schedule_cost_noalloc: null pointer");
    const size_t need = cost_scratch_bytes(ctx->g);
    if (need > kScratchBytes)
        return fail(ctx, GAUS_E_INVALID_ARG,
                    "schedule_cost_noalloc: needs %zu bytes of scratch (B*(4*K*T + 8*(D+1) + 8*T) + 12*B, "
                    "each part rounded up to 256), more than the library's %zu",
                    need, kScratchBytes);
    hipError_t e = enqueue_schedule_cost_scratch(ctx->g, ctx->w, ctx->hp, ctx->scratch, sched, cost, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "schedule_cost_noalloc launch");
    return GAUS_OK;
}

gaus_status gaus_solve(gaus_ctx *ctx, const gaus_solve_params *prm, int32_t *best_sched, double *best_cost,
                       gaus_solve_stats *stats) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!ctx->bound) return fail(ctx, GAUS_E_INVALID_ARG, "solve: state not bound");
    if (!prm || !best_sched || !best_cost || !stats) return fail(ctx, GAUS_E_INVALID_ARG, "solve: null pointer");
    if (prm->max_iters < 1 || prm->check_every < 1)
        return fail(ctx, GAUS_E_INVALID_ARG, "solve: need max_iters >= 1 and check_every >= 1");
    const auto t0 = std::chrono::steady_clock::now();
    auto elapsed = [&]() { return std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count(); };
    hipError_t e = enqueue_best_init(ctx->g, ctx->w, best_cost, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "solve init");
    *stats = gaus_solve_stats{};
    int it = 0, checks = 0;
    while (it < prm->max_iters) {
        const int n = std::min(prm->check_every, prm->max_iters - it);
        gaus_status s = gaus_step(ctx, n, nullptr);
        if (s != GAUS_OK) return s;
        it += n;
        e = enqueue_check(ctx->g, ctx->w, ctx->hp, ctx->mu, ctx->sigma, ctx->m, ctx->v, best_sched, best_cost,
                          prm->reinit_sigma ? 1 : 0, ctx->stream);
        if (e != hipSuccess) return hip_fail(ctx, e, "solve check");
        ++checks;
        if (prm->time_limit_s > 0.0) {
            e = hipStreamSynchronize(ctx->stream);
            if (e != hipSuccess) return hip_fail(ctx, e, "solve");
            if (elapsed() >= prm->time_limit_s) break;
        }
    }
    const int B = ctx->g.B;
    std::vector<int> nre(B), nim(B);
    std::vector<double> bc((size_t)B * kCost);
    e = hipMemcpyAsync(nre.data(), ctx->w.n_reinit, sizeof(int) * B, hipMemcpyDeviceToHost, ctx->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(nim.data(), ctx->w.n_improve, sizeof(int) * B, hipMemcpyDeviceToHost, ctx->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(bc.data(), best_cost, sizeof(double) * bc.size(), hipMemcpyDeviceToHost, ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "solve");
    stats->iters = it;
    stats->checks = checks;
    for (int b = 0; b < B; ++b) { stats->reinits += nre[b]; stats->improvements += nim[b]; }
    // best restart: the same order the device uses per restart
    auto better = [](const double *a, const double *c) {
        const bool fa = a[5] != 0.0 && a[4] == 0.0, fc = c[5] != 0.0 && c[4] == 0.0;
        if (fa != fc) return fa;
        if (fa) return a[0] < c[0];
        if (a[5] != c[5]) return a[5] != 0.0;
        if (a[4] != c[4]) return a[4] < c[4];
        return a[0] < c[0];
    };
    int best = -1;
    for (int b = 0; b < B; ++b) {
        const double *cb = &bc[(size_t)b * kCost];
        if (cb[5] == 0.0) continue;   // never legal
        if (best < 0 || better(cb, &bc[(size_t)best * kCost])) best = b;
    }
    stats->best_restart = best;
    stats->seconds = elapsed();
    return GAUS_OK;
}

gaus_status gaus_solve_check(gaus_ctx *ctx, int32_t *best_sched, double *best_cost, int32_t reinit_sigma,
                             int32_t *mode) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!ctx->bound) return fail(ctx, GAUS_E_INVALID_ARG, "solve_check: state not bound");
    if (!best_sched || !best_cost) return fail(ctx, GAUS_E_INVALID_ARG, "solve_check: null pointer");
    hipError_t e = enqueue_check(ctx->g, ctx->w, ctx->hp, ctx->mu, ctx->sigma, ctx->m, ctx->v, best_sched,
                                 best_cost, reinit_sigma ? 1 : 0, ctx->stream);
    if (e == hipSuccess && mode)
        e = hipMemcpyAsync(mode, ctx->w.mode, sizeof(int) * ctx->g.B, hipMemcpyDeviceToHost, ctx->stream);
    if (e == hipSuccess && mode) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "solve_check");
    return GAUS_OK;
}

gaus_status gaus_init_state(gaus_ctx *ctx, const double *u, float *mu, float *sigma) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!mu || !sigma) return fail(ctx, GAUS_E_INVALID_ARG, "init_state: null pointer");
    const int B = ctx->g.B, N = ctx->g.N;
    if (B > 1 && !u) return fail(ctx, GAUS_E_INVALID_ARG, "init_state: u is required when B > 1");
    std::vector<float> hm((size_t)B * N), hs((size_t)B * N);
    for (int b = 0; b < B; ++b)
        for (int i = 0; i < N; ++i) {
            const double slack = (double)ctx->alap[i] - ctx->asap[i];
            const double sg = std::max((double)ctx->hp.kappa * slack, (double)ctx->hp.sigma_min);
            const double m = b == 0 ? 0.5 * ((double)ctx->asap[i] + ctx->alap[i])
                                    : ctx->asap[i] + u[(size_t)b * N + i] * slack;
            hm[(size_t)b * N + i] = (float)m;
            hs[(size_t)b * N + i] = (float)sg;
        }
    hipError_t e = hipMemcpyAsync(mu, hm.data(), hm.size() * sizeof(float), hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(sigma, hs.data(), hs.size() * sizeof(float), hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "init_state");
    return GAUS_OK;
}

gaus_status gaus_asap_alap(const gaus_ctx *ctx, int32_t *asap, int32_t *alap) {
    if (!ctx || !asap || !alap) return GAUS_E_INVALID_ARG;
    std::copy(ctx->asap.begin(), ctx->asap.end(), asap);
    std::copy(ctx->alap.begin(), ctx->alap.end(), alap);
    return GAUS_OK;
}

gaus_status gaus_get_usage(gaus_ctx *ctx, float *U) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!U) return fail(ctx, GAUS_E_INVALID_ARG, "get_usage: null pointer");
    const size_t bytes = sizeof(float) * (size_t)ctx->g.B * ctx->g.K * ctx->g.T;
    hipError_t e = hipMemcpyAsync(U, ctx->w.U, bytes, hipMemcpyDeviceToDevice, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "get_usage");
    return GAUS_OK;
}

gaus_status gaus_get_storage(gaus_ctx *ctx, float *M) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!M) return fail(ctx, GAUS_E_INVALID_ARG, "get_storage: null pointer");
    if (!(ctx->hp.gamma > 0.0f)) return fail(ctx, GAUS_E_INVALID_ARG, "get_storage: the storage term is off (gamma_mem = 0)");
    const size_t bytes = sizeof(float) * (size_t)ctx->g.B * ctx->g.T;
    hipError_t e = hipMemcpyAsync(M, ctx->w.mreg, bytes, hipMemcpyDeviceToDevice, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "get_storage");
    return GAUS_OK;
}

gaus_status gaus_kernel_timing(gaus_ctx *ctx, int32_t enable) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "kernel_timing");
    if (enable < 0) return fail(ctx, GAUS_E_INVALID_ARG, "kernel_timing: enable < 0");
    ctx->timing = enable != 0;
    ctx->timing_every = enable > 0 ? enable : 1;
    ctx->timing_iter = 0;
    ctx->ev_used = 0;
    return GAUS_OK;
}

gaus_status gaus_kernel_timing_read(gaus_ctx *ctx, double *total_ms, int32_t *launches) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!total_ms || !launches) return fail(ctx, GAUS_E_INVALID_ARG, "kernel_timing_read: null pointer");
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "kernel_timing_read");
    double tot[2] = {0.0, 0.0};
    for (size_t k = 0; k < ctx->ev_used; ++k)
        for (int q = 0; q < (ctx->pa.enabled ? 2 : 1); ++q) {
            float ms = 0.0f;
            e = hipEventElapsedTime(&ms, ctx->ev_pool[4 * k + 2 * q], ctx->ev_pool[4 * k + 2 * q + 1]);
            if (e != hipSuccess) return hip_fail(ctx, e, "kernel_timing_read");
            tot[q] += ms;
        }
    total_ms[0] = tot[0]; total_ms[1] = tot[1];
    launches[0] = (int32_t)ctx->ev_used;
    launches[1] = ctx->pa.enabled ? (int32_t)ctx->ev_used : 0;
    ctx->ev_used = 0;
    return GAUS_OK;
}

gaus_status gaus_sync(gaus_ctx *ctx) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "sync");
    return GAUS_OK;
}

gaus_status gaus_get_dims(const gaus_ctx *ctx, int32_t dims[8]) {
    if (!ctx || !dims) return GAUS_E_INVALID_ARG;
    const Graph &g = ctx->g;
    dims[0] = g.N; dims[1] = g.E; dims[2] = g.K; dims[3] = g.D; dims[4] = g.II; dims[5] = g.T;
    dims[6] = g.nb; dims[7] = g.B;
    return GAUS_OK;
}

gaus_status gaus_get_poly_config(const gaus_ctx *ctx, int32_t cfg[4]) {
    if (!ctx || !cfg) return GAUS_E_INVALID_ARG;
    cfg[0] = ctx->pa.enabled; cfg[1] = ctx->pa.W; cfg[2] = ctx->pa.nc; cfg[3] = ctx->pa.L0;
    return GAUS_OK;
}

gaus_status gaus_poly_census(gaus_ctx *ctx, int64_t counts[2]) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!counts) return fail(ctx, GAUS_E_INVALID_ARG, "poly_census: null pointer");
    const Graph &g = ctx->g;
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "poly_census");
    std::vector<unsigned char> cls((size_t)g.B * g.N);
    std::vector<int> rp(g.N + 1), col(std::max(g.E, 1));
    e = hipMemcpy(cls.data(), ctx->w.cls, cls.size(), hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(rp.data(), g.row_ptr, sizeof(int) * rp.size(), hipMemcpyDeviceToHost);
    if (e == hipSuccess && g.E > 0) e = hipMemcpy(col.data(), g.col, sizeof(int) * g.E, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(ctx, e, "poly_census");
    int64_t nop = 0, ned = 0;
    for (int b = 0; b < g.B; ++b) {
        const unsigned char *c = cls.data() + (size_t)b * g.N;
        for (int i = 0; i < g.N; ++i) {
            if (!c[i]) continue;
            ++nop;
            for (int q = rp[i]; q < rp[i + 1]; ++q) ned += c[col[q]] ? 1 : 0;
        }
    }
    counts[0] = nop;
    counts[1] = ned;
    return GAUS_OK;
}

gaus_status gaus_get_poly_grids(const gaus_ctx *ctx, int32_t cfg[15]) {
    if (!ctx || !cfg) return GAUS_E_INVALID_ARG;
    for (int gi = 0; gi < kGrids; ++gi) {
        const GridArgs &gr = ctx->pa.gr[gi];
        int32_t *q = cfg + 5 * gi;
        q[0] = gr.on; q[1] = kGridP[gi]; q[2] = gr.W; q[3] = gr.nc; q[4] = gr.L0;
    }
    return GAUS_OK;
}

gaus_status gaus_poly_grid_census(gaus_ctx *ctx, int64_t counts[3]) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!counts) return fail(ctx, GAUS_E_INVALID_ARG, "poly_grid_census: null pointer");
    const size_t BN = (size_t)ctx->g.B * ctx->g.N;
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "poly_grid_census");
    std::vector<unsigned char> sel(BN);
    e = hipMemcpy(sel.data(), ctx->w.gsel, BN, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(ctx, e, "poly_grid_census");
    for (int gi = 0; gi < kGrids; ++gi) counts[gi] = 0;
    for (size_t q = 0; q < BN; ++q)
        if (sel[q] < kGrids) ++counts[sel[q]];
    return GAUS_OK;
}

gaus_status gaus_poly_tier_census(gaus_ctx *ctx, int64_t counts[24]) {
    if (!ctx) return GAUS_E_INVALID_ARG;
    if (!counts) return fail(ctx, GAUS_E_INVALID_ARG, "poly_tier_census: null pointer");
    const Graph &g = ctx->g;
    const size_t BN = (size_t)g.B * g.N;
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "poly_tier_census");
    std::vector<unsigned char> sel(BN), tier(BN), cls(BN);
    std::vector<int> rp(g.N + 1), col(std::max(g.E, 1));
    e = hipMemcpy(sel.data(), ctx->w.gsel, BN, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(tier.data(), ctx->w.gtier, BN, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(cls.data(), ctx->w.cls, BN, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(rp.data(), g.row_ptr, sizeof(int) * rp.size(), hipMemcpyDeviceToHost);
    if (e == hipSuccess && g.E > 0) e = hipMemcpy(col.data(), g.col, sizeof(int) * g.E, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(ctx, e, "poly_tier_census");
    for (int q = 0; q < 24; ++q) counts[q] = 0;
    for (int b = 0; b < g.B; ++b)
        for (int i = 0; i < g.N; ++i) {
            const size_t bi = (size_t)b * g.N + i;
            if (sel[bi] >= kGrids || tier[bi] < 1 || tier[bi] > kTiers) continue;
            int64_t *c = counts + (sel[bi] * (kTiers + 1) + tier[bi]) * 2;
            c[0] += 1;
            for (int q = rp[i]; q < rp[i + 1]; ++q) c[1] += cls[(size_t)b * g.N + col[q]] ? 1 : 0;
        }
    return GAUS_OK;
}

}  // extern "C"
