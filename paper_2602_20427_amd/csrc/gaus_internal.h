// Internal declarations shared by the host side (gaus_host.cpp) and the
// gfx950 kernels (gaus_kernels.hip).  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace gaus {

// Partial-sum record widths.
constexpr int kPP = 6;   // per (restart, op, tile): V_dep, L_com, dVdep/dmu_i, dVdep/dsigma_i,
                         //   dLcom/dmu_i, dLcom/dsigma_i  (producer side of the op's out-edges)
constexpr int kCP = 4;   // per (restart, edge, tile): dVdep/dmu_j, dVdep/dsigma_j,
                         //   dLcom/dmu_j, dLcom/dsigma_j (consumer side)
constexpr int kBP = 5;   // per (restart, back edge, tile): V_rec, dVrec/dmu_j, dVrec/dsigma_j
                         //   (producer j), dVrec/dmu_i, dVrec/dsigma_i (consumer i)
constexpr int kHalo = 256;  // largest producer delay handled from the LDS row window
constexpr int kBigIn = 64;  // in-degree above which an op's in-edge records are reduced by a work-group
constexpr int kLegPre = 4;  // predecessors held in a legalization item
constexpr int kCost = 6;    // per schedule: cost, L_com, L_res, L_mem, V_res, legal
constexpr int kTerms = 7;   // per restart: L, V_dep, V_res, V_rec, L_com, L_res, L_mem

// Chunk-polynomial path (dense regime).  On a chunk of W consecutive steps
// with rho = ((W-1)/2)/sigma <= kRhoMax the CDF row of an op is a degree-kDeg
// polynomial in the step offset to ~1e-10; sums over steps become dot products.
// Wider ops need fewer terms for the same accuracy: tier t uses degree
// kTierDeg[t] when rho is at most the tier's bound (set on the host).
constexpr int kDeg = 8;                       // polynomial degree (tier 1, the largest)
constexpr int kTiers = 3;
constexpr int kTierDeg[kTiers + 1] = {0, 8, 6, 5};
constexpr int kNC = kDeg + 1;                 // coefficients per vector
constexpr int kShiftTerms = 4;                // terms of the one-step shift series
constexpr int kTN = kDeg + kShiftTerms + 2;   // scaled derivatives T_0 .. T_{kTN-1}
constexpr int kSmax = 8;                      // largest producer delay on that path
constexpr float kRhoMax = 0.25f;
constexpr int kMaxChunks = 64;                // one chunk per lane of a wave
// chunk widths W of the grids (W <= 256 keeps the degree-16 moments within
// fp32 range; the smallest W gives the lowest sigma threshold of the path,
// about 2 (W - 1) at degree 8).  With the storage term on, a chosen width
// stays >= 16: its holders' gradients lose accuracy at narrower chunks
// (measured at tau = 0.01: 1.2e-7 at W = 16, 7e-6 at 12, 4e-5 at 15).
constexpr int kMinChunk = 12, kMinChunkStorage = 16, kMaxChunk = 256;
constexpr int kStripMax = 320;                 // step-by-step strip positions per op, at most
// Storage term on the chunk polynomials: a holder whose successors are all
// polynomial, at most kMemPolyDeg of them, with rho summed over the holder
// and its successors at most kMemRhoMax for Gaussian start times (the
// product of their series keeps the degree-8 accuracy) and at most the
// family's own degree-8 rho for the others (PolyArgs::mem_rho); every other
// holder is evaluated step by step.
constexpr int kMemPolyDeg = 4;
constexpr float kMemRhoMax = 0.25f;

// Chunk grids: grid g gives each restart 64/P_g lanes of a wave, so P_g
// restarts of one op share a wave (P = 1, 2, 4).  Grid 0 is the per-restart
// layout every polynomial op can take; the packed grids use wider chunks (at
// most 64/P each, a strip of at most 64/P positions) and take an op when
// every restart of its pack, the op and all its consumers are wide enough
// for the grid's degree-8 bound.
constexpr int kGrids = 3;
constexpr int kGridP[kGrids] = {1, 2, 4};
constexpr int kPackMax = 4;   // the largest restart pack
constexpr unsigned char kNoGrid = 255;
// bits of Work::gbits
constexpr unsigned kGbStep = 1u, kGbGrid = 4u;
// bits of Work::gnar: step-by-step ops left to the op kernel / taken by k_group
constexpr unsigned kNarLeft = 1u, kNarTaken = 2u;
// the narrow kernel: threads per work-group (at least the largest group), and
// the longest horizon its fixed-point usage row (8 bytes per step) takes
constexpr int kNarBS = 512;
constexpr int kNarMaxD = 4096;

struct GridArgs {
    int on;               // grid in use
    int W, nc, L0, SP;    // chunk width, chunks, left strip [0, L0), strip positions [0, L0) u {D-2, D-1}
    int split;            // work-groups per op group
    int slot_base;        // first per-work-group output slot of the grid: slot of (restart b, group,
                          // part) = slot_base + (b * ngroups + group) * split + part
    float lam;            // chunk half-width (W-1)/2
    float sig_thr[kTiers + 1];   // sigma >= sig_thr[t]: tier t on this grid
    float H[kDeg + 1];    // even moments of a chunk's points
};

// Work-group segments of the one polynomial launch: [0] packed grid 2
// (P = 4), [1] packed grid 1 (P = 2), [2] grid 0; n = work-groups, nx = their
// x extent (op group slices; the rest is the restart pack).
struct PolySegs {
    int n[3], nx[3];
};

struct PolyArgs {
    int enabled;          // 0: every op takes the per-step path
    int fam;              // CDF family (HP::family): 0 Gaussian, 1 logistic, 3 Cauchy on this path
    int W, nc, L0;        // grid 0: chunk width, chunks, left strip [0, L0); chunks cover [L0, D-2)
    int SP;               // strip positions: [0, L0) and {D-2, D-1}
    int split;            // work-groups per op group in the polynomial kernel
    float lam;            // chunk half-width (W-1)/2
    float sig_thr[kTiers + 1];   // sigma >= sig_thr[t]: tier t (decreasing degree); [1] = path threshold
    float H[kDeg + 1];    // even moments: H[k] = sum over a chunk's points y of y^(2k)
    float mem_rho;        // storage holders: bound of rho summed over a holder and its successors
    GridArgs gr[kGrids];  // [0] = the fields above; [1], [2] = packed grids
};

// Device copy of the preprocessed problem (all pointers are device memory).
struct Graph {
    int N, E, K, D, II, T, nb, B;
    int tile, ntiles;          // steps per tile of the op kernel, tiles per restart
    int ngroups;               // type-pure op groups
    int parts;                 // op-kernel work-groups per (op group, tile): each takes every parts-th op
    int nlevels;               // topological levels (legalization)
    int leg_mode;              // legalization schedule: 0 global int64, 1 LDS int16, 2 LDS int32
    const int *row_ptr, *col;            // CSR by producer
    const int *esrc;                     // producer of each CSR edge (Laplace edges: thread per edge)
    const int *pred_ptr, *pred_eid;      // CSC: CSR edge id of each in-edge
    const int *pred_src;                 // CSC: producer of each in-edge
    const int *delay, *rtype;
    const float *cap;
    const int *bsrc, *bdst, *bdist;      // back edges (producer j, consumer i, k)
    const int *bin_ptr, *bin;            // back edges by consumer
    const int *bout_ptr, *bout;          // back edges by producer
    const int *perm;                     // ops sorted by (type, id)
    const int *grp_start;                // [ngroups+1] ranges of perm
    const int *type_grp;                 // [K+1] groups of type k: [type_grp[k], type_grp[k+1])
    const int *lvl_ptr, *lvl_ops;        // ops by (topological level, id)
    const int *leg_items;                // [N][8] per op in level order: op, delay, predecessor count,
                                         // start of the predecessors past kLegPre in leg_over, the first
                                         // kLegPre predecessors (32-byte aligned)
    const int *leg_over;                 // predecessors past the first kLegPre, in level order
    int leg_ring;                        // 1: II = 0 legalization through the LDS ring (k_legalize_ring)
    int nar_on;                          // 1: short-spread step-by-step ops go to k_group (several
                                         // op-kernel tiles and D <= kNarMaxD)
    int lap_on;                          // 1: Laplace start times: the edge terms in closed form (k_lap_edges)
    int leg_ring_items, leg_ring_over;   // items and overflow predecessors one ring half holds
    int leg_nbatch;                      // ring batches: contiguous ranges of the items of levels >= 1
    const int *leg_batch;                // [nbatch+1][3] level of the first item, first item, first
                                         // overflow predecessor of each batch (last row: the ends)
    const int *grp_of;                   // [N] group of each op
    const float *bmem;                   // [N] storage units b_i
    int nbig;                            // ops with more than kBigIn predecessors
    const int *big_ops, *big_of;         // [nbig] those ops; [N] index into them or -1
    const int *asap, *alap;
};

// Library-owned device workspace.
struct Work {
    float *Upart;     // [B][ngroups][parts][D]   unfolded usage partials of the op kernel
    float *ppart;     // [B][N][ntiles][kPP]
    float *cpart;     // [B][E][ntiles][kCP]
    float *bpart;     // [B][nb][ntiles][kBP]
    float *U;         // [B][K][T]         expected (folded) usage
    int *trans;       // [B][K][D]         signed (t+1) of each ReLU-indicator change at bin edge t
    int *ntrans;      // [B][K]
    float *terms;     // [B][kTerms]       L, V_dep, V_res, V_rec, L_com, L_res of the last forward
    float *lres_part; // [B][K]            smooth peak of one type's usage
    float *soft;      // [B][K][T]         beta * dL_res/dU (softmax over the type's slots)
    float *lmom;      // [B][K][64][kNC]   chunk moments of the softmax differences at the bin edges
    float *lstrip;    // [B][K][kStripMax] the same differences at the strip positions
    float *lpart;     // [B][N][tiles][2]  smooth-peak gradient (mu, sigma) of step-by-step ops, per tile
    float *lpoly;     // [B][N][2]         the same for ops on the polynomial path
    double *Mpart;    // [B][ngroups][D]   expected storage units of a group's ops per step
    unsigned char *mpoly;  // [B][N]       1 = the op's storage term is taken on the chunk polynomials
    double *mcoef;    // [B][ngroups*split][kMaxChunks][kNC]  storage profile coefficients per chunk
    double *mstrip;   // [B][ngroups*split][kStripMax]        storage profile at the strip positions
    double *mcoef_r;  // [B][kMaxChunks*kNC + kStripMax]     the same summed over the work-groups
    float *mmom;      // [B][kMaxChunks][kNC]  chunk moments sum_y c(t) y^n of the storage softmax
    float *mopoly;    // [B][N][2]         storage gradient of a polynomial holder as the holder
    float *mspoly;    // [B][E][2]         storage gradient of the consumer of an edge out of one
    double *mregd;    // [B][T]            expected storage units per (modulo) slot
    float *mreg;      // [B][T]            the same in float (gaus_get_storage)
    float *msoft;     // [B][T]            gamma * dL_mem/dMReg (softmax over the slots)
    float *lmem;      // [B]               smooth peak storage L_mem
    float *mown;      // [B][N][tiles][2]  storage gradient of an op as the holder, per tile
    float *msucc;     // [B][E][tiles][2]  storage gradient of an edge's consumer, per tile
    double *bigsum;   // [B][nbig][6]      in-edge records of the high in-degree ops, reduced
    // discrete schedules (cost of Sec. 2.1; the Alg. 1 driver)
    int *cand;        // [B][N]            legalized rounding of the current means
    double *cand_cost;// [B][kCost]        its cost
    int *hist;        // [B][K][T]         usage counts of a schedule
    long long *mdiff; // [B][D+1]          storage differences (fixed point)
    long long *mprof; // [B][T]            storage profile (fixed point)
    unsigned long long *lcom_acc;  // [B]  sum of (s_j - s_i)^+
    int *illegal;     // [B]               1 if the schedule breaks an edge or the horizon
    int *round_bad;   // [B]               1 if the rounding itself was not legal
    int *mode;        // [B]               re-init: 0 none, 1 from the candidate, 2 from the best
    int *n_reinit, *n_improve;     // [B]  driver counters
    float *wts;       // [B][4]            w_dep, w_res, w_rec, unused
    float *adamf;     // [B][2]            Adam bias corrections 1-beta1^t, 1-beta2^t
    unsigned char *cls;  // [B][N]          1 = op on the chunk-polynomial path this iteration
    float *rsig;           // [B][N]        1/sigma of this iteration (written by k_flags)
    unsigned char *dflag;  // [B][N]        1 = op has step-by-step work (own terms or out-edges),
                           //               2 = that work is done by k_group (records in ppoly / cpoly)
    unsigned *gnar;        // [B][ngroups]  k_group's split of a group with step-by-step work
                           //               (kNarLeft, kNarTaken); valid where gbits has kGbStep
    float *Unar;           // [B][ngroups][D]  usage of the ops k_group took
    float *gsum_nar;       // [B][ngroups][2]  their V_dep, L_com
    float *gsum_lap;       // [B][nlap][2]  V_dep, L_com of each block of edges in closed form (Laplace)
    float *pedge;          // [B][E][4]  producer-side derivatives of each edge in closed form (Laplace)
    unsigned *gbits;  // [B][ngroups]      work of the group this iteration (k_group):
                      //                   kGbStep = some op has step-by-step work,
                      //                   kGbGrid << g = ops on grid g; only such groups'
                      //                   polynomial work-groups write outputs (ppoly / cpoly
                      //                   hold valid records for cls != 0 ops only: readers
                      //                   check cls)
    float *gsum_ops;  // [B][ngroups][parts][ntiles][2]  V_dep, L_com of a k_ops work-group
    float *gsum_poly; // [slots][2]        V_dep, L_com of a k_poly work-group (GridArgs::slot_base)
    unsigned char *gsel;   // [B][N]        grid that evaluates the (restart, op) this iteration (0..2),
                           //               kNoGrid on the step-by-step path
    unsigned char *gtier;  // [B][N]        tier of its vectors on that grid (0 off the polynomial path)
    float *vres_part; // [B][K]            V_res of one resource type
    float *Ucoef_k;   // [B][K][kGrids][64*kNC + 320]  polynomial usage coefficients and strip values per type
    float *ppoly;     // [B][N][kPP]       producer partials of the polynomial path
    float *cpoly;     // [B][E][kCP]       consumer partials of polynomial edges
    float *Ucoef;     // [slots][kMaxChunks][kNC]  usage coefficients per chunk of a k_poly work-group
    float *Ustrip;    // [slots][kStripMax]  usage at the strip positions
    long long *s64;   // [B][N]            legalization workspace
    long long *s64b;  // [B][N]            legalization snapshot (back edges)
    int *status;      // [B]               legalization status
};

struct HP {
    float lr, b1, b2, eps, rho, lambda0, alpha, sigma_min, kappa;
    float beta, tau;   // weight and temperature of the smooth peak usage L_res
    float gamma;       // weight of the smooth peak storage L_mem (same temperature)
    int family;        // CDF family of the start times: 0 Gaussian, 1 logistic, 2 Laplace, 3 Cauchy
};

// Kernel-side configuration chosen on the host from (N, D, B).
struct LaunchCfg {
    int bs;    // threads per work-group of the op kernel (64 or 256)
    int spt;   // steps per thread (1 or 4)
    int fam;   // CDF family (HP::family), a template argument of the step-by-step kernels
};

// Enqueue one forward+backward.  mode 0: write terms/grad to the outputs;
// mode 1: Adam step in place on (mu, sigma, m, v), lambda update, adam_t++.
struct IterArgs {
    const float *mu, *sigma;        // inputs (mode 1: the bound state)
    const float *lambda_in;         // [B][3]
    float *lambda_out;              // mode 1: updated multipliers (may alias lambda_in)
    int *adam_t;                    // mode 1
    float *terms_out;               // [B][kTerms] or null
    float *gmu, *gsig;              // mode 0 outputs
    float *mu_io, *sig_io, *m, *v;  // mode 1 state
    int mode;
    hipEvent_t ops_begin, ops_end;    // optional events around the step-by-step op kernel
    hipEvent_t poly_begin, poly_end;  // optional events around the polynomial kernel
};

hipError_t enqueue_iteration(const Graph &g, const Work &w, const HP &hp, const LaunchCfg &lc,
                             const PolyArgs &pa, const IterArgs &a, hipStream_t st);

// Per-step kernels (gaus_step.hip: step by step; gaus_poly.hip: chunk polynomials).
hipError_t launch_group(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu, hipStream_t st);
// Laplace start times: every forward edge's terms in closed form, a thread per
// edge (records in pedge / cpoly, V_dep and L_com per block of kLapBS edges in gsum_lap).
constexpr int kLapBS = 256;
__host__ __device__ inline int lap_blocks(const Graph &g) { return (g.E + kLapBS - 1) / kLapBS; }
hipError_t launch_lap_edges(const Graph &g, const Work &w, const float *mu, const float *sigma, hipStream_t st);
hipError_t launch_ops(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu, const float *sigma,
                      hipStream_t st);
hipError_t launch_back(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu, const float *sigma,
                       hipStream_t st);
hipError_t launch_lse_ops(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu,
                          const float *sigma, hipStream_t st);
hipError_t launch_mem_fwd(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu,
                          const float *sigma, hipStream_t st);
hipError_t launch_mem_bwd(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu,
                          const float *sigma, hipStream_t st);
hipError_t launch_poly(const Graph &g, const Work &w, const PolyArgs &pa, const float *mu, const float *sigma,
                       hipStream_t st);
hipError_t launch_mem_poly_fwd(const Graph &g, const Work &w, const PolyArgs &pa, const float *mu,
                               hipStream_t st);
hipError_t launch_mem_poly_bwd(const Graph &g, const Work &w, const PolyArgs &pa, const float *mu,
                               hipStream_t st);
hipError_t launch_lse_poly(const Graph &g, const Work &w, const PolyArgs &pa, const float *mu,
                           const float *sigma, hipStream_t st);

// Adam + sigma clamp + lambda += rho*V (from terms) + adam_t++ from a given gradient.
hipError_t enqueue_adam_from_grad(const Graph &g, const Work &w, const HP &hp, const float *gmu,
                                  const float *gsig, const float *terms, float *mu, float *sigma,
                                  float *m, float *v, float *lambda, int *adam_t, hipStream_t st);

// Discrete cost of schedules sched [B][N] (device) into cost [B][kCost] (device).
hipError_t enqueue_schedule_cost(const Graph &g, const Work &w, const HP &hp, const int *sched, double *cost,
                                 hipStream_t st);
// The same with its scratch (usage counts, storage differences and profile,
// edge-length sums, legality flags) in the library's file-scope device array
// of kScratchBytes: cost_scratch_bytes(g) must not exceed it.  scratch_ptr is
// that array's address on the current device (scratch_address, cached per
// device).  Calls that overlap on one device share the array and race.
constexpr size_t kScratchBytes = size_t(8) << 20;
size_t cost_scratch_bytes(const Graph &g);
hipError_t scratch_address(int device, void **out);
hipError_t enqueue_schedule_cost_scratch(const Graph &g, const Work &w, const HP &hp, void *scratch_ptr,
                                         const int *sched, double *cost, hipStream_t st);
// One check of the Alg. 1 driver: legalize the rounded means, cost the
// candidates, keep each restart's best, re-initialize restarts whose
// rounding was not legal (from the candidate if it improved, else from the
// best so far).
hipError_t enqueue_best_init(const Graph &g, const Work &w, double *best_cost, hipStream_t st);
hipError_t enqueue_check(const Graph &g, const Work &w, const HP &hp, float *mu, float *sigma, float *m,
                         float *v, int *best_sched, double *best_cost, int reinit_sigma, hipStream_t st);

// Dynamic LDS of the ring legalization with ready times of ready_bytes each.
size_t legalize_ring_lds(const Graph &g, int ready_bytes);
// Ring batch limits (kernel staging: two 16-byte loads per item, kLegRingV4 of
// them per thread; kLegRingOv overflow predecessors per thread; 512 threads).
constexpr int kLegRingItemsMax = 2048, kLegRingOverMax = 2048;

// Round + legalize every restart; writes sched [B][N] and w.status [B].
hipError_t enqueue_legalize(const Graph &g, const Work &w, const float *mu, int *sched,
                            hipStream_t st);

}  // namespace gaus
