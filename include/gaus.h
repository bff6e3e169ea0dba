/*
 * gaus.h -- C ABI of libgaus, the MI355X (gfx950) hot path of GauS:
 * differentiable scheduling by Gaussian reparameterization
 * (arXiv 2602.20427).
 *
 * Each operator v_i of a DAG G=(V,E) has a Gaussian start time
 * X_i ~ N(mu_i, sigma_i^2) (Sec. 3.1).  Rounding X_i to the nearest step gives
 * per-step masses P_i^d over the horizon {0..D-1} (Sec. 3.2, eq:round; bin 0
 * open to -inf, bin D-1 open to +inf).  One iteration, for each of B
 * independent restarts, evaluates
 *     L = alpha*L_com + sum_{c in {dep,res,rec}} (lambda_c V_c + rho/2 V_c^2)
 * (augmented Lagrangian, Sec. 3.3 eq. (11)), with
 *     V_res = sum_k sum_t ReLU(U_k(t) - C_k)          (App. B.2 eq:relu; usage
 *             U folded modulo II when II > 0, App. B.3)
 *     V_dep = expected violated dependencies          (Sec. 3.2 eq:dep; edge
 *             (i->j) violated iff d_j < d_i + Lat(v_i))
 *     V_rec = expected violated recurrences           (App. B.3; back edge
 *             (j->i,k) violated iff d_j + Lat(v_j) > d_i + k*II)
 *     L_com = expected total edge length E[(d_j-d_i)^+]  (App. B.1)
 * its exact gradient w.r.t. (mu, sigma), and an Adam update (App. C.1), then
 * lambda_c <- lambda_c + rho*V_c (Alg. 1).  Legalization turns rounded means
 * into feasible integer schedules (App. A, Alg. 3 and Alg. 4).
 *
 * Conventions for every entry point:
 *   - Every entry returns a gaus_status; nothing aborts or throws across the
 *     ABI.  gaus_last_error() gives a per-context message.
 *   - Op ids are the caller's.  The library may reorder internally but every
 *     output is indexed by the caller's ids.
 *   - "device" pointers are HIP device memory on the device that was current
 *     at gaus_init; "host" pointers are ordinary host memory.
 *   - Device work is enqueued on the stream given to gaus_init and is
 *     asynchronous unless stated otherwise.  Device faults surface as
 *     GAUS_E_DEVICE at the next synchronizing call.
 *   - A context is used by one host thread at a time; distinct contexts are
 *     independent.
 */
#ifndef GAUS_H
#define GAUS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gaus_ctx gaus_ctx;

typedef enum {
    GAUS_OK = 0,
    GAUS_E_INVALID_ARG = 1,    /* bad pointer, size, range or CSR structure */
    GAUS_E_CYCLE = 2,          /* forward edges are not acyclic */
    GAUS_E_HORIZON = 3,        /* critical path does not fit: some ASAP > ALAP */
    GAUS_E_NOT_CONVERGED = 4,  /* modulo legalization hit its pass cap (N passes) */
    GAUS_E_OVERFLOW = 5,       /* legalized start step beyond D-1 */
    GAUS_E_DEVICE = 6,         /* HIP runtime / kernel error */
    GAUS_E_NOMEM = 7           /* host or device allocation failed */
} gaus_status;

/* Problem statement (Sec. 2.1).  All pointers are HOST memory, read only
 * during gaus_init (copied); the caller may free them afterwards. */
typedef struct {
    int32_t n_ops;             /* N >= 1 */
    int32_t n_edges;           /* E >= 0 */
    const int32_t *row_ptr;    /* [N+1] CSR by producer: row_ptr[0]=0, nondecreasing, row_ptr[N]=E */
    const int32_t *col_idx;    /* [E] consumer of each edge, in [0,N); the graph must be acyclic,
                                  without duplicate edges */
    const int32_t *delay;      /* [N] Lat(v_i), 0 <= Lat <= 2^20 */
    const int32_t *rtype;      /* [N] resource type in [0,K); each op uses one unit of it */
    int32_t n_types;           /* K >= 1 */
    const float *capacity;     /* [K] capacity C_k per step (or per modulo slot), finite, >= 0 */
    int32_t D;                 /* horizon: start steps in [0, D-1]; 1 <= D <= 2^22 */
    int32_t II;                /* 0 = regular scheduling; > 0 = fold usage modulo II */
    int32_t n_back;            /* number of back edges; must be 0 when II == 0 */
    const int32_t *back_src;   /* [n_back] producer v_j of each back edge */
    const int32_t *back_dst;   /* [n_back] consumer v_i (!= v_j) */
    const int32_t *back_dist;  /* [n_back] iteration distance k >= 1, k*II <= 2^30 */
    const float *mem_units;    /* [N] storage units b_i of each op's output (Sec. 2.1 eq:mem),
                                  finite, >= 0; NULL = 1 each.  Used by the storage term. */
} gaus_problem;

/* Hyper-parameters.  gaus_default_hparams() fills the paper's values
 * (App. C.1: Adam lr 1e-2, rho 1e-4, kappa 1/6, LogSumExp temperature 1e-2;
 * Sec. 3.3: lambda0 1e-6) and this library's choices for the unstated ones
 * (Adam betas/eps as in Kingma & Ba, alpha_com 0.01, sigma_min 0.05,
 * beta_res 0 and gamma_mem 0: the smooth peak terms are off unless asked for;
 * family 0, the Gaussian of Sec. 3.1). */
typedef struct {
    float lr, beta1, beta2, eps;   /* Adam */
    float rho;                     /* ALM penalty */
    float lambda0;                 /* initial multipliers */
    float alpha_com;               /* weight alpha of the expected edge length L_com */
    float sigma_min;               /* sigma is clamped to >= sigma_min after each update */
    float kappa;                   /* initial sigma = kappa * (ALAP - ASAP) */
    int32_t poly_chunk;            /* chunk width W of the polynomial evaluation of wide
                                      start-time laws (one restart per wave): 0 = chosen
                                      from D, < 0 = off (every op evaluated step by step),
                                      else W in [12, 256] */
    float beta_res;                /* weight of the smooth peak usage L_res in L (>= 0;
                                      1 with alpha_com gives Formulation A, Sec. 4.1) */
    float tau;                     /* its temperature (> 0): L_res = sum_k tau log sum_t
                                      exp(U_k(t)/tau), App. B.2 and eq:max; slots t < II
                                      when II > 0 (App. B.3) */
    float gamma_mem;               /* weight of the smooth peak storage L_mem in L (>= 0;
                                      1 gives Formulations B and C, Sec. 4.1):
                                      L_mem = tau log sum_t exp(MReg(t)/tau) with MReg the
                                      expected storage units of eq:active folded like the
                                      usage (App. B.3).  Holders with at most 4 successors,
                                      all wide Gaussians, take it on the chunk polynomials,
                                      the others step by step. */
    int32_t family;                /* distribution of the relaxed start times (App. E):
                                      0 Gaussian, 1 logistic (scale sigma sqrt(3)/pi),
                                      2 Laplace (scale sigma/sqrt(2)), 3 Cauchy (scale
                                      sigma sqrt(2 ln 2)); sigma keeps its meaning as the
                                      Gaussian-matched width.  Laplace is evaluated step
                                      by step (its CDF has a kink at the median); the others
                                      take the chunk polynomials when wide enough. */
    int32_t poly_pack;             /* restart packing of the polynomial evaluation: the ops
                                      of 2 or 4 restarts share a wave on wider chunks when
                                      all of them (and their consumers) are wide enough.
                                      0 = on when poly_chunk is 0, > 0 = on, < 0 = off.
                                      Results agree with the unpacked evaluation to fp32
                                      rounding; B < 2 leaves it off. */
} gaus_hparams;

void gaus_default_hparams(gaus_hparams *hp);

/* Validate and preprocess a problem for B restarts, allocate device copies and
 * workspace on the current HIP device.  hip_stream is a hipStream_t (NULL =
 * default stream).  Synchronous.  On failure *out is set to NULL and nothing
 * is allocated; the message is available from gaus_last_error(NULL).
 * Errors: INVALID_ARG, CYCLE, HORIZON, NOMEM, DEVICE. */
gaus_status gaus_init(const gaus_problem *prob, const gaus_hparams *hp, int32_t B,
                      void *hip_stream, gaus_ctx **out);

/* Bind the optimizer state used by gaus_step / gaus_adam_from_grad.  All
 * DEVICE pointers, owned by the caller (the library never frees them) and
 * kept for the context's lifetime or until re-bound:
 *   mu, sigma  [B][N] float;  adam_m, adam_v [2][B][N] float (0 = mu, 1 = sigma);
 *   lambda     [B][3] float (dep, res, rec);  adam_t [1] int32 (steps taken). */
gaus_status gaus_bind_state(gaus_ctx *ctx, float *mu, float *sigma, float *adam_m, float *adam_v,
                            float *lambda, int32_t *adam_t);

/* One forward + backward at (mu, sigma) with multipliers lambda, for all B
 * restarts.  Inputs DEVICE: mu, sigma [B][N], lambda [B][3].  Outputs DEVICE:
 * terms [B][7] = (L, V_dep, V_res, V_rec, L_com, L_res, L_mem), grad_mu,
 * grad_sigma [B][N] (dL/dmu, dL/dsigma), where L = alpha_com L_com +
 * beta_res L_res + gamma_mem L_mem + sum_c (lambda_c V_c + rho/2 V_c^2)
 * (Sec. 3.3 eq. 11; L_res and L_mem are 0 when their weight is 0).
 * Asynchronous.  Errors: INVALID_ARG (null pointer). */
gaus_status gaus_loss_grad(gaus_ctx *ctx, const float *mu, const float *sigma, const float *lambda,
                           float *terms, float *grad_mu, float *grad_sigma);

/* n_iters iterations of Alg. 1's update on the bound state: forward,
 * backward, Adam on mu and sigma, sigma <- max(sigma, sigma_min),
 * lambda_c <- lambda_c + rho * V_c (this iteration's V), adam_t += 1.
 * terms_last (DEVICE [B][7] or NULL) receives the last iteration's terms.
 * Asynchronous.  Errors: INVALID_ARG (state not bound, n_iters < 0). */
gaus_status gaus_step(gaus_ctx *ctx, int32_t n_iters, float *terms_last);

/* The update half of gaus_step from a given gradient: Adam on the bound
 * (mu, sigma) with g_mu, g_sigma (DEVICE [B][N]), the sigma clamp, and
 * lambda_c += rho * terms[b][1+c] with terms DEVICE [B][7]; adam_t += 1.
 * Asynchronous.  Used to check the optimizer step on its own. */
gaus_status gaus_adam_from_grad(gaus_ctx *ctx, const float *g_mu, const float *g_sigma,
                                const float *terms);

/* Round each restart's means half-up to integer steps and legalize them
 * (App. A): II == 0 -> Alg. 3 (clamp to [ASAP, ALAP], one topological pass
 * raising s_v to max over preds u of s_u + Lat(u)); II > 0 -> Alg. 4 (clamp to
 * [0, D-1], passes raising s_v to max(t_min, t_back) until none changes, at
 * most N passes).  mu DEVICE [B][N]; sched DEVICE [B][N] int32 (values above
 * INT32_MAX are saturated); status HOST [B] receives GAUS_OK,
 * GAUS_E_NOT_CONVERGED or GAUS_E_OVERFLOW per restart.  Synchronizes. */
gaus_status gaus_legalize(gaus_ctx *ctx, const float *mu, int32_t *sched, int32_t *status);

/* Discrete cost of integer schedules (Sec. 2.1), the quantity the driver
 * below keeps the best of.  sched DEVICE [B][N] int32; cost DEVICE [B][6]
 * double = (alpha_com L_com + beta_res L_res + gamma_mem L_mem, L_com =
 * sum over edges of (s_j - s_i)^+, L_res = sum over types of the peak usage
 * (folded mod II, eq. (3)/(5)), L_mem = peak storage units (eq:mem, folded),
 * V_res = sum over (type, slot) of usage above capacity, legal = 1 if
 * 0 <= s <= D-1 and every edge and back edge holds, else 0).  Storage units
 * are summed in steps of 2^-20.  Asynchronous. */
gaus_status gaus_schedule_cost(gaus_ctx *ctx, const int32_t *sched, double *cost);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * discrete cost as gaus_schedule_cost (same kernels, bitwise equal results),
 * with its scratch -- usage counts, storage differences and profile,
 * edge-length sums and legality flags -- in a fixed 8 MiB device array of
 * the library instead of its allocations; the call allocates and frees
 * nothing.  It needs B*(4*K*T + 8*(D+1) + 8*T) + 12*B bytes (each part
 * rounded up to 256): INVALID_ARG with a message when that exceeds 8 MiB.
 * Every context on one device shares that device's array and the kernels
 * clear it on each call, so calls that overlap on one device (other
 * streams, other threads) race; calls in stream order do not.  sched DEVICE
 * [B][N] int32, cost DEVICE [B][6] double as gaus_schedule_cost.
 * Asynchronous.  Errors: INVALID_ARG, DEVICE. */
gaus_status gaus_schedule_cost_noalloc(gaus_ctx *ctx, const int32_t *sched, double *cost);

/* Alg. 1 driver (Sec. 3.3) on the bound state. */
typedef struct {
    int32_t max_iters;     /* fused iterations in total, >= 1 */
    int32_t check_every;   /* iterations between checks, >= 1 (App. A reports
                              about two legalizations per run) */
    double time_limit_s;   /* stop at the first check after this much wall
                              time (Sec. 4.1 uses 900 s); <= 0: no limit */
    int32_t reinit_sigma;  /* 1: a re-initialized restart also gets
                              sigma = max(kappa (ALAP - ASAP), sigma_min) */
} gaus_solve_params;

typedef struct {
    int32_t iters;         /* fused iterations run */
    int32_t checks;        /* checks done */
    int32_t reinits;       /* (restart, check) pairs re-initialized */
    int32_t improvements;  /* (restart, check) pairs that improved that restart's best */
    int32_t best_restart;  /* restart holding the best schedule (feasible first), -1 if none legal */
    double seconds;        /* wall time */
} gaus_solve_stats;

/* Runs Alg. 1 on the bound state: blocks of check_every fused iterations
 * (gaus_step); after each block, every restart's means are rounded and
 * legalized (Alg. 3/4) and the result costed (gaus_schedule_cost); a
 * restart keeps the best schedule it has produced (feasible = legal with
 * V_res = 0 first, then lower cost).  A restart whose rounding was not legal
 * is re-initialized (Sec. 3.3 Sampling): mu from the legalized schedule if it
 * improved the restart's best, else from that best ("reset to the prior best",
 * App. A); its Adam moments are cleared.  Stops after max_iters iterations or
 * the time limit.  best_sched DEVICE [B][N] int32 and best_cost DEVICE
 * [B][6] double (as gaus_schedule_cost) receive each restart's best;
 * stats HOST.  Synchronizes.  Errors: INVALID_ARG (state not bound, bad
 * parameters), DEVICE. */
gaus_status gaus_solve(gaus_ctx *ctx, const gaus_solve_params *prm, int32_t *best_sched, double *best_cost,
                       gaus_solve_stats *stats);

/* One check of the Alg. 1 driver on the bound state, the step gaus_solve
 * takes after each block of iterations (Sec. 3.3 "Sampling"; App. A,
 * "Empirical Behavior", reset to the prior best).  For every restart, in
 * order: the means are rounded half-up and legalized (Alg. 3 / Alg. 4) into a
 * candidate; the candidate is costed (gaus_schedule_cost); it replaces the
 * restart's best (best_sched DEVICE [B][N] int32, best_cost DEVICE [B][6]
 * double, as gaus_schedule_cost writes) when it is better in the order
 * gaus_solve documents (equal ones do not replace); if the rounding was not
 * already legal, mu is re-initialized from the candidate when it improved the
 * best, else from the best held before this check, the restart's Adam
 * moments (both halves) are cleared and, with reinit_sigma = 1, sigma is set
 * to max(kappa (ALAP - ASAP), sigma_min).  A best_cost row (+inf, +inf,
 * +inf, +inf, +inf, 0) holds no schedule yet (every candidate replaces it).
 * mode HOST [B] (or NULL) receives per restart 0 (rounding legal, state
 * kept), 1 (re-initialized from the candidate) or 2 (reset to the prior
 * best); when it is given the call synchronizes, else it is asynchronous.
 * Errors: INVALID_ARG (state not bound, null pointer), DEVICE. */
gaus_status gaus_solve_check(gaus_ctx *ctx, int32_t *best_sched, double *best_cost, int32_t reinit_sigma,
                             int32_t *mode);

/* Paper initialization (Sec. 3.3, Alg. 1): sigma = max(kappa*(ALAP-ASAP),
 * sigma_min); restart 0 gets mu = (ASAP+ALAP)/2, restart b >= 1 gets
 * mu = ASAP + u[b][i]*(ALAP-ASAP) with u HOST [B][N] double in [0,1) (may be
 * NULL when B == 1).  mu, sigma DEVICE [B][N].  Synchronizes. */
gaus_status gaus_init_state(gaus_ctx *ctx, const double *u, float *mu, float *sigma);

/* ASAP / ALAP start steps with delays (ASAP of sources 0, ALAP of sinks D-1).
 * asap, alap HOST [N].  Host only. */
gaus_status gaus_asap_alap(const gaus_ctx *ctx, int32_t *asap, int32_t *alap);

/* Expected usage U [B][K][T] (T = II if II > 0 else D) of the last forward
 * pass, copied to DEVICE memory U.  Asynchronous. */
gaus_status gaus_get_usage(gaus_ctx *ctx, float *U);

/* Expected storage units MReg [B][T] of the last forward (Sec. 3.2 eq:active,
 * folded like the usage, App. B.3), copied to DEVICE memory M.  Only when
 * gamma_mem > 0 (else INVALID_ARG).  Asynchronous. */
gaus_status gaus_get_storage(gaus_ctx *ctx, float *M);

/* Profiling hook.  enable = n > 0: in every n-th iteration enqueued from now
 * on (the first, the (n+1)-th, ...), the launches of the two kernels that
 * carry the per-step work -- [0] the step-by-step op kernel and [1] the
 * chunk-polynomial kernel (CDFs, masses, usage, edge terms and their
 * derivatives) -- are bracketed by a pair of HIP events recorded on the
 * context's stream (each recorded event adds a few microseconds between
 * launches, so sampling keeps them out of the iterations' time); 0 = off;
 * negative: INVALID_ARG.  Changing it discards pending events. */
gaus_status gaus_kernel_timing(gaus_ctx *ctx, int32_t enable);

/* Total duration in milliseconds of the bracketed launches of each of the two
 * kernels since timing was enabled or last read, and their numbers (HOST
 * outputs, [2] each; only the sampled iterations count).  Synchronizes the
 * stream, then resets. */
gaus_status gaus_kernel_timing_read(gaus_ctx *ctx, double *total_ms, int32_t *launches);

/* Wait for all work enqueued by this context; reports device errors. */
gaus_status gaus_sync(gaus_ctx *ctx);

/* Problem sizes after preprocessing: N, E, K, D, II, T, n_back, B. */
gaus_status gaus_get_dims(const gaus_ctx *ctx, int32_t dims[8]);

/* Chunk-polynomial configuration of grid 0: enabled (0/1), chunk width W,
 * number of chunks, left strip width.  Ops with Lat <= 8 whose width reaches
 * the degree-8 bound (sigma >= 2(W-1) for the Gaussian) use the path. */
gaus_status gaus_get_poly_config(const gaus_ctx *ctx, int32_t cfg[4]);

/* Census of the last iteration's classification (HOST output, [2]):
 * [0] (restart, op) pairs on the chunk-polynomial path, [1] (restart, edge)
 * pairs whose producer and consumer both are (the edge terms that kernel
 * evaluates).  The rest are evaluated step by step.  Synchronizes the stream;
 * zeros before the first iteration. */
gaus_status gaus_poly_census(gaus_ctx *ctx, int64_t counts[2]);

/* Chunk grids of the polynomial path (HOST output, [3][5]): per grid g
 * (0: one restart per wave, 1 and 2: packs of 2 and 4 restarts sharing a
 * wave) its state (0/1), restarts per wave P, chunk width W, number of chunks
 * and left strip width.  A packed grid takes an op for a whole restart pack
 * when every restart's width, and that of each consumer, reaches the grid's
 * degree-8 bound; the coarsest such grid is used. */
gaus_status gaus_get_poly_grids(const gaus_ctx *ctx, int32_t cfg[15]);

/* Census of the last iteration's grid assignment (HOST output, [3]):
 * (restart, op) pairs evaluated on grid 0, 1, 2.  Synchronizes the stream. */
gaus_status gaus_poly_grid_census(gaus_ctx *ctx, int64_t counts[3]);

/* Census of the last iteration's chunk-polynomial work by grid and series
 * degree tier (HOST output, [3][4][2]): counts[g][t][0] = (restart, op)
 * pairs evaluated on grid g at tier t (1: degree 8, 2: degree 6, 3: degree 5;
 * t = 0 unused), counts[g][t][1] = their out-edges evaluated there (both
 * ends on the polynomial path).  The per-unit work of the polynomial kernel
 * follows from these counts and each grid's chunk and strip sizes
 * (gaus_get_poly_grids).  Synchronizes the stream. */
gaus_status gaus_poly_tier_census(gaus_ctx *ctx, int64_t counts[24]);

/* Message of the last failed call on ctx (or of the last failed gaus_init
 * when ctx is NULL).  Never NULL. */
const char *gaus_last_error(const gaus_ctx *ctx);

/* Static name of a status code. */
const char *gaus_status_string(gaus_status s);

/* Release the context's device copies and workspace (not the caller's
 * buffers).  Synchronizes the stream first.  NULL is ignored. */
void gaus_destroy(gaus_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* GAUS_H */
