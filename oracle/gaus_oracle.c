/*
 * gaus_oracle.c -- CPU oracle for the Gaussian-relaxed scheduling objective.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this code.  It shares no code,
 * header, table or constant with the GPU library: it is a plain, slow, fp64
 * restatement of the method of "GauS: Differentiable Scheduling Optimization
 * via Gaussian Reparameterization" (arXiv 2602.20427), written so that it can
 * be checked against the paper by eye:
 *
 *   - masses P_i^d                : Sec. 3.2, eq:round and its footnote
 *                                   (bin 0 open to -inf, bin D-1 open to +inf);
 *                                   other CDF families of App. E
 *   - expected usage              : App. B.2 (Res^), App. B.3 (modulo fold, MRes^)
 *   - resource violation          : App. B.2, eq:relu
 *   - dependency violation        : Sec. 3.2, eq:dep (with producer delay)
 *   - expected edge length        : App. B.1 (L^_Com)
 *   - recurrence violation        : App. B.3 (V^_Rec, with producer delay)
 *   - smooth peak usage L_Res     : App. B.2 (LogSumExp over steps, temperature
 *                                   tau; Sec. 3.2 eq:max), App. B.3 (modulo slots)
 *   - expected storage Reg^(d)    : Sec. 3.2 eq:active (b_i units held from d_i
 *                                   until the last successor starts), its modulo
 *                                   fold MReg^ (App. B.3) and smooth peak L_Mem
 *                                   (eq:max)
 *   - augmented Lagrangian        : Sec. 3.3, eq. (11) and Alg. 1
 *   - Adam                        : App. C.1 hyper-parameters; Kingma & Ba (2015)
 *   - legalization                : App. A, Alg. 3 (regular), Alg. 4 (modulo)
 *
 * Readings of the paper used here (where it is silent or inconsistent):
 *   R1  a dependency (i->j) is violated iff d_j < d_i + delta_i; delta = 0 gives
 *       eq:dep exactly, delta = 1 matches the "+1" of Alg. 3.
 *   R2  a back edge (j->i, k) (producer j, consumer i) is violated iff
 *       d_j + delta_j > d_i + k*II; the outer sum runs over all d_i >= 0.
 *   R5  the modulo fold only includes steps inside [0, D-1].
 *   R6  each op uses one unit of its own resource type; capacity per type.
 *   R7  ReLU'(0) = 0 (strict indicator U > C).
 *   R8  one multiplier per constraint family (dep, res, rec) per restart.
 *   R12 ASAP/ALAP with delays; sinks' ALAP is D-1 (start steps live in [0,D-1]).
 *   R13 Alg. 4 sources get t_min = 0; predecessors contribute s_u + delta_u.
 *   R14 Alg. 4 first clamps the rounded schedule to [0, D-1]; statuses
 *       NOT_CONVERGED (pass cap N reached) and OVERFLOW (some s > D-1).
 *   R4  rounding is half-up: s = floor(mu) + [mu - floor(mu) >= 1/2].
 *   R17 with K resource types the smooth peak is taken per type over its
 *       usage slots and summed over types: L_Res = sum_k tau log sum_t
 *       exp(U_k(t)/tau) (slots t < II when II > 0: the modulo peak MRes);
 *       it enters the objective with weight beta (Formulation A: beta = 1).
 *   R18 the storage term is eq:active as printed (F_i(d) (1 - prod_succ F_j(d)),
 *       so an op without successors holds nothing; the paper's sink node is
 *       an ordinary op of the caller's graph); folded like usage (R5, k >= 0
 *       as in the printed sum); L_Mem = tau log sum_t exp(MReg(t)/tau) enters
 *       the objective with weight gamma (Formulations B and C: gamma = 1).
 *
 * The gradient is the analytic derivative of the forward below (derived by
 * writing every term as a function of the CDF values at the D-1 interior bin
 * edges and applying the chain rule; see orc_loss_grad).  It is pinned against
 * central finite differences and against fp64 autograd in the tests.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int32_t n, e;              /* ops, forward edges */
    const int32_t *row_ptr;    /* [n+1] CSR by producer */
    const int32_t *col;        /* [e] consumers */
    const int32_t *delay;      /* [n] Lat(v_i) */
    const int32_t *rtype;      /* [n] resource type in [0,K) */
    int32_t K;
    const double *cap;         /* [K] capacity per type */
    int32_t D, II;             /* horizon; initiation interval (0 = regular) */
    int32_t nb;                /* back edges */
    const int32_t *bsrc;       /* [nb] producer v_j */
    const int32_t *bdst;       /* [nb] consumer v_i */
    const int32_t *bdist;      /* [nb] iteration distance k */
    const double *bmem;        /* [n] storage units b_i of each op's output */
} orc_problem;

enum { ORC_OK = 0, ORC_E_INVALID = 1, ORC_E_CYCLE = 2, ORC_E_HORIZON = 3,
       ORC_E_NOT_CONVERGED = 4, ORC_E_OVERFLOW = 5, ORC_E_NOMEM = 7 };

int orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the OpenMP loops that follow (the CPU baseline times 1 and all). */
void orc_set_num_threads(int32_t n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------ distribution family */

/* The relaxed start time is mu + sigma Z with Z of the chosen family
 * (App. E): 0 Gaussian; 1 logistic with scale s = sigma sqrt(3)/pi and
 * 2 Laplace with scale b = sigma/sqrt(2) (variance sigma^2); 3 Cauchy with
 * scale gamma = sigma sqrt(2 ln 2) (the Gaussian's half-maximum width).
 * Below, z is in sigma units and u = z / c the family's own variable. */
static int g_family = 0;

void orc_set_family(int32_t family) { g_family = family; }

static double fam_c(void) {
    switch (g_family) {
    case 1: return sqrt(3.0) / M_PI;
    case 2: return 1.0 / sqrt(2.0);
    case 3: return sqrt(2.0 * log(2.0));
    default: return 1.0;
    }
}

/* P(Z > z) for z >= 0 (the upper tail; by symmetry P(Z <= -z) too) */
static double tail_pos(double z) {
    const double u = z / fam_c();
    switch (g_family) {
    case 1: return exp(-u) / (1.0 + exp(-u));
    case 2: return 0.5 * exp(-u);
    case 3: return u > 1.0 ? atan(1.0 / u) / M_PI : 0.5 - atan(u) / M_PI;
    default: return 0.5 * erfc(z / M_SQRT2);
    }
}

/* CDF, upper tail and density (with respect to z) of Z */
static double Phi(double z) { return z >= 0.0 ? 1.0 - tail_pos(z) : tail_pos(-z); }
static double Qtail(double z) { return z >= 0.0 ? tail_pos(z) : 1.0 - tail_pos(-z); }
static double phi(double z) {
    const double c = fam_c(), u = fabs(z) / c;
    switch (g_family) {
    case 1: return exp(-u) / ((1.0 + exp(-u)) * (1.0 + exp(-u))) / c;
    case 2: return 0.5 * exp(-u) / c;
    case 3: return 1.0 / (M_PI * c * (1.0 + u * u));
    default: return exp(-0.5 * z * z) / sqrt(2.0 * M_PI);
    }
}

/* eq:round: P_i^d = Phi((d+1/2-mu)/sigma) - Phi((d-1/2-mu)/sigma); the lower
 * limit of bin 0 is -inf and the upper limit of bin D-1 is +inf (footnote).
 * When both limits lie in the upper half the difference is taken between
 * upper-tail values, which loses no relative precision. */
double orc_mass(double mu, double sigma, int32_t d, int32_t D) {
    double lo = (d == 0) ? -INFINITY : (d - 0.5 - mu) / sigma;
    double hi = (d == D - 1) ? INFINITY : (d + 0.5 - mu) / sigma;
    if (lo > 0.0) return Qtail(lo) - Qtail(hi);
    return Phi(hi) - Phi(lo);
}

/* CDF of the rounded start step at bin edge t: F(t) = P(d <= t).  Equals the
 * running sum of the masses up to t (telescoping of eq:round); F(t)=0 for
 * t < 0 and F(t)=1 for t >= D-1 because of the open end bins. */
static double cdf_row(const double *F, int64_t u, int32_t D) {
    if (u < 0) return 0.0;
    if (u >= D - 1) return 1.0;
    return F[u];
}

static double mass_row(const double *P, int64_t a, int32_t D) {
    if (a < 0 || a > D - 1) return 0.0;
    return P[a];
}

/* ------------------------------------------------------------ graph helpers */

typedef struct {
    int32_t *pred_ptr, *pred;      /* CSC: predecessors of each op */
    int32_t *bin_ptr, *bin;        /* back edges by consumer (ids into bsrc..) */
    int32_t *bout_ptr, *bout;      /* back edges by producer */
} orc_adj;

static void adj_free(orc_adj *a) {
    free(a->pred_ptr); free(a->pred); free(a->bin_ptr); free(a->bin);
    free(a->bout_ptr); free(a->bout);
}

static int adj_build(const orc_problem *p, orc_adj *a) {
    int32_t n = p->n;
    memset(a, 0, sizeof(*a));
    a->pred_ptr = calloc((size_t)n + 1, sizeof(int32_t));
    a->pred = malloc(sizeof(int32_t) * (size_t)(p->e > 0 ? p->e : 1));
    a->bin_ptr = calloc((size_t)n + 1, sizeof(int32_t));
    a->bout_ptr = calloc((size_t)n + 1, sizeof(int32_t));
    a->bin = malloc(sizeof(int32_t) * (size_t)(p->nb > 0 ? p->nb : 1));
    a->bout = malloc(sizeof(int32_t) * (size_t)(p->nb > 0 ? p->nb : 1));
    if (!a->pred_ptr || !a->pred || !a->bin_ptr || !a->bout_ptr || !a->bin || !a->bout) {
        adj_free(a); return ORC_E_NOMEM;
    }
    for (int32_t i = 0; i < n; ++i)
        for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e) a->pred_ptr[p->col[e] + 1]++;
    for (int32_t i = 0; i < n; ++i) a->pred_ptr[i + 1] += a->pred_ptr[i];
    int32_t *fill = calloc((size_t)n + 1, sizeof(int32_t));
    if (!fill) { adj_free(a); return ORC_E_NOMEM; }
    for (int32_t i = 0; i < n; ++i)              /* producers in id order */
        for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e) {
            int32_t j = p->col[e];
            a->pred[a->pred_ptr[j] + fill[j]++] = i;
        }
    for (int32_t b = 0; b < p->nb; ++b) { a->bin_ptr[p->bdst[b] + 1]++; a->bout_ptr[p->bsrc[b] + 1]++; }
    for (int32_t i = 0; i < n; ++i) { a->bin_ptr[i + 1] += a->bin_ptr[i]; a->bout_ptr[i + 1] += a->bout_ptr[i]; }
    memset(fill, 0, sizeof(int32_t) * ((size_t)n + 1));
    int32_t *fill2 = calloc((size_t)n + 1, sizeof(int32_t));
    if (!fill2) { free(fill); adj_free(a); return ORC_E_NOMEM; }
    for (int32_t b = 0; b < p->nb; ++b) {
        a->bin[a->bin_ptr[p->bdst[b]] + fill[p->bdst[b]]++] = b;
        a->bout[a->bout_ptr[p->bsrc[b]] + fill2[p->bsrc[b]]++] = b;
    }
    free(fill); free(fill2);
    return ORC_OK;
}

/* Kahn's algorithm.  level[v] = 0 for sources, else 1 + max level of its
 * predecessors; order = ops sorted by (level, id).  Returns ORC_E_CYCLE if the
 * forward edges are not acyclic. */
int orc_topo(const orc_problem *p, int32_t *level, int32_t *order) {
    int32_t n = p->n;
    orc_adj a;
    if (adj_build(p, &a)) return ORC_E_NOMEM;
    int32_t *indeg = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    int32_t *queue = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    if (!indeg || !queue) { free(indeg); free(queue); adj_free(&a); return ORC_E_NOMEM; }
    for (int32_t v = 0; v < n; ++v) { indeg[v] = a.pred_ptr[v + 1] - a.pred_ptr[v]; level[v] = 0; }
    int32_t head = 0, tail = 0;
    for (int32_t v = 0; v < n; ++v) if (indeg[v] == 0) queue[tail++] = v;
    while (head < tail) {
        int32_t u = queue[head++];
        for (int32_t e = p->row_ptr[u]; e < p->row_ptr[u + 1]; ++e) {
            int32_t v = p->col[e];
            if (level[u] + 1 > level[v]) level[v] = level[u] + 1;
            if (--indeg[v] == 0) queue[tail++] = v;
        }
    }
    int rc = (tail == n) ? ORC_OK : ORC_E_CYCLE;
    if (rc == ORC_OK) {
        /* counting sort by level, ids ascending inside a level */
        int32_t maxl = 0;
        for (int32_t v = 0; v < n; ++v) if (level[v] > maxl) maxl = level[v];
        int32_t *cnt = calloc((size_t)maxl + 2, sizeof(int32_t));
        if (!cnt) rc = ORC_E_NOMEM;
        else {
            for (int32_t v = 0; v < n; ++v) cnt[level[v] + 1]++;
            for (int32_t l = 0; l <= maxl; ++l) cnt[l + 1] += cnt[l];
            for (int32_t v = 0; v < n; ++v) order[cnt[level[v]]++] = v;
            free(cnt);
        }
    }
    free(indeg); free(queue); adj_free(&a);
    return rc;
}

/* ASAP / ALAP start steps with delays (reading R12):
 *   ASAP_v = max over preds u of ASAP_u + delta_u   (0 for sources)
 *   ALAP_v = min over succs w of ALAP_w - delta_v   (D-1 for sinks)
 * Returns ORC_E_HORIZON when some ASAP_v > ALAP_v (the critical path does not
 * fit in D steps). */
int orc_asap_alap(const orc_problem *p, int64_t *asap, int64_t *alap) {
    int32_t n = p->n;
    int32_t *level = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    int32_t *order = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    if (!level || !order) { free(level); free(order); return ORC_E_NOMEM; }
    int rc = orc_topo(p, level, order);
    if (rc == ORC_OK) {
        for (int32_t v = 0; v < n; ++v) asap[v] = 0;
        for (int32_t q = 0; q < n; ++q) {
            int32_t u = order[q];
            for (int32_t e = p->row_ptr[u]; e < p->row_ptr[u + 1]; ++e) {
                int32_t v = p->col[e];
                if (asap[u] + p->delay[u] > asap[v]) asap[v] = asap[u] + p->delay[u];
            }
        }
        for (int32_t q = n - 1; q >= 0; --q) {
            int32_t v = order[q];
            int64_t best = (int64_t)p->D - 1;
            for (int32_t e = p->row_ptr[v]; e < p->row_ptr[v + 1]; ++e) {
                int64_t c = alap[p->col[e]] - p->delay[v];
                if (c < best) best = c;
            }
            alap[v] = best;
        }
        for (int32_t v = 0; v < n; ++v) if (asap[v] > alap[v]) { rc = ORC_E_HORIZON; break; }
    }
    free(level); free(order);
    return rc;
}

/* -------------------------------------------------------- forward+backward */

/*
 * One restart.  Inputs mu, sigma [n] (float32 values promoted to double),
 * lam[3] = (lambda_dep, lambda_res, lambda_rec), beta and tau of the smooth
 * peak usage term, gamma of the smooth peak storage term.  Outputs:
 *   terms[7] = (L_total, V_dep, V_res, V_rec, L_com, L_res, L_mem)
 *   Mreg[T]  expected (folded) storage units per slot (may be NULL)
 *   U[K*T]   expected (folded) usage, T = II if II > 0 else D
 *   g_mu, g_sigma [n]  dL_total/dmu, dL_total/dsigma (may be NULL: forward only)
 *   n_ties   number of (k, slot) cells with |U - C| < tie_tol * max(1, C)
 */
int orc_loss_grad(const orc_problem *p, const double *mu, const double *sigma,
                  const double *lam, double alpha, double rho, double beta, double tau, double gamma,
                  double tie_tol, double *terms, double *U, double *Mreg, double *g_mu, double *g_sigma,
                  int64_t *n_ties) {
    const int32_t n = p->n, D = p->D, K = p->K, II = p->II;
    const int32_t T = (II > 0) ? II : D;
    if (D < 1 || n < 0 || K < 1) return ORC_E_INVALID;
    orc_adj a;
    if (adj_build(p, &a)) return ORC_E_NOMEM;
    /* F[i][t], t = 0..D-2 (interior bin edges); P[i][d], d = 0..D-1 */
    const int64_t DF = (D > 1) ? D - 1 : 1;
    double *F = malloc(sizeof(double) * (size_t)n * (size_t)DF + 8);
    double *P = malloc(sizeof(double) * (size_t)n * (size_t)D + 8);
    double *vd = calloc((size_t)n + 1, sizeof(double));
    double *lc = calloc((size_t)n + 1, sizeof(double));
    double *vr = calloc((size_t)p->nb + 1, sizeof(double));
    if (!F || !P || !vd || !lc || !vr) {
        free(F); free(P); free(vd); free(lc); free(vr); adj_free(&a); return ORC_E_NOMEM;
    }

    /* eq:round masses and the CDF at interior bin edges */
    #pragma omp parallel for schedule(dynamic, 16)
    for (int32_t i = 0; i < n; ++i) {
        for (int32_t t = 0; t < D - 1; ++t) F[(int64_t)i * DF + t] = Phi((t + 0.5 - mu[i]) / sigma[i]);
        for (int32_t d = 0; d < D; ++d) P[(int64_t)i * D + d] = orc_mass(mu[i], sigma[i], d, D);
    }

    /* expected usage per type and (modulo) slot: App. B.2 / B.3 */
    #pragma omp parallel for schedule(dynamic, 4)
    for (int64_t cell = 0; cell < (int64_t)K * T; ++cell) {
        int32_t k = (int32_t)(cell / T), s = (int32_t)(cell % T);
        double acc = 0.0;
        for (int32_t i = 0; i < n; ++i) {
            if (p->rtype[i] != k) continue;
            for (int32_t d = s; d < D; d += T) acc += P[(int64_t)i * D + d];
        }
        U[cell] = acc;
    }
    double V_res = 0.0;
    int64_t ties = 0;
    for (int64_t cell = 0; cell < (int64_t)K * T; ++cell) {
        double c = p->cap[cell / T];
        double ex = U[cell] - c;
        if (ex > 0.0) V_res += ex;                        /* eq:relu */
        if (fabs(ex) < tie_tol * (c > 1.0 ? c : 1.0)) ties++;
    }
    /* smooth peak per type, tau log sum_t exp(U/tau), shifted by the maximum;
     * soft[k][t] = its derivative with respect to U_k(t) (a softmax) */
    double L_res = 0.0;
    double *soft = calloc((size_t)K * T + 1, sizeof(double));
    if (!soft) { free(F); free(P); free(vd); free(lc); free(vr); adj_free(&a); return ORC_E_NOMEM; }
    if (beta != 0.0) {
        for (int32_t k = 0; k < K; ++k) {
            const double *Uk = U + (int64_t)k * T;
            double m = Uk[0];
            for (int32_t t = 1; t < T; ++t) if (Uk[t] > m) m = Uk[t];
            double z = 0.0;
            for (int32_t t = 0; t < T; ++t) z += exp((Uk[t] - m) / tau);
            L_res += m + tau * log(z);
            for (int32_t t = 0; t < T; ++t) soft[(int64_t)k * T + t] = exp((Uk[t] - m) / tau) / z;
        }
    }

    /* expected storage units per step, eq:active, folded like the usage;
     * L_mem and its derivative with respect to MReg(t) (a softmax) */
    double L_mem = 0.0;
    double *mreg = calloc((size_t)T + 1, sizeof(double));
    double *msoft = calloc((size_t)T + 1, sizeof(double));
    if (!mreg || !msoft) {
        free(mreg); free(msoft); free(soft); free(F); free(P); free(vd); free(lc); free(vr); adj_free(&a);
        return ORC_E_NOMEM;
    }
    if (gamma != 0.0 || Mreg) {
        for (int32_t d = 0; d < D; ++d) {
            double r = 0.0;
            for (int32_t i = 0; i < n; ++i) {
                if (p->row_ptr[i + 1] == p->row_ptr[i]) continue;   /* no successor: holds nothing */
                double q = 1.0;                                     /* P(every successor started by d) */
                for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e)
                    q *= cdf_row(F + (int64_t)p->col[e] * DF, d, D);
                r += p->bmem[i] * cdf_row(F + (int64_t)i * DF, d, D) * (1.0 - q);
            }
            mreg[d % T] += r;
        }
        if (Mreg) for (int32_t t = 0; t < T; ++t) Mreg[t] = mreg[t];
    }
    if (gamma != 0.0) {
        double m = mreg[0];
        for (int32_t t = 1; t < T; ++t) if (mreg[t] > m) m = mreg[t];
        double z = 0.0;
        for (int32_t t = 0; t < T; ++t) z += exp((mreg[t] - m) / tau);
        L_mem = m + tau * log(z);
        for (int32_t t = 0; t < T; ++t) msoft[t] = exp((mreg[t] - m) / tau) / z;
    }

    /* dependency violations and edge lengths, summed per producer */
    #pragma omp parallel for schedule(dynamic, 16)
    for (int32_t i = 0; i < n; ++i) {
        const double *Pi = P + (int64_t)i * D, *Fi = F + (int64_t)i * DF;
        double sd = 0.0, sc = 0.0;
        for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e) {
            const double *Fj = F + (int64_t)p->col[e] * DF;
            /* P(d_j < d_i + delta_i) = sum_a P_i^a * P(d_j <= a + delta_i - 1) */
            for (int32_t aa = 0; aa < D; ++aa) sd += Pi[aa] * cdf_row(Fj, (int64_t)aa + p->delay[i] - 1, D);
            /* E[(d_j - d_i)^+] = sum_t P(d_i <= t) P(d_j > t) */
            for (int32_t t = 0; t < D - 1; ++t) sc += Fi[t] * (1.0 - Fj[t]);
        }
        vd[i] = sd; lc[i] = sc;
    }
    /* recurrence violations: P(d_j + delta_j > d_i + k*II) */
    #pragma omp parallel for schedule(dynamic, 4)
    for (int32_t b = 0; b < p->nb; ++b) {
        int32_t j = p->bsrc[b], i = p->bdst[b];
        int64_t off = (int64_t)p->bdist[b] * II - p->delay[j];
        const double *Pi = P + (int64_t)i * D, *Fj = F + (int64_t)j * DF;
        double s = 0.0;
        for (int32_t aa = 0; aa < D; ++aa) s += Pi[aa] * (1.0 - cdf_row(Fj, aa + off, D));
        vr[b] = s;
    }
    double V_dep = 0.0, L_com = 0.0, V_rec = 0.0;
    for (int32_t i = 0; i < n; ++i) { V_dep += vd[i]; L_com += lc[i]; }
    for (int32_t b = 0; b < p->nb; ++b) V_rec += vr[b];

    /* augmented Lagrangian, eq. (11) */
    double V[3] = {V_dep, V_res, V_rec};
    double L = alpha * L_com + beta * L_res + gamma * L_mem;
    for (int c = 0; c < 3; ++c) L += lam[c] * V[c] + 0.5 * rho * V[c] * V[c];
    terms[0] = L; terms[1] = V_dep; terms[2] = V_res; terms[3] = V_rec; terms[4] = L_com;
    terms[5] = L_res; terms[6] = L_mem;
    if (n_ties) *n_ties = ties;

    if (g_mu && g_sigma) {
        const double w_dep = lam[0] + rho * V_dep, w_res = lam[1] + rho * V_res, w_rec = lam[2] + rho * V_rec;
        #pragma omp parallel
        {
            double *G = malloc(sizeof(double) * (size_t)D + 8);
            #pragma omp for schedule(dynamic, 16)
            for (int32_t i = 0; i < n; ++i) {
                const int32_t k = p->rtype[i];
                /* G(d) = dL/dP_i^d, holding the CDFs of the other ops fixed */
                for (int32_t d = 0; d < D; ++d) {
                    double g = (U[(int64_t)k * T + (d % T)] > p->cap[k]) ? w_res : 0.0;
                    g += beta * soft[(int64_t)k * T + (d % T)];
                    for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e)
                        g += w_dep * cdf_row(F + (int64_t)p->col[e] * DF, (int64_t)d + p->delay[i] - 1, D);
                    for (int32_t q = a.bin_ptr[i]; q < a.bin_ptr[i + 1]; ++q) {
                        int32_t b = a.bin[q], j = p->bsrc[b];
                        int64_t u = (int64_t)d + (int64_t)p->bdist[b] * II - p->delay[j];
                        g += w_rec * (1.0 - cdf_row(F + (int64_t)j * DF, u, D));
                    }
                    G[d] = g;
                }
                /* H(t) = dL/dF_i(t) at the interior bin edges t = 0..D-2 */
                double gm = 0.0, gs = 0.0;
                for (int32_t t = 0; t < D - 1; ++t) {
                    double h = G[t] - G[t + 1];   /* P_i^t = F(t)-F(t-1), P_i^{t+1} = F(t+1)-F(t) */
                    for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e)
                        h += alpha * (1.0 - F[(int64_t)p->col[e] * DF + t]);          /* as producer in L_com */
                    for (int32_t q = a.pred_ptr[i]; q < a.pred_ptr[i + 1]; ++q) {
                        int32_t hh = a.pred[q];
                        h -= alpha * F[(int64_t)hh * DF + t];                           /* as consumer in L_com */
                        h += w_dep * mass_row(P + (int64_t)hh * D, (int64_t)t - p->delay[hh] + 1, D); /* as consumer in V_dep */
                    }
                    for (int32_t q = a.bout_ptr[i]; q < a.bout_ptr[i + 1]; ++q) {      /* as producer in V_rec */
                        int32_t b = a.bout[q], ic = p->bdst[b];
                        int64_t aa = (int64_t)t - (int64_t)p->bdist[b] * II + p->delay[i];
                        h -= w_rec * mass_row(P + (int64_t)ic * D, aa, D);
                    }
                    if (gamma != 0.0) {   /* eq:active: as the op itself and as a successor */
                        double ws = gamma * msoft[t % T], own = 0.0;
                        if (p->row_ptr[i + 1] > p->row_ptr[i]) {
                            double q = 1.0;
                            for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e)
                                q *= F[(int64_t)p->col[e] * DF + t];
                            own = p->bmem[i] * (1.0 - q);
                        }
                        for (int32_t q2 = a.pred_ptr[i]; q2 < a.pred_ptr[i + 1]; ++q2) {
                            int32_t hh = a.pred[q2];
                            double others = 1.0;       /* the other successors of hh, started by t */
                            for (int32_t e = p->row_ptr[hh]; e < p->row_ptr[hh + 1]; ++e)
                                if (p->col[e] != i) others *= F[(int64_t)p->col[e] * DF + t];
                            own -= p->bmem[hh] * F[(int64_t)hh * DF + t] * others;
                        }
                        h += ws * own;
                    }
                    double z = (t + 0.5 - mu[i]) / sigma[i];
                    double dF_dmu = -phi(z) / sigma[i];
                    double dF_dsigma = -phi(z) * z / sigma[i];
                    gm += h * dF_dmu;
                    gs += h * dF_dsigma;
                }
                g_mu[i] = gm; g_sigma[i] = gs;
            }
            free(G);
        }
    }
    free(F); free(P); free(vd); free(lc); free(vr); free(soft); free(mreg); free(msoft); adj_free(&a);
    return ORC_OK;
}

/*
 * Derivative of one expected usage cell U_k(s) (App. B.2; folded modulo II as
 * in App. B.3, steps d = s, s+T, ... inside [0, D-1]) with respect to mu_i and
 * sigma_i of every op i, times w (ops of other types get 0).  With
 * P_i^d = F_i(d) - F_i(d-1) (eq:round) and the constant end values
 * F_i(-1) = 0, F_i(D-1) = 1, each step d of the cell contributes
 * dF_i(d) - dF_i(d-1) over the interior bin edges, where
 * dF/dmu = -phi(z)/sigma and dF/dsigma = -phi(z) z/sigma at z = (t+1/2-mu)/sigma.
 * The ReLU of eq:relu adds w_res times this vector to the gradient exactly
 * when the cell's indicator [U_k(s) > C_k] is 1, so a comparison that meets a
 * cell within rounding of its capacity can accept either indicator value.
 */
int orc_usage_cell_grad(const orc_problem *p, const double *mu, const double *sigma, int32_t k, int32_t s,
                        double w, double *g_mu, double *g_sigma) {
    const int32_t n = p->n, D = p->D, T = (p->II > 0) ? p->II : D;
    if (k < 0 || k >= p->K || s < 0 || s >= T) return ORC_E_INVALID;
    for (int32_t i = 0; i < n; ++i) {
        double gm = 0.0, gs = 0.0;
        if (p->rtype[i] == k) {
            for (int32_t d = s; d < D; d += T) {
                /* +dF(d) at the upper edge of bin d, -dF(d-1) at its lower edge */
                for (int32_t side = 0; side < 2; ++side) {
                    const int32_t t = side == 0 ? d : d - 1;
                    if (t < 0 || t > D - 2) continue;
                    const double z = (t + 0.5 - mu[i]) / sigma[i];
                    const double sg = side == 0 ? 1.0 : -1.0;
                    gm += sg * (-phi(z) / sigma[i]);
                    gs += sg * (-phi(z) * z / sigma[i]);
                }
            }
        }
        g_mu[i] = w * gm;
        g_sigma[i] = w * gs;
    }
    return ORC_OK;
}

/* The paper's formulas written as literal double sums over (d_i, d_j) (with the
 * producer delay of reading R1/R2).  O(E * D^2): tiny instances only. */
void orc_edge_terms_double_sum(const orc_problem *p, const double *mu, const double *sigma, double out[3]) {
    const int32_t D = p->D;
    double vdep = 0.0, lcom = 0.0, vrec = 0.0;
    for (int32_t i = 0; i < p->n; ++i)
        for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e) {
            int32_t j = p->col[e];
            for (int32_t di = 0; di < D; ++di) {
                double pi = orc_mass(mu[i], sigma[i], di, D);
                for (int32_t dj = 0; dj < D; ++dj) {
                    double pj = orc_mass(mu[j], sigma[j], dj, D);
                    if (dj < di + p->delay[i]) vdep += pi * pj;        /* eq:dep */
                    if (dj >= di) lcom += pi * pj * (dj - di);          /* App. B.1 */
                }
            }
        }
    for (int32_t b = 0; b < p->nb; ++b) {
        int32_t j = p->bsrc[b], i = p->bdst[b];
        for (int32_t di = 0; di < D; ++di) {
            double pi = orc_mass(mu[i], sigma[i], di, D);
            for (int32_t dj = 0; dj < D; ++dj)
                if ((int64_t)dj + p->delay[j] > (int64_t)di + (int64_t)p->bdist[b] * p->II)   /* App. B.3 */
                    vrec += pi * orc_mass(mu[j], sigma[j], dj, D);
        }
    }
    out[0] = vdep; out[1] = lcom; out[2] = vrec;
}

/* ------------------------------------------------------------------ Adam */

/* One Adam step (Kingma & Ba 2015, bias-corrected, no weight decay) on n
 * parameters; t is the step number after incrementing (t >= 1). */
void orc_adam(int64_t n, double *theta, double *m, double *v, const double *g, int32_t t,
              double lr, double b1, double b2, double eps) {
    double c1 = 1.0 - pow(b1, t), c2 = 1.0 - pow(b2, t);
    for (int64_t i = 0; i < n; ++i) {
        m[i] = b1 * m[i] + (1.0 - b1) * g[i];
        v[i] = b2 * v[i] + (1.0 - b2) * g[i] * g[i];
        double mh = m[i] / c1, vh = v[i] / c2;
        theta[i] -= lr * mh / (sqrt(vh) + eps);
    }
}

/* ------------------------------------------------- discrete schedule cost */

/*
 * Cost of one integer schedule s [n] (Sec. 2.1), the quantity a driver of
 * Alg. 1 keeps the best of:
 *   out[0] = alpha * L_com + beta * L_res + gamma * L_mem      (the cost)
 *   out[1] = L_com = sum over edges (s_j - s_i)^+              (App. B.1)
 *   out[2] = L_res = sum over types k of max_t U_k(t)          (eq. (3), usage
 *            folded mod II when II > 0 as in eq. (5))
 *   out[3] = L_mem = max_t Mem(t), Mem(d) = sum_i b_i [s_i <= d < max_succ s_j]
 *            (eq:mem), folded like the usage
 *   out[4] = V_res = sum_{k,t} (U_k(t) - C_k)^+                 (eq:relu at sigma -> 0)
 *   out[5] = 1 if the schedule is legal: 0 <= s <= D-1, every edge has
 *            s_j >= s_i + Lat_i and every back edge s_i + k II >= s_j + Lat_j
 * Steps outside [0, D-1] count in neither usage nor storage.
 */
int orc_schedule_cost(const orc_problem *p, const int64_t *s, double alpha, double beta, double gamma,
                      double *out) {
    const int32_t n = p->n, D = p->D, K = p->K, II = p->II;
    const int32_t T = (II > 0) ? II : D;
    double *U = calloc((size_t)K * T + 1, sizeof(double));
    double *M = calloc((size_t)T + 1, sizeof(double));
    if (!U || !M) { free(U); free(M); return ORC_E_NOMEM; }
    int legal = 1;
    double lcom = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        if (s[i] < 0 || s[i] > D - 1) legal = 0;
        else U[(int64_t)p->rtype[i] * T + s[i] % T] += 1.0;
        int64_t last = -1;
        for (int32_t e = p->row_ptr[i]; e < p->row_ptr[i + 1]; ++e) {
            int64_t sj = s[p->col[e]];
            if (sj < s[i] + p->delay[i]) legal = 0;
            if (sj > s[i]) lcom += (double)(sj - s[i]);
            if (sj > last) last = sj;
        }
        for (int64_t d = s[i]; d < last; ++d)
            if (d >= 0 && d <= D - 1) M[d % T] += p->bmem[i];
    }
    for (int32_t b = 0; b < p->nb; ++b) {
        int32_t j = p->bsrc[b], i = p->bdst[b];
        if (s[i] + (int64_t)p->bdist[b] * II < s[j] + p->delay[j]) legal = 0;
    }
    double lres = 0.0, vres = 0.0, lmem = 0.0;
    for (int32_t k = 0; k < K; ++k) {
        double mx = 0.0;
        for (int32_t t = 0; t < T; ++t) {
            double u = U[(int64_t)k * T + t];
            if (u > mx) mx = u;
            if (u > p->cap[k]) vres += u - p->cap[k];
        }
        lres += mx;
    }
    for (int32_t t = 0; t < T; ++t) if (M[t] > lmem) lmem = M[t];
    out[0] = alpha * lcom + beta * lres + gamma * lmem;
    out[1] = lcom; out[2] = lres; out[3] = lmem; out[4] = vres; out[5] = legal;
    free(U); free(M);
    return ORC_OK;
}

/* ------------------------------------------------------------ legalization */

/* half-up rounding of a float32 value, after clamping it to [-1, D]; a NaN
 * is treated as -1 */
static int64_t round_half_up(float muf, int32_t D) {
    double m = (double)muf;
    if (!(m >= -1.0)) m = -1.0;
    if (m > (double)D) m = (double)D;
    double fl = floor(m);
    return (int64_t)fl + ((m - fl) >= 0.5 ? 1 : 0);
}

/*
 * Both legalization heuristics of App. A start from the rounded means, clamp
 * them (Alg. 3 for II = 0: into [ASAP, ALAP]; Alg. 4 for II > 0: into
 * [0, D-1]), and then only ever raise an op, each time to the smallest step
 * its predecessors (and, for Alg. 4, its recurrences) allow; Alg. 4 repeats
 * its sweeps until nothing moves, at most N of them.  What they return is
 * therefore, by definition, the least schedule s >= r (r = the clamped
 * rounding) with
 *     s_v >= s_u + Lat_u              for every edge u -> v,
 *     s_i + k II >= s_j + Lat_j       for every back edge (j -> i, k);
 * the set of such s is closed under componentwise minimum, so when one
 * exists a least one does.  This oracle computes that schedule directly, as
 * the limit of whole-graph rounds s <- max(s, requirement(s)) in which every
 * op reads the previous round's values (no sweep order at all):
 *   - without a cycle of positive weight in the constraint graph a longest
 *     path has at most N-1 edges, so the values settle within N-1 rounds and
 *     a round that changes nothing ends the computation;
 *   - a positive cycle (recurrences no schedule can meet) changes something
 *     in every round: after N rounds the status is NOT_CONVERGED (the pass
 *     cap of Alg. 4; any sweep order settles no later than these rounds, so
 *     the status does not depend on the order);
 *   - OVERFLOW when the least schedule leaves the horizon (some s_v > D-1).
 * Returns ORC_OK, ORC_E_NOT_CONVERGED or ORC_E_OVERFLOW.
 */
static int least_schedule_above(const orc_problem *p, const orc_adj *a, int64_t *s) {
    const int32_t n = p->n;
    int64_t *prev = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!prev) return ORC_E_NOMEM;
    int settled = 0;
    for (int32_t round = 0; round < (n > 0 ? n : 1) && !settled; ++round) {
        memcpy(prev, s, sizeof(int64_t) * (size_t)n);
        settled = 1;
        for (int32_t v = 0; v < n; ++v) {
            int64_t need = prev[v];
            for (int32_t r = a->pred_ptr[v]; r < a->pred_ptr[v + 1]; ++r) {   /* forward edges u -> v */
                const int32_t u = a->pred[r];
                if (prev[u] + p->delay[u] > need) need = prev[u] + p->delay[u];
            }
            for (int32_t r = a->bin_ptr[v]; r < a->bin_ptr[v + 1]; ++r) {     /* back edges (j -> v, k) */
                const int32_t b = a->bin[r], j = p->bsrc[b];
                const int64_t c = prev[j] + p->delay[j] - (int64_t)p->bdist[b] * p->II;
                if (c > need) need = c;
            }
            if (need != prev[v]) settled = 0;
            s[v] = need;
        }
    }
    free(prev);
    if (!settled) return ORC_E_NOT_CONVERGED;
    for (int32_t v = 0; v < n; ++v) if (s[v] > p->D - 1) return ORC_E_OVERFLOW;
    return ORC_OK;
}

/*
 * Legalize one restart (App. A).  mu [n] float32; out s [n] int64; returns the
 * status of least_schedule_above (or ORC_E_CYCLE / ORC_E_HORIZON for a bad
 * problem).  r = half-up rounding of mu (R4), clamped to [ASAP, ALAP] when
 * II == 0 (Alg. 3) and to [0, D-1] when II > 0 (Alg. 4, R14).
 */
int orc_legalize(const orc_problem *p, const float *mu, int64_t *s) {
    const int32_t n = p->n, D = p->D;
    int32_t *level = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    int32_t *order = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    int64_t *asap = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *alap = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    orc_adj a;
    if (!level || !order || !asap || !alap || adj_build(p, &a)) {
        free(level); free(order); free(asap); free(alap); return ORC_E_NOMEM;
    }
    int rc = orc_topo(p, level, order);
    if (rc == ORC_OK && p->II == 0) rc = orc_asap_alap(p, asap, alap);
    if (rc == ORC_OK) {
        for (int32_t v = 0; v < n; ++v) {
            const int64_t lo = p->II == 0 ? asap[v] : 0, hi = p->II == 0 ? alap[v] : (int64_t)D - 1;
            const int64_t r = round_half_up(mu[v], D);
            s[v] = r < lo ? lo : (r > hi ? hi : r);
        }
        rc = least_schedule_above(p, &a, s);
    }
    free(level); free(order); free(asap); free(alap); adj_free(&a);
    return rc;
}

/* --------------------------------------------------- one check of Alg. 1 */

/*
 * The order in which a driver of Alg. 1 keeps schedules (reading R15 of the
 * Sampling paragraph of Sec. 3.3 and App. A's "reset to the prior best"):
 * a schedule is feasible when it is legal and within every capacity
 * (V_res = 0); feasible beats infeasible; two feasible ones compare by cost;
 * among infeasible ones a legal one beats an illegal one, then the lower
 * V_res wins, then the lower cost.  Equal ones do not replace each other.
 * c = (cost, L_com, L_res, L_mem, V_res, legal) as orc_schedule_cost writes.
 */
static int better_schedule(const double *c, const double *b) {
    const int fc = c[5] != 0.0 && c[4] == 0.0, fb = b[5] != 0.0 && b[4] == 0.0;
    if (fc != fb) return fc;
    if (fc) return c[0] < b[0];
    if (c[5] != b[5]) return c[5] != 0.0;
    if (c[4] != b[4]) return c[4] < b[4];
    return c[0] < b[0];
}

/*
 * One check of the Alg. 1 driver for one restart, in the order the driver
 * takes its steps:
 *   1. round the means half-up (R4);
 *   2. legalize (Alg. 3 / Alg. 4 above): the candidate schedule;
 *   3. cost the candidate (Sec. 2.1, orc_schedule_cost);
 *   4. keep it as the restart's best if it is better (better_schedule);
 *   5. if the rounding was not already legal (the candidate differs from it),
 *      re-initialize the means (Sec. 3.3 "Sampling"): from the candidate if
 *      it improved the best, else from the prior best (App. A);
 *   6. clear the re-initialized restart's Adam moments and, with
 *      reinit_sigma, set sigma = max(kappa (ALAP - ASAP), sigma_min) (the
 *      initial rule, Sec. 3.3 "Initialization").
 * In/out: mu, sigma [n] float32; m, v [2][n] float32 (moments of mu, then of
 * sigma); best_s [n] int64 and best_c [6] (a best_c with legal = 0 and
 * V_res = cost = +inf holds no schedule yet).  Out: cand [n], cand_c [6],
 * *mode (0 kept, 1 from the candidate, 2 from the prior best), *improved.
 * kappa and sigma_min are the float32 hyper-parameters.
 */
int orc_check(const orc_problem *p, float *mu, float *sigma, float *m, float *v, int64_t *best_s,
              double *best_c, double alpha, double beta, double gamma, int32_t reinit_sigma, float kappa,
              float sigma_min, int64_t *cand, double *cand_c, int32_t *mode, int32_t *improved) {
    const int32_t n = p->n;
    int64_t *asap = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *alap = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!asap || !alap) { free(asap); free(alap); return ORC_E_NOMEM; }
    int rc = orc_asap_alap(p, asap, alap);
    if (rc != ORC_OK && p->II == 0) { free(asap); free(alap); return rc; }
    (void)orc_legalize(p, mu, cand);                        /* steps 1-2; the status is not used */
    rc = orc_schedule_cost(p, cand, alpha, beta, gamma, cand_c);   /* step 3 */
    if (rc != ORC_OK) { free(asap); free(alap); return rc; }
    int rounding_legal = 1;
    for (int32_t i = 0; i < n; ++i) if (round_half_up(mu[i], p->D) != cand[i]) rounding_legal = 0;
    *improved = better_schedule(cand_c, best_c);            /* step 4 */
    if (*improved) {
        memcpy(best_s, cand, sizeof(int64_t) * (size_t)n);
        memcpy(best_c, cand_c, sizeof(double) * 6);
    }
    *mode = rounding_legal ? 0 : (*improved ? 1 : 2);
    if (*mode) {                                            /* steps 5-6 */
        const int64_t *src = (*mode == 1) ? cand : best_s;  /* after step 4, best_s is the prior best
                                                               whenever mode is 2 */
        for (int32_t i = 0; i < n; ++i) {
            mu[i] = (float)src[i];
            if (reinit_sigma) {
                const double w = (double)kappa * (double)(alap[i] - asap[i]);
                const float sg = (float)w;
                sigma[i] = sg > sigma_min ? sg : sigma_min;
            }
            m[i] = 0.0f; m[n + i] = 0.0f;
            v[i] = 0.0f; v[n + i] = 0.0f;
        }
    }
    free(asap); free(alap);
    return ORC_OK;
}

/* ---------------------------------------------------------- initial state */

/* Paper's initialization (Sec. 3.3 "Initialization", Alg. 1):
 *   sigma = max(kappa * (ALAP - ASAP), sigma_min)
 *   mu    = (ASAP + ALAP) / 2 for restart 0; restarts b >= 1 place mu at
 *           ASAP + u * (ALAP - ASAP) with u ~ U[0,1) given by the caller. */
int orc_init_state(const orc_problem *p, int32_t B, const double *u, double kappa, double sigma_min,
                   double *mu, double *sigma) {
    const int32_t n = p->n;
    int64_t *asap = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *alap = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!asap || !alap) { free(asap); free(alap); return ORC_E_NOMEM; }
    int rc = orc_asap_alap(p, asap, alap);
    if (rc == ORC_OK) {
        for (int32_t b = 0; b < B; ++b)
            for (int32_t v = 0; v < n; ++v) {
                double slack = (double)(alap[v] - asap[v]);
                double sg = kappa * slack;
                sigma[(int64_t)b * n + v] = sg > sigma_min ? sg : sigma_min;
                mu[(int64_t)b * n + v] = (b == 0) ? 0.5 * (double)(asap[v] + alap[v])
                                                  : (double)asap[v] + u[(int64_t)b * n + v] * slack;
            }
    }
    free(asap); free(alap);
    return rc;
}
