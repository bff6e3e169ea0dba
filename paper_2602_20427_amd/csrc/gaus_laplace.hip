// gfx950 kernel of the edge terms for the Laplace start times (App. E) in
// closed form.  See gaus_kernels.hip for the notation.
//
// With the Laplace law an op's CDF at the bin edges v is, in u-space
// u = lam (v - m), lam = sqrt(2)/sigma, m = mu - 1/2,
//   F(v) = exp(u)/2 (v < m),   1 - exp(-u)/2 (v >= m),
// with F = 0 for v < 0 and F = 1 for v >= D-1 (the open end bins), and
//   dF/dmu = -lam exp(-|u|)/2,   dF/dsigma = dF/dmu (v - m)/sigma.
// On any run of steps where none of these cases changes, every factor of
// the edge sums (F_i(u), F_i(u-s), F_i(u-s+1), F_j(u), F_j(u-1) and their
// derivatives) is a constant plus one exponential in u, so every summand is
// a short sum of terms c e^(g u) (u - a)^p with p <= 1 and each sum over the
// run is a geometric (p = 0) or arithmetico-geometric (p = 1) series in
// closed form.  The runs are cut where a case changes: nine growth rates
// per run (producer slot x consumer slot) and a handful of runs per edge,
// against D steps on the step path.  Everything here is fp64 (the series in
// expm1 form; no term exceeds its largest summand, which keeps every
// exponent bounded).
#include "gaus_device.h"

namespace gaus {

namespace {

// A factor on the run [a, b]: a constant c plus the exponential growing with
// u (the op's CDF below its median, rate +lam) and the one decaying with u
// (above it, rate -lam), each given by its values at a and at b (weights
// included; 0 when absent).  Differences of factors are taken slot by slot.
struct LF {
    double c, loA, loB, upA, upB;
};
__device__ __forceinline__ LF fsub(const LF &f, const LF &h) {
    return LF{f.c - h.c, f.loA - h.loA, f.loB - h.loB, f.upA - h.upA, f.upB - h.upB};
}

// Sums over k = 0 .. n-1 of e^(g k) (G0) and k e^(g k) (G1), g <= 0, n >= 2.
__device__ __forceinline__ void geo_sums(double g, int n, double &G0, double &G1) {
    const double x = -g, xn = x * n;
    if (x == 0.0) {
        G0 = n;
        G1 = 0.5 * n * (n - 1.0);
        return;
    }
    const double e1 = -expm1(-x);   // 1 - e^(-x)
    if (xn < 0.5) {
        const double en = -expm1(-xn);   // 1 - e^(-x n)
        G0 = en / e1;
        if (xn < 0.02) {   // power sums S_p = sum k^p, k < n, and the series of e^(-x k)
            const double nn = n, s1 = 0.5 * nn * (nn - 1.0), s2 = (nn - 1.0) * nn * (2.0 * nn - 1.0) / 6.0;
            const double s3 = s1 * s1, s4 = (nn - 1.0) * nn * (2.0 * nn - 1.0) * (3.0 * nn * nn - 3.0 * nn - 1.0) / 30.0;
            const double s5 = s1 * s1 * (2.0 * nn * nn - 2.0 * nn - 1.0) / 3.0;
            G1 = s1 - x * s2 + x * x * s3 / 2.0 - x * x * x * s4 / 6.0 + x * x * x * x * s5 / 24.0;
        } else {
            // sum k q^k = q (1 - q^(n-1) (1 + (n-1)(1-q))) / (1-q)^2, q = e^(-x);
            // here q > 0.6 and q^(n-1) > 0.6, both exact enough from e1, en
            const double q = 1.0 - e1, qn1 = (1.0 - en) / q;
            G1 = q * (1.0 - qn1 * (1.0 + (n - 1.0) * e1)) / (e1 * e1);
        }
    } else {
        // e^(-x n) < 0.61: 1 - e^(-x n) from the product without cancellation.
        // q^(n-1), and q once x >= 0.5, come from exp itself: through e1 and
        // en they would carry an absolute error of an ulp of 1, which is no
        // small error once they are tiny (0/0 once e1 rounds to 1)
        const double q = x < 0.5 ? 1.0 - e1 : exp(-x), qn1 = exp(-x * (n - 1.0));
        G0 = (1.0 - q * qn1) / e1;
        G1 = q * (1.0 - qn1 * (1.0 + (n - 1.0) * e1)) / (e1 * e1);
    }
}

// Weights of the run for a product of slots with growth g: the sums over
// the run of the product (S0) and of the product times (u - a) (S1) are
// V w0 and V w1, V the product's value at a (g <= 0) or at b (g > 0, the
// series then taken from b: every term at most V).
struct GW {
    double w0, w1;
    bool atB;
};
__device__ __attribute__((noinline)) GW run_weights(double g, int n) {   // (a call: fewer live registers)
    GW r;
    if (n == 1) { r.w0 = 1.0; r.w1 = 0.0; r.atB = false; return r; }
    if (n <= 4) {   // a few steps: the powers of e^(-|g|) from the larger end
        const double q = exp(-fabs(g));
        double G0 = 1.0, G1 = 0.0, qk = 1.0;
        for (int k = 1; k < n; ++k) { qk *= q; G0 += qk; G1 = fma((double)k, qk, G1); }
        r.w0 = G0;
        r.w1 = g <= 0.0 ? G1 : (n - 1.0) * G0 - G1;
        r.atB = g > 0.0;
        return r;
    }
    double G0, G1;
    if (g <= 0.0) {
        geo_sums(g, n, G0, G1);
        r.w0 = G0; r.w1 = G1; r.atB = false;
    } else {
        geo_sums(-g, n, G0, G1);
        r.w0 = G0; r.w1 = (n - 1.0) * G0 - G1; r.atB = true;
    }
    return r;
}

// The nine slot pairs (producer slot x, consumer slot y) of a run.
struct RunW {
    GW w[3][3];
};
__device__ __forceinline__ RunW run_table(double li, double lj, int n, const bool ui[3], const bool uj[3]) {
    RunW t;
    const double gi[3] = {0.0, li, -li}, gj[3] = {0.0, lj, -lj};
#pragma unroll
    for (int x = 0; x < 3; ++x)
#pragma unroll
        for (int y = 0; y < 3; ++y) {
            if (ui[x] && uj[y]) t.w[x][y] = run_weights(gi[x] + gj[y], n);
            else t.w[x][y] = GW{0.0, 0.0, false};   // no factor of the run has these slots
        }
    return t;
}
// the slots a factor holds (constant, growing, decaying)
__device__ __forceinline__ void mark(const LF &f, bool u[3]) {
    u[0] = u[0] || f.c != 0.0;
    u[1] = u[1] || f.loA != 0.0 || f.loB != 0.0;
    u[2] = u[2] || f.upA != 0.0 || f.upB != 0.0;
}

// sums over the run of f*h (f a producer factor, h a consumer factor):
// S0 = sum f h, S1 = sum f h (u - a)
__device__ __forceinline__ void prod_sums(const LF &f, const LF &h, const RunW &t, double &S0, double &S1) {
    const double fa[3] = {f.c, f.loA, f.upA}, fb[3] = {f.c, f.loB, f.upB};
    const double ha[3] = {h.c, h.loA, h.upA}, hb[3] = {h.c, h.loB, h.upB};
    S0 = 0.0;
    S1 = 0.0;
#pragma unroll
    for (int x = 0; x < 3; ++x)
#pragma unroll
        for (int y = 0; y < 3; ++y) {
            const GW &w = t.w[x][y];
            const double V = w.atB ? fb[x] * hb[y] : fa[x] * ha[y];
            S0 = fma(V, w.w0, S0);
            S1 = fma(V, w.w1, S1);
        }
}

// The op at the bin edges u + off, u in [a, b] (one case throughout): past
// an end of the horizon (F = 0 below it, 1 at its last edge and beyond) or
// on one side of the median, with e/2 at both ends, e = e^(-lam |v - m|).
struct LOp {
    double m, lam;
};
struct LV {
    int endv;   // 0: F = 0, 1: F = 1, -1: inside
    bool up;    // at or above the median
    double ea, eb;
};
__device__ __forceinline__ LV lval(const LOp &o, int off, int a, int b, int D) {
    LV v;
    const int va = a + off, vb = b + off;
    v.endv = va < 0 ? 0 : va >= D - 1 ? 1 : -1;
    v.up = (double)va >= o.m;
    v.ea = v.eb = 0.0;
    if (v.endv < 0) {
        const double sg = v.up ? -1.0 : 1.0;   // e^(+lam (v-m)) below the median, e^(-lam (v-m)) above
        v.ea = 0.5 * exp(sg * o.lam * ((double)va - o.m));
        v.eb = 0.5 * exp(sg * o.lam * ((double)vb - o.m));
    }
    return v;
}
// kind 0: F, 1: 1 - F, 2: dF/dmu
__device__ __forceinline__ LF factor(const LV &v, double lam, int kind) {
    LF f{0.0, 0.0, 0.0, 0.0, 0.0};
    if (v.endv >= 0) {
        f.c = ((kind == 0 && v.endv == 1) || (kind == 1 && v.endv == 0)) ? 1.0 : 0.0;
        return f;
    }
    // F: e/2 below, 1 - e/2 above; 1 - F: the complement; dF/dmu = -lam e/2
    const double w = kind == 2 ? -lam : (kind == 0) == v.up ? -1.0 : 1.0;
    f.c = kind == 2 ? 0.0 : (kind == 0) == v.up ? 1.0 : 0.0;
    if (v.up) { f.upA = w * v.ea; f.upB = w * v.eb; }
    else { f.loA = w * v.ea; f.loB = w * v.eb; }
    return f;
}

__device__ __forceinline__ double cdf_lap(const LOp &o, int v, int D) {
    if (v < 0) return 0.0;
    if (v >= D - 1) return 1.0;
    const double u = o.lam * ((double)v - o.m);
    return u < 0.0 ? 0.5 * exp(u) : 1.0 - 0.5 * exp(-u);
}

}  // namespace

// One edge (i -> j), producer delay s: the ten sums of the op kernel's
// description (gaus_step.hip) over the whole horizon.
//   P[0] V_dep, P[1] L_com, P[2..3] dVdep/d(mu_i, sigma_i), P[4..5] dLcom/d(mu_i, sigma_i)
//   C[0..1] dVdep/d(mu_j, sigma_j), C[2..3] dLcom/d(mu_j, sigma_j)
__device__ void laplace_edge(const LOp &oi, double sg_i, int s, const LOp &oj, double sg_j, int D, double P[6],
                             double C[4]) {
    // the steps where a case changes (the first step of the new case),
    // taken in increasing order by a scan over the candidates
    // (medians clamped to +-2^50 before the conversion: cuts that far out
    // never fall inside the horizon)
    const double mcl = 1125899906842624.0;
    const long long ci = (long long)ceil(fmin(fmax(oi.m, -mcl), mcl)), cj = (long long)ceil(fmin(fmax(oj.m, -mcl), mcl));
    const long long cand[12] = {s, (long long)s - 1, D - 1, (long long)D - 1 + s, (long long)D - 2 + s,
                                ci, ci + s, ci + s - 1, 1, D, cj, cj + 1};
    for (int k = 0; k < 6; ++k) P[k] = 0.0;
    for (int k = 0; k < 4; ++k) C[k] = 0.0;
    for (int a = 0; a < D;) {
        long long nx = D;   // the first cut past a
#pragma unroll
        for (int k = 0; k < 12; ++k) nx = cand[k] > a && cand[k] < nx ? cand[k] : nx;
        const int b = (int)nx - 1;
        const int n = b - a + 1;
        // each op's values at the five shifts, once (ten exponentials per run)
        const LV vi = lval(oi, 0, a, b, D), vis = lval(oi, -s, a, b, D), vis1 = lval(oi, 1 - s, a, b, D);
        const LV vj = lval(oj, 0, a, b, D), vjm = lval(oj, -1, a, b, D);
        const LF Fi = factor(vi, oi.lam, 0), dFi = factor(vi, oi.lam, 2);
        const LF dFis = factor(vis, oi.lam, 2);
        const LF A = fsub(factor(vis1, oi.lam, 0), factor(vis, oi.lam, 0));
        const LF Fj = factor(vj, oj.lam, 0), Rj = factor(vj, oj.lam, 1), dFj = factor(vj, oj.lam, 2);
        const LF dSj = fsub(Fj, factor(vjm, oj.lam, 0));
        bool ui[3] = {false, false, false}, uj[3] = {false, false, false};
        mark(Fi, ui); mark(dFi, ui); mark(dFis, ui); mark(A, ui);
        mark(Fj, uj); mark(Rj, uj); mark(dFj, uj); mark(dSj, uj);
        const RunW t = run_table(oi.lam, oj.lam, n, ui, uj);
        double s0, s1;
        if (b <= D - 2) {   // the interior edges u <= D-2
            prod_sums(A, Fj, t, s0, s1);
            P[0] += s0;
            prod_sums(Fi, Rj, t, s0, s1);
            P[1] += s0;
            prod_sums(A, dFj, t, s0, s1);
            C[0] += s0;
            C[1] += (s1 + ((double)a - oj.m) * s0) / sg_j;
            prod_sums(Fi, dFj, t, s0, s1);
            C[2] -= s0;
            C[3] -= (s1 + ((double)a - oj.m) * s0) / sg_j;
            prod_sums(dFi, Rj, t, s0, s1);
            P[4] += s0;
            P[5] += (s1 + ((double)a - oi.m) * s0) / sg_i;
        }
        // dVdep/dth_i runs to u = D-1, with F_j(D-1) = 1
        prod_sums(dFis, dSj, t, s0, s1);
        P[2] -= s0;
        P[3] -= (s1 + ((double)(a - s) - oi.m) * s0) / sg_i;
        a = b + 1;
    }
    P[0] += 1.0 - cdf_lap(oi, D - 1 - s, D);
}

// Work-group = (block of kLapBS edges, restart), thread per edge: its sums
// in closed form.  Records: the producer-side derivatives in pedge, the
// consumer-side ones in the edge's single cpoly slot (the op kernel leaves
// the forward edges to this kernel); V_dep and L_com of the block per restart
// in gsum_lap.  Work-group x serves restart x mod B (as the op kernel).
__global__ __launch_bounds__(kLapBS) __attribute__((amdgpu_waves_per_eu(2))) void k_lap_edges(Graph G, const float *__restrict__ mu,
                                                      const float *__restrict__ sigma, Work W) {
    const int b = blockIdx.x % G.B, blk = blockIdx.x / G.B, tid = threadIdx.x;
    const int N = G.N, D = G.D;
    const int e = blk * kLapBS + tid;
    double vdep = 0.0, lcom = 0.0;
    if (e < G.E) {
        const int i = G.esrc[e], j = G.col[e];
        const size_t bi = (size_t)b * N + i, bj = (size_t)b * N + j;
        const double sg_i = sigma[bi], sg_j = sigma[bj];
        const LOp oi{(double)mu[bi] - 0.5, 1.4142135623730951 / sg_i};
        const LOp oj{(double)mu[bj] - 0.5, 1.4142135623730951 / sg_j};
        double P[6], C[4];
        laplace_edge(oi, sg_i, G.delay[i], oj, sg_j, D, P, C);
        const size_t be = (size_t)b * G.E + e;
        *reinterpret_cast<float4 *>(W.cpoly + be * kCP) = make_float4((float)C[0], (float)C[1], (float)C[2], (float)C[3]);
        *reinterpret_cast<float4 *>(W.pedge + be * 4) = make_float4((float)P[2], (float)P[3], (float)P[4], (float)P[5]);
        vdep = P[0];
        lcom = P[1];
    }
    // the block's sums: per wave, then the waves in order
    __shared__ double sW[kLapBS / 64][2];
    const int lane = tid & 63, w = tid >> 6;
    for (int o = 32; o >= 1; o >>= 1) {
        vdep += __shfl_xor(vdep, o, 64);
        lcom += __shfl_xor(lcom, o, 64);
    }
    if (lane == 0) { sW[w][0] = vdep; sW[w][1] = lcom; }
    __syncthreads();
    if (tid < 2) {
        double v = 0.0;
        for (int k = 0; k < kLapBS / 64; ++k) v += sW[k][tid];
        W.gsum_lap[((size_t)b * lap_blocks(G) + blk) * 2 + tid] = (float)v;
    }
}

hipError_t launch_lap_edges(const Graph &g, const Work &w, const float *mu, const float *sigma, hipStream_t st) {
    if (g.E == 0) return hipSuccess;
    hipLaunchKernelGGL(k_lap_edges, dim3((unsigned)((size_t)lap_blocks(g) * g.B)), dim3(kLapBS), 0, st, g, mu, sigma, w);
    return hipGetLastError();
}

}  // namespace gaus
