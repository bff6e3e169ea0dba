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
    const double e1 = -expm1(-x), en = -expm1(-xn);   // 1 - e^(-x), 1 - e^(-x n)
    G0 = en / e1;
    if (xn < 0.02) {   // power sums S_p = sum k^p, k < n, and the series of e^(-x k)
        const double nn = n, s1 = 0.5 * nn * (nn - 1.0), s2 = (nn - 1.0) * nn * (2.0 * nn - 1.0) / 6.0;
        const double s3 = s1 * s1, s4 = (nn - 1.0) * nn * (2.0 * nn - 1.0) * (3.0 * nn * nn - 3.0 * nn - 1.0) / 30.0;
        const double s5 = s1 * s1 * (2.0 * nn * nn - 2.0 * nn - 1.0) / 3.0;
        G1 = s1 - x * s2 + x * x * s3 / 2.0 - x * x * x * s4 / 6.0 + x * x * x * x * s5 / 24.0;
    } else {
        // sum k q^k = q (1 - q^(n-1) (1 + (n-1)(1-q))) / (1-q)^2, q = e^(-x)
        const double q = 1.0 - e1, qn1 = (1.0 - en) / q;
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
__device__ __forceinline__ GW run_weights(double g, int n) {
    GW r;
    if (n == 1) { r.w0 = 1.0; r.w1 = 0.0; r.atB = false; return r; }
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
__device__ __forceinline__ RunW run_table(double li, double lj, int n) {
    RunW t;
    const double gi[3] = {0.0, li, -li}, gj[3] = {0.0, lj, -lj};
#pragma unroll
    for (int x = 0; x < 3; ++x)
#pragma unroll
        for (int y = 0; y < 3; ++y) t.w[x][y] = run_weights(gi[x] + gj[y], n);
    return t;
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

// The op's CDF at the bin edges u + off, u in [a, b] (one case throughout):
// kind 0: F, 1: 1 - F, 2: dF/dmu.
struct LOp {
    double m, lam;
};
__device__ __forceinline__ LF factor(const LOp &o, int kind, int off, int a, int b, int D) {
    LF f{0.0, 0.0, 0.0, 0.0, 0.0};
    const int va = a + off, vb = b + off;
    const bool zero = va < 0, one = va >= D - 1;
    if (zero || one) {
        f.c = ((kind == 0 && one) || (kind == 1 && zero)) ? 1.0 : 0.0;
        return f;
    }
    const bool up = (double)va >= o.m;
    const double sg = up ? -1.0 : 1.0;   // e^(+lam (v-m)) below the median, e^(-lam (v-m)) above
    const double ea = 0.5 * exp(sg * o.lam * ((double)va - o.m)), eb = 0.5 * exp(sg * o.lam * ((double)vb - o.m));
    // F: e/2 below, 1 - e/2 above; 1 - F: the complement; dF/dmu = -lam e/2
    const double w = kind == 2 ? -o.lam : (kind == 0) == up ? -1.0 : 1.0;
    f.c = kind == 2 ? 0.0 : (kind == 0) == up ? 1.0 : 0.0;
    if (up) { f.upA = w * ea; f.upB = w * eb; }
    else { f.loA = w * ea; f.loB = w * eb; }
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
    const long long ci = (long long)ceil(oi.m), cj = (long long)ceil(oj.m);
    long long cand[15] = {s, (long long)s - 1, D - 1, (long long)D - 1 + s, (long long)D - 2 + s,
                          ci, ci + s, ci + s - 1, 1, D, cj, cj + 1, 0, 0, 0};
    for (int k = 0; k < 6; ++k) P[k] = 0.0;
    for (int k = 0; k < 4; ++k) C[k] = 0.0;
    for (int a = 0; a < D;) {
        long long nx = D;   // the first cut past a
#pragma unroll
        for (int k = 0; k < 12; ++k) nx = cand[k] > a && cand[k] < nx ? cand[k] : nx;
        const int b = (int)nx - 1;
        const int n = b - a + 1;
        const RunW t = run_table(oi.lam, oj.lam, n);
        const LF Fi = factor(oi, 0, 0, a, b, D), dFi = factor(oi, 2, 0, a, b, D);
        const LF dFis = factor(oi, 2, -s, a, b, D);
        const LF A = fsub(factor(oi, 0, 1 - s, a, b, D), factor(oi, 0, -s, a, b, D));
        const LF Fj = factor(oj, 0, 0, a, b, D), Rj = factor(oj, 1, 0, a, b, D), dFj = factor(oj, 2, 0, a, b, D);
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
        const LF dSj = fsub(Fj, factor(oj, 0, -1, a, b, D));
        prod_sums(dFis, dSj, t, s0, s1);
        P[2] -= s0;
        P[3] -= (s1 + ((double)(a - s) - oi.m) * s0) / sg_i;
        a = b + 1;
    }
    P[0] += 1.0 - cdf_lap(oi, D - 1 - s, D);
}

// Work-group = (op group, restart), thread per op: the op's out-edges in
// closed form.  Records: the op's producer sums in its single ppoly slot,
// each edge's consumer sums in its single cpoly slot (the op kernel leaves
// the edges to this kernel and writes zero producer records per tile); V_dep
// and L_com of the group per restart in gsum_lap.
constexpr int kLapBS = 256;
__global__ __launch_bounds__(kLapBS) void k_lap_edges(Graph G, const float *__restrict__ mu,
                                                      const float *__restrict__ sigma, Work W) {
    const int b = blockIdx.x % G.B, grp = blockIdx.x / G.B, tid = threadIdx.x;
    const int N = G.N, D = G.D;
    const int q0 = G.grp_start[grp], nq = G.grp_start[grp + 1] - q0;
    double vdep = 0.0, lcom = 0.0;
    if (tid < nq) {
        const int i = G.perm[q0 + tid];
        const size_t bi = (size_t)b * N + i;
        const double sg_i = sigma[bi];
        const LOp oi{(double)mu[bi] - 0.5, 1.4142135623730951 / sg_i};
        const int s = G.delay[i];
        double P[6] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
        for (int e = G.row_ptr[i]; e < G.row_ptr[i + 1]; ++e) {
            const int j = G.col[e];
            const size_t bj = (size_t)b * N + j;
            const double sg_j = sigma[bj];
            const LOp oj{(double)mu[bj] - 0.5, 1.4142135623730951 / sg_j};
            double Pe[6], Ce[4];
            laplace_edge(oi, sg_i, s, oj, sg_j, D, Pe, Ce);
            for (int k = 0; k < 6; ++k) P[k] += Pe[k];
            float4 c4;
            c4.x = (float)Ce[0]; c4.y = (float)Ce[1]; c4.z = (float)Ce[2]; c4.w = (float)Ce[3];
            *reinterpret_cast<float4 *>(W.cpoly + ((size_t)b * G.E + e) * kCP) = c4;
        }
        float *pp = W.ppoly + bi * kPP;
        for (int k = 0; k < kPP; ++k) pp[k] = (float)P[k];
        vdep = P[0];
        lcom = P[1];
    }
    // the group's sums: per wave, then the waves in order
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
        W.gsum_lap[((size_t)b * G.ngroups + grp) * 2 + tid] = (float)v;
    }
}

hipError_t launch_lap_edges(const Graph &g, const Work &w, const float *mu, const float *sigma, hipStream_t st) {
    hipLaunchKernelGGL(k_lap_edges, dim3((unsigned)((size_t)g.ngroups * g.B)), dim3(kLapBS), 0, st, g, mu, sigma, w);
    return hipGetLastError();
}

}  // namespace gaus
