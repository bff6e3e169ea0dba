// gfx950 kernels of the GauS hot path: masses, folded usage, resource /
// dependency / recurrence penalties, expected edge length, their analytic
// gradient, Adam, and Alg. 3/4 legalization.
//
// Notation (arXiv 2602.20427): op i has start step d_i ~ round(N(mu_i, sigma_i^2)).
// F_i(t) = P(d_i <= t) at the interior bin edges t = 0..D-2 (eq:round with the
// open end bins: F_i(t) = 0 for t < 0 and 1 for t >= D-1), P_i^d = F_i(d) - F_i(d-1).
// Every term of the objective is a sum over steps of products of F's and P's
// of the two end points of an edge, so all kernels iterate over a step index u
// and evaluate F, dF/dmu, dF/dsigma from (mu, sigma) on the fly: nothing of size
// B*N*D is ever stored.
//
// Reductions use fixed trees and per-(tile, group) partial buffers, never
// floating-point atomics, so results are bitwise reproducible.
#include "gaus_internal.h"
#include "gaus_erfcx_coeffs.h"

#include <algorithm>

namespace gaus {

namespace {

constexpr float kInvSqrt2 = 0.70710678118654752f;
constexpr float kInvSqrt2Pi = 0.39894228040143268f;
constexpr float kHalfLog2e = 0.72134752044448170f;  // log2(e)/2

// Tail of the standard normal and the Gaussian factor: tail = Phi(-|z|),
// g = exp(-z^2/2).  Phi(-|z|) = erfc(x)/2 with x = |z|/sqrt(2) and
// erfc(x) = exp(-x^2) * t * Q(t), t = 1/(1 + p x), Q a fitted polynomial
// (gaus_erfcx_coeffs.h).  exp(-x^2) equals g, which the gradient needs, so
// both come from one exp.
__device__ __forceinline__ void normal_tail_pdf(float z, float &tail, float &g) {
    const float x = fabsf(z) * kInvSqrt2;
    g = __builtin_amdgcn_exp2f(-(z * z) * kHalfLog2e);
    const float t = __builtin_amdgcn_rcpf(fmaf(GAUS_ERFCX_P, x, 1.0f));
    float q = gaus_erfcx_q[GAUS_ERFCX_DEG];
#pragma unroll
    for (int k = GAUS_ERFCX_DEG - 1; k >= 0; --k) q = fmaf(q, t, gaus_erfcx_q[k]);
    tail = 0.5f * g * (t * q);
}

// A CDF value F is kept as a signed tail: +Phi(-|z|) below the median
// (F = tail) and -Phi(-|z|) at or above it (F = 1 - tail; -0.0 for F = 1).
// Differences of neighbouring CDF values (the masses P_i^d) are then formed
// from tails, without the cancellation of 1 - F near F = 1.
__device__ __forceinline__ bool st_upper(float st) { return __builtin_signbit(st); }
__device__ __forceinline__ float st_F(float st) { return st_upper(st) ? 1.0f + st : st; }
__device__ __forceinline__ float st_1mF(float st) { return st_upper(st) ? -st : 1.0f - st; }
// F(hi) - F(lo) for bin edges lo < hi
__device__ __forceinline__ float st_mass(float lo, float hi) {
    const bool ul = st_upper(lo), uh = st_upper(hi);
    if (ul) return hi - lo;                  // both above: tail(lo) - tail(hi)
    if (!uh) return hi - lo;                 // both below: tail(hi) - tail(lo)
    return (1.0f + hi) - lo;                 // straddles the median
}

// Signed-tail CDF and its derivatives at bin edge v of an op (mu, rs = 1/sigma,
// cinv = 1/(sigma sqrt(2 pi))): dF/dmu = -phi(z)/sigma, dF/dsigma = -phi(z) z/sigma.
// Outside the interior edges F is the constant 0 (v < 0) or 1 (v >= D-1).
__device__ __forceinline__ void cdf_at(long long v, int D, float mu, float rs, float cinv, float &st,
                                       float &Fm, float &Fs) {
    if (v < 0) { st = 0.0f; Fm = 0.0f; Fs = 0.0f; return; }
    if (v >= D - 1) { st = -0.0f; Fm = 0.0f; Fs = 0.0f; return; }
    const float z = ((float)v + 0.5f - mu) * rs;
    float tail, g;
    normal_tail_pdf(z, tail, g);
    st = (z >= 0.0f) ? -tail : tail;
    Fm = -g * cinv;
    Fs = Fm * z;
}

__device__ __forceinline__ float st_at(long long v, int D, float mu, float rs) {
    if (v < 0) return 0.0f;
    if (v >= D - 1) return -0.0f;
    const float z = ((float)v + 0.5f - mu) * rs;
    float tail, g;
    normal_tail_pdf(z, tail, g);
    return (z >= 0.0f) ? -tail : tail;
}

// Wave-wide sums with DPP lane moves (fused into the adds) inside rows of 16
// lanes and the gfx950 lane-swap instructions across rows.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;
constexpr int kDppRor4 = 0x124;
constexpr int kDppRor8 = 0x128;

// sum over lanes l, l^16, l^32, l^48 (LDS swizzle inside halves, LDS
// permute across them); each pair is added in both lanes in the same order
__device__ __forceinline__ float cross_rows_sum(float x) {
    constexpr int kSwizzleXor16 = 0x1F | (0x10 << 10);   // bit mode: and 31, xor 16
    x += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), kSwizzleXor16));
    const int lane = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
    x += __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, __builtin_bit_cast(int, x)));
    return x;
}

// Sum over the 64 lanes; every lane receives the same total.
__device__ __forceinline__ float wave_sum(float x) {
    x += dpp_mov<kDppXor1>(x);
    x += dpp_mov<kDppXor2>(x);
    x += dpp_mov<kDppHalfMirror>(x);
    x += dpp_mov<kDppMirror>(x);
    return cross_rows_sum(x);
}

// Four sums at once: lane l < 4 receives the total of value wave4_comp(l).
__device__ __forceinline__ int wave4_comp(int lane) { return 2 * (lane & 1) + ((lane >> 1) & 1); }

__device__ __forceinline__ float wave_sum4(float v0, float v1, float v2, float v3, int lane) {
    const bool b0 = lane & 1, b1 = lane & 2;
    const float a = (b0 ? v2 : v0) + dpp_mov<kDppXor1>(b0 ? v0 : v2);   // value 2*b0
    const float c = (b0 ? v3 : v1) + dpp_mov<kDppXor1>(b0 ? v1 : v3);   // value 2*b0+1
    float x = (b1 ? c : a) + dpp_mov<kDppXor2>(b1 ? a : c);             // value 2*b0+b1
    x += dpp_mov<kDppRor4>(x);
    x += dpp_mov<kDppRor8>(x);
    return cross_rows_sum(x);
}

// Maximum over the 64 lanes; every lane receives it.
__device__ __forceinline__ float wave_max(float x) {
    x = fmaxf(x, dpp_mov<kDppXor1>(x));
    x = fmaxf(x, dpp_mov<kDppXor2>(x));
    x = fmaxf(x, dpp_mov<kDppHalfMirror>(x));
    x = fmaxf(x, dpp_mov<kDppMirror>(x));
    constexpr int kSwizzleXor16 = 0x1F | (0x10 << 10);
    x = fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), kSwizzleXor16)));
    const int lane = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
    return fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, __builtin_bit_cast(int, x))));
}

// Two sums at once: lane l < 2 receives the total of value l.
__device__ __forceinline__ float wave_sum2(float v0, float v1, int lane) {
    const bool b0 = lane & 1;
    float x = (b0 ? v1 : v0) + dpp_mov<kDppXor1>(b0 ? v0 : v1);
    x += dpp_mov<kDppXor2>(x);
    x += dpp_mov<kDppRor4>(x);
    x += dpp_mov<kDppRor8>(x);
    return cross_rows_sum(x);
}

// Sum NV values over the work-group; thread c < NV receives total c.
// slot: LDS scratch [NW][8]; callers alternate between two slots so that only
// one barrier per reduction is needed.
template <int NV, int BS>
__device__ __forceinline__ float block_sum(float (&v)[NV], float (*slot)[8]) {
    constexpr int NW = BS / 64;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
    for (int c = 0; c < NV; ++c) v[c] = wave_sum(v[c]);
    if (lane == 0) {
#pragma unroll
        for (int c = 0; c < NV; ++c) slot[wid][c] = v[c];
    }
    __syncthreads();
    float r = 0.0f;
    if (threadIdx.x < NV) {
#pragma unroll
        for (int w = 0; w < NW; ++w) r += slot[w][threadIdx.x];
    }
    return r;
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

}  // namespace

// ---------------------------------------------------------------------------
// Op kernel.  Work-group = (op group, step tile, restart).  Threads own steps
// u = t0 + k*BS + tid (k < SPT).  For each op i of the group (all of one
// resource type, out-degree m, delay s = Lat(v_i)):
//   * its CDF row over the tile plus a left halo of s steps goes to LDS; the
//     mass P_i^u is added to the group's usage;
//   * for each out-edge (i -> j) the consumer's CDF and Gaussian factor are
//     evaluated once per step.  The consumer-side derivatives of this edge are
//       dVdep/dth_j = sum_u A(u) F_j'(u),   A(u) = P_i^{u-s+1}
//       dLcom/dth_j = -sum_u F_i(u) F_j'(u)
//     and the successor CDF sum S_i(u) = sum_j F_j(u) is accumulated split
//     into lower-side CDFs, upper tails and a count of successors past their
//     median, so that S_i, m - S_i and S_i(u) - S_i(u-1) keep full precision;
//   * after the out-edges the producer-side terms follow from S_i:
//       V_dep          = sum_u A(u) S_i(u) + m (1 - F_i(D-1-s))
//       L_com          = sum_u F_i(u) (m - S_i(u))
//       dVdep/dth_i    = -sum_u F_i'(u-s) (S_i(u) - S_i(u-1))
//       dLcom/dth_i    = sum_u F_i'(u) (m - S_i(u))
//     (u over the interior edges 0..D-2 except in dVdep/dth_i, which runs to
//     u = D-1 with S_i(D-1) = m: the consumers' bin D-1 is open to +inf).
// ---------------------------------------------------------------------------
template <int BS, int SPT>
__global__ __launch_bounds__(BS) void k_ops(Graph G, const float *__restrict__ mu,
                                            const float *__restrict__ sigma, Work W) {
    constexpr int TILE = BS * SPT;
    constexpr int WIN = TILE + kHalo + 1;
    __shared__ float sT[WIN], sFm[WIN], sFs[WIN];
    __shared__ float sRed[2][BS / 64][8];
    __shared__ float sPrev[3];

    const int grp = blockIdx.x, tile = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x;
    const int D = G.D, N = G.N;
    const int t0 = tile * TILE;
    const float *mub = mu + (size_t)b * N;
    const float *sgb = sigma + (size_t)b * N;

    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    float accU[SPT];
#pragma unroll
    for (int k = 0; k < SPT; ++k) accU[k] = 0.0f;
    int par = 0;

    // Groups without step-by-step work leave nothing here: their readers skip
    // them (group and op flags).  Otherwise thread t looks at op q0+t (groups
    // hold at most as many ops as the work-group has threads); ops and edges
    // on the chunk-polynomial path are left to k_poly.
    if (!W.gflag[(size_t)b * G.ngroups + grp]) return;
    __shared__ int sDirect[BS];   // 0: nothing; else 1 + number of step-by-step out-edges
    const unsigned char *clsb = W.cls + (size_t)b * N;
    {
        int flag = 0;
        if (q0 + tid < q1) {
            const int i = G.perm[q0 + tid];
            if (W.dflag[(size_t)b * N + i]) {
                const int e0 = G.row_ptr[i], e1 = G.row_ptr[i + 1];
                const bool poly_i = clsb[i] != 0;
                int m = 0;
                for (int e = e0; e < e1; ++e) m += (poly_i && clsb[G.col[e]]) ? 0 : 1;
                flag = 1 + m;
            }
        }
        sDirect[tid] = flag;
    }
    float gsum0 = 0.0f, gsum1 = 0.0f;  // V_dep, L_com of the work-group (threads 0, 1)
    __syncthreads();

    for (int q = q0; q < q1; ++q) {
        const int flag = sDirect[q - q0];
        if (flag == 0) continue;
        const int i = uniform(G.perm[q]);
        const int e0 = uniform(G.row_ptr[i]), e1 = uniform(G.row_ptr[i + 1]);
        const bool poly_i = clsb[i] != 0;
        const int m = uniform(flag - 1);
        const float m_i = mub[i], s_i = sgb[i];
        const float rs = 1.0f / s_i;
        const float cinv = rs * kInvSqrt2Pi;
        const int s = uniform(G.delay[i]);
        const bool win_shift = (m > 0) && (s <= kHalo);
        const int Lh = win_shift ? (s > 1 ? s : 1) : 1;

        // row window: positions v = t0 - Lh + p, p in [0, TILE + Lh]
        for (int p = tid; p < TILE + Lh + 1; p += BS) {
            float st, Fm, Fs;
            cdf_at(t0 - Lh + p, D, m_i, rs, cinv, st, Fm, Fs);
            sT[p] = st; sFm[p] = Fm; sFs[p] = Fs;
        }
        __syncthreads();

        float rF[SPT], rFm[SPT], rFs[SPT], rA[SPT], rFms[SPT], rFss[SPT];
        float tail1mF = 0.0f;  // 1 - F_i(D-1-s), held by the thread owning u = D-1
#pragma unroll
        for (int k = 0; k < SPT; ++k) {
            const int u = t0 + k * BS + tid;
            const int p = u - t0 + Lh;
            rF[k] = st_F(sT[p]); rFm[k] = sFm[p]; rFs[k] = sFs[p];
            if (u < D && !poly_i) accU[k] += st_mass(sT[p - 1], sT[p]);
            rA[k] = 0.0f; rFms[k] = 0.0f; rFss[k] = 0.0f;
            if (m > 0 && u < D) {
                if (win_shift) {
                    rA[k] = st_mass(sT[p - s], sT[p - s + 1]);
                    rFms[k] = sFm[p - s]; rFss[k] = sFs[p - s];
                    if (u == D - 1) tail1mF = st_1mF(sT[p - s]);
                } else {
                    float st0, Fm0, Fs0, st1, Fm1, Fs1;
                    cdf_at((long long)u - s, D, m_i, rs, cinv, st0, Fm0, Fs0);
                    cdf_at((long long)u - s + 1, D, m_i, rs, cinv, st1, Fm1, Fs1);
                    rA[k] = st_mass(st0, st1); rFms[k] = Fm0; rFss[k] = Fs0;
                    if (u == D - 1) tail1mF = st_1mF(st0);
                }
            }
        }
        __syncthreads();  // the window may be overwritten from here on

        float SL[SPT], SU[SPT], SC[SPT];
#pragma unroll
        for (int k = 0; k < SPT; ++k) { SL[k] = 0.0f; SU[k] = 0.0f; SC[k] = 0.0f; }
        float pL = 0.0f, pU = 0.0f, pC = 0.0f;   // S_i(t0-1), thread 0 only

        for (int e = e0; e < e1; ++e) {
            const int j = uniform(G.col[e]);
            if (poly_i && clsb[j]) continue;  // polynomial edge
            const float m_j = mub[j], s_j = sgb[j];
            const float rsj = 1.0f / s_j;
            float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int k = 0; k < SPT; ++k) {
                const int u = t0 + k * BS + tid;
                if (u < D - 1) {
                    const float z = ((float)u + 0.5f - m_j) * rsj;
                    float tl, gj;
                    normal_tail_pdf(z, tl, gj);
                    const bool up = z >= 0.0f;
                    SL[k] += up ? 0.0f : tl;
                    SU[k] += up ? tl : 0.0f;
                    SC[k] += up ? 1.0f : 0.0f;
                    const float gz = gj * z;
                    acc[0] = fmaf(rA[k], gj, acc[0]);
                    acc[1] = fmaf(rA[k], gz, acc[1]);
                    acc[2] = fmaf(rF[k], gj, acc[2]);
                    acc[3] = fmaf(rF[k], gz, acc[3]);
                }
            }
            if (tid == 0 && t0 > 0) {
                const float z = ((float)(t0 - 1) + 0.5f - m_j) * rsj;
                float tl, gj;
                normal_tail_pdf(z, tl, gj);
                if (z >= 0.0f) { pU += tl; pC += 1.0f; } else { pL += tl; }
            }
            const float r = block_sum<4, BS>(acc, sRed[par]);
            par ^= 1;
            if (tid < 4) {
                // F_j'(u) = -g_j/(sigma_j sqrt(2 pi)) [* z for sigma]; L_com enters with a minus
                const float cj = rsj * kInvSqrt2Pi;
                const float val = (tid < 2) ? -cj * r : cj * r;
                W.cpart[(((size_t)b * G.E + e) * G.ntiles + tile) * kCP + tid] = val;
            }
        }

        float pr[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
        if (m > 0) {
            const float mf = (float)m;
            // S_i(D-1) = m: every consumer is at or before step D-1
#pragma unroll
            for (int k = 0; k < SPT; ++k) {
                const int u = t0 + k * BS + tid;
                if (u == D - 1) { SL[k] = 0.0f; SU[k] = 0.0f; SC[k] = mf; }
                if (u < D) { sT[u - t0] = SL[k]; sFm[u - t0] = SU[k]; sFs[u - t0] = SC[k]; }
            }
            if (tid == 0) { sPrev[0] = pL; sPrev[1] = pU; sPrev[2] = pC; }
            __syncthreads();
#pragma unroll
            for (int k = 0; k < SPT; ++k) {
                const int u = t0 + k * BS + tid;
                if (u >= D) continue;
                const int ix = u - t0;
                const float L1 = ix ? sT[ix - 1] : sPrev[0];
                const float U1 = ix ? sFm[ix - 1] : sPrev[1];
                const float C1 = ix ? sFs[ix - 1] : sPrev[2];
                const float dS = ((SL[k] - L1) + (SC[k] - C1)) - (SU[k] - U1);
                pr[2] = fmaf(-rFms[k], dS, pr[2]);
                pr[3] = fmaf(-rFss[k], dS, pr[3]);
                if (u < D - 1) {
                    const float S = (SL[k] + SC[k]) - SU[k];
                    const float rest = ((mf - SC[k]) - SL[k]) + SU[k];
                    pr[0] = fmaf(rA[k], S, pr[0]);
                    pr[1] = fmaf(rF[k], rest, pr[1]);
                    pr[4] = fmaf(rFm[k], rest, pr[4]);
                    pr[5] = fmaf(rFs[k], rest, pr[5]);
                } else {
                    pr[0] = fmaf(mf, tail1mF, pr[0]);
                }
            }
            const float r = block_sum<6, BS>(pr, sRed[par]);
            par ^= 1;
            if (tid < kPP) W.ppart[(((size_t)b * N + i) * G.ntiles + tile) * kPP + tid] = r;
            if (tid == 0) gsum0 += r;
            if (tid == 1) gsum1 += r;
        } else if (tid < kPP) {
            W.ppart[(((size_t)b * N + i) * G.ntiles + tile) * kPP + tid] = 0.0f;
        }
    }
    {
        float *gs = W.gsum_ops + (((size_t)b * G.ngroups + grp) * G.ntiles + tile) * 2;
        if (tid == 0) gs[0] = gsum0;
        if (tid == 1) gs[1] = gsum1;
    }

    float *up = W.Upart + ((size_t)b * G.ngroups + grp) * D;
#pragma unroll
    for (int k = 0; k < SPT; ++k) {
        const int u = t0 + k * BS + tid;
        if (u < D) up[u] = accU[k];
    }
}

// ---------------------------------------------------------------------------
// Chunk-polynomial path (dense regime).
//
// Chunks of W steps tile [L0, D-2); a chunk's points are y = u - t_mid in
// [-lam, lam], lam = (W-1)/2.  Around the chunk centre an op's CDF is
// F(u) = Phi(z0 + r y), r = 1/sigma, and its Taylor coefficients in y are
// T_n = Phi^(n)(z0) r^n / n!, which obey
//   T_1 = phi(z0) r,
//   T_{n+1} = -(z0 r/(n+1)) T_n - ((n-1) r^2/(n(n+1))) T_{n-1}
// (the Hermite recursion of the derivatives of phi, scaled).  From one set of
// T's follow, with constant integer coefficients (one step = 1 in y):
//   F:         f_k = T_k
//   dF/dmu:    a_k = -(k+1) T_{k+1}
//   dF/dsigma: e_k = z0 a_k + r a_{k-1}           (dF/dsigma = z dF/dmu)
//   mass F(v) - F(v-1):  m_k = -sum_{j>=1} C(k+j,j) (-1)^j T_{k+j}
//   dF/dmu at v-1:       a1_k = -sum_{j>=0} (k+j+1) C(k+j,j) (-1)^j T_{k+1+j}
// The series converge like powers of rho = lam r; with rho <= kRhoMax the
// truncation error is ~1e-10.  Every sum over the chunk's steps of a product
// p(u) q(u) equals sum_k (H p)_k q_k with the chunk moments H_n = sum_y y^n,
// so an edge costs 10 dot products of length kNC.
// The strip [0, L0) u {D-2, D-1} (boundary conventions of the open end bins,
// zero derivatives outside the interior edges) is evaluated step by step.
// ---------------------------------------------------------------------------
__global__ void k_classify(Graph G, PolyArgs pa, const float *__restrict__ sigma, Work W) {
    const int b = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < G.ngroups) W.gflag[(size_t)b * G.ngroups + i] = 0;
    if (i >= G.N) return;
    const float s = sigma[(size_t)b * G.N + i];
    W.cls[(size_t)b * G.N + i] = (pa.enabled && s >= pa.sig_thr && G.delay[i] <= kSmax) ? 1 : 0;
}

// Which ops (and groups) have step-by-step work this iteration: ops off the
// polynomial path, and polynomial ops with an out-edge to such an op.
__global__ void k_flags(Graph G, Work W) {
    const int b = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= G.N) return;
    const unsigned char *clsb = W.cls + (size_t)b * G.N;
    int d = clsb[i] ? 0 : 1;
    for (int e = G.row_ptr[i]; e < G.row_ptr[i + 1] && !d; ++e) d = clsb[G.col[e]] ? 0 : 1;
    W.dflag[(size_t)b * G.N + i] = (unsigned char)d;
    if (d) atomicOr(&W.gflag[(size_t)b * G.ngroups + G.grp_of[i]], 1);
}

namespace {

struct Expansion {
    float T[kTN];   // Taylor coefficients in y, T[0] = F(z0)
    float G0;       // 1 - F(z0), from the tail
    float z0, r;
};

constexpr double binom_d(int n, int k) {
    double v = 1.0;
    for (int q = 1; q <= k; ++q) v = v * (double)(n - k + q) / (double)q;
    return v;
}
// coefficient of T_{k+j} in the mass coefficient m_k (j >= 1)
constexpr float mass_coef(int k, int j) { return (float)(-binom_d(k + j, j) * ((j & 1) ? -1.0 : 1.0)); }
// coefficient of T_{k+1+j} in dF/dmu one step back, a1_k (j >= 0)
constexpr float back_coef(int k, int j) {
    return (float)(-(double)(k + j + 1) * binom_d(k + j, j) * ((j & 1) ? -1.0 : 1.0));
}

__device__ __forceinline__ void expand(float mu, float rs, float tcen, Expansion &e) {
    e.r = rs;
    e.z0 = (tcen + 0.5f - mu) * rs;
    float tail, g;
    normal_tail_pdf(e.z0, tail, g);
    const bool up = e.z0 >= 0.0f;
    e.T[0] = up ? 1.0f - tail : tail;
    e.G0 = up ? tail : 1.0f - tail;
    e.T[1] = g * (kInvSqrt2Pi * rs);
    const float zr = e.z0 * rs, r2 = rs * rs;
    e.T[2] = (zr * -0.5f) * e.T[1];
#pragma unroll
    for (int n = 2; n < kTN - 1; ++n) {
        const float c1 = -1.0f / (float)(n + 1);
        const float c2 = -(float)(n - 1) / (float)(n * (n + 1));
        e.T[n + 1] = fmaf(zr * c1, e.T[n], (r2 * c2) * e.T[n - 1]);
    }
}

__device__ __forceinline__ void vec_dFdmu(const Expansion &e, float (&a)[kNC]) {
#pragma unroll
    for (int k = 0; k < kNC; ++k) a[k] = -(float)(k + 1) * e.T[k + 1];
}

__device__ __forceinline__ void vec_times_z(const float (&a)[kNC], float zc, float r, float (&o)[kNC]) {
    o[0] = zc * a[0];
#pragma unroll
    for (int k = 1; k < kNC; ++k) o[k] = fmaf(zc, a[k], r * a[k - 1]);
}

__device__ __forceinline__ void vec_mass(const Expansion &e, float (&m)[kNC]) {
#pragma unroll
    for (int k = 0; k < kNC; ++k) {
        float acc = 0.0f;
#pragma unroll
        for (int j = kShiftTerms; j >= 1; --j) acc = fmaf(mass_coef(k, j), e.T[k + j], acc);
        m[k] = acc;
    }
}

__device__ __forceinline__ void vec_dFdmu_back(const Expansion &e, float (&a)[kNC]) {
#pragma unroll
    for (int k = 0; k < kNC; ++k) {
        float acc = 0.0f;
#pragma unroll
        for (int j = kShiftTerms; j >= 0; --j) acc = fmaf(back_coef(k, j), e.T[k + 1 + j], acc);
        a[k] = acc;
    }
}

// (H p)_k = sum_l H_{k+l} p_l; the chunk points are symmetric, odd moments vanish
__device__ __forceinline__ void vec_moments(const float (&p)[kNC], const PolyArgs &pa, float (&o)[kNC]) {
#pragma unroll
    for (int k = 0; k < kNC; ++k) {
        float acc = 0.0f;
#pragma unroll
        for (int l = 0; l < kNC; ++l)
            if (((k + l) & 1) == 0) acc = fmaf(pa.H[(k + l) / 2], p[l], acc);
        o[k] = acc;
    }
}

__device__ __forceinline__ float vdot(const float (&a)[kNC], const float (&b)[kNC]) {
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < kNC; ++k) acc = fmaf(a[k], b[k], acc);
    return acc;
}

// dot with 1 - F given F's coefficients and the precise 1 - F(z0)
__device__ __forceinline__ float vdot_1mF(const float (&a)[kNC], const Expansion &e) {
    float acc = a[0] * e.G0;
#pragma unroll
    for (int k = 1; k < kNC; ++k) acc = fmaf(-a[k], e.T[k], acc);
    return acc;
}

__device__ __forceinline__ float vdot_F(const float (&a)[kNC], const Expansion &e) {
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < kNC; ++k) acc = fmaf(a[k], e.T[k], acc);
    return acc;
}

}  // namespace

constexpr int kPolyWaves = 4;
constexpr int kStripPassesMax = (kStripMax + 63) / 64;
constexpr int kOpsPerWaveMax = 64;              // group size <= kPolyWaves * 64

// Work-group = (op group, restart), kPolyWaves waves; each wave takes the
// group's ops in turn.  For a polynomial op: lanes = strip positions for the
// step-by-step part, lanes = chunks for the polynomial part; per polynomial
// out-edge the consumer-side derivatives of both parts are reduced together.
// NP: strip passes of 64 lanes, ceil(SP / 64).
template <int NP>
__global__ __launch_bounds__(64 * kPolyWaves) __attribute__((amdgpu_waves_per_eu(3)))
void k_poly(Graph G, PolyArgs pa, const float *__restrict__ mu, const float *__restrict__ sigma, Work W) {
    // dynamic LDS: per wave 7 rows of SP strip values, then per wave SP strip usages
    extern __shared__ float sDyn[];
    __shared__ float sUc[kPolyWaves][kMaxChunks][kNC];
    __shared__ float sGs[kPolyWaves][2];
    const int SP = pa.SP, split = pa.split;
    const int grp = blockIdx.x / split, sub = blockIdx.x - grp * split, b = blockIdx.y;
    const size_t slot_id = ((size_t)b * G.ngroups + grp) * split + sub;   // per-work-group outputs
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int N = G.N, D = G.D;
    const float *mub = mu + (size_t)b * N;
    const float *sgb = sigma + (size_t)b * N;
    const unsigned char *clsb = W.cls + (size_t)b * N;
    const bool cact = lane < pa.nc;
    const float tcen = (float)(pa.L0 + lane * pa.W) + pa.lam;

    float uc[kNC];
#pragma unroll
    for (int k = 0; k < kNC; ++k) uc[k] = 0.0f;
    float us[NP];
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) us[ps] = 0.0f;
    float *own = sDyn + (size_t)wv * 7 * SP;
    float *sUs = sDyn + (size_t)kPolyWaves * 7 * SP;

    // the work-group's ops are q = q0 + sub + split*j; this wave's are
    // j = wv + kPolyWaves*l, parameters loaded by lane l
    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    const int nj = (q1 - q0 - sub + split - 1) / split;
    const int nq = (nj - wv + kPolyWaves - 1) / kPolyWaves;
    int l_i = 0, l_cls = 0, l_s = 0, l_e0 = 0, l_e1 = 0;
    float l_mu = 0.0f, l_sg = 1.0f;
    if (lane < nq) {
        l_i = G.perm[q0 + sub + split * (wv + kPolyWaves * lane)];
        l_cls = clsb[l_i];
        l_mu = mub[l_i]; l_sg = sgb[l_i];
        l_s = G.delay[l_i];
        l_e0 = G.row_ptr[l_i]; l_e1 = G.row_ptr[l_i + 1];
    }
    float gsum = 0.0f;  // V_dep, L_com of this wave's ops (lanes 0 and 2)
    for (int oq = 0; oq < nq; ++oq) {
        const int i = __builtin_amdgcn_readlane(l_i, oq);
        float *pp = W.ppoly + ((size_t)b * N + i) * kPP;
        if (!__builtin_amdgcn_readlane(l_cls, oq)) {
            if (lane < kPP) pp[lane] = 0.0f;
            continue;
        }
        const float m_i = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, l_mu), oq));
        const float s_i = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, l_sg), oq));
        const float rs = 1.0f / s_i, cinv = rs * kInvSqrt2Pi;
        const int s = __builtin_amdgcn_readlane(l_s, oq);
        const int e0 = __builtin_amdgcn_readlane(l_e0, oq), e1 = __builtin_amdgcn_readlane(l_e1, oq);
        float pr[kPP] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
        // the op's polynomial out-edges, loaded by lane (batches of 64)
        int x_j = 0, x_ok = 0;
        float x_mu = 0.0f, x_sg = 1.0f;

        // (1) strip: own CDF values per position, kept in this wave's LDS rows
#pragma unroll
        for (int ps = 0; ps < NP; ++ps) {
            const int p = ps * 64 + lane;
            if (p < SP) {
                const int u = p < pa.L0 ? p : D - 2 + (p - pa.L0);
                float st, Fm, Fs, st0, Fm0, Fs0;
                cdf_at(u, D, m_i, rs, cinv, st, Fm, Fs);
                us[ps] += st_mass(st_at((long long)u - 1, D, m_i, rs), st);
                cdf_at((long long)u - s, D, m_i, rs, cinv, st0, Fm0, Fs0);
                const float st1 = st_at((long long)u - s + 1, D, m_i, rs);
                own[0 * SP + p] = st_F(st);
                own[1 * SP + p] = Fm;
                own[2 * SP + p] = Fs;
                own[3 * SP + p] = st_mass(st0, st1);
                own[4 * SP + p] = Fm0;
                own[5 * SP + p] = Fs0;
                own[6 * SP + p] = st_1mF(st0);
            }
        }

        // (2) chunk: producer vectors multiplied by the chunk moments
        float HF[kNC], HFm[kNC], HFs[kNC], HA[kNC], HFm1[kNC], HFs1[kNC];
        if (cact) {
            Expansion ea;
            expand(m_i, rs, tcen, ea);
            float v[kNC], w[kNC];
            vec_mass(ea, v);
#pragma unroll
            for (int k = 0; k < kNC; ++k) uc[k] += v[k];
#pragma unroll
            for (int k = 0; k < kNC; ++k) w[k] = ea.T[k];
            vec_moments(w, pa, HF);
            vec_dFdmu(ea, v);
            vec_moments(v, pa, HFm);
            vec_times_z(v, ea.z0, ea.r, w);
            vec_moments(w, pa, HFs);
            // shifted functions: A(u) = mass at u-s+1, dF(u-s)
            Expansion es;
            if (s != 1) expand(m_i, rs, tcen - (float)(s - 1), es);
            const Expansion &ex = (s != 1) ? es : ea;
            vec_mass(ex, v);
            vec_moments(v, pa, HA);
            vec_dFdmu_back(ex, v);
            vec_moments(v, pa, HFm1);
            vec_times_z(v, ex.z0 - rs, ex.r, w);
            vec_moments(w, pa, HFs1);
        } else {
#pragma unroll
            for (int k = 0; k < kNC; ++k) { HF[k] = HFm[k] = HFs[k] = HA[k] = HFm1[k] = HFs1[k] = 0.0f; }
        }

        // (3) polynomial out-edges
        for (int e = e0; e < e1; ++e) {
            const int eb = (e - e0) & 63;
            if (eb == 0) {
                x_ok = 0;
                if (e + lane < e1) {
                    x_j = G.col[e + lane];
                    x_ok = clsb[x_j];
                    x_mu = mub[x_j]; x_sg = sgb[x_j];
                }
            }
            if (!__builtin_amdgcn_readlane(x_ok, eb)) continue;  // step-by-step edge, done by k_ops
            const float m_j = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x_mu), eb));
            const float s_j = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x_sg), eb));
            const float rsj = 1.0f / s_j, cj = rsj * kInvSqrt2Pi;
            float cc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ps = 0; ps < NP; ++ps) {
                const int p = ps * 64 + lane;
                if (p < SP) {
                    const int u = p < pa.L0 ? p : D - 2 + (p - pa.L0);
                    float stj, Fmj, Fsj;
                    cdf_at(u, D, m_j, rsj, cj, stj, Fmj, Fsj);
                    const float Pj = st_mass(st_at((long long)u - 1, D, m_j, rsj), stj);
                    const float F = own[0 * SP + p], Fm = own[1 * SP + p];
                    const float Fs = own[2 * SP + p], A = own[3 * SP + p];
                    pr[2] = fmaf(-own[4 * SP + p], Pj, pr[2]);
                    pr[3] = fmaf(-own[5 * SP + p], Pj, pr[3]);
                    if (u < D - 1) {
                        const float omF = st_1mF(stj);
                        pr[0] = fmaf(A, st_F(stj), pr[0]);
                        pr[1] = fmaf(F, omF, pr[1]);
                        pr[4] = fmaf(Fm, omF, pr[4]);
                        pr[5] = fmaf(Fs, omF, pr[5]);
                        cc[0] = fmaf(A, Fmj, cc[0]);
                        cc[1] = fmaf(A, Fsj, cc[1]);
                        cc[2] = fmaf(-F, Fmj, cc[2]);
                        cc[3] = fmaf(-F, Fsj, cc[3]);
                    } else {
                        pr[0] += own[6 * SP + p];
                    }
                }
            }
            if (cact) {
                Expansion ej;
                expand(m_j, rsj, tcen, ej);
                float a[kNC], v[kNC];
                pr[0] += vdot_F(HA, ej);
                pr[1] += vdot_1mF(HF, ej);
                pr[4] += vdot_1mF(HFm, ej);
                pr[5] += vdot_1mF(HFs, ej);
                vec_dFdmu(ej, a);
                cc[0] += vdot(HA, a);
                cc[2] -= vdot(HF, a);
                vec_times_z(a, ej.z0, ej.r, v);
                cc[1] += vdot(HA, v);
                cc[3] -= vdot(HF, v);
                vec_mass(ej, v);
                pr[2] -= vdot(HFm1, v);
                pr[3] -= vdot(HFs1, v);
            }
            const float ct = wave_sum4(cc[0], cc[1], cc[2], cc[3], lane);
            if (lane < kCP) W.cpoly[((size_t)b * G.E + e) * kCP + wave4_comp(lane)] = ct;
        }
        const float pt4 = wave_sum4(pr[0], pr[1], pr[2], pr[3], lane);
        const float pt2 = wave_sum2(pr[4], pr[5], lane);
        if (lane < 4) pp[wave4_comp(lane)] = pt4;
        if (lane < 2) pp[4 + lane] = pt2;
        gsum += pt4;   // lane 0: V_dep, lane 2: L_com
    }
    if (lane == 0) sGs[wv][0] = gsum;
    if (lane == 2) sGs[wv][1] = gsum;

    // usage of the group: combine the waves' chunk coefficients and strip values
#pragma unroll
    for (int k = 0; k < kNC; ++k) sUc[wv][lane][k] = uc[k];
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) {
        const int p = ps * 64 + lane;
        if (p < SP) sUs[wv * SP + p] = us[ps];
    }
    __syncthreads();
    float *ucg = W.Ucoef + slot_id * kMaxChunks * kNC;
    for (int x = threadIdx.x; x < kMaxChunks * kNC; x += 64 * kPolyWaves) {
        const int c = x / kNC, k = x % kNC;
        float acc = 0.0f;
#pragma unroll
        for (int w = 0; w < kPolyWaves; ++w) acc += sUc[w][c][k];
        ucg[x] = acc;
    }
    if (threadIdx.x < 2) {
        float acc = 0.0f;
#pragma unroll
        for (int w = 0; w < kPolyWaves; ++w) acc += sGs[w][threadIdx.x];
        W.gsum_poly[slot_id * 2 + threadIdx.x] = acc;
    }
    float *usg = W.Ustrip + slot_id * kStripMax;
    for (int p = threadIdx.x; p < kStripMax; p += 64 * kPolyWaves) {
        float acc = 0.0f;
        if (p < SP) {
#pragma unroll
            for (int w = 0; w < kPolyWaves; ++w) acc += sUs[w * SP + p];
        }
        usg[p] = acc;
    }
}

// ---------------------------------------------------------------------------
// Gradient of the smooth peak usage.  With c_k(d) = beta dL_res/dU_k(d mod T)
// (the softmax written by k_vres), summation by parts onto the interior bin
// edges gives
//   dL/dth_i += sum_{t=0}^{D-2} (c(t) - c(t+1)) dF_i(t)/dth_i,
// a dense weight per bin edge.  Step-by-step ops take it per step
// (k_lse_ops); polynomial ops take it per chunk as the moments
// M_n = sum_y (c(t) - c(t+1)) y^n (k_lse_mom), dotted with the chunk
// coefficients of dF/dmu and dF/dsigma (k_lse_poly).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float soft_diff(const float *sk, int t, int T) {
    return sk[t % T] - sk[(t + 1) % T];
}

template <int BS, int SPT>
__global__ __launch_bounds__(BS) void k_lse_ops(Graph G, const float *__restrict__ mu,
                                                const float *__restrict__ sigma, Work W) {
    constexpr int TILE = BS * SPT;
    __shared__ float sW[TILE];
    __shared__ int sI[BS];
    __shared__ float sMu[BS], sRs[BS];
    __shared__ float sRed[2][BS / 64][8];
    const int grp = blockIdx.x, tile = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    const int N = G.N, D = G.D, T = G.T;
    const int t0 = tile * TILE;
    int direct = 0;
    if (q0 + tid < q1) {
        const int i = G.perm[q0 + tid];
        const size_t bi = (size_t)b * N + i;
        direct = W.cls[bi] ? 0 : 1;
        sI[tid] = direct ? i : -1;
        sMu[tid] = mu[bi];
        sRs[tid] = 1.0f / sigma[bi];
    } else if (tid < BS) {
        sI[tid] = -1;
    }
    if (!__syncthreads_or(direct)) return;   // every op of the group is polynomial
    const float *sk = W.soft + ((size_t)b * G.K + G.rtype[G.perm[q0]]) * T;
    for (int x = tid; x < TILE; x += BS) {
        const int t = t0 + x;
        sW[x] = t <= D - 2 ? soft_diff(sk, t, T) : 0.0f;
    }
    __syncthreads();
    int par = 0;
    for (int q = 0; q < q1 - q0; ++q) {
        const int i = sI[q];
        if (i < 0) continue;
        const float m = sMu[q], rs = sRs[q], cinv = rs * kInvSqrt2Pi;
        float acc[2] = {0.0f, 0.0f};
#pragma unroll
        for (int j = 0; j < SPT; ++j) {
            const int x = tid + j * BS;
            const float w = sW[x];
            if (w != 0.0f) {
                const float z = ((float)(t0 + x) + 0.5f - m) * rs;
                const float Fm = -__builtin_amdgcn_exp2f(-(z * z) * kHalfLog2e) * cinv;
                acc[0] = fmaf(w, Fm, acc[0]);
                acc[1] = fmaf(w, Fm * z, acc[1]);
            }
        }
        const float r = block_sum<2, BS>(acc, sRed[par]);
        par ^= 1;
        if (tid < 2) W.lpart[(((size_t)b * N + i) * G.ntiles + tile) * 2 + tid] = r;
    }
}

__global__ __launch_bounds__(256) void k_lse_mom(Graph G, PolyArgs pa, Work W) {
    __shared__ float sRed[4][kNC];
    const int c = blockIdx.x, k = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int T = G.T, D = G.D;
    const float *sk = W.soft + ((size_t)b * G.K + k) * T;
    if (c == pa.nc) {   // the strip: weights per position (none at D-1, not a bin edge)
        float *dst = W.lstrip + ((size_t)b * G.K + k) * kStripMax;
        for (int p = tid; p < pa.SP; p += 256) {
            const int u = p < pa.L0 ? p : D - 2 + (p - pa.L0);
            dst[p] = u <= D - 2 ? soft_diff(sk, u, T) : 0.0f;
        }
        return;
    }
    float mom[kNC];
#pragma unroll
    for (int n = 0; n < kNC; ++n) mom[n] = 0.0f;
    if (tid < pa.W) {
        const int t = pa.L0 + c * pa.W + tid;
        const float y = (float)tid - pa.lam;
        float yp = soft_diff(sk, t, T);
#pragma unroll
        for (int n = 0; n < kNC; ++n) { mom[n] = yp; yp *= y; }
    }
#pragma unroll
    for (int n = 0; n < kNC; ++n) {
        const float r = wave_sum(mom[n]);
        if (lane == 0) sRed[wid][n] = r;
    }
    __syncthreads();
    if (tid < kNC)
        W.lmom[(((size_t)b * G.K + k) * kMaxChunks + c) * kNC + tid] =
            (sRed[0][tid] + sRed[1][tid]) + (sRed[2][tid] + sRed[3][tid]);
}

template <int NP>
__global__ __launch_bounds__(64 * kPolyWaves) void k_lse_poly(Graph G, PolyArgs pa, const float *__restrict__ mu,
                                                              const float *__restrict__ sigma, Work W) {
    const int SP = pa.SP, split = pa.split;
    const int grp = blockIdx.x / split, sub = blockIdx.x - grp * split, b = blockIdx.y;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int N = G.N, D = G.D;
    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    if (q1 <= q0) return;
    const int nj = (q1 - q0 - sub + split - 1) / split;
    const int nq = (nj - wv + kPolyWaves - 1) / kPolyWaves;
    int l_i = 0, l_cls = 0;
    float l_mu = 0.0f, l_sg = 1.0f;
    if (lane < nq) {
        l_i = G.perm[q0 + sub + split * (wv + kPolyWaves * lane)];
        const size_t bi = (size_t)b * N + l_i;
        l_cls = W.cls[bi];
        l_mu = mu[bi]; l_sg = sigma[bi];
    }
    // this lane's chunk moments and strip weights of the group's type
    const int k = G.rtype[G.perm[q0]];
    const bool cact = lane < pa.nc;
    float mom[kNC];
    const float *msrc = W.lmom + (((size_t)b * G.K + k) * kMaxChunks + lane) * kNC;
#pragma unroll
    for (int n = 0; n < kNC; ++n) mom[n] = cact ? msrc[n] : 0.0f;
    float sw[NP];
    const float *ssrc = W.lstrip + ((size_t)b * G.K + k) * kStripMax;
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) {
        const int p = ps * 64 + lane;
        sw[ps] = p < SP ? ssrc[p] : 0.0f;
    }
    const float tcen = (float)(pa.L0 + lane * pa.W) + pa.lam;
    for (int oq = 0; oq < nq; ++oq) {
        if (!__builtin_amdgcn_readlane(l_cls, oq)) continue;
        const int i = __builtin_amdgcn_readlane(l_i, oq);
        const float m_i = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, l_mu), oq));
        const float s_i = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, l_sg), oq));
        const float rs = 1.0f / s_i, cinv = rs * kInvSqrt2Pi;
        float gm = 0.0f, gs = 0.0f;
#pragma unroll
        for (int ps = 0; ps < NP; ++ps) {
            const int p = ps * 64 + lane;
            if (p < SP) {
                const int u = p < pa.L0 ? p : D - 2 + (p - pa.L0);
                const float z = ((float)u + 0.5f - m_i) * rs;
                const float Fm = -__builtin_amdgcn_exp2f(-(z * z) * kHalfLog2e) * cinv;
                gm = fmaf(sw[ps], Fm, gm);
                gs = fmaf(sw[ps], Fm * z, gs);
            }
        }
        if (cact) {
            Expansion e;
            expand(m_i, rs, tcen, e);
            float a[kNC], v[kNC];
            vec_dFdmu(e, a);
            vec_times_z(a, e.z0, e.r, v);
            gm += vdot(a, mom);
            gs += vdot(v, mom);
        }
        const float r = wave_sum2(gm, gs, lane);
        if (lane < 2) W.lpoly[((size_t)b * N + i) * 2 + lane] = r;
    }
}

// ---------------------------------------------------------------------------
// Back-edge kernel (modulo scheduling).  Work-group = (back-edge block, tile,
// restart); one back edge (j -> i, k) at a time, c = k*II - Lat_j:
//   V_rec       = F_i(-c-1) + sum_u P_i^{u-c} (1 - F_j(u))
//   dVrec/dth_j = -sum_u F_j'(u) P_i^{u-c}
//   dVrec/dth_i =  sum_t F_i'(t) P_j^{t+c+1}
// with u, t over the interior edges 0..D-2.
// ---------------------------------------------------------------------------
template <int BS, int SPT>
__global__ __launch_bounds__(BS) void k_back(Graph G, const float *__restrict__ mu,
                                             const float *__restrict__ sigma, Work W,
                                             int edges_per_block) {
    constexpr int TILE = BS * SPT;
    __shared__ float sRed[2][BS / 64][8];
    const int tile = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int D = G.D, N = G.N;
    const int t0 = tile * TILE;
    const int be0 = blockIdx.x * edges_per_block;
    const int be1 = min(be0 + edges_per_block, G.nb);
    int par = 0;
    for (int e = be0; e < be1; ++e) {
        const int j = uniform(G.bsrc[e]), i = uniform(G.bdst[e]);
        const long long c = (long long)G.bdist[e] * G.II - G.delay[j];
        const float mj = mu[(size_t)b * N + j], sj = sigma[(size_t)b * N + j];
        const float mi = mu[(size_t)b * N + i], si = sigma[(size_t)b * N + i];
        const float rsj = 1.0f / sj, rsi = 1.0f / si;
        const float cj = rsj * kInvSqrt2Pi, ci = rsi * kInvSqrt2Pi;
        float acc[5] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k = 0; k < SPT; ++k) {
            const int u = t0 + k * BS + tid;
            if (u < D - 1) {
                float sj_, Fmj, Fsj, si_, Fmi, Fsi;
                cdf_at(u, D, mj, rsj, cj, sj_, Fmj, Fsj);
                cdf_at(u, D, mi, rsi, ci, si_, Fmi, Fsi);
                const float Pi = st_mass(st_at((long long)u - c - 1, D, mi, rsi), st_at((long long)u - c, D, mi, rsi));
                const float Pj = st_mass(st_at((long long)u + c, D, mj, rsj), st_at((long long)u + c + 1, D, mj, rsj));
                acc[0] = fmaf(Pi, st_1mF(sj_), acc[0]);
                acc[1] = fmaf(-Fmj, Pi, acc[1]);
                acc[2] = fmaf(-Fsj, Pi, acc[2]);
                acc[3] = fmaf(Fmi, Pj, acc[3]);
                acc[4] = fmaf(Fsi, Pj, acc[4]);
            }
        }
        if (tile == 0 && tid == 0) acc[0] += st_F(st_at(-c - 1, D, mi, rsi));
        const float r = block_sum<5, BS>(acc, sRed[par]);
        par ^= 1;
        if (tid < kBP) W.bpart[(((size_t)b * G.nb + e) * G.ntiles + tile) * kBP + tid] = r;
    }
}

// ---------------------------------------------------------------------------
// Usage: U[b][k][slot] = sum over type-k groups and steps t = slot (mod T).
// ---------------------------------------------------------------------------
// Polynomial usage per (type, restart): the groups' chunk coefficients and
// strip values summed over the type's groups (64 entries x 4 group slices per
// work-group, combined in a fixed order).
constexpr int kUcEntries = kMaxChunks * kNC + kStripMax;   // per (restart, type)

__global__ __launch_bounds__(256) void k_ucoef(Graph G, PolyArgs pa, Work W) {
    __shared__ float part[4][64];
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int x = blockIdx.x * 64 + tx, k = blockIdx.y, b = blockIdx.z;
    // the type's polynomial work-groups: slots [g0*split, g1*split) of restart b
    const int g0 = G.type_grp[k] * pa.split, g1 = G.type_grp[k + 1] * pa.split;
    const size_t rb = (size_t)b * G.ngroups * pa.split;
    const int ncoef = pa.nc * kNC;
    float acc = 0.0f;
    if (x < ncoef) {
        for (int g = g0 + ty; g < g1; g += 4) acc += W.Ucoef[(rb + g) * kMaxChunks * kNC + x];
    } else if (x < ncoef + pa.SP) {
        for (int g = g0 + ty; g < g1; g += 4) acc += W.Ustrip[(rb + g) * kStripMax + (x - ncoef)];
    }
    part[ty][tx] = acc;
    __syncthreads();
    if (ty == 0 && x < ncoef + pa.SP)
        W.Ucoef_k[((size_t)b * G.K + k) * kUcEntries + x] = (part[0][tx] + part[1][tx]) + (part[2][tx] + part[3][tx]);
}

// Usage U(slot) per (slot block, type, restart): step-by-step partials of the
// type's active groups plus the polynomial part (chunk polynomial at t, or
// the strip value), summed over t = slot mod T.
constexpr int kUsageBS = 256;

__global__ __launch_bounds__(kUsageBS) void k_usage(Graph G, PolyArgs pa, Work W) {
    constexpr int kMaxAct = 1024;
    __shared__ float sC[kUcEntries];
    __shared__ int sAct[kMaxAct];
    __shared__ int wcount[kUsageBS / 64];
    __shared__ int base;
    const int k = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int g0 = G.type_grp[k], g1 = G.type_grp[k + 1];
    const int D = G.D, T = G.T;

    // the type's groups with step-by-step partials, compacted in order
    if (tid == 0) base = 0;
    __syncthreads();
    for (int c0 = g0; c0 < g1; c0 += kUsageBS) {
        const int g = c0 + tid;
        const bool f = g < g1 && W.gflag[(size_t)b * G.ngroups + g] != 0;
        const unsigned long long bal = __ballot(f);
        const int before = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) wcount[wid] = __popcll(bal);
        __syncthreads();
        int off = base;
        for (int w = 0; w < wid; ++w) off += wcount[w];
        if (f && off + before < kMaxAct) sAct[off + before] = g;
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < kUsageBS / 64; ++w) tot += wcount[w];
            base += tot;
        }
        __syncthreads();
    }
    const int nact = base;   // > kMaxAct: scan the flags instead of the list
    if (pa.enabled) {
        const float *src = W.Ucoef_k + ((size_t)b * G.K + k) * kUcEntries;
        const int n = pa.nc * kNC + pa.SP;
        for (int x = tid; x < n; x += kUsageBS) sC[x] = src[x];
    }
    __syncthreads();
    const int slot = blockIdx.x * kUsageBS + tid;
    if (slot >= T) return;
    const int ncoef = pa.nc * kNC;
    float acc = 0.0f;
    for (int t = slot; t < D; t += T) {
        float ut = 0.0f;
        if (nact <= kMaxAct) {
            for (int q = 0; q < nact; ++q) ut += W.Upart[((size_t)b * G.ngroups + sAct[q]) * D + t];
        } else {
            for (int g = g0; g < g1; ++g)
                if (W.gflag[(size_t)b * G.ngroups + g]) ut += W.Upart[((size_t)b * G.ngroups + g) * D + t];
        }
        if (pa.enabled) {
            if (t >= pa.L0 && t < D - 2) {
                const int c = (t - pa.L0) / pa.W;
                const float x = (float)(t - pa.L0 - c * pa.W) - pa.lam;
                const float *cf = sC + c * kNC;
                float v = cf[kNC - 1];
#pragma unroll
                for (int q = kNC - 2; q >= 0; --q) v = fmaf(v, x, cf[q]);
                ut += v;
            } else {
                ut += sC[ncoef + (t < pa.L0 ? t : pa.L0 + (t - (D - 2)))];
            }
        }
        acc += ut;
    }
    W.U[((size_t)b * G.K + k) * T + slot] = acc;
}

// ---------------------------------------------------------------------------
// Per (type, restart): the type's share of V_res (eq:relu) and the bin edges
// t = 0..D-2 where its ReLU indicator I(t mod T) != I((t+1) mod T) changes,
// compacted in increasing t (wave ballots + a work-group prefix).
// ---------------------------------------------------------------------------
constexpr int kTermsBS = 1024;

__device__ float block_sum1024(float x, float *scratch /*[16]*/) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    x = wave_sum(x);
    if (lane == 0) scratch[wid] = x;
    __syncthreads();
    float r = 0.0f;
#pragma unroll
    for (int w = 0; w < kTermsBS / 64; ++w) r += scratch[w];
    __syncthreads();
    return r;
}

__device__ float block_max1024(float x, float *scratch /*[16]*/) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    x = wave_max(x);
    if (lane == 0) scratch[wid] = x;
    __syncthreads();
    float r = scratch[0];
#pragma unroll
    for (int w = 1; w < kTermsBS / 64; ++w) r = fmaxf(r, scratch[w]);
    __syncthreads();
    return r;
}

// Per (type, restart) also the smooth peak (App. B.2, eq:max)
//   L_res,k = tau log sum_t exp(U_k(t)/tau) = M + tau log sum_t exp((U_k(t) - M)/tau),
// M = max_t U_k(t), and beta times its derivative (the softmax) per slot.
__global__ __launch_bounds__(kTermsBS) void k_vres(Graph G, Work W, HP hp) {
    __shared__ float scratch[kTermsBS / 64];
    __shared__ int wcount[kTermsBS / 64];
    __shared__ int base;
    const int k = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int T = G.T, D = G.D;
    const float ck = G.cap[k];
    const float *Uk = W.U + ((size_t)b * G.K + k) * T;

    float vres = 0.0f;
    for (int c = tid; c < T; c += kTermsBS) {
        const float ex = Uk[c] - ck;
        if (ex > 0.0f) vres += ex;
    }
    vres = block_sum1024(vres, scratch);
    if (tid == 0) W.vres_part[(size_t)b * G.K + k] = vres;

    if (hp.beta != 0.0f) {
        float mx = -INFINITY;
        for (int c = tid; c < T; c += kTermsBS) mx = fmaxf(mx, Uk[c]);
        mx = block_max1024(mx, scratch);
        const float itau = 1.0f / hp.tau;
        float z = 0.0f;
        for (int c = tid; c < T; c += kTermsBS) z += expf((Uk[c] - mx) * itau);
        z = block_sum1024(z, scratch);
        if (tid == 0) W.lres_part[(size_t)b * G.K + k] = mx + hp.tau * logf(z);
        const float bz = hp.beta / z;
        float *sk = W.soft + ((size_t)b * G.K + k) * T;
        for (int c = tid; c < T; c += kTermsBS) sk[c] = bz * expf((Uk[c] - mx) * itau);
    } else if (tid == 0) {
        W.lres_part[(size_t)b * G.K + k] = 0.0f;
    }

    int *out = W.trans + ((size_t)b * G.K + k) * D;
    if (tid == 0) base = 0;
    __syncthreads();
    for (int t0 = 0; t0 < D - 1; t0 += kTermsBS) {
        const int t = t0 + tid;
        int sgn = 0;
        if (t < D - 1) {
            const int a = Uk[t % T] > ck, c = Uk[(t + 1) % T] > ck;
            sgn = a - c;
        }
        const unsigned long long bal = __ballot(sgn != 0);
        const int before = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) wcount[wid] = __popcll(bal);
        __syncthreads();
        int off = base;
        for (int w = 0; w < wid; ++w) off += wcount[w];
        if (sgn != 0) out[off + before] = sgn * (t + 1);
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < kTermsBS / 64; ++w) tot += wcount[w];
            base += tot;
        }
        __syncthreads();
    }
    if (tid == 0) W.ntrans[(size_t)b * G.K + k] = base;
}

// ---------------------------------------------------------------------------
// Per restart: V_res, V_dep, L_com, V_rec from the partials, the augmented
// Lagrangian (eq. 11), the weights w_c = lambda_c + rho V_c, and in step mode
// the multiplier update lambda_c += rho V_c and the Adam bias corrections.
// ---------------------------------------------------------------------------
constexpr int kCombineBS = 256;

__device__ float block_sum256(float x, float *scratch /*[4]*/) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    x = wave_sum(x);
    if (lane == 0) scratch[wid] = x;
    __syncthreads();
    const float r = (scratch[0] + scratch[1]) + (scratch[2] + scratch[3]);
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(kCombineBS) void k_combine(Graph G, PolyArgs pa, Work W, HP hp,
                                                        const float *__restrict__ lambda_in,
                                                        float *lambda_out, const int *adam_t,
                                                        float *terms_out) {
    __shared__ float scratch[kCombineBS / 64];
    const int b = blockIdx.x, tid = threadIdx.x;
    float vres = 0.0f, vdep = 0.0f, lcom = 0.0f, vrec = 0.0f, lres = 0.0f;
    for (int k = tid; k < G.K; k += kCombineBS) {
        vres += W.vres_part[(size_t)b * G.K + k];
        lres += W.lres_part[(size_t)b * G.K + k];
    }
    const int npoly = G.ngroups * pa.split;
    for (int g = tid; g < npoly; g += kCombineBS) {
        const float *gp = W.gsum_poly + ((size_t)b * npoly + g) * 2;
        vdep += gp[0]; lcom += gp[1];
    }
    for (int g = tid; g < G.ngroups; g += kCombineBS) {
        if (W.gflag[(size_t)b * G.ngroups + g]) {
            const float *go = W.gsum_ops + ((size_t)b * G.ngroups + g) * G.ntiles * 2;
            for (int tl = 0; tl < G.ntiles; ++tl) { vdep += go[2 * tl]; lcom += go[2 * tl + 1]; }
        }
    }
    const size_t nbp = (size_t)G.nb * G.ntiles;
    const float *bp = W.bpart + (size_t)b * nbp * kBP;
    for (size_t r = tid; r < nbp; r += kCombineBS) vrec += bp[r * kBP + 0];
    vres = block_sum256(vres, scratch);
    vdep = block_sum256(vdep, scratch);
    lcom = block_sum256(lcom, scratch);
    vrec = block_sum256(vrec, scratch);
    lres = block_sum256(lres, scratch);

    if (tid == 0) {
        const float V[3] = {vdep, vres, vrec};
        const float *lam = lambda_in + (size_t)b * 3;
        float L = fmaf(hp.beta, lres, hp.alpha * lcom);
        float w[3];
        for (int c = 0; c < 3; ++c) {
            L += lam[c] * V[c] + 0.5f * hp.rho * V[c] * V[c];
            w[c] = lam[c] + hp.rho * V[c];
        }
        float *tm = W.terms + (size_t)b * kTerms;
        tm[0] = L; tm[1] = vdep; tm[2] = vres; tm[3] = vrec; tm[4] = lcom; tm[5] = lres;
        if (terms_out) for (int c = 0; c < kTerms; ++c) terms_out[(size_t)b * kTerms + c] = tm[c];
        float *wt = W.wts + (size_t)b * 4;
        wt[0] = w[0]; wt[1] = w[1]; wt[2] = w[2]; wt[3] = 0.0f;
        if (lambda_out) for (int c = 0; c < 3; ++c) lambda_out[(size_t)b * 3 + c] = fmaf(hp.rho, V[c], lam[c]);
        if (adam_t) {
            const int t = *adam_t + 1;
            W.adamf[(size_t)b * 2 + 0] = 1.0f - powf(hp.b1, (float)t);
            W.adamf[(size_t)b * 2 + 1] = 1.0f - powf(hp.b2, (float)t);
        }
    }
}

// Adam (Kingma & Ba), bias-corrected.  Every rounding step is spelled out
// (no implicit multiply-add contraction) so that the fused step and the
// separate optimizer kernel produce identical bits.
__device__ __forceinline__ void adam_update(float &th, float &m, float &v, float g, float lr, float b1,
                                            float b2, float eps, float c1, float c2) {
    m = fmaf(b1, m, __fmul_rn(1.0f - b1, g));
    v = fmaf(b2, v, __fmul_rn(__fmul_rn(1.0f - b2, g), g));
    const float denom = __fadd_rn(sqrtf(__fdiv_rn(v, c2)), eps);
    th = __fsub_rn(th, __fdiv_rn(__fmul_rn(lr, __fdiv_rn(m, c1)), denom));
}

// dL/dtheta from the four constraint/objective derivatives, fixed rounding order.
__device__ __forceinline__ float combine_grad(float w_res, float r, float w_dep, float d, float w_rec,
                                              float q, float alpha, float c) {
    return fmaf(alpha, c, fmaf(w_rec, q, fmaf(w_dep, d, __fmul_rn(w_res, r))));
}

// ---------------------------------------------------------------------------
// Gradient assembly (+ Adam in step mode).  Thread per (restart, op):
//   dL/dth_i = w_res dVres/dth_i + w_dep dVdep/dth_i + w_rec dVrec/dth_i + alpha dLcom/dth_i
// dVres/dth_i = sum over bin edges t where the ReLU indicator of the op's type
// changes of (I(t) - I(t+1)) F_i'(t); the other pieces are sums of partials
// (own tiles, in-edges through the CSC, back edges on either side).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_final(Graph G, Work W, HP hp, const float *mu,
                                               const float *sigma, float *gmu,
                                               float *gsig, float *mu_io, float *sig_io, float *am,
                                               float *av, int *adam_t, int mode) {
    const int b = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= G.N) return;
    const int N = G.N, nt = G.ntiles;
    const size_t bi = (size_t)b * N + i;
    const float m_i = mu[bi], s_i = sigma[bi];
    const float rs = 1.0f / s_i, cinv = rs * kInvSqrt2Pi;
    const float *wt = W.wts + (size_t)b * 4;
    const float w_dep = wt[0], w_res = wt[1], w_rec = wt[2];

    // resource term through the indicator changes of this op's type
    const int k = G.rtype[i];
    const int nt_k = W.ntrans[(size_t)b * G.K + k];
    const int *tr = W.trans + ((size_t)b * G.K + k) * G.D;
    float rm = 0.0f, rsg = 0.0f;
    for (int q = 0; q < nt_k; ++q) {
        const int code = tr[q];
        const float sgn = code > 0 ? 1.0f : -1.0f;
        const int t = (code > 0 ? code : -code) - 1;
        const float z = ((float)t + 0.5f - m_i) * rs;
        const float g = __builtin_amdgcn_exp2f(-(z * z) * kHalfLog2e);
        const float Fm = -g * cinv;
        rm = fmaf(sgn, Fm, rm);
        rsg = fmaf(sgn, Fm * z, rsg);
    }

    float dm = 0.0f, ds = 0.0f, cm = 0.0f, cs = 0.0f;
    if (W.dflag[bi]) {
        const float *pp = W.ppart + bi * nt * kPP;
        for (int tl = 0; tl < nt; ++tl) {
            dm += pp[tl * kPP + 2]; ds += pp[tl * kPP + 3];
            cm += pp[tl * kPP + 4]; cs += pp[tl * kPP + 5];
        }
    }
    const float *ppy = W.ppoly + bi * kPP;
    dm += ppy[2]; ds += ppy[3]; cm += ppy[4]; cs += ppy[5];
    const bool poly_i = W.cls[bi] != 0;
    for (int q = G.pred_ptr[i]; q < G.pred_ptr[i + 1]; ++q) {
        const int e = G.pred_eid[q];
        if (poly_i && W.cls[(size_t)b * N + G.pred_src[q]]) {
            const float *cp = W.cpoly + ((size_t)b * G.E + e) * kCP;
            dm += cp[0]; ds += cp[1]; cm += cp[2]; cs += cp[3];
            continue;
        }
        const float *cp = W.cpart + (((size_t)b * G.E + e) * nt) * kCP;
        for (int tl = 0; tl < nt; ++tl) {
            dm += cp[tl * kCP + 0]; ds += cp[tl * kCP + 1];
            cm += cp[tl * kCP + 2]; cs += cp[tl * kCP + 3];
        }
    }
    float qm = 0.0f, qs = 0.0f;
    for (int q = G.bout_ptr[i]; q < G.bout_ptr[i + 1]; ++q) {
        const float *bp = W.bpart + (((size_t)b * G.nb + G.bout[q]) * nt) * kBP;
        for (int tl = 0; tl < nt; ++tl) { qm += bp[tl * kBP + 1]; qs += bp[tl * kBP + 2]; }
    }
    for (int q = G.bin_ptr[i]; q < G.bin_ptr[i + 1]; ++q) {
        const float *bp = W.bpart + (((size_t)b * G.nb + G.bin[q]) * nt) * kBP;
        for (int tl = 0; tl < nt; ++tl) { qm += bp[tl * kBP + 3]; qs += bp[tl * kBP + 4]; }
    }
    float g_mu = combine_grad(w_res, rm, w_dep, dm, w_rec, qm, hp.alpha, cm);
    float g_sg = combine_grad(w_res, rsg, w_dep, ds, w_rec, qs, hp.alpha, cs);
    if (hp.beta != 0.0f) {   // smooth peak usage, already weighted by beta
        float lm = 0.0f, ls = 0.0f;
        if (poly_i) {
            lm = W.lpoly[bi * 2 + 0]; ls = W.lpoly[bi * 2 + 1];
        } else {
            const float *lp = W.lpart + bi * nt * 2;
            for (int tl = 0; tl < nt; ++tl) { lm += lp[tl * 2 + 0]; ls += lp[tl * 2 + 1]; }
        }
        g_mu = __fadd_rn(g_mu, lm);
        g_sg = __fadd_rn(g_sg, ls);
    }

    if (mode == 0) {
        gmu[bi] = g_mu;
        gsig[bi] = g_sg;
    } else {
        const float c1 = W.adamf[(size_t)b * 2 + 0], c2 = W.adamf[(size_t)b * 2 + 1];
        const size_t half = (size_t)G.B * N;
        float th = mu_io[bi], mm = am[bi], vv = av[bi];
        adam_update(th, mm, vv, g_mu, hp.lr, hp.b1, hp.b2, hp.eps, c1, c2);
        mu_io[bi] = th; am[bi] = mm; av[bi] = vv;
        th = sig_io[bi]; mm = am[half + bi]; vv = av[half + bi];
        adam_update(th, mm, vv, g_sg, hp.lr, hp.b1, hp.b2, hp.eps, c1, c2);
        sig_io[bi] = fmaxf(th, hp.sigma_min);
        am[half + bi] = mm; av[half + bi] = vv;
        if (b == 0 && i == 0) *adam_t += 1;
    }
}

// lambda += rho V (V from terms) and the Adam bias corrections; one thread per restart.
__global__ void k_lambda_from_terms(int B, HP hp, const float *terms, float *lambda,
                                    const int *adam_t, float *adamf) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    for (int c = 0; c < 3; ++c)
        lambda[(size_t)b * 3 + c] = fmaf(hp.rho, terms[(size_t)b * kTerms + 1 + c], lambda[(size_t)b * 3 + c]);
    const int t = *adam_t + 1;
    adamf[(size_t)b * 2 + 0] = 1.0f - powf(hp.b1, (float)t);
    adamf[(size_t)b * 2 + 1] = 1.0f - powf(hp.b2, (float)t);
}

__global__ __launch_bounds__(256) void k_adam(int B, int N, HP hp, const float *adamf,
                                              const float *gmu, const float *gsig, float *mu,
                                              float *sigma, float *am, float *av, int *adam_t) {
    const int b = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N) return;
    const size_t bi = (size_t)b * N + i, half = (size_t)B * N;
    const float c1 = adamf[(size_t)b * 2 + 0], c2 = adamf[(size_t)b * 2 + 1];
    float th = mu[bi], mm = am[bi], vv = av[bi];
    adam_update(th, mm, vv, gmu[bi], hp.lr, hp.b1, hp.b2, hp.eps, c1, c2);
    mu[bi] = th; am[bi] = mm; av[bi] = vv;
    th = sigma[bi]; mm = am[half + bi]; vv = av[half + bi];
    adam_update(th, mm, vv, gsig[bi], hp.lr, hp.b1, hp.b2, hp.eps, c1, c2);
    sigma[bi] = fmaxf(th, hp.sigma_min);
    am[half + bi] = mm; av[half + bi] = vv;
    if (b == 0 && i == 0) *adam_t += 1;
}

// ---------------------------------------------------------------------------
// Legalization (App. A).  One work-group per restart sweeps the topological
// levels; ops of one level have no forward edges between them, so a level is
// processed in parallel and the sweep equals the paper's sequential pass.
// Modulo: back-edge requirements read the schedule as it was at the start of
// the pass; the iteration is monotone and inflationary, so when it stops it has
// reached the least fixed point above the clamped rounding, as Alg. 4 does.
// ---------------------------------------------------------------------------
constexpr int kLegBS = 1024;

__device__ __forceinline__ long long round_half_up(float mu, int D) {
    float m = fmaxf(mu, -1.0f);              // NaN -> -1
    m = fminf(m, (float)D);
    const float fl = floorf(m);
    return (long long)fl + ((m - fl) >= 0.5f ? 1 : 0);
}

__global__ __launch_bounds__(kLegBS) void k_legalize(Graph G, Work W, const float *__restrict__ mu,
                                                     int *sched) {
    __shared__ int changed, over;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = G.N, D = G.D;
    long long *s = W.s64 + (size_t)b * N;
    long long *sp = W.s64b + (size_t)b * N;
    for (int v = tid; v < N; v += kLegBS) {
        long long r = round_half_up(mu[(size_t)b * N + v], D);
        const long long lo = G.II == 0 ? G.asap[v] : 0, hi = G.II == 0 ? G.alap[v] : D - 1;
        r = r < lo ? lo : (r > hi ? hi : r);
        s[v] = r;
    }
    __syncthreads();
    int st = 0;
    if (G.II == 0) {
        for (int l = 1; l < G.nlevels; ++l) {
            for (int q = G.lvl_ptr[l] + tid; q < G.lvl_ptr[l + 1]; q += kLegBS) {
                const int v = G.lvl_ops[q];
                long long req = s[v];
                for (int r = G.pred_ptr[v]; r < G.pred_ptr[v + 1]; ++r) {
                    const int u = G.pred_src[r];
                    const long long c = s[u] + G.delay[u];
                    req = c > req ? c : req;
                }
                s[v] = req;
            }
            __syncthreads();
        }
    } else {
        int converged = 0;
        for (int pass = 0; pass < (N > 0 ? N : 1); ++pass) {
            for (int v = tid; v < N; v += kLegBS) sp[v] = s[v];
            if (tid == 0) changed = 0;
            __syncthreads();
            for (int l = 0; l < G.nlevels; ++l) {
                for (int q = G.lvl_ptr[l] + tid; q < G.lvl_ptr[l + 1]; q += kLegBS) {
                    const int v = G.lvl_ops[q];
                    long long req = 0;
                    for (int r = G.pred_ptr[v]; r < G.pred_ptr[v + 1]; ++r) {
                        const int u = G.pred_src[r];
                        const long long c = s[u] + G.delay[u];
                        req = c > req ? c : req;
                    }
                    for (int r = G.bin_ptr[v]; r < G.bin_ptr[v + 1]; ++r) {
                        const int e = G.bin[r], j = G.bsrc[e];
                        const long long c = sp[j] + G.delay[j] - (long long)G.bdist[e] * G.II;
                        req = c > req ? c : req;
                    }
                    if (req > s[v]) { s[v] = req; changed = 1; }
                }
                __syncthreads();
            }
            const int ch = changed;
            __syncthreads();
            if (!ch) { converged = 1; break; }
        }
        if (!converged) {
            st = 4;  // GAUS_E_NOT_CONVERGED
        } else {
            if (tid == 0) over = 0;
            __syncthreads();
            for (int v = tid; v < N; v += kLegBS)
                if (s[v] > D - 1) over = 1;
            __syncthreads();
            st = over ? 5 : 0;  // GAUS_E_OVERFLOW
        }
    }
    for (int v = tid; v < N; v += kLegBS) {
        const long long x = s[v];
        sched[(size_t)b * N + v] = x > 2147483647LL ? 2147483647 : (int)x;
    }
    if (tid == 0) W.status[b] = st;
}

// ---------------------------------------------------------------------------
// Host-side enqueue helpers
// ---------------------------------------------------------------------------
template <int BS, int SPT>
static void launch_ops(const Graph &g, const Work &w, const float *mu, const float *sigma,
                       hipStream_t st) {
    dim3 grid(g.ngroups, g.ntiles, g.B);
    hipLaunchKernelGGL((k_ops<BS, SPT>), grid, dim3(BS), 0, st, g, mu, sigma, w);
}

template <int BS, int SPT>
static void launch_back(const Graph &g, const Work &w, const float *mu, const float *sigma,
                        hipStream_t st) {
    const int epb = 4;
    dim3 gb((g.nb + epb - 1) / epb, g.ntiles, g.B);
    hipLaunchKernelGGL((k_back<BS, SPT>), gb, dim3(BS), 0, st, g, mu, sigma, w, epb);
}

hipError_t enqueue_iteration(const Graph &g, const Work &w, const HP &hp, const LaunchCfg &lc,
                             const PolyArgs &pa, const IterArgs &a, hipStream_t st) {
    {
        dim3 grid((std::max(g.N, g.ngroups) + 255) / 256, g.B);
        hipLaunchKernelGGL(k_classify, grid, dim3(256), 0, st, g, pa, a.sigma, w);
        dim3 grid2((g.N + 255) / 256, g.B);
        hipLaunchKernelGGL(k_flags, grid2, dim3(256), 0, st, g, w);
    }
    if (a.ops_begin) (void)hipEventRecord(a.ops_begin, st);
    if (lc.bs == 64 && lc.spt == 1) launch_ops<64, 1>(g, w, a.mu, a.sigma, st);
    else if (lc.bs == 256 && lc.spt == 1) launch_ops<256, 1>(g, w, a.mu, a.sigma, st);
    else if (lc.bs == 256 && lc.spt == 4) launch_ops<256, 4>(g, w, a.mu, a.sigma, st);
    else return hipErrorInvalidValue;
    if (a.ops_end) (void)hipEventRecord(a.ops_end, st);
    if (pa.enabled) {
        if (a.poly_begin) (void)hipEventRecord(a.poly_begin, st);
        const size_t lds = sizeof(float) * (size_t)kPolyWaves * 8 * pa.SP;
        const dim3 grid(g.ngroups * pa.split, g.B), block(64 * kPolyWaves);
        switch ((pa.SP + 63) / 64) {
        case 1: hipLaunchKernelGGL(k_poly<1>, grid, block, lds, st, g, pa, a.mu, a.sigma, w); break;
        case 2: hipLaunchKernelGGL(k_poly<2>, grid, block, lds, st, g, pa, a.mu, a.sigma, w); break;
        case 3: hipLaunchKernelGGL(k_poly<3>, grid, block, lds, st, g, pa, a.mu, a.sigma, w); break;
        case 4: hipLaunchKernelGGL(k_poly<4>, grid, block, lds, st, g, pa, a.mu, a.sigma, w); break;
        case kStripPassesMax: hipLaunchKernelGGL(k_poly<kStripPassesMax>, grid, block, lds, st, g, pa, a.mu, a.sigma, w); break;
        default: return hipErrorInvalidValue;
        }
        if (a.poly_end) (void)hipEventRecord(a.poly_end, st);
    }
    if (g.nb > 0) {
        if (lc.bs == 64) launch_back<64, 1>(g, w, a.mu, a.sigma, st);
        else if (lc.spt == 1) launch_back<256, 1>(g, w, a.mu, a.sigma, st);
        else launch_back<256, 4>(g, w, a.mu, a.sigma, st);
    }
    if (pa.enabled)
        hipLaunchKernelGGL(k_ucoef, dim3((pa.nc * kNC + pa.SP + 63) / 64, g.K, g.B), dim3(256), 0, st, g, pa, w);
    hipLaunchKernelGGL(k_usage, dim3((g.T + kUsageBS - 1) / kUsageBS, g.K, g.B), dim3(kUsageBS), 0, st, g, pa, w);
    hipLaunchKernelGGL(k_vres, dim3(g.K, g.B), dim3(kTermsBS), 0, st, g, w, hp);
    hipLaunchKernelGGL(k_combine, dim3(g.B), dim3(kCombineBS), 0, st, g, pa, w, hp, a.lambda_in,
                       a.mode == 1 ? a.lambda_out : nullptr, a.mode == 1 ? a.adam_t : nullptr,
                       a.terms_out);
    if (hp.beta != 0.0f) {   // gradient of the smooth peak usage
        const dim3 gops(g.ngroups, g.ntiles, g.B);
        if (lc.bs == 64) hipLaunchKernelGGL((k_lse_ops<64, 1>), gops, dim3(64), 0, st, g, a.mu, a.sigma, w);
        else if (lc.spt == 1) hipLaunchKernelGGL((k_lse_ops<256, 1>), gops, dim3(256), 0, st, g, a.mu, a.sigma, w);
        else hipLaunchKernelGGL((k_lse_ops<256, 4>), gops, dim3(256), 0, st, g, a.mu, a.sigma, w);
        if (pa.enabled) {
            hipLaunchKernelGGL(k_lse_mom, dim3(pa.nc + 1, g.K, g.B), dim3(256), 0, st, g, pa, w);
            const dim3 grid(g.ngroups * pa.split, g.B), block(64 * kPolyWaves);
            switch ((pa.SP + 63) / 64) {
            case 1: hipLaunchKernelGGL(k_lse_poly<1>, grid, block, 0, st, g, pa, a.mu, a.sigma, w); break;
            case 2: hipLaunchKernelGGL(k_lse_poly<2>, grid, block, 0, st, g, pa, a.mu, a.sigma, w); break;
            case 3: hipLaunchKernelGGL(k_lse_poly<3>, grid, block, 0, st, g, pa, a.mu, a.sigma, w); break;
            case 4: hipLaunchKernelGGL(k_lse_poly<4>, grid, block, 0, st, g, pa, a.mu, a.sigma, w); break;
            case kStripPassesMax:
                hipLaunchKernelGGL(k_lse_poly<kStripPassesMax>, grid, block, 0, st, g, pa, a.mu, a.sigma, w);
                break;
            default: return hipErrorInvalidValue;
            }
        }
    }
    {
        dim3 grid((g.N + 255) / 256, g.B);
        hipLaunchKernelGGL(k_final, grid, dim3(256), 0, st, g, w, hp, a.mu, a.sigma, a.gmu, a.gsig,
                           a.mu_io, a.sig_io, a.m, a.v, a.adam_t, a.mode);
    }
    return hipGetLastError();
}

hipError_t enqueue_adam_from_grad(const Graph &g, const Work &w, const HP &hp, const float *gmu,
                                  const float *gsig, const float *terms, float *mu, float *sigma,
                                  float *m, float *v, float *lambda, int *adam_t, hipStream_t st) {
    hipLaunchKernelGGL(k_lambda_from_terms, dim3((g.B + 255) / 256), dim3(256), 0, st, g.B, hp,
                       terms, lambda, adam_t, w.adamf);
    dim3 grid((g.N + 255) / 256, g.B);
    hipLaunchKernelGGL(k_adam, grid, dim3(256), 0, st, g.B, g.N, hp, w.adamf, gmu, gsig, mu, sigma,
                       m, v, adam_t);
    return hipGetLastError();
}

hipError_t enqueue_legalize(const Graph &g, const Work &w, const float *mu, int *sched,
                            hipStream_t st) {
    hipLaunchKernelGGL(k_legalize, dim3(g.B), dim3(kLegBS), 0, st, g, w, mu, sched);
    return hipGetLastError();
}

}  // namespace gaus
