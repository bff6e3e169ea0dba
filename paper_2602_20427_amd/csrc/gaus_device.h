// Device-side helpers shared by the gfx950 kernels of the GauS hot path:
// the normal CDF / density, signed-tail CDF values, wave and work-group
// reductions, and the chunk-polynomial expansions.  Header-only, included by
// every kernel source.
#pragma once

#include "gaus_internal.h"
#include "gaus_erfcx_coeffs.h"

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

// Families of the relaxed start time (App. E).  Each is the CDF of a
// symmetric law of z = (v + 1/2 - mu)/sigma; the non-Gaussian ones are taken
// at u = z/c, with c matching them to the Gaussian: logistic c = sqrt(3)/pi and
// Laplace c = 1/sqrt(2) (equal variance), Cauchy c = sqrt(2 ln 2) (equal
// half-width at half maximum).  fam_tail_h<FAM>(z, tail, h) returns the tail
// P(Z > |z|) and a density factor h with density(z) = fam_k<FAM>() * h;
// fam_h<FAM>(z) returns h alone.
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kInvPi = 0.31830988618379067f;

template <int FAM>
__host__ __device__ constexpr float fam_cinv() {   // 1/c
    return FAM == 1 ? 1.81379936423421785f : FAM == 2 ? 1.41421356237309505f
         : FAM == 3 ? 0.84932180028801904f : 1.0f;
}
template <int FAM>
__host__ __device__ constexpr float fam_k() {
    return FAM == 1 ? 1.81379936423421785f    // logistic: h = e/(1+e)^2, e = exp(-|u|); k = 1/c
         : FAM == 2 ? 0.70710678118654752f    // Laplace:  h = exp(-|u|); k = 1/(2c)
         : FAM == 3 ? 0.27034752558309155f    // Cauchy:   h = 1/(1+u^2); k = 1/(pi c)
         : kInvSqrt2Pi;                       // Gaussian: h = exp(-z^2/2)
}

template <int FAM>
__device__ __forceinline__ void fam_tail_h(float z, float &tail, float &h) {
    if constexpr (FAM == 0) {
        normal_tail_pdf(z, tail, h);
    } else if constexpr (FAM == 1) {
        const float e = __builtin_amdgcn_exp2f(-fabsf(z) * (fam_cinv<1>() * kLog2e));
        const float r = __builtin_amdgcn_rcpf(1.0f + e);
        tail = e * r;                 // e/(1+e) = 1/(1+exp|u|)
        h = tail * r;
    } else if constexpr (FAM == 2) {
        const float e = __builtin_amdgcn_exp2f(-fabsf(z) * (fam_cinv<2>() * kLog2e));
        tail = 0.5f * e;
        h = e;
    } else {
        // P(U > u) = atan(1/u)/pi for u > 1 (no cancellation), 1/2 - atan(u)/pi below
        const float u = fabsf(z) * fam_cinv<3>();
        const bool far = u > 1.0f;
        const float a = atanf(far ? __builtin_amdgcn_rcpf(u) : u);
        tail = far ? a * kInvPi : fmaf(-a, kInvPi, 0.5f);
        h = __builtin_amdgcn_rcpf(fmaf(u, u, 1.0f));
    }
}

template <int FAM>
__device__ __forceinline__ float fam_h(float z) {
    if constexpr (FAM == 0) {
        return __builtin_amdgcn_exp2f(-(z * z) * kHalfLog2e);
    } else if constexpr (FAM == 1) {
        const float e = __builtin_amdgcn_exp2f(-fabsf(z) * (fam_cinv<1>() * kLog2e));
        const float r = __builtin_amdgcn_rcpf(1.0f + e);
        return e * r * r;
    } else if constexpr (FAM == 2) {
        return __builtin_amdgcn_exp2f(-fabsf(z) * (fam_cinv<2>() * kLog2e));
    } else {
        const float u = z * fam_cinv<3>();
        return __builtin_amdgcn_rcpf(fmaf(u, u, 1.0f));
    }
}

// |z| beyond which the step-by-step evaluations flush the tail and the
// density factor to exactly 0 (fam_tail_h_fl): both are below 3e-16 there
// (relative to the peak density for the factor: Gaussian e^-32, logistic
// and Laplace e^-35), far below fp32 resolution.  A CDF value is then
// exactly 0 or 1 and its derivatives exactly 0, which the spread tests below
// rely on.  The Cauchy tails never vanish.
template <int FAM>
__host__ __device__ constexpr float fam_zflush() {
    return FAM == 0 ? 8.0f       // Phi(-8) = 6.2e-16
         : FAM == 1 ? 20.0f      // exp(-20 pi/sqrt(3)) = 1.7e-16
         : FAM == 2 ? 25.0f      // exp(-25 sqrt(2))/2 = 2.0e-16
         : 3.0e38f;
}

// fam_tail_h with the far tails flushed (every step-by-step evaluation)
template <int FAM>
__device__ __forceinline__ void fam_tail_h_fl(float z, float &tail, float &g) {
    fam_tail_h<FAM>(z, tail, g);
    if constexpr (FAM != 3) {
        const bool far = fabsf(z) > fam_zflush<FAM>();
        tail = far ? 0.0f : tail;
        g = far ? 0.0f : g;
    }
}

// Bin edges [lo, hi] (clamped into [a - 1 .. b + 1]) outside which an op's CDF
// is the exact constant: 0 below lo, 1 above hi (kZF = fam_zflush of its
// family).  Widened by one step for the rounding of the float bounds; a NaN
// mean gives [a, b].
__device__ __forceinline__ void spread_z(float kZF, float mu, float rs, int a, int b, int &lo, int &hi) {
    const float w = kZF / rs, c = mu - 0.5f;
    float l = floorf(c - w) - 1.0f, h = ceilf(c + w) + 1.0f;
    l = fminf(fmaxf(l, (float)a), (float)b + 1.0f);
    h = fmaxf(fminf(h, (float)b), (float)a - 1.0f);
    lo = (int)l;
    hi = (int)h;
}

// Tiles [t0, tb) of the step-by-step op kernel that hold records: an op's
// producer-side derivatives (of F_i at u and of A(u) and F_i' at u - s) can
// be nonzero only where its spread, or the spread shifted by its delay s,
// meets the tile; the consumer-side derivatives of an edge into an op only
// where the consumer's spread does.  Elsewhere they are exactly 0: the op
// kernel writes no record there and its readers skip the tile.  (These are
// the op kernel's own spread tests, so writer and readers agree.)
__device__ __forceinline__ bool tile_prod_rec(float kZF, float mu, float rs, int s, int t0, int tb) {
    int pl, ph;
    spread_z(kZF, mu, rs, t0 - s - 1, tb, pl, ph);
    const int n1 = min(ph + 1, tb - 1) - max(pl, t0) + 1;
    const int n2 = min(ph + s, tb - 1) - max(pl + s - 1, t0) + 1;
    return n1 > 0 || n2 > 0;
}
__device__ __forceinline__ bool tile_cons_rec(float kZF, float mu, float rs, int t0, int tb) {
    int cl, ch;
    spread_z(kZF, mu, rs, t0 - 1, tb, cl, ch);
    return min(ch + 1, tb - 1) - max(cl, t0) + 1 > 0;
}

// The same with the family chosen at run time (kernels outside the inner loops).
__device__ __forceinline__ float fam_k_rt(int fam) {
    switch (fam) {
        case 1: return fam_k<1>();
        case 2: return fam_k<2>();
        case 3: return fam_k<3>();
        default: return fam_k<0>();
    }
}
__device__ __forceinline__ float fam_zflush_rt(int fam) {
    switch (fam) {
        case 1: return fam_zflush<1>();
        case 2: return fam_zflush<2>();
        case 3: return fam_zflush<3>();
        default: return fam_zflush<0>();
    }
}
__device__ __forceinline__ float fam_h_rt(int fam, float z) {
    switch (fam) {
        case 1: return fam_h<1>(z);
        case 2: return fam_h<2>(z);
        case 3: return fam_h<3>(z);
        default: return fam_h<0>(z);
    }
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
// cinv = fam_k<FAM>()/sigma, i.e. 1/(sigma sqrt(2 pi)) for the Gaussian):
// dF/dmu = -phi(z)/sigma, dF/dsigma = -phi(z) z/sigma.  Outside the interior
// edges F is the constant 0 (v < 0) or 1 (v >= D-1).
template <int FAM = 0>
__device__ __forceinline__ void cdf_at(long long v, int D, float mu, float rs, float cinv, float &st,
                                       float &Fm, float &Fs) {
    if (v < 0) { st = 0.0f; Fm = 0.0f; Fs = 0.0f; return; }
    if (v >= D - 1) { st = -0.0f; Fm = 0.0f; Fs = 0.0f; return; }
    const float z = ((float)v + 0.5f - mu) * rs;
    float tail, g;
    fam_tail_h_fl<FAM>(z, tail, g);
    st = (z >= 0.0f) ? -tail : tail;
    Fm = -g * cinv;
    Fs = Fm * z;
}

// the same for 32-bit positions (no 64-bit integer conversion)
template <int FAM = 0>
__device__ __forceinline__ void cdf_at(int v, int D, float mu, float rs, float cinv, float &st, float &Fm,
                                       float &Fs) {
    if (v < 0) { st = 0.0f; Fm = 0.0f; Fs = 0.0f; return; }
    if (v >= D - 1) { st = -0.0f; Fm = 0.0f; Fs = 0.0f; return; }
    const float z = ((float)v + 0.5f - mu) * rs;
    float tail, g;
    fam_tail_h_fl<FAM>(z, tail, g);
    st = (z >= 0.0f) ? -tail : tail;
    Fm = -g * cinv;
    Fs = Fm * z;
}

template <int FAM = 0>
__device__ __forceinline__ float st_at(long long v, int D, float mu, float rs) {
    if (v < 0) return 0.0f;
    if (v >= D - 1) return -0.0f;
    const float z = ((float)v + 0.5f - mu) * rs;
    float tail, g;
    fam_tail_h_fl<FAM>(z, tail, g);
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

// Sums over groups of 64/P consecutive lanes (P = 1, 2, 4 restarts per wave):
// rows of 16 lanes are summed by the DPP steps, then across rows inside the
// group (ds_swizzle within 32 lanes, ds_bpermute across the halves).
template <int P>
__device__ __forceinline__ float group_rows_sum(float x) {
    if constexpr (P == 1) {
        return cross_rows_sum(x);
    } else if constexpr (P == 2) {
        constexpr int kSwizzleXor16 = 0x1F | (0x10 << 10);
        return x + __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), kSwizzleXor16));
    } else {
        static_assert(P == 4, "groups of 64, 32 or 16 lanes");
        return x;
    }
}

// wave_sum4 per lane group: lane l of a group (l < 4) receives the group's
// total of value wave4_comp(l).  P = 1 is wave_sum4.
template <int P>
__device__ __forceinline__ float group_sum4(float v0, float v1, float v2, float v3, int lane) {
    const bool b0 = lane & 1, b1 = lane & 2;
    const float a = (b0 ? v2 : v0) + dpp_mov<kDppXor1>(b0 ? v0 : v2);
    const float c = (b0 ? v3 : v1) + dpp_mov<kDppXor1>(b0 ? v1 : v3);
    float x = (b1 ? c : a) + dpp_mov<kDppXor2>(b1 ? a : c);
    x += dpp_mov<kDppRor4>(x);
    x += dpp_mov<kDppRor8>(x);
    return group_rows_sum<P>(x);
}

// wave_sum2 per lane group: lane l < 2 of a group receives total l.
template <int P>
__device__ __forceinline__ float group_sum2(float v0, float v1, int lane) {
    const bool b0 = lane & 1;
    float x = (b0 ? v1 : v0) + dpp_mov<kDppXor1>(b0 ? v0 : v1);
    x += dpp_mov<kDppXor2>(x);
    x += dpp_mov<kDppRor4>(x);
    x += dpp_mov<kDppRor8>(x);
    return group_rows_sum<P>(x);
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
    static_assert(NV <= 8, "at most 8 values");
    constexpr int NW = BS / 64;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    // wave totals four and two values at a time
#pragma unroll
    for (int c = 0; c + 4 <= NV; c += 4) {
        const float r = wave_sum4(v[c], v[c + 1], v[c + 2], v[c + 3], lane);
        if (lane < 4) slot[wid][c + wave4_comp(lane)] = r;
    }
    constexpr int c2 = NV / 4 * 4;
    if constexpr (NV - c2 >= 2) {
        const float r = wave_sum2(v[c2], v[c2 + 1], lane);
        if (lane < 2) slot[wid][c2 + lane] = r;
    }
    if constexpr ((NV - c2) % 2 == 1) {
        const float r = wave_sum(v[NV - 1]);
        if (lane == 0) slot[wid][NV - 1] = r;
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



// Expansion of an op's CDF around a chunk centre, NC coefficients per vector
// (degree NC-1): T[n] = Phi^(n)(z0) r^n / n!, n < NC + kShiftTerms + 1, the
// terms the one-step shift series reach.
// NT: coefficients kept (the shift series need NC + kShiftTerms + 1; dF/dmu
// alone needs NC + 1).
template <int NC = kNC, int NT = NC + kShiftTerms + 1>
struct Expansion {
    float T[NT];                     // Taylor coefficients in y, T[0] = F(z0)
    float G0;                        // 1 - F(z0), from the tail
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

// Taylor coefficients in y of F(z0 + r y) for each family (App. E), from one
// tail/density evaluation at the chunk centre:
//   Gaussian: the Hermite recursion above;
//   logistic: F = S(q y + u0), q = r/c, S' = S (1 - S), so with the
//     coefficients of 1 - F being 1 - T_0 and -T_n,
//     (n+1) T_{n+1} = q (T_n (1 - 2 T_0) - sum_{k=1}^{n-1} T_k T_{n-k});
//   Cauchy: F' = 1/(pi (1 + u^2)) = Im(1/(u - i))/pi, whose expansion about
//     u0 is a geometric series, so T_n = -Im((-w)^n)/(pi n) with
//     w = q/(u0 - i) = q (u0 + i)/(1 + u0^2).
// 1 - T_0 is taken from the precise tail (G0), never as 1 - F.
template <int FAM = 0, int NC, int NT>
__device__ __forceinline__ void expand(float mu, float rs, float tcen, Expansion<NC, NT> &e) {
    static_assert(FAM == 0 || FAM == 1 || FAM == 3, "no chunk expansion for this family");
    constexpr int TN = NT;
    e.r = rs;
    e.z0 = (tcen + 0.5f - mu) * rs;
    float tail, g;
    fam_tail_h<FAM>(e.z0, tail, g);
    const bool up = e.z0 >= 0.0f;
    e.T[0] = up ? 1.0f - tail : tail;
    e.G0 = up ? tail : 1.0f - tail;
    e.T[1] = g * (fam_k<FAM>() * rs);
    if constexpr (FAM == 0) {
        const float zr = e.z0 * rs, r2 = rs * rs;
        e.T[2] = (zr * -0.5f) * e.T[1];
#pragma unroll
        for (int n = 2; n < TN - 1; ++n) {
            const float c1 = -1.0f / (float)(n + 1);
            const float c2 = -(float)(n - 1) / (float)(n * (n + 1));
            e.T[n + 1] = fmaf(zr * c1, e.T[n], (r2 * c2) * e.T[n - 1]);
        }
    } else if constexpr (FAM == 1) {
        const float q = rs * fam_cinv<1>();
        const float d0 = e.G0 - e.T[0];   // 1 - 2 F(z0)
#pragma unroll
        for (int n = 1; n < TN - 1; ++n) {
            // sum_{k=1}^{n-1} T_k T_{n-k}, each pair once
            float acc = 0.0f;
#pragma unroll
            for (int k = 1; 2 * k < n; ++k) acc = fmaf(e.T[k], e.T[n - k], acc);
            acc += acc;
            if (n % 2 == 0) acc = fmaf(e.T[n / 2], e.T[n / 2], acc);
            e.T[n + 1] = fmaf(e.T[n], d0, -acc) * (q * (1.0f / (float)(n + 1)));
        }
    } else {
        const float q = rs * fam_cinv<3>();
        const float qh = q * g;                          // g = 1/(1 + u0^2)
        const float wr = -qh * (e.z0 * fam_cinv<3>()), wi = -qh;   // -w
        float pr = wr, pim = wi;
#pragma unroll
        for (int n = 2; n < TN; ++n) {
            const float nr = fmaf(pr, wr, -pim * wi);
            const float ni = fmaf(pr, wi, pim * wr);
            pr = nr; pim = ni;
            e.T[n] = -pim * (kInvPi / (float)n);
        }
    }
}

template <int NC, int NT>
__device__ __forceinline__ void vec_dFdmu(const Expansion<NC, NT> &e, float (&a)[NC]) {
    static_assert(NT >= NC + 1, "dF/dmu needs NC + 1 coefficients");
#pragma unroll
    for (int k = 0; k < NC; ++k) a[k] = -(float)(k + 1) * e.T[k + 1];
}

template <int NC>
__device__ __forceinline__ void vec_times_z(const float (&a)[NC], float zc, float r, float (&o)[NC]) {
    o[0] = zc * a[0];
#pragma unroll
    for (int k = 1; k < NC; ++k) o[k] = fmaf(zc, a[k], r * a[k - 1]);
}

// The shift series take the coefficients the expansion holds (T_n, n < NT):
// with NT = NC + 1 a coefficient of degree k gets min(kShiftTerms, NC - k)
// terms, the rest being of the order of the series' own truncation.
template <int NC, int NT>
__device__ __forceinline__ void vec_mass(const Expansion<NC, NT> &e, float (&m)[NC]) {
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        float acc = 0.0f;
#pragma unroll
        for (int j = kShiftTerms; j >= 1; --j)
            if (k + j < NT) acc = fmaf(mass_coef(k, j), e.T[k + j], acc);
        m[k] = acc;
    }
}

template <int NC, int NT>
__device__ __forceinline__ void vec_dFdmu_back(const Expansion<NC, NT> &e, float (&a)[NC]) {
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        float acc = 0.0f;
#pragma unroll
        for (int j = kShiftTerms; j >= 0; --j)
            if (k + 1 + j < NT) acc = fmaf(back_coef(k, j), e.T[k + 1 + j], acc);
        a[k] = acc;
    }
}

// (H p)_k = sum_l H_{k+l} p_l; the chunk points are symmetric, odd moments
// vanish.  Only terms with k + l <= NC - 1 are kept: the dot product with a
// consumer vector q then sums p_l q_k H_{k+l} over total degree k + l <= d
// (the series degree), i.e. the product p q truncated at degree d like p and
// q themselves; the dropped terms are O(rho^(d+2)) against O(rho^(d+1)) for
// the truncation of either series.
template <int NC>
__device__ __forceinline__ void vec_moments(const float (&p)[NC], const float (&H)[kDeg + 1], float (&o)[NC]) {
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        float acc = 0.0f;
#pragma unroll
        for (int l = 0; l < NC; ++l)
            if (((k + l) & 1) == 0 && k + l <= NC - 1) acc = fmaf(H[(k + l) / 2], p[l], acc);
        o[k] = acc;
    }
}

template <int NC>
__device__ __forceinline__ float vdot(const float (&a)[NC], const float (&b)[NC]) {
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < NC; ++k) acc = fmaf(a[k], b[k], acc);
    return acc;
}

// dot with 1 - F given F's coefficients and the precise 1 - F(z0)
template <int NC, int NT>
__device__ __forceinline__ float vdot_1mF(const float (&a)[NC], const Expansion<NC, NT> &e) {
    float acc = a[0] * e.G0;
#pragma unroll
    for (int k = 1; k < NC; ++k) acc = fmaf(-a[k], e.T[k], acc);
    return acc;
}

template <int NC, int NT>
__device__ __forceinline__ float vdot_F(const float (&a)[NC], const Expansion<NC, NT> &e) {
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < NC; ++k) acc = fmaf(a[k], e.T[k], acc);
    return acc;
}

// c = a b truncated to NC coefficients (the Cauchy product of two series)
template <int NC>
__device__ __forceinline__ void poly_mul(const float (&a)[NC], const float (&b)[NC], float (&c)[NC]) {
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        float acc = 0.0f;
#pragma unroll
        for (int i = 0; i <= k; ++i) acc = fmaf(a[i], b[k - i], acc);
        c[k] = acc;
    }
}

// weight difference c(t) - c(t+1) of a per-slot table folded mod T
__device__ __forceinline__ float soft_diff(const float *sk, int t, int T) {
    return sk[t % T] - sk[(t + 1) % T];
}

}  // namespace

constexpr int kPolyWaves = 4;
constexpr int kStripPassesMax = (kStripMax + 63) / 64;
constexpr int kOpsPerWaveMax = 64;              // group size <= kPolyWaves * 64

}  // namespace gaus
