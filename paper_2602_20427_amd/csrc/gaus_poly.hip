// gfx950 kernels of the chunk-polynomial evaluation (dense regime): k_poly
// (forward terms, usage coefficients and the edge derivatives of ops whose
// width allows it) and k_lse_mom / k_lse_poly (gradient of the smooth peak
// usage for those ops).  The method is described before poly_tier in
// gaus_kernels.hip.
#include <type_traits>

#include "gaus_device.h"

namespace gaus {


constexpr int kStripExtra = 8;   // row slots past SP: [SP] = D-3, [SP+1 .. SP+4] = helper values
constexpr int kStripPad = kSmax; // zero slots before position 0 (positions -kSmax .. -1, F = 0)

// Taylor coefficients kept past the degree (the shift series' extra terms)
constexpr int kPolyExtraT = 2;

// LDS floats per (wave, restart) of k_poly: 6 rows of SP strip values and 3
// rows of SP + kStripExtra raw CDF values after kStripPad zeros; with P > 1
// rounded so that the restarts' rows start 64/P banks apart (lane c of every
// restart then reads and writes a bank of its own).
template <int P>
__host__ __device__ constexpr int row_stride(int SP) {
    const int n = 6 * SP + 3 * (kStripPad + SP + kStripExtra);
    return P == 1 ? n : n + ((64 / P - n % 64) % 64 + 64) % 64;
}

// Value of lane h*(64/P) + src (the lane holding item src of this lane's
// restart h), for P > 1; P = 1 reads lane src.
template <int P>
__device__ __forceinline__ float from_lane(float v, int src, int h) {
    if constexpr (P == 1) {
        return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), src));
    } else {
        const int addr = (h * (64 / P) + src) << 2;
        return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(addr, __builtin_bit_cast(int, v)));
    }
}

// Work-group = (op group slice, restart pack), kPolyWaves waves; each wave
// takes the slice's ops in turn.  P restarts of the op share the wave: lane
// = (restart h of the pack, index c < 64/P); for each restart, lanes = strip
// positions for the step-by-step part and lanes = chunks of grid GI for the
// polynomial part; per polynomial out-edge the consumer-side derivatives of
// both parts are reduced together over the restart's lanes.
// NP: strip passes of 64/P lanes, ceil(SP / (64/P)).
//
// Strip values are evaluated once per position and shared between lanes
// through per-(wave, restart) LDS rows: CDF values one step back (for the
// masses) and Lat steps back (for the delay-shifted functions) are read from
// the lanes that own those positions.  Position D-1 has the constant F = 1,
// so its lane evaluates D-3 instead (the step before D-2, the first position
// of the upper segment); the shifted values of the two upper positions and,
// for Lat = 0, the value at L0 come from one more evaluation on four lanes.
// One work-group of grid GI: (bx, by) = (op group slice, restart pack); sUc,
// sGs: the work-group's LDS for the chunk coefficients and the edge sums.
template <int NP, int FAM, int P>
__device__ __forceinline__ void poly_wg(const Graph &G, const PolyArgs &pa, const float *__restrict__ mu,
                                        const float *__restrict__ sigma, const Work &W, int bx, int by,
                                        float (*sUc)[64][kNC], float (*sGs)[kPackMax][2]) {
    static_assert(P == 1 || NP == 1, "packed grids: one strip pass");
    static_assert(P <= kPackMax, "restart pack");
    constexpr int GI = P == 1 ? 0 : P == 2 ? 1 : 2;   // grid
    constexpr int L = 64 / P;                          // lanes per restart
    const GridArgs &gd = pa.gr[GI];
    const int split = gd.split;
    const int grp = bx / split, sub = bx - grp * split;
    const int N = G.N, D = G.D, B = G.B;
    // no op of the group on this grid (in every restart of the pack): nothing
    // to write, the readers skip the group
    if (!(W.gbits[(size_t)by * P * G.ngroups + grp] & (kGbGrid << GI))) return;
    // dynamic LDS: per (wave, restart) 6 rows of SP strip values and 3 rows of
    // SP + kStripExtra raw CDF values, then per (wave, restart) SP strip usages
    extern __shared__ float sDyn[];
    const int SP = gd.SP, L0 = gd.L0;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int h = P == 1 ? 0 : lane / L, c = P == 1 ? lane : lane % L;
    const int b0 = by * P, bh = b0 + h;    // this lane's restart
    const bool hact = P == 1 || bh < B;
    const bool cact = hact && c < gd.nc;
    const float tcen = (float)(L0 + c * gd.W) + gd.lam;
    // per-work-group output slot of restart b
    auto slot_of = [&](int b) { return (size_t)gd.slot_base + ((size_t)b * G.ngroups + grp) * split + sub; };

    float uc[kNC];
#pragma unroll
    for (int k = 0; k < kNC; ++k) uc[k] = 0.0f;
    float us[NP];
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) us[ps] = 0.0f;
    const int SPX = kStripPad + SP + kStripExtra;
    const int RS = row_stride<P>(SP);
    float *own = sDyn + (size_t)(wv * P + h) * RS;
    float *rSt = own + 6 * SP + kStripPad, *rFm = rSt + SPX, *rFs = rFm + SPX;
    float *sUs = sDyn + (size_t)kPolyWaves * P * RS;
    if (c < kStripPad) {   // never overwritten: positions before 0 have F = 0, dF = 0
        rSt[c - kStripPad] = 0.0f; rFm[c - kStripPad] = 0.0f; rFs[c - kStripPad] = 0.0f;
    }

    // the work-group's ops are q = q0 + sub + split*j; this wave's are
    // j = wv + kPolyWaves*l (at most 16, as split keeps 64 ops per work-group):
    // lane l < nq loads op l's restart-independent data, lane h*(64/P) + l its
    // mean and 1/sigma in restart h of the pack
    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    const int nj = (q1 - q0 - sub + split - 1) / split;
    const int nq = (nj - wv + kPolyWaves - 1) / kPolyWaves;
    int l_i = 0, l_cls = 0, l_mine = 0, l_s = 0, l_e0 = 0, l_e1 = 0;
    float l_mu = 0.0f, l_sg = 1.0f;   // l_sg holds 1/sigma
    if (c < nq) {
        const int i = G.perm[q0 + sub + split * (wv + kPolyWaves * c)];
        if (hact) { l_mu = mu[(size_t)bh * N + i]; l_sg = W.rsig[(size_t)bh * N + i]; }
        if (lane < nq) {
            l_i = i;
            // tier on its grid (0: step by step); every restart of a pack has the same
            l_cls = W.gtier[(size_t)b0 * N + i];
            l_mine = W.gsel[(size_t)b0 * N + i] == GI;
            l_s = G.delay[i];
            l_e0 = G.row_ptr[i]; l_e1 = G.row_ptr[i + 1];
        }
    }
    float gsum = 0.0f;  // V_dep, L_com of this wave's ops (lanes c = 0 and 2)
    // polynomial ops, one pass per degree tier (NC coefficients per vector)
    auto tier_pass = [&](auto nc_tag, int tier) {
    constexpr int NC = decltype(nc_tag)::value;
    for (int oq = 0; oq < nq; ++oq) {
        if (!__builtin_amdgcn_readlane(l_mine, oq) || __builtin_amdgcn_readlane(l_cls, oq) != tier) continue;
        const int i = __builtin_amdgcn_readlane(l_i, oq);
        float *pp = W.ppoly + ((size_t)bh * N + i) * kPP;
        const float m_i = from_lane<P>(l_mu, oq, h);
        const float rs = from_lane<P>(l_sg, oq, h);
        const float cinv = rs * fam_k<FAM>();
        const int s = __builtin_amdgcn_readlane(l_s, oq);
        const int e0 = __builtin_amdgcn_readlane(l_e0, oq), e1 = __builtin_amdgcn_readlane(l_e1, oq);
        float pr[kPP] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
        // the op's polynomial out-edges in batches of 64/P: lane h*(64/P) + l
        // loads edge l's consumer in restart h
        int x_ok = 0;
        float x_mu = 0.0f, x_sg = 1.0f;   // x_sg: 1/sigma of the consumer

        // (1) strip: own CDF values per position (raw rows), then the derived
        // rows the out-edges read: F, dF(u), A(u) = mass at u-s+1 (at u = D-1
        // instead 1 - F(u-s), the weight of the consumers' open last bin), dF(u-s)
#pragma unroll
        for (int ps = 0; ps < NP; ++ps) {
            const int p = ps * L + c;
            if (p < SP) {
                const bool last = p == SP - 1;   // position D-1: evaluates D-3
                const int u = p < L0 ? p : D - 2 + (p - L0);
                float st, Fm, Fs;
                cdf_at<FAM>(last ? D - 3 : u, D, m_i, rs, cinv, st, Fm, Fs);
                if (last) { rSt[SP] = st; st = -0.0f; Fm = 0.0f; Fs = 0.0f; }
                rSt[p] = st; rFm[p] = Fm; rFs[p] = Fs;
            }
        }
        if (c < 4) {   // D-2-s, D-1-s, D-s (upper shifted positions) and L0
            const int v = c < 3 ? D - 2 - s + c : L0;
            float st, Fm, Fs;
            cdf_at<FAM>(v, D, m_i, rs, cinv, st, Fm, Fs);
            rSt[SP + 1 + c] = st; rFm[SP + 1 + c] = Fm; rFs[SP + 1 + c] = Fs;
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int ps = 0; ps < NP; ++ps) {
            const int p = ps * L + c;
            if (p < SP) {
                const float st = rSt[p];
                const float stm1 = rSt[p == L0 ? SP : p - 1];
                us[ps] += st_mass(stm1, st);
                // positions u-s and u-s+1: lanes p-s, p-s+1 below L0 (negative
                // ones in the zero pad, L0 itself from the helper slot), helper
                // slots for the upper two
                int i0, i1;
                if (p < L0) { i0 = p - s; i1 = p - s + 1 == L0 ? SP + 4 : p - s + 1; }
                else { i0 = SP + 1 + (p - L0); i1 = i0 + 1; }
                const float st0 = rSt[i0], Fm0 = rFm[i0], Fs0 = rFs[i0], st1 = rSt[i1];
                own[0 * SP + p] = st_F(st);
                own[1 * SP + p] = rFm[p];
                own[2 * SP + p] = rFs[p];
                own[3 * SP + p] = p == SP - 1 ? st_1mF(st0) : st_mass(st0, st1);
                own[4 * SP + p] = Fm0;
                own[5 * SP + p] = Fs0;
            }
        }
        __builtin_amdgcn_wave_barrier();

        // (2) chunk: producer vectors multiplied by the chunk moments
        // (every lane: lanes past the last chunk compute finite values that the
        // out-edges below and the usage readers never use)
        float HF[NC], HFm[NC], HFs[NC], HA[NC], HFm1[NC], HFs1[NC];
        {
            Expansion<NC, NC + kPolyExtraT> ea;
            expand<FAM>(m_i, rs, tcen, ea);
            float v[NC], w[NC];
            vec_mass(ea, v);
#pragma unroll
            for (int k = 0; k < NC; ++k) uc[k] += v[k];
#pragma unroll
            for (int k = 0; k < NC; ++k) w[k] = ea.T[k];
            vec_moments(w, gd.H, HF);
            vec_dFdmu(ea, v);
            vec_moments(v, gd.H, HFm);
            vec_times_z(v, ea.z0, ea.r, w);
            vec_moments(w, gd.H, HFs);
            // shifted functions: A(u) = mass at u-s+1, dF(u-s)
            Expansion<NC, NC + kPolyExtraT> es;
            if (s != 1) expand<FAM>(m_i, rs, tcen - (float)(s - 1), es);
            const Expansion<NC, NC + kPolyExtraT> &ex = (s != 1) ? es : ea;
            vec_mass(ex, v);
            vec_moments(v, gd.H, HA);
            vec_dFdmu_back(ex, v);
            vec_moments(v, gd.H, HFm1);
            vec_times_z(v, ex.z0 - rs, ex.r, w);
            vec_moments(w, gd.H, HFs1);
        }

        // (3) polynomial out-edges
        for (int e = e0; e < e1; ++e) {
            const int eb = (e - e0) % L;
            if (eb == 0) {
                x_ok = 0;
                if (e + c < e1) {
                    const int x_j = G.col[e + c];
                    // packed ops have only polynomial consumers (every restart)
                    x_ok = P == 1 ? W.cls[(size_t)b0 * N + x_j] : 1;
                    if (hact) { x_mu = mu[(size_t)bh * N + x_j]; x_sg = W.rsig[(size_t)bh * N + x_j]; }
                }
            }
            if (!__builtin_amdgcn_readlane(x_ok, eb)) continue;  // step-by-step edge, done by k_ops
            const float m_j = from_lane<P>(x_mu, eb, h);
            const float rsj = from_lane<P>(x_sg, eb, h);
            const float cj = rsj * fam_k<FAM>();
            float cc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            // the consumer's CDF per strip position (D-1's lane evaluates D-3)
            float xst[NP], xFm[NP], xFs[NP];
#pragma unroll
            for (int ps = 0; ps < NP; ++ps) {
                const int p = ps * L + c;
                if (p < SP) {
                    const bool last = p == SP - 1;
                    const int u = p < L0 ? p : D - 2 + (p - L0);
                    cdf_at<FAM>(last ? D - 3 : u, D, m_j, rsj, cj, xst[ps], xFm[ps], xFs[ps]);
                    if (last) { rSt[SP] = xst[ps]; xst[ps] = -0.0f; xFm[ps] = 0.0f; xFs[ps] = 0.0f; }
                    rSt[p] = xst[ps];
                }
            }
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int ps = 0; ps < NP; ++ps) {
                const int p = ps * L + c;
                if (p < SP) {
                    // at u = D-1 the consumer's F = 1 and dF = 0: only
                    // pr[0] += 1 - F_i(D-1-s) remains, the rest adds zeros
                    const float stj = xst[ps], Fmj = xFm[ps], Fsj = xFs[ps];
                    const float Pj = st_mass(rSt[p == L0 ? SP : p - 1], stj);
                    const float F = own[0 * SP + p], Fm = own[1 * SP + p];
                    const float Fs = own[2 * SP + p], A = own[3 * SP + p];
                    pr[2] = fmaf(-own[4 * SP + p], Pj, pr[2]);
                    pr[3] = fmaf(-own[5 * SP + p], Pj, pr[3]);
                    const float omF = st_1mF(stj);
                    pr[0] = fmaf(A, st_F(stj), pr[0]);
                    pr[1] = fmaf(F, omF, pr[1]);
                    pr[4] = fmaf(Fm, omF, pr[4]);
                    pr[5] = fmaf(Fs, omF, pr[5]);
                    cc[0] = fmaf(A, Fmj, cc[0]);
                    cc[1] = fmaf(A, Fsj, cc[1]);
                    cc[2] = fmaf(-F, Fmj, cc[2]);
                    cc[3] = fmaf(-F, Fsj, cc[3]);
                }
            }
            if (cact) {
                Expansion<NC, NC + kPolyExtraT> ej;
                expand<FAM>(m_j, rsj, tcen, ej);
                float a[NC], v[NC];
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
            const float ct = group_sum4<P>(cc[0], cc[1], cc[2], cc[3], lane);
            if (c < kCP && hact) W.cpoly[((size_t)bh * G.E + e) * kCP + wave4_comp(c)] = ct;
        }
        const float pt4 = group_sum4<P>(pr[0], pr[1], pr[2], pr[3], lane);
        const float pt2 = group_sum2<P>(pr[4], pr[5], lane);
        if (hact) {
            if (c < 4) pp[wave4_comp(c)] = pt4;
            if (c < 2) pp[4 + c] = pt2;
        }
        gsum += pt4;   // lane c = 0: V_dep, c = 2: L_com
    }
    };
    // every degree tier: 5, 6, then 8
    tier_pass(std::integral_constant<int, kTierDeg[3] + 1>{}, 3);
    tier_pass(std::integral_constant<int, kTierDeg[2] + 1>{}, 2);
    tier_pass(std::integral_constant<int, kTierDeg[1] + 1>{}, 1);
    if (c == 0) sGs[wv][h][0] = gsum;
    if (c == 2) sGs[wv][h][1] = gsum;

    // usage of the group: combine the waves' chunk coefficients and strip values
#pragma unroll
    for (int k = 0; k < kNC; ++k) sUc[wv][lane][k] = uc[k];
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) {
        const int p = ps * L + c;
        if (p < SP) sUs[(wv * P + h) * SP + p] = us[ps];
    }
    __syncthreads();
    // entries (restart hh of the pack, chunk cc < 64/P, coefficient k)
    for (int x = threadIdx.x; x < 64 * kNC; x += 64 * kPolyWaves) {
        const int ln = x / kNC, k = x % kNC;
        const int hh = ln / L, cx = ln % L;
        if (b0 + hh >= B) continue;
        float acc = 0.0f;
#pragma unroll
        for (int w = 0; w < kPolyWaves; ++w) acc += sUc[w][ln][k];
        float *dst = W.Ucoef + slot_of(b0 + hh) * kMaxChunks * kNC + cx * kNC + k;
        *dst = acc;
    }
    if (threadIdx.x < 2 * P) {
        const int hh = threadIdx.x >> 1, v = threadIdx.x & 1;
        if (b0 + hh < B) {
            float acc = 0.0f;
#pragma unroll
            for (int w = 0; w < kPolyWaves; ++w) acc += sGs[w][hh][v];
            float *gs = W.gsum_poly + slot_of(b0 + hh) * 2 + v;
            *gs = acc;
        }
    }
    for (int x = threadIdx.x; x < P * SP; x += 64 * kPolyWaves) {
        const int hh = x / SP, p = x % SP;
        if (b0 + hh >= B) continue;
        float acc = 0.0f;
#pragma unroll
        for (int w = 0; w < kPolyWaves; ++w) acc += sUs[(w * P + hh) * SP + p];
        float *usg = W.Ustrip + slot_of(b0 + hh) * kStripMax + p;
        *usg = acc;
    }
}

// The polynomial path in one launch: the work-groups of the packed grids
// (P = 4, then P = 2) and of grid 0 (every tier) one after the other in x, so
// a grid with no op costs its early exits inside the launch, not a launch of
// its own.  Segment sizes in PolySegs (host: poly_segs).
template <int NPV, int FAM>
__global__ __launch_bounds__(64 * kPolyWaves) __attribute__((amdgpu_waves_per_eu(3)))
void k_poly(Graph G, PolyArgs pa, const float *__restrict__ mu, const float *__restrict__ sigma, Work W,
            PolySegs sg) {
    __shared__ float sUc[kPolyWaves][64][kNC];
    __shared__ float sGs[kPolyWaves][kPackMax][2];
    int x = blockIdx.x;
    if (x < sg.n[0]) {
        poly_wg<1, FAM, 4>(G, pa, mu, sigma, W, x % sg.nx[0], x / sg.nx[0], sUc, sGs);
        return;
    }
    x -= sg.n[0];
    if (x < sg.n[1]) {
        poly_wg<1, FAM, 2>(G, pa, mu, sigma, W, x % sg.nx[1], x / sg.nx[1], sUc, sGs);
        return;
    }
    x -= sg.n[1];
    poly_wg<NPV, FAM, 1>(G, pa, mu, sigma, W, x % sg.nx[2], x / sg.nx[2], sUc, sGs);
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


template <int NP, int FAM>
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
        l_mu = mu[bi]; l_sg = W.rsig[bi];   // 1/sigma
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
        const float rs = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, l_sg), oq));
        const float cinv = rs * fam_k<FAM>();
        float gm = 0.0f, gs = 0.0f;
#pragma unroll
        for (int ps = 0; ps < NP; ++ps) {
            const int p = ps * 64 + lane;
            if (p < SP) {
                const int u = p < pa.L0 ? p : D - 2 + (p - pa.L0);
                const float z = ((float)u + 0.5f - m_i) * rs;
                const float Fm = -fam_h<FAM>(z) * cinv;
                gm = fmaf(sw[ps], Fm, gm);
                gs = fmaf(sw[ps], Fm * z, gs);
            }
        }
        // the op's own degree tier (its chunk expansion meets no consumer here)
        auto chunk = [&](auto nc_tag) {
            constexpr int NC = decltype(nc_tag)::value;
            Expansion<NC, NC + 1> e;
            expand<FAM>(m_i, rs, tcen, e);
            float a[NC], v[NC], mm[NC];
            vec_dFdmu(e, a);
            vec_times_z(a, e.z0, e.r, v);
#pragma unroll
            for (int n = 0; n < NC; ++n) mm[n] = mom[n];
            gm += vdot(a, mm);
            gs += vdot(v, mm);
        };
        if (cact) {
            const int tier = __builtin_amdgcn_readlane(l_cls, oq);
            if (tier == 3) chunk(std::integral_constant<int, kTierDeg[3] + 1>{});
            else if (tier == 2) chunk(std::integral_constant<int, kTierDeg[2] + 1>{});
            else chunk(std::integral_constant<int, kTierDeg[1] + 1>{});
        }
        const float r = wave_sum2(gm, gs, lane);
        if (lane < 2) W.lpoly[((size_t)b * N + i) * 2 + lane] = r;
    }
}

// ---------------------------------------------------------------------------
// Storage term of the polynomial holders (eq:active): on a chunk the holder's
// CDF F_h and its successors' F_j are degree-8 series in the step offset, and
//   R = 1 - prod_j F_j = sum_j (prod_{k<j} F_k) (1 - F_j),   Reg_h = b_h F_h R
// are formed as truncated series products, 1 - F_j from the precise tail at
// the chunk centre, so R keeps full precision where every F_j is near 1.
// The strip positions are evaluated step by step.  Work-group = (op group,
// restart, split slot) as in k_poly; per work-group the chunk coefficients and
// strip values of its holders are summed in fp64.
// ---------------------------------------------------------------------------
template <int NP, int FAM>
__global__ __launch_bounds__(64 * kPolyWaves) void k_mem_poly_fwd(Graph G, PolyArgs pa, const float *__restrict__ mu,
                                                                  Work W) {
    __shared__ double sMc[kPolyWaves][kNC][kMaxChunks];
    __shared__ double sMs[kPolyWaves][NP * 64];
    const int SP = pa.SP, split = pa.split, L0 = pa.L0;
    const int grp = blockIdx.x / split, sub = blockIdx.x - grp * split, b = blockIdx.y;
    const size_t slot_id = ((size_t)b * G.ngroups + grp) * split + sub;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int N = G.N, D = G.D;
    const float *mub = mu + (size_t)b * N;
    const float *rsb = W.rsig + (size_t)b * N;
    const float tcen = (float)(L0 + lane * pa.W) + pa.lam;

    double mc[kNC], ms[NP];
#pragma unroll
    for (int k = 0; k < kNC; ++k) mc[k] = 0.0;
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) ms[ps] = 0.0;

    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    const int nj = (q1 - q0 - sub + split - 1) / split;
    const int nq = (nj - wv + kPolyWaves - 1) / kPolyWaves;
    int l_i = 0, l_ok = 0;
    if (lane < nq) {
        l_i = G.perm[q0 + sub + split * (wv + kPolyWaves * lane)];
        l_ok = W.mpoly[(size_t)b * N + l_i];
    }
    for (int oq = 0; oq < nq; ++oq) {
        if (!__builtin_amdgcn_readlane(l_ok, oq)) continue;
        const int i = __builtin_amdgcn_readlane(l_i, oq);
        const float m_i = mub[i], rs = rsb[i], bh = G.bmem[i];
        const int e0 = G.row_ptr[i], e1 = G.row_ptr[i + 1];
        // strip: Reg_h(u) step by step
#pragma unroll
        for (int ps = 0; ps < NP; ++ps) {
            const int p = ps * 64 + lane;
            if (p < SP) {
                const int u = p < L0 ? p : D - 2 + (p - L0);
                const float Fh = st_F(st_at<FAM>(u, D, m_i, rs));
                float Q = 1.0f, R = 0.0f;
                for (int e = e0; e < e1; ++e) {
                    const int j = G.col[e];
                    const float st = st_at<FAM>(u, D, mub[j], rsb[j]);
                    R = fmaf(Q, st_1mF(st), R);
                    Q *= st_F(st);
                }
                ms[ps] += (double)(bh * Fh * R);
            }
        }
        // chunks: truncated series products
        Expansion<kNC, kNC> eh;
        expand<FAM>(m_i, rs, tcen, eh);
        float Q[kNC], R[kNC];
#pragma unroll
        for (int k = 0; k < kNC; ++k) { Q[k] = k == 0 ? 1.0f : 0.0f; R[k] = 0.0f; }
        for (int e = e0; e < e1; ++e) {
            const int j = G.col[e];
            Expansion<kNC, kNC> ej;
            expand<FAM>(mub[j], rsb[j], tcen, ej);
            float omF[kNC], Fj[kNC], t[kNC];
#pragma unroll
            for (int k = 0; k < kNC; ++k) { omF[k] = k == 0 ? ej.G0 : -ej.T[k]; Fj[k] = ej.T[k]; }
            poly_mul(Q, omF, t);
#pragma unroll
            for (int k = 0; k < kNC; ++k) R[k] += t[k];
            poly_mul(Q, Fj, t);
#pragma unroll
            for (int k = 0; k < kNC; ++k) Q[k] = t[k];
        }
        float Fh[kNC], reg[kNC];
#pragma unroll
        for (int k = 0; k < kNC; ++k) Fh[k] = eh.T[k];
        poly_mul(Fh, R, reg);
#pragma unroll
        for (int k = 0; k < kNC; ++k) mc[k] += (double)(bh * reg[k]);
    }
    // combine the waves in a fixed order; every slot is written (zeros if the
    // work-group holds no polynomial holder)
#pragma unroll
    for (int k = 0; k < kNC; ++k) sMc[wv][k][lane] = mc[k];
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) sMs[wv][ps * 64 + lane] = ms[ps];
    __syncthreads();
    double *mcg = W.mcoef + slot_id * kMaxChunks * kNC;
    for (int x = threadIdx.x; x < kMaxChunks * kNC; x += 64 * kPolyWaves) {
        const int c = x / kNC, k = x % kNC;
        double acc = 0.0;
#pragma unroll
        for (int w = 0; w < kPolyWaves; ++w) acc += sMc[w][k][c];
        mcg[x] = acc;
    }
    double *msg = W.mstrip + slot_id * kStripMax;
    for (int p = threadIdx.x; p < kStripMax; p += 64 * kPolyWaves) {
        double acc = 0.0;
        if (p < SP) {
#pragma unroll
            for (int w = 0; w < kPolyWaves; ++w) acc += sMs[w][p];
        }
        msg[p] = acc;
    }
}


// Chunk moments of the storage softmax c(t) = gamma dL_mem/dMReg(t mod T) at
// the bin edges: mmom[c][n] = sum_y c(t_mid + y) y^n.  Work-group per (chunk,
// restart).
__global__ __launch_bounds__(256) void k_mem_mom(Graph G, PolyArgs pa, Work W) {
    __shared__ float sRed[4][kNC];
    const int c = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const float *ms = W.msoft + (size_t)b * G.T;
    float mom[kNC];
#pragma unroll
    for (int n = 0; n < kNC; ++n) mom[n] = 0.0f;
    if (tid < pa.W) {
        const int t = pa.L0 + c * pa.W + tid;
        const float y = (float)tid - pa.lam;
        float yp = ms[t % G.T];
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
        W.mmom[((size_t)b * kMaxChunks + c) * kNC + tid] = (sRed[0][tid] + sRed[1][tid]) + (sRed[2][tid] + sRed[3][tid]);
}

// Gradient of gamma L_mem for the polynomial holders, c(t) as above:
//   holder h:      sum_t c(t) b_h R_h(t) dF_h(t)
//   successor j:  -sum_t c(t) b_h F_h(t) prod_{k != j} F_k(t) dF_j(t)
// (dF = dF/dmu or dF/dsigma).  Chunks: the products as truncated series,
// dotted with the chunk moments; strip: step by step.  DEG successors.
template <int DEG, int NP, int FAM>
__device__ __forceinline__ void mem_poly_holder(const Graph &G, const PolyArgs &pa, const Work &W, int b, int h,
                                                int e0, const float *mub, const float *rsb, const float *ms,
                                                const float (&cm)[kNC], bool cact, float tcen, int lane) {
    const int SP = pa.SP, L0 = pa.L0, D = G.D, T = G.T;
    const float m_h = mub[h], rs_h = rsb[h], bh = G.bmem[h];
    const float cinv_h = rs_h * fam_k<FAM>();
    float mj[DEG], rj[DEG];
#pragma unroll
    for (int q = 0; q < DEG; ++q) {
        const int j = G.col[e0 + q];
        mj[q] = mub[j]; rj[q] = rsb[j];
    }
    float own[2] = {0.0f, 0.0f}, sc[DEG][2];
#pragma unroll
    for (int q = 0; q < DEG; ++q) { sc[q][0] = 0.0f; sc[q][1] = 0.0f; }
    // strip, step by step
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) {
        const int p = ps * 64 + lane;
        if (p < SP) {
            const int u = p < L0 ? p : D - 2 + (p - L0);
            const float c = u <= D - 2 ? ms[u % T] : 0.0f;
            float st, Fm, Fs;
            cdf_at<FAM>(u, D, m_h, rs_h, cinv_h, st, Fm, Fs);
            const float Fh = st_F(st);
            float F[DEG], Fmj[DEG], Fsj[DEG];
            float Q = 1.0f, R = 0.0f;
#pragma unroll
            for (int q = 0; q < DEG; ++q) {
                float sj;
                cdf_at<FAM>(u, D, mj[q], rj[q], rj[q] * fam_k<FAM>(), sj, Fmj[q], Fsj[q]);
                F[q] = st_F(sj);
                R = fmaf(Q, st_1mF(sj), R);
                Q *= F[q];
            }
            const float wr = c * bh * R;
            own[0] = fmaf(wr, Fm, own[0]);
            own[1] = fmaf(wr, Fs, own[1]);
            const float wf = -c * bh * Fh;
#pragma unroll
            for (int q = 0; q < DEG; ++q) {
                float others = 1.0f;
#pragma unroll
                for (int k = 0; k < DEG; ++k) others *= (k == q) ? 1.0f : F[k];
                sc[q][0] = fmaf(wf * others, Fmj[q], sc[q][0]);
                sc[q][1] = fmaf(wf * others, Fsj[q], sc[q][1]);
            }
        }
    }
    // chunks
    if (cact) {
        Expansion<kNC, kNC + 1> eh;
        expand<FAM>(m_h, rs_h, tcen, eh);
        float T_[DEG][kNC + 1], G0[DEG], Z0[DEG];
#pragma unroll
        for (int q = 0; q < DEG; ++q) {
            Expansion<kNC, kNC + 1> ej;
            expand<FAM>(mj[q], rj[q], tcen, ej);
#pragma unroll
            for (int k = 0; k <= kNC; ++k) T_[q][k] = ej.T[k];
            G0[q] = ej.G0; Z0[q] = ej.z0;
        }
        // R = 1 - prod F_j (from the precise tails), own gradient
        float Q[kNC], R[kNC], t[kNC];
#pragma unroll
        for (int k = 0; k < kNC; ++k) { Q[k] = k == 0 ? 1.0f : 0.0f; R[k] = 0.0f; }
#pragma unroll
        for (int q = 0; q < DEG; ++q) {
            float omF[kNC], Fq[kNC];
#pragma unroll
            for (int k = 0; k < kNC; ++k) { omF[k] = k == 0 ? G0[q] : -T_[q][k]; Fq[k] = T_[q][k]; }
            poly_mul(Q, omF, t);
#pragma unroll
            for (int k = 0; k < kNC; ++k) R[k] += t[k];
            poly_mul(Q, Fq, t);
#pragma unroll
            for (int k = 0; k < kNC; ++k) Q[k] = t[k];
        }
        float a[kNC], v[kNC];
        vec_dFdmu(eh, a);
        vec_times_z(a, eh.z0, eh.r, v);
        poly_mul(R, a, t);
        own[0] += bh * vdot(t, cm);
        poly_mul(R, v, t);
        own[1] += bh * vdot(t, cm);
        // successors: W_q = b_h F_h prod_{k != q} F_k, times dF_q
        float Fh[kNC];
#pragma unroll
        for (int k = 0; k < kNC; ++k) Fh[k] = eh.T[k];
#pragma unroll
        for (int q = 0; q < DEG; ++q) {
            float Wq[kNC];
#pragma unroll
            for (int k = 0; k < kNC; ++k) Wq[k] = Fh[k];
#pragma unroll
            for (int k = 0; k < DEG; ++k) {
                if (k == q) continue;
                float Fk[kNC];
#pragma unroll
                for (int n = 0; n < kNC; ++n) Fk[n] = T_[k][n];
                poly_mul(Wq, Fk, t);
#pragma unroll
                for (int n = 0; n < kNC; ++n) Wq[n] = t[n];
            }
#pragma unroll
            for (int k = 0; k < kNC; ++k) a[k] = -(float)(k + 1) * T_[q][k + 1];
            vec_times_z(a, Z0[q], rj[q], v);
            poly_mul(Wq, a, t);
            sc[q][0] -= bh * vdot(t, cm);
            poly_mul(Wq, v, t);
            sc[q][1] -= bh * vdot(t, cm);
        }
    }
    const float r = wave_sum2(own[0], own[1], lane);
    if (lane < 2) W.mopoly[((size_t)b * G.N + h) * 2 + lane] = r;
#pragma unroll
    for (int q = 0; q < DEG; ++q) {
        const float rq = wave_sum2(sc[q][0], sc[q][1], lane);
        if (lane < 2) W.mspoly[((size_t)b * G.E + e0 + q) * 2 + lane] = rq;
    }
}

template <int NP, int FAM>
__global__ __launch_bounds__(64 * kPolyWaves) void k_mem_poly_bwd(Graph G, PolyArgs pa, const float *__restrict__ mu,
                                                                  Work W) {
    const int split = pa.split;
    const int grp = blockIdx.x / split, sub = blockIdx.x - grp * split, b = blockIdx.y;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int N = G.N;
    const float *mub = mu + (size_t)b * N;
    const float *rsb = W.rsig + (size_t)b * N;
    const float *ms = W.msoft + (size_t)b * G.T;
    const bool cact = lane < pa.nc;
    const float tcen = (float)(pa.L0 + lane * pa.W) + pa.lam;
    float cm[kNC];
    const float *msrc = W.mmom + ((size_t)b * kMaxChunks + lane) * kNC;
#pragma unroll
    for (int n = 0; n < kNC; ++n) cm[n] = cact ? msrc[n] : 0.0f;
    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    const int nj = (q1 - q0 - sub + split - 1) / split;
    const int nq = (nj - wv + kPolyWaves - 1) / kPolyWaves;
    int l_i = 0, l_ok = 0;
    if (lane < nq) {
        l_i = G.perm[q0 + sub + split * (wv + kPolyWaves * lane)];
        l_ok = W.mpoly[(size_t)b * N + l_i];
    }
    for (int oq = 0; oq < nq; ++oq) {
        if (!__builtin_amdgcn_readlane(l_ok, oq)) continue;
        const int h = __builtin_amdgcn_readlane(l_i, oq);
        const int e0 = G.row_ptr[h], deg = G.row_ptr[h + 1] - e0;   // 1 .. kMemPolyDeg
        switch (deg) {
            case 1: mem_poly_holder<1, NP, FAM>(G, pa, W, b, h, e0, mub, rsb, ms, cm, cact, tcen, lane); break;
            case 2: mem_poly_holder<2, NP, FAM>(G, pa, W, b, h, e0, mub, rsb, ms, cm, cact, tcen, lane); break;
            case 3: mem_poly_holder<3, NP, FAM>(G, pa, W, b, h, e0, mub, rsb, ms, cm, cact, tcen, lane); break;
            default: mem_poly_holder<kMemPolyDeg, NP, FAM>(G, pa, W, b, h, e0, mub, rsb, ms, cm, cact, tcen, lane); break;
        }
    }
}


// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
hipError_t launch_poly(const Graph &g, const Work &w, const PolyArgs &pa, const float *mu, const float *sigma,
                       hipStream_t st) {
    // segments: packed grid 2 (P = 4), packed grid 1 (P = 2), grid 0; dynamic
    // LDS for the largest of them
    PolySegs sg{};
    size_t lds = sizeof(float) * (size_t)kPolyWaves * (row_stride<1>(pa.SP) + pa.SP);
    auto packed = [&](int gi, int P, auto p_tag) {
        constexpr int P_ = decltype(p_tag)::value;
        const GridArgs &gd = pa.gr[gi];
        const int s = gi == 2 ? 0 : 1;
        if (!gd.on) return;
        sg.nx[s] = g.ngroups * gd.split;
        sg.n[s] = sg.nx[s] * ((g.B + P - 1) / P);
        lds = std::max(lds, sizeof(float) * (size_t)kPolyWaves * P_ * (row_stride<P_>(gd.SP) + gd.SP));
    };
    packed(2, 4, std::integral_constant<int, 4>{});
    packed(1, 2, std::integral_constant<int, 2>{});
    sg.nx[2] = g.ngroups * pa.split;
    sg.n[2] = sg.nx[2] * g.B;
    const dim3 grid((unsigned)(sg.n[0] + sg.n[1] + sg.n[2])), block(64 * kPolyWaves);
    auto run = [&](auto fam_tag) -> hipError_t {
        constexpr int FAM = decltype(fam_tag)::value;
        switch ((pa.SP + 63) / 64) {
        case 1: hipLaunchKernelGGL((k_poly<1, FAM>), grid, block, lds, st, g, pa, mu, sigma, w, sg); break;
        case 2: hipLaunchKernelGGL((k_poly<2, FAM>), grid, block, lds, st, g, pa, mu, sigma, w, sg); break;
        case 3: hipLaunchKernelGGL((k_poly<3, FAM>), grid, block, lds, st, g, pa, mu, sigma, w, sg); break;
        case 4: hipLaunchKernelGGL((k_poly<4, FAM>), grid, block, lds, st, g, pa, mu, sigma, w, sg); break;
        case kStripPassesMax:
            hipLaunchKernelGGL((k_poly<kStripPassesMax, FAM>), grid, block, lds, st, g, pa, mu, sigma, w, sg); break;
        default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    };
    switch (pa.fam) {
    case 0: return run(std::integral_constant<int, 0>{});
    case 1: return run(std::integral_constant<int, 1>{});
    case 3: return run(std::integral_constant<int, 3>{});
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_mem_poly_fwd(const Graph &g, const Work &w, const PolyArgs &pa, const float *mu,
                               hipStream_t st) {
    const dim3 grid(g.ngroups * pa.split, g.B), block(64 * kPolyWaves);
    auto run = [&](auto fam_tag) -> hipError_t {
        constexpr int FAM = decltype(fam_tag)::value;
        switch ((pa.SP + 63) / 64) {
        case 1: hipLaunchKernelGGL((k_mem_poly_fwd<1, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        case 2: hipLaunchKernelGGL((k_mem_poly_fwd<2, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        case 3: hipLaunchKernelGGL((k_mem_poly_fwd<3, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        case 4: hipLaunchKernelGGL((k_mem_poly_fwd<4, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        case kStripPassesMax:
            hipLaunchKernelGGL((k_mem_poly_fwd<kStripPassesMax, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        default: return hipErrorInvalidValue;
        }
        return hipSuccess;
    };
    switch (pa.fam) {
    case 0: return run(std::integral_constant<int, 0>{});
    case 1: return run(std::integral_constant<int, 1>{});
    case 3: return run(std::integral_constant<int, 3>{});
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_mem_poly_bwd(const Graph &g, const Work &w, const PolyArgs &pa, const float *mu,
                               hipStream_t st) {
    hipLaunchKernelGGL(k_mem_mom, dim3(pa.nc, g.B), dim3(256), 0, st, g, pa, w);
    const dim3 grid(g.ngroups * pa.split, g.B), block(64 * kPolyWaves);
    auto run = [&](auto fam_tag) -> hipError_t {
        constexpr int FAM = decltype(fam_tag)::value;
        switch ((pa.SP + 63) / 64) {
        case 1: hipLaunchKernelGGL((k_mem_poly_bwd<1, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        case 2: hipLaunchKernelGGL((k_mem_poly_bwd<2, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        case 3: hipLaunchKernelGGL((k_mem_poly_bwd<3, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        case 4: hipLaunchKernelGGL((k_mem_poly_bwd<4, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        case kStripPassesMax:
            hipLaunchKernelGGL((k_mem_poly_bwd<kStripPassesMax, FAM>), grid, block, 0, st, g, pa, mu, w); break;
        default: return hipErrorInvalidValue;
        }
        return hipSuccess;
    };
    switch (pa.fam) {
    case 0: return run(std::integral_constant<int, 0>{});
    case 1: return run(std::integral_constant<int, 1>{});
    case 3: return run(std::integral_constant<int, 3>{});
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_lse_poly(const Graph &g, const Work &w, const PolyArgs &pa, const float *mu,
                           const float *sigma, hipStream_t st) {
    hipLaunchKernelGGL(k_lse_mom, dim3(pa.nc + 1, g.K, g.B), dim3(256), 0, st, g, pa, w);
    const dim3 grid(g.ngroups * pa.split, g.B), block(64 * kPolyWaves);
    auto run = [&](auto fam_tag) -> hipError_t {
        constexpr int FAM = decltype(fam_tag)::value;
        switch ((pa.SP + 63) / 64) {
        case 1: hipLaunchKernelGGL((k_lse_poly<1, FAM>), grid, block, 0, st, g, pa, mu, sigma, w); break;
        case 2: hipLaunchKernelGGL((k_lse_poly<2, FAM>), grid, block, 0, st, g, pa, mu, sigma, w); break;
        case 3: hipLaunchKernelGGL((k_lse_poly<3, FAM>), grid, block, 0, st, g, pa, mu, sigma, w); break;
        case 4: hipLaunchKernelGGL((k_lse_poly<4, FAM>), grid, block, 0, st, g, pa, mu, sigma, w); break;
        case kStripPassesMax:
            hipLaunchKernelGGL((k_lse_poly<kStripPassesMax, FAM>), grid, block, 0, st, g, pa, mu, sigma, w); break;
        default: return hipErrorInvalidValue;
        }
        return hipSuccess;
    };
    switch (pa.fam) {
    case 0: return run(std::integral_constant<int, 0>{});
    case 1: return run(std::integral_constant<int, 1>{});
    case 3: return run(std::integral_constant<int, 3>{});
    default: return hipErrorInvalidValue;
    }
}

}  // namespace gaus
