// gfx950 kernels of the step-by-step evaluation: every (restart, op, step)
// evaluated directly (k_ops for the forward edges, k_back for back edges,
// k_lse_ops for the gradient of the smooth peak usage).  See gaus_kernels.hip
// for the notation.
#include <type_traits>

#include "gaus_device.h"

namespace gaus {

// ---------------------------------------------------------------------------
// Op kernel.  Work-group = (op group, step tile, restart).  Its ops (all of
// one resource type) are sorted by how far their spreads reach into the tile
// (below) and taken by lane groups, by single waves, or by the row path.
// Row path: threads own steps u = t0 + k*BS + tid (k < SPT).  For each op i
// (out-degree m, delay s = Lat(v_i)):
//   * its CDF row over the tile plus a left halo of s steps goes to LDS; the
//     mass P_i^u is added to the group's usage;
//   * for each out-edge (i -> j) the consumer's CDF and density factor are
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
// Narrow ops.  An op's CDF is the exact constant 0 below and 1 above the
// bin edges where |z| <= fam_zflush, so an edge i -> j varies over a tile only
// near the two ops' spreads and the horizon's ends; elsewhere each summand
// above is 0, except F_i(u)(1 - F_j(u)) = 1 between the spreads (i done, j
// not started).  When these spreads are short, a lane group takes the op (a
// quarter of a wave when every spread has at most kTinySpan steps, half a
// wave up to kMidSpan, else the whole wave): it evaluates every summand on
// the steps where one may vary
// (the spread of F_i(u), that of A(u) and F_i'(u-s), that of F_j(u), and the
// steps 0, s-1, D-2, D-1) and counts the steps between the spreads, with no
// work-group barrier.  Wider ops take a wave each (wide_ops below) when their
// consumers' spreads cover less than half the tile on average (the summands
// are then evaluated on those spreads only), else the row path above.
// When no spread meets the tile at all, every term is an integer (counts and
// the unit masses at the horizon's ends) and the op's own thread finishes it
// while the group is sorted.
constexpr int kNarrowSpan = 128;   // widest spread (in steps) on the narrow path
constexpr int kMidSpan = 64;       // widest spread of the ops taken two per wave
constexpr int kTinySpan = 16;      // widest spread of the ops taken four per wave
constexpr int kNarrowPass = 4;     // passes of a lane group over the producer's steps (2 for four per wave)

template <int FAM>
__device__ __forceinline__ void spread(float mu, float rs, int a, int b, int &lo, int &hi) {
    spread_z(fam_zflush<FAM>(), mu, rs, a, b, lo, hi);
}

// classes of an op in a step tile
enum : unsigned char { kNone = 0, kConst = 1, kTiny = 2, kNarrow = 3, kWide = 4, kMid = 5, kRow = 6, kLapU = 7 };

// A group's ops and their consumers as the op and group kernels read them,
// staged in LDS once per work-group (the consumers of at most kStage edges in
// k_group, kStageOps in k_ops, whose LDS also holds the wide ops' rows; an op
// whose edges do not fit reads them from global memory).
constexpr int kStage = 1024;
constexpr int kStageOps = 512;
struct OpStage {
    int *i, *e0, *deg, *s, *off;   // op id, first edge, out-degree, delay, first staged edge (-1: none)
    float *mu, *rs;                // mean and 1/sigma
    unsigned char *poly;           // op on the chunk-polynomial path
    float *emu, *ers;              // consumer mean and 1/sigma, per staged edge
    unsigned char *eon;            // edge on the step-by-step path
};

__device__ __forceinline__ float uniformf(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, x)));
}

// Narrow ops of class `want` from the group's list, NP at a time by each wave,
// one op per lane group of 64/NP lanes (the loads of the ops and their
// consumers overlap; loops run to the lane groups' maximum).  Its V_dep and
// L_com go to g0 and g1 of the lanes 0 and 2 of each lane group.  The usage
// goes to sU64, the work-group's row of the steps from t0 in fixed point
// (2^-40 units, integer LDS atomics: the sum does not depend on the order).
// In a step tile of the op kernel (ONE = false) the records go to the
// per-tile ppart / cpart; over the whole horizon (ONE = true, k_group) to the
// single ppoly / cpoly slots of the op and its edges.
constexpr float kUsageFix = 1099511627776.0f;   // 2^40

// Maximum over the wave of a value that is the same on every lane of each
// lane group of 64/NP lanes: one read per lane group, no cross-lane traffic.
template <int NP>
__device__ __forceinline__ int group_max(int v) {
    int m = __builtin_amdgcn_readlane(v, 0);
#pragma unroll
    for (int k = 1; k < NP; ++k) m = max(m, __builtin_amdgcn_readlane(v, k * (64 / NP)));
    return m;
}
template <int FAM, int NP, int BS, bool ONE = false>
__device__ __forceinline__ void narrow_ops(const Graph &G, const Work &W, const float *__restrict__ mub,
                                           const float *__restrict__ rsb, const unsigned char *__restrict__ clsb,
                                           const OpStage &st, const unsigned char *sCls, const int *sDirect,
                                           long long *sU64, unsigned char want, int nq, int t0, int tb,
                                           int tile, int b, float &g0, float &g1) {
    constexpr int NW = BS / 64, GL = 64 / NP;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int grl = lane / GL, gl = lane % GL;   // lane group, lane in the group
    const int D = G.D, N = G.N;
    // lane groups run their edge loops to the longest: ops are taken in
    // bins of similar step-by-step out-degree (NP > 1)
    constexpr int NBIN = NP > 1 ? 3 : 1;
    for (int pass = 0; pass < (nq + 64 * NW - 1) / (64 * NW) * NBIN; ++pass) {
        const int base = pass / NBIN * 64 * NW, bin = pass % NBIN;
        const int xl = base + lane * NW + w;
        bool sel = xl < nq && sCls[xl] == want;
        if (NBIN > 1 && sel) {
            const int md = sDirect[xl] - 1;
            sel = (md <= 1 ? 0 : md <= 3 ? 1 : 2) == bin;
        }
        unsigned long long todo = __ballot(sel);
        while (todo) {
            int myl = -1;
            for (int k = 0; k < NP && todo; ++k) {
                const int l = __builtin_ctzll(todo);
                todo &= todo - 1;
                if (grl == k) myl = l;
            }
            const bool ok = myl >= 0;
            const int x = base + myl * NW + w;   // the op's index in the work-group's list
            int i = 0, e0 = 0, e1 = 0, m = 0, s = 0, off = -1;
            float m_i = 0.0f, rs = 1.0f;
            bool poly_i = false;
            if (ok) {
                i = st.i[x]; e0 = st.e0[x]; e1 = e0 + st.deg[x];
                poly_i = st.poly[x] != 0;
                m = sDirect[x] - 1;
                m_i = st.mu[x]; rs = st.rs[x];
                s = st.s[x]; off = st.off[x];
            }
            const float cinv = rs * fam_k<FAM>();
            int pl, ph;   // F_i is read at the bin edges u - s .. u (u in the tile)
            spread<FAM>(m_i, rs, t0 - s - 1, tb, pl, ph);
            // steps where F_i(u), F_i'(u) or P_i^u may vary (X1), and where
            // A(u) or F_i'(u-s) may (X2)
            const int x1l = max(pl, t0), x1h = min(ph + 1, tb - 1);
            const int x2l = max(pl + s - 1, t0), x2h = min(ph + s, tb - 1);
            const int n1 = ok ? max(x1h - x1l + 1, 0) : 0, n2 = ok ? max(x2h - x2l + 1, 0) : 0;

            // usage: P_i^u = F_i(u) - F_i(u-1) is 0 off X1 but at u = 0 and D-1
            const int nu = (ok && !poly_i) ? n1 + 2 : 0;
            const int nu_max = group_max<NP>(nu);
            for (int x0 = 0; x0 < nu_max; x0 += GL) {
                const int xx = x0 + gl;
                int u = x1l + xx;
                bool take = xx < nu;
                if (take && xx >= n1) {
                    u = xx == n1 ? 0 : D - 1;
                    take = u >= t0 && u < tb && !(u >= x1l && u <= x1h) && !(xx > n1 && u == 0);
                }
                const float P = take ? st_mass(st_at<FAM>(u - 1, D, m_i, rs), st_at<FAM>(u, D, m_i, rs)) : 0.0f;
                if (take)
                    atomicAdd(reinterpret_cast<unsigned long long *>(sU64 + (u - t0)),
                              (unsigned long long)__float2ll_rn(P * kUsageFix));
            }

            // F_i off its spread (every step of the tile outside X1 u X2 sees
            // F_i(u), A(u) and the tail 1 - F_i(D-1-s) only through it)
            auto Fc = [&](int v) { return v < 0 ? 0 : (v >= D - 1 || v > ph) ? 1 : 0; };
            // Producer values on X1 and X2 \ X1, the same steps for every
            // out-edge: kNarrowPass passes of GL lanes (x < n1: X1; then X2,
            // less the steps of X1).  At u = D-1 the A slot holds 1 - F_i(D-1-s).
            constexpr int R = NP == 4 ? 2 : kNarrowPass;
            static_assert(R * GL >= 2 * (NP == 1 ? kNarrowSpan : NP == 2 ? kMidSpan : kTinySpan),
                          "passes cover X1 and X2");
            const int n12 = n1 + n2;
            const int n12_max = group_max<NP>(n12);
            float cSt[R], cFm[R], cFs[R], cA[R], cFms[R], cFss[R];
            int cu[R];
            bool cin2[R];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int xx = r * GL + gl;
                int u = xx < n1 ? x1l + xx : x2l + (xx - n1);
                const bool in1 = u >= x1l && u <= x1h, in2 = u >= x2l && u <= x2h;
                const bool take = xx < n12 && (xx < n1 || !in1);
                cu[r] = take ? u : -1;
                cin2[r] = take && in2;
                cSt[r] = 0.0f; cFm[r] = 0.0f; cFs[r] = 0.0f; cA[r] = 0.0f; cFms[r] = 0.0f; cFss[r] = 0.0f;
                if (r * GL >= n12_max || !take) continue;
                if (in1) cdf_at<FAM>(u, D, m_i, rs, cinv, cSt[r], cFm[r], cFs[r]);
                else cSt[r] = Fc(u) ? -0.0f : 0.0f;
                if (in2) {
                    float st0;
                    cdf_at<FAM>(u - s, D, m_i, rs, cinv, st0, cFms[r], cFss[r]);
                    cA[r] = u < D - 1 ? st_mass(st0, st_at<FAM>(u - s + 1, D, m_i, rs)) : st_1mF(st0);
                } else {
                    cA[r] = (float)(u < D - 1 ? Fc(u - s + 1) - Fc(u - s) : 1 - Fc(D - 1 - s));
                }
            }

            float pr[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
            int cnt = 0;   // steps between the spreads, summed over the edges
            const int deg = ok ? e1 - e0 : 0;
            const int deg_max = group_max<NP>(deg);
            for (int t = 0; t < deg_max; ++t) {
                const int e = e0 + t;
                bool ev = t < deg;
                float m_j = 0.0f, rsj = 1.0f;
                if (ev && off >= 0) {
                    ev = st.eon[off + t] != 0;
                    m_j = st.emu[off + t]; rsj = st.ers[off + t];
                } else if (ev) {
                    const int j = G.col[e];
                    ev = !(poly_i && clsb[j]) && !G.lap_on;
                    if (ev) { m_j = mub[j]; rsj = rsb[j]; }
                }
                const float cj = rsj * fam_k<FAM>();
                int cl, ch;
                spread<FAM>(m_j, rsj, t0 - 1, tb, cl, ch);
                const int x3l = max(cl, t0), x3h = min(ch + 1, tb - 1);
                const int n3 = max(x3h - x3l + 1, 0);
                // off X3 the consumer's CDF is the exact constant cdf_at returns
                // there (0 below its spread, 1 above it and at D-1; zero
                // derivatives), so only steps of X3 evaluate it
                auto Fcj = [&](int v) { return v < 0 ? 0 : (v >= D - 1 || v > ch) ? 1 : 0; };
                // F_i(u) (1 - F_j(u)) = 1 on [r0, r1) off the evaluated steps
                const int r0 = max(t0, ph + 1), r1 = min(min(tb, D - 1), cl);
                if (ev) cnt += max(r1 - r0, 0);
                float c4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                // X1 u X2 with the cached producer values
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    if (r * GL >= n12_max) break;
                    const int u = cu[r];
                    if (!ev || u < 0) continue;
                    const bool vary = u >= x3l && u <= x3h;
                    float st_j = Fcj(u) ? -0.0f : 0.0f, Fmj = 0.0f, Fsj = 0.0f;
                    if (vary) cdf_at<FAM>(u, D, m_j, rsj, cj, st_j, Fmj, Fsj);
                    if (cin2[r]) {
                        const float dS = vary ? st_mass(st_at<FAM>(u - 1, D, m_j, rsj), st_j)
                                              : (float)(Fcj(u) - Fcj(u - 1));
                        pr[2] = fmaf(-cFms[r], dS, pr[2]);
                        pr[3] = fmaf(-cFss[r], dS, pr[3]);
                    }
                    if (u < D - 1) {
                        const float Fi = st_F(cSt[r]), Rj = st_1mF(st_j);
                        pr[0] = fmaf(cA[r], st_F(st_j), pr[0]);
                        pr[1] += fmaf(Fi, Rj, (u >= r0 && u < r1) ? -1.0f : 0.0f);
                        pr[4] = fmaf(cFm[r], Rj, pr[4]);
                        pr[5] = fmaf(cFs[r], Rj, pr[5]);
                        c4[0] = fmaf(cA[r], Fmj, c4[0]);
                        c4[1] = fmaf(cA[r], Fsj, c4[1]);
                        c4[2] = fmaf(-Fi, Fmj, c4[2]);
                        c4[3] = fmaf(-Fi, Fsj, c4[3]);
                    } else {
                        pr[0] += cA[r];   // 1 - F_i(D-1-s)
                    }
                }
                // X3 \ (X1 u X2), then the steps 0, s-1, D-2, D-1 off all three:
                // F_i is constant there (no producer derivatives)
                const int ntot = ev ? n3 + 4 : 0;
                const int ntot_max = group_max<NP>(ntot);
                for (int x0 = 0; x0 < ntot_max; x0 += GL) {
                    const int xx = x0 + gl;
                    int u;
                    bool take = xx < ntot;
                    if (xx < n3) {
                        u = x3l + xx;
                        take = take && !(u >= x1l && u <= x1h) && !(u >= x2l && u <= x2h);
                    } else {
                        const int k = xx - n3;
                        u = k == 0 ? 0 : k == 1 ? s - 1 : k == 2 ? D - 2 : D - 1;
                        take = take && u >= t0 && u < tb && !(u >= x1l && u <= x1h) && !(u >= x2l && u <= x2h) &&
                               !(u >= x3l && u <= x3h) && !(k >= 1 && u == 0) && !(k >= 2 && u == s - 1) &&
                               !(k == 3 && u == D - 2);
                    }
                    if (!take) continue;
                    float st_j = Fcj(u) ? -0.0f : 0.0f, Fmj = 0.0f, Fsj = 0.0f;   // the four steps: off X3
                    if (xx < n3) cdf_at<FAM>(u, D, m_j, rsj, cj, st_j, Fmj, Fsj);
                    if (u < D - 1) {
                        const float Fi = (float)Fc(u), A = (float)(Fc(u - s + 1) - Fc(u - s));
                        const float Rj = st_1mF(st_j);
                        pr[0] = fmaf(A, st_F(st_j), pr[0]);
                        pr[1] += fmaf(Fi, Rj, (u >= r0 && u < r1) ? -1.0f : 0.0f);
                        c4[0] = fmaf(A, Fmj, c4[0]);
                        c4[1] = fmaf(A, Fsj, c4[1]);
                        c4[2] = fmaf(-Fi, Fmj, c4[2]);
                        c4[3] = fmaf(-Fi, Fsj, c4[3]);
                    } else {
                        pr[0] += (float)(1 - Fc(D - 1 - s));   // 1 - F_i(D-1-s)
                    }
                }
                const float r = group_sum4<NP>(c4[0], c4[1], c4[2], c4[3], lane);
                if (ev && gl < 4) {
                    if constexpr (ONE) W.cpoly[((size_t)b * G.E + e) * kCP + wave4_comp(gl)] = r;
                    else W.cpart[(((size_t)b * G.E + e) * G.ntiles + tile) * kCP + wave4_comp(gl)] = r;
                }
            }
            if (gl == 0) pr[1] += (float)cnt;
            const float ra = group_sum4<NP>(pr[0], pr[1], pr[2], pr[3], lane);
            const float rb = group_sum2<NP>(pr[4], pr[5], lane);
            if (ok) {
                float *pp = ONE ? W.ppoly + ((size_t)b * N + i) * kPP
                                : W.ppart + (((size_t)b * N + i) * G.ntiles + tile) * kPP;
                if (gl < 4) pp[wave4_comp(gl)] = m > 0 ? ra : 0.0f;
                if (gl < 2) pp[4 + gl] = m > 0 ? rb : 0.0f;
                if (m > 0 && gl == 0) g0 += ra;   // V_dep (component 0 at lane 0 of the group)
                if (m > 0 && gl == 2) g1 += ra;   // L_com (component 1 at lane 2)
            }
        }
    }
}

// Wide ops (a spread past kNarrowSpan steps in the tile): one wave per op,
// lanes over steps, no work-group barrier.  The producer's signed-tail CDF on
// the positions of its spread within [t0 - kWideHalo - 1, tb] goes to the wave's
// LDS row once (positions below it are evaluated directly).  For each
// step-by-step out-edge (i -> j), the summands are evaluated one by one only
// on X3 (the tile's steps where F_j(u) or F_j(u) - F_j(u-1) may vary: the
// consumer's spread and the step after it) and at u = D-1.  Off X3, F_j is
// the exact constant 0 (below) or 1 (above), so
//   * below X3 the summands of L_com and dLcom/dth_i are F_i(u) and F_i'(u)
//     (sums over the producer's row, densities recomputed from z), those of
//     V_dep and dVdep/dth_i are 0;
//   * above X3 the summands A(u) of V_dep add up to F_i(b - s) - F_i(a - s)
//     over [a, b) (a telescoping sum), the others are 0;
//   * the consumer-side derivatives are 0.
// The usage of an op off the polynomial path goes to the fixed-point row sU64.
constexpr int kWideHalo = 8;   // producer positions held below the tile start (delays up to this)
constexpr float kGsumFix = 4294967296.0f;   // 2^32

template <int FAM>
__device__ __forceinline__ float dens_at(int v, int D, float z) {   // density factor, 0 where cdf_at's is
    const bool off = v < 0 || v >= D - 1 || (FAM != 3 && fabsf(z) > fam_zflush<FAM>());
    return off ? 0.0f : fam_h<FAM>(z);
}

// cdf_at without branches (both sides are evaluated, then selected)
template <int FAM>
__device__ __forceinline__ void cdf_sel(int v, int D, float mu, float rs, float cinv, float &st, float &Fm,
                                        float &Fs) {
    const float z = ((float)v + 0.5f - mu) * rs;
    float tail, g;
    fam_tail_h_fl<FAM>(z, tail, g);
    const bool lo = v < 0, hi = v >= D - 1;
    st = hi ? -0.0f : lo ? 0.0f : (z >= 0.0f ? -tail : tail);
    Fm = (lo || hi) ? 0.0f : -g * cinv;
    Fs = (lo || hi) ? 0.0f : Fm * z;
}
template <int FAM>
__device__ __forceinline__ float st_sel(int v, int D, float mu, float rs) {
    const float z = ((float)v + 0.5f - mu) * rs;
    float tail, g;
    fam_tail_h_fl<FAM>(z, tail, g);
    return v >= D - 1 ? -0.0f : v < 0 ? 0.0f : (z >= 0.0f ? -tail : tail);
}

template <int FAM, int BS, int RS>
__device__ __forceinline__ void wide_ops(const Graph &G, const Work &W, const float *__restrict__ mub,
                                         const float *__restrict__ rsb, const unsigned char *__restrict__ clsb,
                                         const OpStage &st, const int *sDirect, const int *sWide, int nWide,
                                         int *sNext, float *sRows, long long *sU64, long long *sG64, int t0,
                                         int tb, int tile, int b) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int D = G.D, N = G.N;
    float *row = sRows + w * RS;          // positions rb .. rb + RS - 1
    const int rb = t0 - kWideHalo - 1;
    // the waves take the next op of the list as they come free (the results
    // do not depend on which wave takes which: per-op records, fixed-point sums)
    while (true) {
        int kk = 0;
        if (lane == 0) kk = atomicAdd(sNext, 1);
        kk = __shfl(kk, 0, 64);
        if (kk >= nWide) break;
        const int x = uniform(sWide[kk]);
        const int i = uniform(st.i[x]), e0 = uniform(st.e0[x]), deg = uniform(st.deg[x]);
        const bool poly_i = uniform(st.poly[x]) != 0;
        const int m = uniform(sDirect[x] - 1), s = uniform(st.s[x]), off = uniform(st.off[x]);
        const float m_i = uniformf(st.mu[x]), rs = uniformf(st.rs[x]);
        const float cinv = rs * fam_k<FAM>();
        int pl, ph;   // F_i is read at the bin edges u - s - 1 .. u (u in the tile)
        spread<FAM>(m_i, rs, t0 - s - 1, tb, pl, ph);
        const int R0 = max(pl, rb), R1 = min(ph, tb);       // held in the row (s <= kWideHalo)
        __asm__ volatile("" ::: "memory");   // the previous op's reads of the row come first
        for (int v = R0 + lane; v <= R1; v += 64) row[v - rb] = st_sel<FAM>(v, D, m_i, rs);
        __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // a wave's LDS accesses complete in order
        auto stv = [&](int v) {   // signed tail of F_i at bin edge v in [t0 - s - 1, tb]
            const float r = row[min(max(v - rb, 0), RS - 1)];
            const float c = (v >= 0 && (v >= D - 1 || v > ph)) ? -0.0f : 0.0f;   // off the spread
            return (v >= R0 && v <= R1) ? r : c;
        };

        // usage P_i^u: 0 off the spread X1 but at u = 0 and D-1
        if (!poly_i) {
            const int x1l = max(pl, t0), x1h = min(ph + 1, tb - 1);
            const int n1 = max(x1h - x1l + 1, 0);
            for (int x0 = 0; x0 < n1 + 2; x0 += 64) {
                const int xx = x0 + lane;
                int u = x1l + xx;
                bool take = xx < n1 + 2;
                if (take && xx >= n1) {
                    u = xx == n1 ? 0 : D - 1;
                    take = u >= t0 && u < tb && !(u >= x1l && u <= x1h) && !(xx > n1 && u == 0);
                }
                if (take) {
                    const float P = st_mass(stv(u - 1), stv(u));
                    atomicAdd(reinterpret_cast<unsigned long long *>(sU64 + (u - t0)),
                              (unsigned long long)__float2ll_rn(P * kUsageFix));
                }
            }
        }

        float pr[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
        float cnt = 0.0f;   // below X3 and past the producer's spread: F_i = 1
        for (int t = 0; t < deg; ++t) {
            const int e = e0 + t;
            bool ev;
            float m_j = 0.0f, rsj = 1.0f;
            if (off >= 0) {
                ev = uniform(st.eon[off + t]) != 0;
                m_j = uniformf(st.emu[off + t]); rsj = uniformf(st.ers[off + t]);
            } else {
                const int j = uniform(G.col[e]);
                ev = !(poly_i && clsb[j]) && !G.lap_on;
                if (ev) { m_j = uniformf(mub[j]); rsj = uniformf(rsb[j]); }
            }
            if (!ev) continue;   // both ends on the polynomial path
            const float cj = rsj * fam_k<FAM>();
            int cl, ch;
            spread<FAM>(m_j, rsj, t0 - 1, tb, cl, ch);
            const int x3l = max(cl, t0), x3h = min(ch + 1, tb - 1);
            const int n3 = max(x3h - x3l + 1, 0);
            float c4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            // one step u of X3 or u = D-1, with the consumer's signed tails at
            // u and u-1 and its derivatives at u
            // (at u = D-1, F_j = 1 and F_j' = 0 make every summand but V_dep's
            // and dVdep/dth_i's vanish by themselves; V_dep takes 1 - F_i(D-1-s))
            auto term = [&](int u, float st_j, float st_jm, float Fmj, float Fsj) __attribute__((always_inline)) {
                const float dS = st_mass(st_jm, st_j);   // F_j(u) - F_j(u-1)
                const float ss0 = stv(u - s);
                const float zs = ((float)(u - s) + 0.5f - m_i) * rs;
                const float Fms = -dens_at<FAM>(u - s, D, zs) * cinv;   // F_i'(u - s)
                pr[2] = fmaf(-Fms, dS, pr[2]);
                pr[3] = fmaf(-Fms * zs, dS, pr[3]);
                const bool last = u >= D - 1;
                const float A = st_mass(ss0, stv(u - s + 1));
                const float Fi = st_F(stv(u)), Rj = st_1mF(st_j);
                const float zi = ((float)u + 0.5f - m_i) * rs;
                const float Fmi = -dens_at<FAM>(u, D, zi) * cinv;
                pr[0] = fmaf(last ? st_1mF(ss0) : A, last ? 1.0f : st_F(st_j), pr[0]);
                pr[1] = fmaf(Fi, Rj, pr[1]);
                pr[4] = fmaf(Fmi, Rj, pr[4]);
                pr[5] = fmaf(Fmi * zi, Rj, pr[5]);
                c4[0] = fmaf(A, Fmj, c4[0]);
                c4[1] = fmaf(A, Fsj, c4[1]);
                c4[2] = fmaf(-Fi, Fmj, c4[2]);
                c4[3] = fmaf(-Fi, Fsj, c4[3]);
            };
            // X3: lanes over the positions x3l - 1 .. x3h, one evaluation of
            // F_j each; the step u takes F_j(u-1) from the lane below (lane 0
            // from lane 63 of the previous pass)
            float carry = 0.0f;
            for (int x0 = 0; x0 < n3 + 1 && n3 > 0; x0 += 64) {
                const int p = x3l - 1 + x0 + lane;
                float st_j, Fmj, Fsj;
                cdf_sel<FAM>(p, D, m_j, rsj, cj, st_j, Fmj, Fsj);
                float stm = __shfl_up(st_j, 1, 64);
                if (lane == 0) stm = carry;
                carry = __shfl(st_j, 63, 64);
                if (x0 + lane >= 1 && x0 + lane <= n3) term(p, st_j, stm, Fmj, Fsj);
            }
            // u = D-1 off X3 (F_j(D-1) = 1 by the open end bin)
            if (D - 1 >= t0 && D - 1 < tb && !(D - 1 >= x3l && D - 1 <= x3h) && lane == 0)
                term(D - 1, -0.0f, st_sel<FAM>(D - 2, D, m_j, rsj), 0.0f, 0.0f);
            // below X3: u in [t0, lo), F_j(u) = 0 (u < D-1)
            const int lo = min(n3 > 0 ? x3l : (cl > tb - 1 ? tb : t0), D - 1);
            const int q0 = max(t0, pl), q1 = min(lo, ph + 1);
            float sg = 0.0f, sgz = 0.0f;
            for (int u = q0 + lane; u < q1; u += 64) {
                const float z = ((float)u + 0.5f - m_i) * rs;
                const float g = dens_at<FAM>(u, D, z);
                pr[1] += st_F(stv(u));
                sg += g;
                sgz = fmaf(g, z, sgz);
            }
            pr[4] = fmaf(-cinv, sg, pr[4]);
            pr[5] = fmaf(-cinv, sgz, pr[5]);
            cnt += (float)max(lo - max(t0, ph + 1), 0);
            // above X3: u in [a, bb), F_j(u) = 1
            const int a = n3 > 0 ? x3h + 1 : (cl > tb - 1 ? tb : t0), bb = min(tb, D - 1);
            if (lane == 0 && a < bb) pr[0] += st_mass(stv(a - s), stv(bb - s));
            const float r = wave_sum4(c4[0], c4[1], c4[2], c4[3], lane);
            if (lane < 4) W.cpart[(((size_t)b * G.E + e) * G.ntiles + tile) * kCP + wave4_comp(lane)] = r;
        }
        if (lane == 0) pr[1] += cnt;
        const float ra = wave_sum4(pr[0], pr[1], pr[2], pr[3], lane);
        const float rc = wave_sum2(pr[4], pr[5], lane);
        float *pp = W.ppart + (((size_t)b * N + i) * G.ntiles + tile) * kPP;
        if (lane < 4) pp[wave4_comp(lane)] = m > 0 ? ra : 0.0f;
        if (lane < 2) pp[4 + lane] = m > 0 ? rc : 0.0f;
        // V_dep and L_com of the work-group in fixed point (2^-32 units)
        if (m > 0 && lane == 0) atomicAdd(reinterpret_cast<unsigned long long *>(sG64),
                                          (unsigned long long)__float2ll_rn(ra * kGsumFix));
        if (m > 0 && lane == 2) atomicAdd(reinterpret_cast<unsigned long long *>(sG64 + 1),
                                          (unsigned long long)__float2ll_rn(ra * kGsumFix));
    }
}

// Usage of the wide Laplace ops (their edges are in closed form): wave w takes
// every NW-th op of the list, lane l the TILE/64 consecutive steps from
// t0 + l TILE/64.  A lane whose steps have their bin edges (one step below
// them included) all on one side of the median gets the masses from one
// evaluation and the ratio e^(-lam) per step (lam = sqrt(2)/sigma, the
// Laplace masses being geometric there): from its last step down on the
// lower side, from its first step up on the upper side, so the series runs
// from the largest value; the steps of the other lanes are evaluated one by
// one, a lane's steps at a time across the wave.  The sums go to the
// fixed-point row sU64.
template <int BS, int TILE>
__device__ __forceinline__ void lap_usage(const Graph &G, const unsigned char *sCls, const OpStage &st, int nq,
                                          int t0, int tb, long long *sU64) {
    constexpr int NW = BS / 64, L = TILE / 64;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int D = G.D;
    const int u0 = t0 + L * lane;
    float acc[L];
#pragma unroll
    for (int k = 0; k < L; ++k) acc[k] = 0.0f;
    for (int x = w; x < nq; x += NW) {
        if (uniform(sCls[x]) != kLapU) continue;
        const float m_i = uniformf(st.mu[x]), rs = uniformf(st.rs[x]);
        auto direct = [&](int u) {   // P_i^u, 0 past the tile
            return u < tb ? st_mass(st_sel<2>(u - 1, D, m_i, rs), st_sel<2>(u, D, m_i, rs)) : 0.0f;
        };
        const int ul = u0 + L - 1;
        const bool inner = u0 - 1 >= 0 && ul <= D - 2 && ul < tb;   // bin edges u0-1 .. ul interior, in the tile
        const bool below = inner && (float)ul + 0.5f - m_i < 0.0f;           // edge ul below the median
        const bool above = inner && (float)(u0 - 1) + 0.5f - m_i >= 0.0f;   // edge u0-1 at or above it
        if (below || above) {
            const float r = __builtin_amdgcn_exp2f(-1.4142135623730951f * rs * kLog2e);   // e^(-lam)
            float P = direct(below ? ul : u0);
            // (fixed register indices in both branches: an index that differs
            // between lanes would make the compiler walk the lanes)
            if (below) {
#pragma unroll
                for (int k = L - 1; k >= 0; --k) { acc[k] += P; P *= r; }
            } else {
#pragma unroll
                for (int k = 0; k < L; ++k) { acc[k] += P; P *= r; }
            }
        }
        // the other lanes' steps (the median's, the horizon ends'): every
        // step evaluated, one lane each, one such lane at a time
        unsigned long long rest = __ballot(u0 < tb && !(below || above));
        while (rest) {
            const int l = __builtin_ctzll(rest);
            rest &= rest - 1;
            const int u = t0 + L * l + lane;
            if (lane < L && u < tb)
                atomicAdd(reinterpret_cast<unsigned long long *>(sU64 + (u - t0)),
                          (unsigned long long)__float2ll_rn(direct(u) * kUsageFix));
        }
    }
#pragma unroll
    for (int k = 0; k < L; ++k)
        if (u0 + k < tb && acc[k] != 0.0f)
            atomicAdd(reinterpret_cast<unsigned long long *>(sU64 + (u0 + k - t0)),
                      (unsigned long long)__float2ll_rn(acc[k] * kUsageFix));
}

template <int FAM, int BS, int SPT>
__global__ __launch_bounds__(BS) __attribute__((amdgpu_waves_per_eu(4))) void k_ops(Graph G, const float *__restrict__ mu,
                                            const float *__restrict__ sigma, Work W) {
    constexpr int TILE = BS * SPT;
    constexpr int NW = BS / 64;
    constexpr int RS = TILE + kWideHalo + 2;   // a wave's row of producer values: positions t0-kWideHalo-1 .. t0+TILE
    constexpr int WIN = TILE + kHalo + 1;      // the row path's window
    constexpr int kBuf = NW * RS > 3 * WIN ? NW * RS : 3 * WIN;
    __shared__ long long sU64[TILE];           // the tile's usage, 2^-40 units
    __shared__ float sBuf[kBuf];               // the wide ops' rows, then the row path's window
    float *sRows = sBuf, *sT = sBuf, *sFm = sBuf + WIN, *sFs = sBuf + 2 * WIN;
    __shared__ float sRed[2][BS / 64][8];
    __shared__ float sPrev[3];
    constexpr int kEdgeBatch = 8;
    __shared__ float sCp[2][kEdgeBatch][NW][4];   // wave partials of the out-edges' derivatives
    __shared__ int sCpE[2][kEdgeBatch];           // their edges
    __shared__ float sCpC[2][kEdgeBatch];         // and fam_k/sigma_j
    __shared__ float sLast[NW][SPT][3];           // each wave's last S_i(u) terms (lower, upper, count)
    int cpar = 0, par = 0;

    // work-group x serves restart x mod B (the XCDs receive work-groups in
    // turn: with B a multiple of 8 a restart's gathered means and widths stay
    // in one XCD's L2), then (group, part) and tile
    const int b = blockIdx.x % G.B, xr = blockIdx.x / G.B;
    const int gp = xr % (G.ngroups * G.parts), tile = xr / (G.ngroups * G.parts);
    const int grp = gp / G.parts, part = gp % G.parts;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int D = G.D, N = G.N;
    const int t0 = tile * TILE;
    const float *mub = mu + (size_t)b * N;
    const float *rsb = W.rsig + (size_t)b * N;   // 1/sigma

    // this work-group's ops: every parts-th op of the group, from op q0 + part
    const int q0 = G.grp_start[grp] + part, q1 = G.grp_start[grp + 1];
    const int nq = q1 > q0 ? (q1 - q0 + G.parts - 1) / G.parts : 0;
    float accU[SPT];
#pragma unroll
    for (int k = 0; k < SPT; ++k) accU[k] = 0.0f;

    // Groups without step-by-step work leave nothing here: their readers skip
    // them (group and op flags).  Otherwise thread t looks at op q0 + t*parts
    // (groups hold at most as many ops as the work-group has threads); ops and
    // edges on the chunk-polynomial path are left to k_poly.
    if (!(W.gbits[(size_t)b * G.ngroups + grp] & kGbStep)) return;
    // with the narrow kernel on, only the ops it left (step-by-step flag 1)
    if (G.nar_on && !(W.gnar[(size_t)b * G.ngroups + grp] & kNarLeft)) return;
    // Each op is sorted for this tile by its thread: nothing to do (no
    // step-by-step work), constant (every spread misses the tile: its terms
    // are integer counts, finished here), tiny or narrow (lane groups, below),
    // wide (a wave each) or the row path.
    __shared__ int sDirect[BS];   // 1 + number of step-by-step out-edges
    __shared__ unsigned char sCls[BS];
    __shared__ int sConst[4];     // constant ops: V_dep, L_com, P^0, P^{D-1}
    __shared__ int sWide[BS], sWcnt[NW];   // the wide ops in list order
    __shared__ int sNextWide;
    __shared__ long long sG64[2];          // the wide ops' V_dep and L_com, 2^-32 units
    __shared__ int sOpI[BS], sOpE0[BS], sOpDeg[BS], sOpS[BS], sOpOff[BS], sWsum[NW];
    __shared__ float sOpMu[BS], sOpRs[BS], sEmu[kStageOps], sErs[kStageOps];
    __shared__ unsigned char sOpPoly[BS], sEon[kStageOps];
    const OpStage st{sOpI, sOpE0, sOpDeg, sOpS, sOpOff, sOpMu, sOpRs, sOpPoly, sEmu, sErs, sEon};
    const unsigned char *clsb = W.cls + (size_t)b * N;
    const int tb = min(t0 + TILE, D);   // the tile's steps are [t0, tb)
    if (tid < 4) sConst[tid] = 0;
    if (tid < 2) sG64[tid] = 0;
    if (tid == 0) sNextWide = 0;
    for (int p = tid; p < TILE; p += BS) sU64[p] = 0;
    {
        const int lane = tid & 63, w = tid >> 6;
        int i = 0, e0 = 0, deg = 0, s = 0;
        float m_i = 0.0f, rs = 1.0f;
        bool poly_i = false, on = false;
        if (tid < nq) {
            i = G.perm[q0 + tid * G.parts];
            on = W.dflag[(size_t)b * N + i] == 1;
            if (on) {
                e0 = G.row_ptr[i]; deg = G.row_ptr[i + 1] - e0;
                poly_i = clsb[i] != 0;
                s = G.delay[i];
                m_i = mub[i]; rs = rsb[i];
            }
        }
        // LDS offsets of the ops' edges: exclusive scan of the out-degrees
        int x = deg;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(x, o, 64);
            if (lane >= o) x += y;
        }
        if (lane == 63) sWsum[w] = x;
        __syncthreads();
        int off = x - deg;
        for (int k = 0; k < w; ++k) off += sWsum[k];
        if (!on || off + deg > kStageOps) off = -1;
        sOpI[tid] = i; sOpE0[tid] = e0; sOpDeg[tid] = deg; sOpS[tid] = s; sOpOff[tid] = off;
        sOpMu[tid] = m_i; sOpRs[tid] = rs; sOpPoly[tid] = poly_i ? 1 : 0;

        unsigned char c = kNone;
        int flag = 0;
        if (on) {
            const int e1 = e0 + deg;
            int pl, ph;   // F_i is read at the bin edges u - s .. u (u in the tile)
            spread<FAM>(m_i, rs, t0 - s - 1, tb, pl, ph);
            // the tile's steps where F_i(u), F_i'(u) or P_i^u may vary, and
            // where A(u) or F_i'(u-s) may
            const int n1 = min(ph + 1, tb - 1) - max(pl, t0) + 1;
            const int n2 = min(ph + s, tb - 1) - max(pl + s - 1, t0) + 1;
            int span = max(max(n1, n2), 0);
            bool act = n1 > 0 || n2 > 0;
            // F_i off its spread, and A(u) at the steps 0, s-1, D-2 (where
            // the bins open to -inf and +inf meet it)
            auto Fc = [&](int v) { return v < 0 ? 0 : (v >= D - 1 || v > ph) ? 1 : 0; };
            const int us[3] = {0, s - 1, D - 2};
            int ua[3];
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                const int u = us[k];
                const bool fresh = (k < 1 || u != us[0]) && (k < 2 || u != us[1]);
                ua[k] = (fresh && u >= t0 && u < tb && u < D - 1) ? Fc(u - s + 1) - Fc(u - s) : 0;
            }
            int m = 0, cnt = 0, dep = 0, sum3 = 0;
            for (int e = e0; e < e1; ++e) {
                const int j = G.col[e];
                const bool sbs = !(poly_i && clsb[j]) && !G.lap_on;   // Laplace: edges in closed form
                float m_j = 0.0f, rsj = 1.0f;
                if (sbs) { m_j = mub[j]; rsj = rsb[j]; }
                if (off >= 0) {
                    sEmu[off + e - e0] = m_j; sErs[off + e - e0] = rsj; sEon[off + e - e0] = sbs ? 1 : 0;
                }
                if (!sbs) continue;
                ++m;
                int cl, ch;
                spread<FAM>(m_j, rsj, t0 - 1, tb, cl, ch);
                const int n3 = min(ch + 1, tb - 1) - max(cl, t0) + 1;
                span = max(span, n3);
                sum3 += max(n3, 0);
                act = act || n3 > 0;
                // F_i(u) (1 - F_j(u)) = 1 for ph < u < cl
                cnt += max(min(min(tb, D - 1), cl) - max(t0, ph + 1), 0);
#pragma unroll
                for (int k = 0; k < 3; ++k) dep += ua[k] * (us[k] > ch ? 1 : 0);
            }
            flag = 1 + m;
            // wide: one wave per op when the consumers' spreads cover less
            // than half the tile on average (and the delay fits the wave's
            // row), else the row path (its producer values serve every edge
            // at every step of the tile)
            c = !act ? kConst
                : span <= kTinySpan ? kTiny
                : span <= kMidSpan ? kMid
                : span <= kNarrowSpan ? kNarrow
                : G.lap_on ? kLapU   // Laplace: usage only (the edges are in closed form)
                : (s <= kWideHalo && (m == 0 || 2 * sum3 < m * (tb - t0))) ? kWide : kRow;
            if (c == kConst) {
                // no records: every derivative is 0 here, and the readers skip
                // this tile (tile_prod_rec / tile_cons_rec are false for it)
                if (D - 1 >= t0 && D - 1 < tb) dep += m * (1 - Fc(D - 1 - s));
                if (m == 0) dep = cnt = 0;
                if (dep) atomicAdd(&sConst[0], dep);
                if (cnt) atomicAdd(&sConst[1], cnt);
                // P_i^0 = F_i(0), P_i^{D-1} = 1 - F_i(D-2): integers off the spread
                if (!poly_i && t0 == 0 && Fc(0)) atomicAdd(&sConst[2], 1);
                if (!poly_i && D - 1 >= t0 && D - 1 < tb && D > 1 && !Fc(D - 2)) atomicAdd(&sConst[3], 1);
            }
        }
        sDirect[tid] = flag;
        sCls[tid] = c;
        const unsigned long long bw = __ballot(c == kWide);
        if (lane == 0) sWcnt[w] = __popcll(bw);
        __syncthreads();
        int ow = __popcll(bw & ((1ull << lane) - 1ull));
        for (int k = 0; k < w; ++k) ow += sWcnt[k];
        if (c == kWide) sWide[ow] = tid;
    }
    float gsum0 = 0.0f, gsum1 = 0.0f;  // V_dep, L_com of the work-group (threads 0, 1)
    __syncthreads();

    // Narrow ops: the shortest spreads four at a time per wave, then two, the
    // others one at a time; then the wide ops, one per wave.
    __shared__ float sGw[NW][2];          // the narrow ops' V_dep and L_com per wave
    {
        const int lane = tid & 63, w = tid >> 6;
        int nWide = 0;
#pragma unroll
        for (int k = 0; k < NW; ++k) nWide += sWcnt[k];
        float g0 = 0.0f, g1 = 0.0f;
        narrow_ops<FAM, 4, BS>(G, W, mub, rsb, clsb, st, sCls, sDirect, sU64, kTiny, nq, t0, tb, tile, b, g0, g1);
        narrow_ops<FAM, 2, BS>(G, W, mub, rsb, clsb, st, sCls, sDirect, sU64, kMid, nq, t0, tb, tile, b, g0, g1);
        narrow_ops<FAM, 1, BS>(G, W, mub, rsb, clsb, st, sCls, sDirect, sU64, kNarrow, nq, t0, tb, tile, b, g0,
                               g1);
        wide_ops<FAM, BS, RS>(G, W, mub, rsb, clsb, st, sDirect, sWide, nWide, &sNextWide, sRows, sU64, sG64, t0, tb,
                              tile, b);
        if (FAM == 2 && G.lap_on) lap_usage<BS, TILE>(G, sCls, st, nq, t0, tb, sU64);
        const float s0 = wave_sum((lane & 15) == 0 ? g0 : 0.0f), s1 = wave_sum((lane & 15) == 2 ? g1 : 0.0f);
        if (lane == 0) { sGw[w][0] = s0; sGw[w][1] = s1; }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < SPT; ++k) accU[k] += (float)((double)sU64[k * BS + tid] * (1.0 / 1099511627776.0));

    // Row path: the other wide ops one at a time by the whole work-group
    // (the op kernel's description at the top of this file).
    for (int x = 0; x < nq; ++x) {
        if (sCls[x] != kRow) continue;
        const int i = uniform(sOpI[x]);
        const int e0 = uniform(sOpE0[x]), e1 = e0 + uniform(sOpDeg[x]);
        const int off = uniform(sOpOff[x]);
        const bool poly_i = uniform(sOpPoly[x]) != 0;
        const int m = uniform(sDirect[x] - 1);
        const float m_i = uniformf(sOpMu[x]), rs = uniformf(sOpRs[x]);
        const float cinv = rs * fam_k<FAM>();
        const int s = uniform(sOpS[x]);
        const bool win_shift = (m > 0) && (s <= kHalo);
        const int Lh = win_shift ? (s > 1 ? s : 1) : 1;

        // row window: positions v = t0 - Lh + p, p in [0, TILE + Lh].  When
        // all of it lies past fam_zflush on one side of the mean, its values
        // are the exact constants (F = 0 or 1, zero derivatives).
        constexpr float kZF = fam_zflush<FAM>();
        const int wside = uniform(((float)(t0 + TILE) + 0.5f - m_i) * rs < -kZF ? -1
                                  : ((float)(t0 - Lh) + 0.5f - m_i) * rs > kZF ? 1 : 0);
        for (int p = tid; p < TILE + Lh + 1; p += BS) {
            float st, Fm, Fs;
            const int v = t0 - Lh + p;
            if (wside == 0) {
                cdf_at<FAM>(v, D, m_i, rs, cinv, st, Fm, Fs);
            } else {
                st = v < 0 ? 0.0f : (v >= D - 1 || wside > 0) ? -0.0f : 0.0f;
                Fm = 0.0f; Fs = 0.0f;
            }
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
                    cdf_at<FAM>((long long)u - s, D, m_i, rs, cinv, st0, Fm0, Fs0);
                    cdf_at<FAM>((long long)u - s + 1, D, m_i, rs, cinv, st1, Fm1, Fs1);
                    rA[k] = st_mass(st0, st1); rFms[k] = Fm0; rFss[k] = Fs0;
                    if (u == D - 1) tail1mF = st_1mF(st0);
                }
            }
        }

        // Out-edges.  Each wave sums its part of an edge's consumer-side
        // derivatives at once; the work-group totals of a batch of kEdgeBatch
        // edges are formed after one barrier.
        float SL[SPT], SU[SPT], SC[SPT];
#pragma unroll
        for (int k = 0; k < SPT; ++k) { SL[k] = 0.0f; SU[k] = 0.0f; SC[k] = 0.0f; }
        float pL = 0.0f, pU = 0.0f, pC = 0.0f;   // S_i(t0-1), thread 0 only
        int ne = 0;                              // edges of the open batch
        auto flush = [&](int n) {   // after a barrier: the batch's totals to cpart
            if (tid < 4 * n) {
                const int slot = tid >> 2, c = tid & 3;
                float r = sCp[cpar][slot][0][c];
#pragma unroll
                for (int w2 = 1; w2 < NW; ++w2) r += sCp[cpar][slot][w2][c];
                // F_j'(u) = -k g_j/sigma_j (k = fam_k, g_j the density factor) [* z for sigma]; L_com enters with a minus
                const float cj = sCpC[cpar][slot];
                W.cpart[(((size_t)b * G.E + sCpE[cpar][slot]) * G.ntiles + tile) * kCP + c] = c < 2 ? -cj * r : cj * r;
            }
            cpar ^= 1;
        };

        for (int e = e0; e < e1; ++e) {
            float m_j, rsj;
            if (off >= 0) {
                if (!uniform(sEon[off + e - e0])) continue;   // polynomial edge
                m_j = uniformf(sEmu[off + e - e0]); rsj = uniformf(sErs[off + e - e0]);
            } else {
                const int j = uniform(G.col[e]);
                if ((poly_i && clsb[j]) || G.lap_on) continue;
                m_j = mub[j]; rsj = rsb[j];
            }
            // steps t0-1 .. t0+TILE-1 all past fam_zflush on one side of the
            // consumer's mean: its tail and density are exactly 0 there, so
            // the edge adds only the count of consumers past their median
            const int side = uniform(((float)(t0 + TILE - 1) + 0.5f - m_j) * rsj < -kZF ? -1
                                     : ((float)(t0 - 1) + 0.5f - m_j) * rsj > kZF ? 1 : 0);
            if (side != 0) {
                if (side > 0) {
#pragma unroll
                    for (int k = 0; k < SPT; ++k)
                        if (t0 + k * BS + tid < D - 1) SC[k] += 1.0f;
                    if (tid == 0 && t0 > 0) pC += 1.0f;
                }
                if (tid < 4) W.cpart[(((size_t)b * G.E + e) * G.ntiles + tile) * kCP + tid] = 0.0f;
                continue;
            }
            float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int k = 0; k < SPT; ++k) {
                const int u = t0 + k * BS + tid;
                if (u < D - 1) {
                    const float z = ((float)u + 0.5f - m_j) * rsj;
                    float tl, gj;
                    fam_tail_h_fl<FAM>(z, tl, gj);
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
                fam_tail_h_fl<FAM>(z, tl, gj);
                if (z >= 0.0f) { pU += tl; pC += 1.0f; } else { pL += tl; }
            }
            const float r = wave_sum4(acc[0], acc[1], acc[2], acc[3], lane);
            if (lane < 4) sCp[cpar][ne][wid][wave4_comp(lane)] = r;
            if (tid == 0) { sCpE[cpar][ne] = e; sCpC[cpar][ne] = rsj * fam_k<FAM>(); }
            if (++ne == kEdgeBatch) {
                __syncthreads();
                flush(ne);
                ne = 0;
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
            }
            // S_i(u-1) of each step: from the lane below, across waves and
            // steps-per-thread blocks through LDS (each wave's last lane)
            if (lane == 63) {
#pragma unroll
                for (int k = 0; k < SPT; ++k) { sLast[wid][k][0] = SL[k]; sLast[wid][k][1] = SU[k]; sLast[wid][k][2] = SC[k]; }
            }
            if (tid == 0) { sPrev[0] = pL; sPrev[1] = pU; sPrev[2] = pC; }
            __syncthreads();
            flush(ne);
            ne = 0;
#pragma unroll
            for (int k = 0; k < SPT; ++k) {
                const int u = t0 + k * BS + tid;
                float L1 = __shfl_up(SL[k], 1, 64), U1 = __shfl_up(SU[k], 1, 64), C1 = __shfl_up(SC[k], 1, 64);
                if (lane == 0) {
                    const int w2 = wid > 0 ? wid - 1 : NW - 1, k2 = wid > 0 ? k : k - 1;
                    L1 = k2 >= 0 ? sLast[w2][k2 < 0 ? 0 : k2][0] : sPrev[0];
                    U1 = k2 >= 0 ? sLast[w2][k2 < 0 ? 0 : k2][1] : sPrev[1];
                    C1 = k2 >= 0 ? sLast[w2][k2 < 0 ? 0 : k2][2] : sPrev[2];
                }
                if (u >= D) continue;
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
        } else {
            __syncthreads();   // every wave is done with the window
            if (tid < kPP) W.ppart[(((size_t)b * N + i) * G.ntiles + tile) * kPP + tid] = 0.0f;
        }
    }
    // the constant ops' usage, and the narrow and constant ops' sums
#pragma unroll
    for (int k = 0; k < SPT; ++k) {
        const int u = t0 + k * BS + tid;
        if (u == 0) accU[k] += (float)sConst[2];
        if (u == D - 1) accU[k] += (float)sConst[3];
    }
    if (tid < 2) {
        float v = sGw[0][tid];
#pragma unroll
        for (int w = 1; w < NW; ++w) v += sGw[w][tid];
        v += (float)sConst[tid];
        v += (float)((double)sG64[tid] * (1.0 / 4294967296.0));
        if (tid == 0) gsum0 += v; else gsum1 += v;
    }
    {
        float *gs = W.gsum_ops + ((((size_t)b * G.ngroups + grp) * G.parts + part) * G.ntiles + tile) * 2;
        if (tid == 0) gs[0] = gsum0;
        if (tid == 1) gs[1] = gsum1;
    }

    float *up = W.Upart + (((size_t)b * G.ngroups + grp) * G.parts + part) * D;
#pragma unroll
    for (int k = 0; k < SPT; ++k) {
        const int u = t0 + k * BS + tid;
        if (u < D) up[u] = accU[k];
    }
}


// ---------------------------------------------------------------------------
// Group kernel.  Work-group = (op group, restart).
// (1) The group's work bits this iteration (gbits): the OR over its ops of
//     kGbStep (step-by-step work) and kGbGrid << grid; one plain store per
//     (restart, group).
// (2) With the narrow path on (G.nar_on): the step-by-step ops whose spreads
//     are short, each taken once over the whole horizon instead of once per
//     step tile.  Thread per op for the sorting (the op kernel's spread tests
//     with one tile [0, D)): an op off the polynomial path whose own spreads
//     and whose consumers' spreads span at most kNarrowSpan steps is taken
//     here (its step-by-step flag becomes 2, and the op kernel leaves it); the
//     others stay with the op kernel.  The taken ops run through narrow_ops
//     over the horizon: usage into one fixed-point LDS row of D steps, records
//     into the single ppoly / cpoly slots (free for ops off the polynomial
//     path), V_dep and L_com per (restart, group).  gnar[b][group] tells the
//     readers which parts exist.
// ---------------------------------------------------------------------------
template <int FAM>
__global__ __launch_bounds__(kNarBS) void k_group(Graph G, const float *__restrict__ mu, Work W) {
    constexpr int BS = kNarBS, NW = BS / 64;
    extern __shared__ long long sRow[];   // [D] usage of the taken ops, 2^-40 units
    __shared__ int sDirect[BS];
    __shared__ unsigned char sCls[BS];
    __shared__ int sOpI[BS], sOpE0[BS], sOpDeg[BS], sOpS[BS], sOpOff[BS], sWsum[NW];
    __shared__ float sOpMu[BS], sOpRs[BS], sEmu[kStage], sErs[kStage];
    __shared__ unsigned char sOpPoly[BS], sEon[kStage];
    __shared__ int sAny[2];                // an op left to the op kernel / taken here
    __shared__ float sGw[NW][2];
    const OpStage st{sOpI, sOpE0, sOpDeg, sOpS, sOpOff, sOpMu, sOpRs, sOpPoly, sEmu, sErs, sEon};
    // work-group x serves restart x mod B (as in the op kernel)
    const int b = blockIdx.x % G.B, grp = blockIdx.x / G.B, tid = threadIdx.x;
    const int lane = tid & 63, w = tid >> 6;
    const int D = G.D, N = G.N;
    const size_t bg = (size_t)b * G.ngroups + grp;
    const int q0 = G.grp_start[grp], nq = G.grp_start[grp + 1] - q0;
    {   // (1) work bits
        __shared__ unsigned sW[NW];
        unsigned bits = 0u;
        for (int q = tid; q < nq; q += BS) {
            const size_t bi = (size_t)b * N + G.perm[q0 + q];
            const int gs = W.gsel[bi];
            bits |= W.dflag[bi] ? kGbStep : 0u;
            bits |= gs < kGrids ? kGbGrid << gs : 0u;
        }
        unsigned v = 0u;
#pragma unroll
        for (int k = 0; k < 2 + kGrids; ++k) v |= __ballot((bits >> k) & 1u) ? 1u << k : 0u;
        if (lane == 0) sW[w] = v;
        __syncthreads();
        v = 0u;
#pragma unroll
        for (int k = 0; k < NW; ++k) v |= sW[k];
        if (tid == 0) W.gbits[bg] = v;
        // no step-by-step work in the group: the readers skip it before reading gnar
        if (!(v & kGbStep) || !G.nar_on) return;
    }
    const float *mub = mu + (size_t)b * N;
    const float *rsb = W.rsig + (size_t)b * N;
    const unsigned char *clsb = W.cls + (size_t)b * N;
    for (int u = tid; u < D; u += BS) sRow[u] = 0;
    if (tid < 2) sAny[tid] = 0;
    {
        int i = 0, e0 = 0, deg = 0, s = 0;
        float m_i = 0.0f, rs = 1.0f;
        bool poly_i = false, on = false;
        if (tid < nq) {
            i = G.perm[q0 + tid];
            on = W.dflag[(size_t)b * N + i] == 1;
            if (on) {
                e0 = G.row_ptr[i]; deg = G.row_ptr[i + 1] - e0;
                poly_i = clsb[i] != 0;
                s = G.delay[i];
                m_i = mub[i]; rs = rsb[i];
            }
        }
        // LDS offsets of the ops' edges: exclusive scan of the out-degrees
        int x = deg;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(x, o, 64);
            if (lane >= o) x += y;
        }
        if (lane == 63) sWsum[w] = x;
        __syncthreads();
        int off = x - deg;
        for (int k = 0; k < w; ++k) off += sWsum[k];
        if (!on || off + deg > kStage) off = -1;
        sOpI[tid] = i; sOpE0[tid] = e0; sOpDeg[tid] = deg; sOpS[tid] = s; sOpOff[tid] = off;
        sOpMu[tid] = m_i; sOpRs[tid] = rs; sOpPoly[tid] = poly_i ? 1 : 0;
        unsigned char c = kNone;
        int flag = 0;
        if (on) {
            int pl, ph;   // F_i is read at the bin edges u - s .. u (u in [0, D))
            spread<FAM>(m_i, rs, -s - 1, D, pl, ph);
            const int n1 = min(ph + 1, D - 1) - max(pl, 0) + 1;
            const int n2 = min(ph + s, D - 1) - max(pl + s - 1, 0) + 1;
            int span = max(max(n1, n2), 0);
            int m = 0;
            for (int e = e0; e < e0 + deg; ++e) {
                const int j = G.col[e];
                const bool sbs = !(poly_i && clsb[j]) && !G.lap_on;   // Laplace: edges in closed form
                float m_j = 0.0f, rsj = 1.0f;
                if (sbs) { m_j = mub[j]; rsj = rsb[j]; }
                if (off >= 0) {
                    sEmu[off + e - e0] = m_j; sErs[off + e - e0] = rsj; sEon[off + e - e0] = sbs ? 1 : 0;
                }
                if (!sbs) continue;
                ++m;
                int cl, ch;
                spread<FAM>(m_j, rsj, -1, D, cl, ch);
                span = max(span, min(ch + 1, D - 1) - max(cl, 0) + 1);
            }
            flag = 1 + m;
            const bool take = !poly_i && span <= kNarrowSpan;
            c = take ? (span <= kTinySpan ? kTiny : span <= kMidSpan ? kMid : kNarrow) : kNone;
            if (take) W.dflag[(size_t)b * N + i] = 2;
            sAny[take ? 1 : 0] = 1;
        }
        sDirect[tid] = flag;
        sCls[tid] = c;
    }
    __syncthreads();
    if (tid == 0) W.gnar[bg] = (sAny[0] ? kNarLeft : 0u) | (sAny[1] ? kNarTaken : 0u);
    if (!sAny[1]) return;
    float g0 = 0.0f, g1 = 0.0f;
    narrow_ops<FAM, 4, BS, true>(G, W, mub, rsb, clsb, st, sCls, sDirect, sRow, kTiny, nq, 0, D, 0, b,
                                 g0, g1);
    narrow_ops<FAM, 2, BS, true>(G, W, mub, rsb, clsb, st, sCls, sDirect, sRow, kMid, nq, 0, D, 0, b,
                                 g0, g1);
    narrow_ops<FAM, 1, BS, true>(G, W, mub, rsb, clsb, st, sCls, sDirect, sRow, kNarrow, nq, 0, D, 0, b,
                                 g0, g1);
    const float s0 = wave_sum((lane & 15) == 0 ? g0 : 0.0f), s1 = wave_sum((lane & 15) == 2 ? g1 : 0.0f);
    if (lane == 0) { sGw[w][0] = s0; sGw[w][1] = s1; }
    __syncthreads();
    float *row = W.Unar + bg * D;
    for (int u = tid; u < D; u += BS) row[u] = (float)((double)sRow[u] * (1.0 / 1099511627776.0));
    if (tid < 2) {
        float v = sGw[0][tid];
#pragma unroll
        for (int k = 1; k < NW; ++k) v += sGw[k][tid];
        W.gsum_nar[bg * 2 + tid] = v;
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
template <int FAM, int BS, int SPT>
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
        const float mj = mu[(size_t)b * N + j], rsj = W.rsig[(size_t)b * N + j];
        const float mi = mu[(size_t)b * N + i], rsi = W.rsig[(size_t)b * N + i];
        const float cj = rsj * fam_k<FAM>(), ci = rsi * fam_k<FAM>();
        float acc[5] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k = 0; k < SPT; ++k) {
            const int u = t0 + k * BS + tid;
            if (u < D - 1) {
                float sj_, Fmj, Fsj, si_, Fmi, Fsi;
                cdf_at<FAM>(u, D, mj, rsj, cj, sj_, Fmj, Fsj);
                cdf_at<FAM>(u, D, mi, rsi, ci, si_, Fmi, Fsi);
                const float Pi = st_mass(st_at<FAM>((long long)u - c - 1, D, mi, rsi), st_at<FAM>((long long)u - c, D, mi, rsi));
                const float Pj = st_mass(st_at<FAM>((long long)u + c, D, mj, rsj), st_at<FAM>((long long)u + c + 1, D, mj, rsj));
                acc[0] = fmaf(Pi, st_1mF(sj_), acc[0]);
                acc[1] = fmaf(-Fmj, Pi, acc[1]);
                acc[2] = fmaf(-Fsj, Pi, acc[2]);
                acc[3] = fmaf(Fmi, Pj, acc[3]);
                acc[4] = fmaf(Fsi, Pj, acc[4]);
            }
        }
        if (tile == 0 && tid == 0) acc[0] += st_F(st_at<FAM>(-c - 1, D, mi, rsi));
        const float r = block_sum<5, BS>(acc, sRed[par]);
        par ^= 1;
        if (tid < kBP) W.bpart[(((size_t)b * G.nb + e) * G.ntiles + tile) * kBP + tid] = r;
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
template <int FAM, int BS, int SPT>
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
        sRs[tid] = W.rsig[bi];
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
        const float m = sMu[q], rs = sRs[q], cinv = rs * fam_k<FAM>();
        float acc[2] = {0.0f, 0.0f};
#pragma unroll
        for (int j = 0; j < SPT; ++j) {
            const int x = tid + j * BS;
            const float w = sW[x];
            if (w != 0.0f) {
                const float z = ((float)(t0 + x) + 0.5f - m) * rs;
                const float Fm = -fam_h<FAM>(z) * cinv;
                acc[0] = fmaf(w, Fm, acc[0]);
                acc[1] = fmaf(w, Fm * z, acc[1]);
            }
        }
        const float r = block_sum<2, BS>(acc, sRed[par]);
        par ^= 1;
        if (tid < 2) W.lpart[(((size_t)b * N + i) * G.ntiles + tile) * 2 + tid] = r;
    }
}


// ---------------------------------------------------------------------------
// Expected storage units (eq:active): op h holds b_h units at step t with
// probability F_h(t) (1 - Q_h(t)), Q_h(t) = prod over successors F_j(t).
// Q and R = 1 - Q are carried together (R += Q (1 - F_j), Q *= F_j) with
// 1 - F_j from the tail, so R keeps full precision when every F_j is near 1.
// Work-group = (type-pure op group, tile of steps, restart); each thread
// owns SPT steps and sums the group's ops into Mpart (no atomics).  The sums
// are kept in fp64: the profile reaches 1e5 units and more, and its
// LogSumExp weights amplify absolute errors by 1/tau.
// ---------------------------------------------------------------------------
template <int FAM, int BS, int SPT>
__global__ __launch_bounds__(BS) void k_mem_fwd(Graph G, const float *__restrict__ mu,
                                                const float *__restrict__ sigma, Work W) {
    constexpr int TILE = BS * SPT;
    __shared__ int sI[BS];
    __shared__ float sMu[BS], sRs[BS];
    const int grp = blockIdx.x, tile = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    const int N = G.N, D = G.D;
    const int t0 = tile * TILE;
    const float *mub = mu + (size_t)b * N, *rsb = W.rsig + (size_t)b * N;
    sI[tid] = -1;
    if (q0 + tid < q1) {
        const int i = G.perm[q0 + tid];
        // an op without successors holds nothing; polynomial holders are taken elsewhere
        if (G.row_ptr[i + 1] > G.row_ptr[i] && !W.mpoly[(size_t)b * N + i]) sI[tid] = i;
        sMu[tid] = mub[i];
        sRs[tid] = rsb[i];
    }
    __syncthreads();
    double acc[SPT];
#pragma unroll
    for (int j = 0; j < SPT; ++j) acc[j] = 0.0;
    for (int q = 0; q < q1 - q0; ++q) {
        const int i = sI[q];
        if (i < 0) continue;
        const float m = sMu[q], rs = sRs[q], bi = G.bmem[i];
        float Fi[SPT], Q[SPT], R[SPT];
#pragma unroll
        for (int j = 0; j < SPT; ++j) {
            Fi[j] = st_F(st_at<FAM>((long long)t0 + tid + j * BS, D, m, rs));
            Q[j] = 1.0f; R[j] = 0.0f;
        }
        for (int e = G.row_ptr[i]; e < G.row_ptr[i + 1]; ++e) {
            const int k = G.col[e];
            const float mk = mub[k], rk = rsb[k];
#pragma unroll
            for (int j = 0; j < SPT; ++j) {
                const float st = st_at<FAM>((long long)t0 + tid + j * BS, D, mk, rk);
                R[j] = fmaf(Q[j], st_1mF(st), R[j]);
                Q[j] *= st_F(st);
            }
        }
#pragma unroll
        for (int j = 0; j < SPT; ++j) acc[j] += (double)(bi * Fi[j] * R[j]);
    }
    double *mp = W.Mpart + ((size_t)b * G.ngroups + grp) * D;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int t = t0 + tid + j * BS;
        if (t < D) mp[t] = acc[j];
    }
}

// Gradient of gamma L_mem with c(t) = gamma softmax(MReg / tau) at slot
// t mod T, over the interior bin edges t = 0..D-2:
//   as the holder:      c(t) b_h (1 - Q_h(t)) dF_h(t)/dth_h
//   as a successor i:  -c(t) b_h F_h(t) prod_{j != i} F_j(t) dF_i(t)/dth_i
// with prod_{j != i} F_j = Q_h / F_i (taken as 0 when F_i < 2^-100: dF_i is
// then as small up to a bounded factor, far below fp32 resolution).
template <int FAM, int BS, int SPT>
__global__ __launch_bounds__(BS) void k_mem_bwd(Graph G, const float *__restrict__ mu,
                                                const float *__restrict__ sigma, Work W) {
    constexpr int TILE = BS * SPT;
    __shared__ float sW[TILE];
    __shared__ int sI[BS];
    __shared__ float sMu[BS], sRs[BS];
    __shared__ float sRed[2][BS / 64][8];
    const int grp = blockIdx.x, tile = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int q0 = G.grp_start[grp], q1 = G.grp_start[grp + 1];
    const int N = G.N, D = G.D, T = G.T, nt = G.ntiles;
    const int t0 = tile * TILE;
    const float *mub = mu + (size_t)b * N, *rsb = W.rsig + (size_t)b * N;
    sI[tid] = -1;
    if (q0 + tid < q1) {
        const int i = G.perm[q0 + tid];
        if (G.row_ptr[i + 1] > G.row_ptr[i] && !W.mpoly[(size_t)b * N + i]) sI[tid] = i;
        sMu[tid] = mub[i];
        sRs[tid] = rsb[i];
    }
    const float *ms = W.msoft + (size_t)b * T;
    for (int x = tid; x < TILE; x += BS) {
        const int t = t0 + x;
        sW[x] = t <= D - 2 ? ms[t % T] : 0.0f;
    }
    __syncthreads();
    int par = 0;
    for (int q = 0; q < q1 - q0; ++q) {
        const int h = sI[q];
        if (h < 0) continue;
        const float m = sMu[q], rs = sRs[q], cinv = rs * fam_k<FAM>(), bh = G.bmem[h];
        const int e0 = G.row_ptr[h], e1 = G.row_ptr[h + 1];
        float Fh[SPT], Fmh[SPT], Fsh[SPT], Q[SPT], R[SPT], own[2] = {0.0f, 0.0f};
#pragma unroll
        for (int j = 0; j < SPT; ++j) {
            float st;
            cdf_at<FAM>((long long)t0 + tid + j * BS, D, m, rs, cinv, st, Fmh[j], Fsh[j]);
            Fh[j] = st_F(st);
            Q[j] = 1.0f; R[j] = 0.0f;
        }
        for (int e = e0; e < e1; ++e) {
            const int k = uniform(G.col[e]);
            const float mk = mub[k], rk = rsb[k];
#pragma unroll
            for (int j = 0; j < SPT; ++j) {
                const float sk = st_at<FAM>((long long)t0 + tid + j * BS, D, mk, rk);
                R[j] = fmaf(Q[j], st_1mF(sk), R[j]);
                Q[j] *= st_F(sk);
            }
        }
#pragma unroll
        for (int j = 0; j < SPT; ++j) {
            const float wr = sW[tid + j * BS] * bh * R[j];
            own[0] = fmaf(wr, Fmh[j], own[0]);
            own[1] = fmaf(wr, Fsh[j], own[1]);
        }
        {
            const float r = block_sum<2, BS>(own, sRed[par]);
            par ^= 1;
            if (tid < 2) W.mown[(((size_t)b * N + h) * nt + tile) * 2 + tid] = r;
        }
        for (int e = e0; e < e1; ++e) {
            const int k = uniform(G.col[e]);
            const float mk = mub[k], rk = rsb[k], ck = rk * fam_k<FAM>();
            float acc[2] = {0.0f, 0.0f};
#pragma unroll
            for (int j = 0; j < SPT; ++j) {
                float st, Fm, Fs;
                cdf_at<FAM>((long long)t0 + tid + j * BS, D, mk, rk, ck, st, Fm, Fs);
                const float Fk = st_F(st);
                // prod over the other successors; below 2^-100 the term is far
                // under fp32 resolution (dF_k vanishes with F_k)
                const float others = Fk > 0x1p-100f ? Q[j] * __builtin_amdgcn_rcpf(Fk) : 0.0f;
                const float c = -sW[tid + j * BS] * bh * Fh[j] * others;
                acc[0] = fmaf(c, Fm, acc[0]);
                acc[1] = fmaf(c, Fs, acc[1]);
            }
            const float r = block_sum<2, BS>(acc, sRed[par]);
            par ^= 1;
            if (tid < 2) W.msucc[(((size_t)b * G.E + e) * nt + tile) * 2 + tid] = r;
        }
    }
}

// ---------------------------------------------------------------------------
// Launchers.  The CDF family and the work-group shape are template arguments;
// dispatch() calls f(FAM, BS, SPT) with them as integral constants.
// ---------------------------------------------------------------------------
template <int V> using IC = std::integral_constant<int, V>;

template <int FAM, class F>
hipError_t dispatch_shape(const LaunchCfg &lc, F &&f) {
    if (lc.bs == 64 && lc.spt == 1) f(IC<FAM>{}, IC<64>{}, IC<1>{});
    else if (lc.bs == 256 && lc.spt == 1) f(IC<FAM>{}, IC<256>{}, IC<1>{});
    else if (lc.bs == 256 && lc.spt == 4) f(IC<FAM>{}, IC<256>{}, IC<4>{});
    else return hipErrorInvalidValue;
    return hipSuccess;
}

template <class F>
hipError_t dispatch(const LaunchCfg &lc, F &&f) {
    switch (lc.fam) {
        case 0: return dispatch_shape<0>(lc, f);
        case 1: return dispatch_shape<1>(lc, f);
        case 2: return dispatch_shape<2>(lc, f);
        case 3: return dispatch_shape<3>(lc, f);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_ops(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu, const float *sigma,
                      hipStream_t st) {
    const size_t nwg = (size_t)g.ngroups * g.parts * g.ntiles * g.B;
    if (nwg > 0x7fffffffu) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)nwg);
    return dispatch(lc, [&](auto fam, auto bs, auto spt) {
        hipLaunchKernelGGL((k_ops<decltype(fam)::value, decltype(bs)::value, decltype(spt)::value>), grid,
                           dim3(decltype(bs)::value), 0, st, g, mu, sigma, w);
    });
}

hipError_t launch_group(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu, hipStream_t st) {
    const dim3 grid((unsigned)((size_t)g.ngroups * g.B));
    const size_t lds = g.nar_on ? sizeof(long long) * (size_t)g.D : 0;
    switch (lc.fam) {
        case 0: hipLaunchKernelGGL(k_group<0>, grid, dim3(kNarBS), lds, st, g, mu, w); break;
        case 1: hipLaunchKernelGGL(k_group<1>, grid, dim3(kNarBS), lds, st, g, mu, w); break;
        case 2: hipLaunchKernelGGL(k_group<2>, grid, dim3(kNarBS), lds, st, g, mu, w); break;
        case 3: hipLaunchKernelGGL(k_group<3>, grid, dim3(kNarBS), lds, st, g, mu, w); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_back(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu, const float *sigma,
                       hipStream_t st) {
    const int epb = 4;
    const dim3 grid((g.nb + epb - 1) / epb, g.ntiles, g.B);
    return dispatch(lc, [&](auto fam, auto bs, auto spt) {
        hipLaunchKernelGGL((k_back<decltype(fam)::value, decltype(bs)::value, decltype(spt)::value>), grid,
                           dim3(decltype(bs)::value), 0, st, g, mu, sigma, w, epb);
    });
}

hipError_t launch_lse_ops(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu,
                          const float *sigma, hipStream_t st) {
    const dim3 grid(g.ngroups, g.ntiles, g.B);
    return dispatch(lc, [&](auto fam, auto bs, auto spt) {
        hipLaunchKernelGGL((k_lse_ops<decltype(fam)::value, decltype(bs)::value, decltype(spt)::value>), grid,
                           dim3(decltype(bs)::value), 0, st, g, mu, sigma, w);
    });
}

hipError_t launch_mem_fwd(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu,
                          const float *sigma, hipStream_t st) {
    const dim3 grid(g.ngroups, g.ntiles, g.B);
    return dispatch(lc, [&](auto fam, auto bs, auto spt) {
        hipLaunchKernelGGL((k_mem_fwd<decltype(fam)::value, decltype(bs)::value, decltype(spt)::value>), grid,
                           dim3(decltype(bs)::value), 0, st, g, mu, sigma, w);
    });
}

hipError_t launch_mem_bwd(const Graph &g, const Work &w, const LaunchCfg &lc, const float *mu,
                          const float *sigma, hipStream_t st) {
    const dim3 grid(g.ngroups, g.ntiles, g.B);
    return dispatch(lc, [&](auto fam, auto bs, auto spt) {
        hipLaunchKernelGGL((k_mem_bwd<decltype(fam)::value, decltype(bs)::value, decltype(spt)::value>), grid,
                           dim3(decltype(bs)::value), 0, st, g, mu, sigma, w);
    });
}

}  // namespace gaus
