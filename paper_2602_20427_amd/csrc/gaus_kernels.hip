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
//
// This file: classification, usage, penalties and the per-restart scalars,
// gradient assembly with Adam, and legalization; the per-step work is in
// gaus_step.hip (step by step) and gaus_poly.hip (chunk polynomials).
#include "gaus_device.h"

#include <algorithm>
#include <map>
#include <mutex>

namespace gaus {

// ---------------------------------------------------------------------------
// Chunk-polynomial path (dense regime).
//
// Chunks of W steps tile [L0, D-2); a chunk's points are y = u - t_mid in
// [-lam, lam], lam = (W-1)/2.  Around the chunk centre an op's CDF is
// F(u) = Phi(z0 + r y), r = 1/sigma, and its Taylor coefficients in y are
// T_n = Phi^(n)(z0) r^n / n!, which obey
//   T_1 = phi(z0) r,
//   T_{n+1} = -(z0 r/(n+1)) T_n - ((n-1) r^2/(n(n+1))) T_{n-1}
// (the Hermite recursion of the derivatives of phi, scaled).  The logistic
// and Cauchy laws of App. E have recursions of their own (expand in the
// device header); everything below uses only the T's and holds for any
// location-scale family.  From one set of T's follow, with constant integer
// coefficients (one step = 1 in y):
//   F:         f_k = T_k
//   dF/dmu:    a_k = -(k+1) T_{k+1}
//   dF/dsigma: e_k = z0 a_k + r a_{k-1}           (dF/dsigma = z dF/dmu)
//   mass F(v) - F(v-1):  m_k = -sum_{j>=1} C(k+j,j) (-1)^j T_{k+j}
//   dF/dmu at v-1:       a1_k = -sum_{j>=0} (k+j+1) C(k+j,j) (-1)^j T_{k+1+j}
// The series converge like powers of rho = lam r; each family's tier bounds
// (set on the host) keep the truncation error of the density series below
// ~8e-8 of the peak density.  Every sum over the chunk's steps of a product
// p(u) q(u) equals sum_k (H p)_k q_k with the chunk moments H_n = sum_y y^n,
// so an edge costs 10 dot products of length kNC.
// The strip [0, L0) u {D-2, D-1} (boundary conventions of the open end bins,
// zero derivatives outside the interior edges) is evaluated step by step.
// ---------------------------------------------------------------------------
// Path of an op this iteration: 0 = step by step, else the polynomial tier
// (wider sigma: higher tier, lower degree).
__device__ __forceinline__ int poly_tier(const PolyArgs &pa, float s, int delay) {
    int t = 0;
    if (pa.enabled && delay <= kSmax)
        for (int q = 1; q <= kTiers; ++q) t = s >= pa.sig_thr[q] ? q : t;
    return t;
}

// The same on packed grid g (0 when the grid is off).
__device__ __forceinline__ int grid_tier(const GridArgs &gr, float s, int delay) {
    int t = 0;
    if (gr.on && delay <= kSmax)
        for (int q = 1; q <= kTiers; ++q) t = s >= gr.sig_thr[q] ? q : t;
    return t;
}

// Classification and work flags.  Work-group = (64 consecutive ops, pack of
// kFlagPack restarts), one wave per restart of the pack and thread per
// (restart, op), so every per-op array is read and written in op order:
//   * 1/sigma and the op's path (tier) for the other kernels;
//   * step-by-step work of the op: its own path, or an out-edge to an op off
//     the polynomial path;
//   * a polynomial producer's tier: the highest degree among itself and its
//     polynomial consumers;
//   * its grid: the coarsest packed grid whose whole restart pack (the
//     restarts < B of [P floor(b/P), P floor(b/P) + P)) has the op and all
//     its consumers reach the grid's degree-8 bound, with the pack's tier
//     (the highest degree of its members'); else grid 0 with the op's own
//     tier, or kNoGrid on the step-by-step path.  Polynomial records (ppoly,
//     cpoly) are written only for ops on a grid; every reader checks cls.
// The per-(restart, group) OR of these flags (gbits) follows in k_group.
// The consumers' tiers are recomputed here from their sigmas.  With the
// storage term on, also whether a holder's storage term is taken on the
// chunk polynomials (kMemPolyDeg, PolyArgs::mem_rho).
constexpr int kFlagPack = 4;   // the largest restart pack of a grid
static_assert(kGridP[kGrids - 1] == kFlagPack, "packs nest in the flag kernel's restarts");

__global__ __launch_bounds__(64 * kFlagPack) void k_flags(Graph G, PolyArgs pa, const float *__restrict__ sigma,
                                                          Work W, int mem_on) {
    __shared__ unsigned char sTp[kFlagPack][kGrids][64];   // tier on each packed grid, 0 if not eligible
    const int q = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int i = blockIdx.x * 64 + lane;
    const int b = blockIdx.y * kFlagPack + q;
    const int N = G.N, nb = min(kFlagPack, G.B - (int)blockIdx.y * kFlagPack);
    const bool act = q < nb && i < N;
    int d = 0, t = 0, ci = 0;
    size_t bi = 0;
    if (act) {
        bi = (size_t)b * N + i;
        const float *sgb = sigma + (size_t)b * N;
        const float s = sgb[i];
        W.rsig[bi] = 1.0f / s;
        const int di = G.delay[i];
        ci = poly_tier(pa, s, di);
        W.cls[bi] = (unsigned char)ci;
        d = ci ? 0 : 1;
        t = ci;
        // packed-grid tiers count only for ops on the polynomial path of grid 0
        // (an explicit grid-0 chunk width can make a packed grid's threshold
        // the lower one: such an op stays step by step in every restart)
        int tp[kGrids];   // [0] unused
#pragma unroll
        for (int g = 1; g < kGrids; ++g) tp[g] = ci ? grid_tier(pa.gr[g], s, di) : 0;
        const int e0 = G.row_ptr[i], e1 = G.row_ptr[i + 1];
        float rsum = 1.0f / s;   // sum of 1/sigma over the holder and its successors
        for (int e = e0; e < e1; ++e) {
            const int j = G.col[e];
            const float sj = sgb[j];
            const int dj = G.delay[j];
            const int cj = poly_tier(pa, sj, dj);
            d |= cj ? 0 : 1;
            t = cj ? min(t, cj) : t;
#pragma unroll
            for (int g = 1; g < kGrids; ++g) {
                const int c = cj ? grid_tier(pa.gr[g], sj, dj) : 0;   // a step-by-step consumer
                tp[g] = c ? min(tp[g], c) : 0;                         // keeps the op off the packs
            }
            if (mem_on) rsum += 1.0f / sj;
        }
#pragma unroll
        for (int g = 1; g < kGrids; ++g) sTp[q][g][lane] = (unsigned char)tp[g];
        W.dflag[bi] = (unsigned char)d;
        W.mpoly[bi] = (unsigned char)(mem_on && ci != 0 && d == 0 && e1 > e0 &&
                                      e1 - e0 <= kMemPolyDeg && pa.lam * rsum <= pa.mem_rho);
    }
    __syncthreads();
    if (act) {   // grid: the coarsest packed grid whose pack qualifies
        int g_sel = ci ? 0 : kNoGrid, tier = t;
#pragma unroll
        for (int g = kGrids - 1; g >= 1; --g) {
            if (!pa.gr[g].on || g_sel != 0) continue;
            const int P = kGridP[g], p0 = q - q % P;
            int tt = kTiers;
            bool ok = true;
            for (int r = p0; r < p0 + P && r < nb; ++r) {
                const int v = sTp[r][g][lane];
                ok = ok && v != 0;
                tt = min(tt, v);
            }
            if (ok) { g_sel = g; tier = tt; }
        }
        W.gsel[bi] = (unsigned char)g_sel;
        W.gtier[bi] = (unsigned char)(g_sel == kNoGrid ? 0 : tier);
    }
}

// ---------------------------------------------------------------------------
// Usage: U[b][k][slot] = sum over type-k groups and steps t = slot (mod T).
// ---------------------------------------------------------------------------
// Polynomial usage per (type, restart, grid): the groups' chunk coefficients
// and strip values summed over the type's groups (64 entries x 16 group
// slices per work-group, combined in a fixed order).
constexpr int kUcEntries = kMaxChunks * kNC + kStripMax;   // per (restart, type, grid)

constexpr int kUcoefRows = 16;   // work-group = 64 entries x 16 strided partial sums
constexpr int kUcoefMaxSlots = 4096;   // slots of one type listed in LDS

__global__ __launch_bounds__(64 * kUcoefRows) void k_ucoef(Graph G, PolyArgs pa, Work W) {
    __shared__ float part[kUcoefRows][64];
    __shared__ int sGrp[64 * kUcoefRows];
    __shared__ int sSlot[kUcoefMaxSlots];
    __shared__ int wcnt[kUcoefRows];
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int x = blockIdx.x * 64 + tx, k = blockIdx.y, b = blockIdx.z / kGrids, gi = blockIdx.z % kGrids;
    const GridArgs &gd = pa.gr[gi];
    const int ncoef = gd.nc * kNC, nent = ncoef + gd.SP;
    if (!gd.on || blockIdx.x * 64 >= nent) return;
    const int split = gd.split;
    const size_t rb = (size_t)gd.slot_base + (size_t)b * G.ngroups * split;
    // the type's groups with ops on the grid, compacted in order (their
    // work-groups wrote every slot; the others wrote nothing)
    const unsigned *gb = W.gbits + (size_t)b * G.ngroups;
    const unsigned gmask = kGbGrid << gi;
    auto work = [&](int q) { return (gb[q] & gmask) != 0u; };
    const int t0 = G.type_grp[k], t1 = G.type_grp[k + 1];
    float acc = 0.0f;
    if (t1 - t0 <= 64 * kUcoefRows) {
        const int q = t0 + (int)threadIdx.x;
        const bool f = q < t1 && work(q);
        const unsigned long long bal = __ballot(f);
        if (tx == 0) wcnt[ty] = __popcll(bal);
        __syncthreads();
        int off = 0, ng = 0;
#pragma unroll
        for (int w = 0; w < kUcoefRows; ++w) { off += w < ty ? wcnt[w] : 0; ng += wcnt[w]; }
        if (f) sGrp[off + __popcll(bal & ((1ull << tx) - 1ull))] = q;
        __syncthreads();
        const int nsl = ng * split;
        if (nsl <= kUcoefMaxSlots) {
            // the listed groups' slots, then row ty sums slots ty, ty + 16, ...
            for (int q2 = threadIdx.x; q2 < nsl; q2 += 64 * kUcoefRows)
                sSlot[q2] = sGrp[q2 / split] * split + q2 % split;
            __syncthreads();
            if (x < ncoef) {
#pragma unroll 8
                for (int q2 = ty; q2 < nsl; q2 += kUcoefRows) acc += W.Ucoef[(rb + sSlot[q2]) * kMaxChunks * kNC + x];
            } else if (x < nent) {
#pragma unroll 8
                for (int q2 = ty; q2 < nsl; q2 += kUcoefRows) acc += W.Ustrip[(rb + sSlot[q2]) * kStripMax + (x - ncoef)];
            }
        } else {
            for (int j = ty; j < ng; j += kUcoefRows) {
                const size_t s0 = rb + (size_t)sGrp[j] * split;
                if (x < ncoef) {
                    for (int u = 0; u < split; ++u) acc += W.Ucoef[(s0 + u) * kMaxChunks * kNC + x];
                } else if (x < nent) {
                    for (int u = 0; u < split; ++u) acc += W.Ustrip[(s0 + u) * kStripMax + (x - ncoef)];
                }
            }
        }
    } else {   // more groups than one pass lists: test each
        for (int g = t0 + ty; g < t1; g += kUcoefRows) {
            if (!work(g)) continue;
            const size_t s0 = rb + (size_t)g * split;
            if (x < ncoef) {
                for (int u = 0; u < split; ++u) acc += W.Ucoef[(s0 + u) * kMaxChunks * kNC + x];
            } else if (x < nent) {
                for (int u = 0; u < split; ++u) acc += W.Ustrip[(s0 + u) * kStripMax + (x - ncoef)];
            }
        }
    }
    part[ty][tx] = acc;
    __syncthreads();
    if (ty == 0 && x < nent) {
        float t = 0.0f;
#pragma unroll
        for (int r = 0; r < kUcoefRows; ++r) t += part[r][tx];
        W.Ucoef_k[(((size_t)b * G.K + k) * kGrids + gi) * kUcEntries + x] = t;
    }
}

// Usage U(slot) per (slot block, type, restart): step-by-step partials of the
// type's active groups plus the polynomial part (chunk polynomial at t, or
// the strip value), summed over t = slot mod T.
constexpr int kUsageBS = 256;

template <int RP>   // threads per slot, each summing every RP-th step-by-step row
__global__ __launch_bounds__(kUsageBS) void k_usage(Graph G, PolyArgs pa, Work W) {
    constexpr int kMaxAct = 1024;
    __shared__ float sC[kGrids][kUcEntries];
    __shared__ int sAct[kMaxAct], sActN[kMaxAct];
    __shared__ int wcount[2][kUsageBS / 64];
    __shared__ int base[2];
    const int k = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int g0 = G.type_grp[k], g1 = G.type_grp[k + 1];
    const int D = G.D, T = G.T;

    // the type's groups with step-by-step partials of the op kernel (sAct) and
    // of the narrow kernel (sActN), compacted in order
    auto has_rows = [&](int g, int which) {
        const size_t bg = (size_t)b * G.ngroups + g;
        if (!(W.gbits[bg] & kGbStep)) return false;
        if (!G.nar_on) return which == 0;
        return (W.gnar[bg] & (which == 0 ? kNarLeft : kNarTaken)) != 0u;
    };
    if (tid < 2) base[tid] = 0;
    __syncthreads();
    for (int c0 = g0; c0 < g1; c0 += kUsageBS) {
        const int g = c0 + tid;
#pragma unroll
        for (int which = 0; which < 2; ++which) {
            const bool f = g < g1 && has_rows(g, which);
            const unsigned long long bal = __ballot(f);
            const int before = __popcll(bal & ((1ull << lane) - 1ull));
            if (lane == 0) wcount[which][wid] = __popcll(bal);
            __syncthreads();
            int off = base[which];
            for (int w = 0; w < wid; ++w) off += wcount[which][w];
            if (f && off + before < kMaxAct) (which == 0 ? sAct : sActN)[off + before] = g;
            __syncthreads();
            if (tid == 0) {
                int tot = 0;
                for (int w = 0; w < kUsageBS / 64; ++w) tot += wcount[which][w];
                base[which] += tot;
            }
            __syncthreads();
        }
    }
    const int nact = base[0], nactN = base[1];   // > kMaxAct: scan the flags instead of the list
    for (int gi = 0; gi < kGrids; ++gi) {
        const GridArgs &gd = pa.gr[gi];
        if (!gd.on) continue;
        const float *src = W.Ucoef_k + (((size_t)b * G.K + k) * kGrids + gi) * kUcEntries;
        const int n = gd.nc * kNC + gd.SP;
        for (int x = tid; x < n; x += kUsageBS) sC[gi][x] = src[x];
    }
    __syncthreads();
    // thread (row part ry, slot): the step-by-step rows ry, ry + RP, ... of
    // the slot's steps, then the row parts are added in order by ry = 0
    constexpr int NS = kUsageBS / RP;   // slots per work-group
    const int ry = tid / NS, sl = tid % NS, slot = blockIdx.x * NS + sl;
    __shared__ double sPart[RP][NS];
    // fp64 sums: the softmax of the smooth peak terms amplifies a usage error
    // dU by about dU/tau, so U is formed to well below fp32 rounding of its sum
    double rows = 0.0;
    const int P = G.parts;
    if (slot < T) {
        for (int t = slot; t < D; t += T) {
            if (nact <= kMaxAct && P == 1) {
                // four rows in flight at a time (the sum order stays the row order)
                const float *ub = W.Upart + (size_t)b * G.ngroups * D + t;
                int r = ry;
                for (; r + 3 * RP < nact; r += 4 * RP) {
                    const float u0 = ub[(size_t)sAct[r] * D], u1 = ub[(size_t)sAct[r + RP] * D];
                    const float u2 = ub[(size_t)sAct[r + 2 * RP] * D], u3 = ub[(size_t)sAct[r + 3 * RP] * D];
                    rows += u0; rows += u1; rows += u2; rows += u3;
                }
                for (; r < nact; r += RP) rows += ub[(size_t)sAct[r] * D];
            } else if (nact <= kMaxAct) {
                for (int r = ry; r < nact * P; r += RP)
                    rows += W.Upart[(((size_t)b * G.ngroups + sAct[r / P]) * P + r % P) * D + t];
            } else if (ry == 0) {
                for (int g = g0; g < g1; ++g)
                    if (has_rows(g, 0))
                        for (int pt = 0; pt < P; ++pt) rows += W.Upart[(((size_t)b * G.ngroups + g) * P + pt) * D + t];
            }
            // the narrow kernel's rows (one per group), eight loads in flight
            // (the sum order stays the row order)
            if (nactN <= kMaxAct) {
                const float *nb = W.Unar + (size_t)b * G.ngroups * D + t;
                int r = ry;
                for (; r + 7 * RP < nactN; r += 8 * RP) {
                    float u8[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) u8[k] = nb[(size_t)sActN[r + k * RP] * D];
#pragma unroll
                    for (int k = 0; k < 8; ++k) rows += u8[k];
                }
                for (; r < nactN; r += RP) rows += nb[(size_t)sActN[r] * D];
            } else if (ry == 0) {
                for (int g = g0; g < g1; ++g)
                    if (has_rows(g, 1)) rows += W.Unar[((size_t)b * G.ngroups + g) * D + t];
            }
        }
    }
    sPart[ry][sl] = rows;
    __syncthreads();
    if (ry != 0 || slot >= T) return;
    double acc = 0.0;
#pragma unroll
    for (int y = 0; y < RP; ++y) acc += sPart[y][sl];
    for (int t = slot; t < D; t += T) {
        double ut = 0.0;
        for (int gi = 0; gi < kGrids; ++gi) {
            const GridArgs &gd = pa.gr[gi];
            if (!gd.on) continue;
            if (t >= gd.L0 && t < D - 2) {
                const int c = (t - gd.L0) / gd.W;
                const float x = (float)(t - gd.L0 - c * gd.W) - gd.lam;
                const float *cf = sC[gi] + c * kNC;
                float v = cf[kNC - 1];
#pragma unroll
                for (int q = kNC - 2; q >= 0; --q) v = fmaf(v, x, cf[q]);
                ut += (double)v;
            } else {
                ut += (double)sC[gi][gd.nc * kNC + (t < gd.L0 ? t : gd.L0 + (t - (D - 2)))];
            }
        }
        acc += ut;
    }
    W.U[((size_t)b * G.K + k) * T + slot] = (float)acc;
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
// Expected storage units per (modulo) slot: the groups' partials summed and
// folded (eq:active, App. B.3); then per restart the smooth peak
// L_mem = M + tau log sum_t exp((MReg(t) - M)/tau) and gamma times its
// derivative (a softmax) per slot.
// ---------------------------------------------------------------------------
// Storage profile coefficients of the polynomial holders summed over the
// work-groups of a restart (16 strided partial sums per entry, fp64).
__global__ __launch_bounds__(64 * kUcoefRows) void k_mcoef(Graph G, PolyArgs pa, Work W) {
    __shared__ double part[kUcoefRows][64];
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int x = blockIdx.x * 64 + tx, b = blockIdx.y;
    const int nslot = G.ngroups * pa.split;
    const size_t rb = (size_t)b * nslot;
    const int ncoef = pa.nc * kNC;
    double acc = 0.0;
    if (x < ncoef) {
        for (int g = ty; g < nslot; g += kUcoefRows) acc += W.mcoef[(rb + g) * kMaxChunks * kNC + x];
    } else if (x < ncoef + pa.SP) {
        for (int g = ty; g < nslot; g += kUcoefRows) acc += W.mstrip[(rb + g) * kStripMax + (x - ncoef)];
    }
    part[ty][tx] = acc;
    __syncthreads();
    if (ty == 0 && x < ncoef + pa.SP) {
        double t = 0.0;
#pragma unroll
        for (int r = 0; r < kUcoefRows; ++r) t += part[r][tx];
        W.mcoef_r[(size_t)b * (kMaxChunks * kNC + kStripMax) + x] = t;
    }
}

// Storage profile per (modulo) slot: the step-by-step holders' group partials
// plus, with the polynomial path on, the polynomial holders' chunk
// polynomial at t (or their strip value), in fp64.
__global__ __launch_bounds__(256) void k_mreg(Graph G, PolyArgs pa, Work W) {
    const int slot = blockIdx.x * 256 + threadIdx.x, b = blockIdx.y;
    if (slot >= G.T) return;
    const double *mc = W.mcoef_r + (size_t)b * (kMaxChunks * kNC + kStripMax);
    const int D = G.D, ncoef = pa.nc * kNC;
    double acc = 0.0;
    for (int t = slot; t < D; t += G.T) {
        for (int g = 0; g < G.ngroups; ++g) acc += W.Mpart[((size_t)b * G.ngroups + g) * D + t];
        if (pa.enabled) {
            if (t >= pa.L0 && t < D - 2) {
                const int c = (t - pa.L0) / pa.W;
                const double y = (double)(t - pa.L0 - c * pa.W) - (double)pa.lam;
                double v = mc[c * kNC + kNC - 1];
                for (int k = kNC - 2; k >= 0; --k) v = fma(v, y, mc[c * kNC + k]);
                acc += v;
            } else {
                acc += mc[ncoef + (t < pa.L0 ? t : pa.L0 + (t - (D - 2)))];
            }
        }
    }
    W.mregd[(size_t)b * G.T + slot] = acc;
    W.mreg[(size_t)b * G.T + slot] = (float)acc;
}

__global__ __launch_bounds__(kTermsBS) void k_mem_lse(Graph G, Work W, HP hp) {
    __shared__ float scratch[kTermsBS / 64];
    const int b = blockIdx.x, tid = threadIdx.x, T = G.T;
    const double *mr = W.mregd + (size_t)b * T;
    // the maximum in fp64 (the profile's own precision), exponents in fp32
    __shared__ double dmax[kTermsBS / 64];
    double mx = -INFINITY;
    for (int c = tid; c < T; c += kTermsBS) mx = fmax(mx, mr[c]);
    for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off, 64));
    if ((tid & 63) == 0) dmax[tid >> 6] = mx;
    __syncthreads();
    mx = dmax[0];
    for (int w = 1; w < kTermsBS / 64; ++w) mx = fmax(mx, dmax[w]);
    const float itau = 1.0f / hp.tau;
    float z = 0.0f;
    for (int c = tid; c < T; c += kTermsBS) z += expf((float)(mr[c] - mx) * itau);
    z = block_sum1024(z, scratch);
    if (tid == 0) W.lmem[b] = (float)(mx + (double)hp.tau * log((double)z));
    const float gz = hp.gamma / z;
    float *ms = W.msoft + (size_t)b * T;
    for (int c = tid; c < T; c += kTermsBS) ms[c] = gz * expf((float)(mr[c] - mx) * itau);
}

// ---------------------------------------------------------------------------
// Per restart: V_res, V_dep, L_com, V_rec from the partials, the augmented
// Lagrangian (eq. 11), the weights w_c = lambda_c + rho V_c, and in step mode
// the multiplier update lambda_c += rho V_c and the Adam bias corrections.
// ---------------------------------------------------------------------------
constexpr int kCombineBS = 1024;

__global__ __launch_bounds__(kCombineBS) void k_combine(Graph G, PolyArgs pa, Work W, HP hp,
                                                        const float *__restrict__ lambda_in,
                                                        float *lambda_out, const int *adam_t,
                                                        float *terms_out) {
    __shared__ float scratch[5][kCombineBS / 64];
    const int b = blockIdx.x, tid = threadIdx.x;
    float vres = 0.0f, vdep = 0.0f, lcom = 0.0f, vrec = 0.0f, lres = 0.0f;
    for (int k = tid; k < G.K; k += kCombineBS) {
        vres += W.vres_part[(size_t)b * G.K + k];
        lres += W.lres_part[(size_t)b * G.K + k];
    }
    for (int gi = 0; gi < kGrids; ++gi) {
        const GridArgs &gd = pa.gr[gi];
        if (!gd.on) continue;
        const int npoly = G.ngroups * gd.split;
        const unsigned *gb = W.gbits + (size_t)b * G.ngroups;
        for (int g = tid; g < npoly; g += kCombineBS) {
            if (!(gb[g / gd.split] & (kGbGrid << gi))) continue;
            const size_t sl = (size_t)gd.slot_base + (size_t)b * npoly + g;
            vdep += W.gsum_poly[sl * 2]; lcom += W.gsum_poly[sl * 2 + 1];
        }
    }
    for (int g = tid; g < G.ngroups; g += kCombineBS) {
        const size_t bg = (size_t)b * G.ngroups + g;
        if (!(W.gbits[bg] & kGbStep)) continue;
        const unsigned nar = G.nar_on ? W.gnar[bg] : kNarLeft;
        if (nar & kNarLeft) {
            const float *go = W.gsum_ops + bg * G.parts * G.ntiles * 2;
            for (int tl = 0; tl < G.parts * G.ntiles; ++tl) { vdep += go[2 * tl]; lcom += go[2 * tl + 1]; }
        }
        if (nar & kNarTaken) { vdep += W.gsum_nar[bg * 2]; lcom += W.gsum_nar[bg * 2 + 1]; }
    }
    if (G.lap_on)   // Laplace: the closed-form edge sums per block of edges
        for (int k = tid; k < lap_blocks(G); k += kCombineBS) {
            vdep += W.gsum_lap[((size_t)b * lap_blocks(G) + k) * 2];
            lcom += W.gsum_lap[((size_t)b * lap_blocks(G) + k) * 2 + 1];
        }
    const size_t nbp = (size_t)G.nb * G.ntiles;
    const float *bp = W.bpart + (size_t)b * nbp * kBP;
    for (size_t r = tid; r < nbp; r += kCombineBS) vrec += bp[r * kBP + 0];
    // the five sums: per wave, then over the waves in order (one barrier)
    {
        const int lane = tid & 63, wid = tid >> 6;
        const float v5[5] = {vres, vdep, lcom, vrec, lres};
#pragma unroll
        for (int c = 0; c < 5; ++c) {
            const float r = wave_sum(v5[c]);
            if (lane == 0) scratch[c][wid] = r;
        }
    }
    __syncthreads();
    if (tid == 0) {
        float t5[5];
#pragma unroll
        for (int c = 0; c < 5; ++c) {
            float r = 0.0f;
            for (int w = 0; w < kCombineBS / 64; ++w) r += scratch[c][w];
            t5[c] = r;
        }
        vres = t5[0]; vdep = t5[1]; lcom = t5[2]; vrec = t5[3]; lres = t5[4];

        const float V[3] = {vdep, vres, vrec};
        const float *lam = lambda_in + (size_t)b * 3;
        const float lmem = hp.gamma != 0.0f ? W.lmem[b] : 0.0f;
        float L = fmaf(hp.gamma, lmem, fmaf(hp.beta, lres, hp.alpha * lcom));
        float w[3];
        for (int c = 0; c < 3; ++c) {
            L += lam[c] * V[c] + 0.5f * hp.rho * V[c] * V[c];
            w[c] = lam[c] + hp.rho * V[c];
        }
        float *tm = W.terms + (size_t)b * kTerms;
        tm[0] = L; tm[1] = vdep; tm[2] = vres; tm[3] = vrec; tm[4] = lcom; tm[5] = lres; tm[6] = lmem;
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
// In-edge records of the ops with more than kBigIn predecessors (a sink
// joined to every leaf has thousands), reduced by one work-group each in
// fp64 and a fixed order: consumer-side dependency / edge-length derivatives
// and, with the storage term, the successor-side storage derivatives.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_gather_big(Graph G, Work W, HP hp, const float *__restrict__ mu) {
    __shared__ double sRed[4][6];
    const int x = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int i = G.big_ops[x], N = G.N, nt = G.ntiles;
    const bool poly_i = W.cls[(size_t)b * N + i] != 0;
    // step-by-step in-edge records exist only in the tiles the op's spread
    // meets (tile_cons_rec, the op kernel's own test)
    const float kZF = fam_zflush_rt(hp.family), m_i = mu[(size_t)b * N + i], rs = W.rsig[(size_t)b * N + i];
    double acc[6] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    for (int q = G.pred_ptr[i] + tid; q < G.pred_ptr[i + 1]; q += 256) {
        const int e = G.pred_eid[q];
        const size_t bs = (size_t)b * N + G.pred_src[q];
        if ((poly_i && W.cls[bs]) || W.dflag[bs] == 2 || G.lap_on) {   // single record of the edge
            const float *cp = W.cpoly + ((size_t)b * G.E + e) * kCP;
            for (int c = 0; c < 4; ++c) acc[c] += cp[c];
        } else {
            const float *cp = W.cpart + (((size_t)b * G.E + e) * nt) * kCP;
            for (int tl = 0; tl < nt; ++tl) {
                const int t0 = tl * G.tile;
                if (!tile_cons_rec(kZF, m_i, rs, t0, min(t0 + G.tile, G.D))) continue;
                for (int c = 0; c < 4; ++c) acc[c] += cp[tl * kCP + c];
            }
        }
        if (hp.gamma != 0.0f) {
            if (W.mpoly[(size_t)b * N + G.pred_src[q]]) {   // producer's storage term on the polynomials
                acc[4] += W.mspoly[((size_t)b * G.E + e) * 2 + 0];
                acc[5] += W.mspoly[((size_t)b * G.E + e) * 2 + 1];
            } else {
                const float *sp = W.msucc + ((size_t)b * G.E + e) * nt * 2;
                for (int tl = 0; tl < nt; ++tl) { acc[4] += sp[tl * 2 + 0]; acc[5] += sp[tl * 2 + 1]; }
            }
        }
    }
#pragma unroll
    for (int c = 0; c < 6; ++c) {
        double v = acc[c];
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
        if (lane == 0) sRed[wid][c] = v;
    }
    __syncthreads();
    if (tid < 6)
        W.bigsum[((size_t)b * G.nbig + x) * 6 + tid] = (sRed[0][tid] + sRed[1][tid]) + (sRed[2][tid] + sRed[3][tid]);
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
    // work-group x serves restart x mod B: work-groups are dealt to the 8 XCDs
    // in turn, so with B a multiple of 8 each restart's records (gathered at
    // random through the in-edges) stay in one XCD's L2
    const int b = blockIdx.x % G.B;
    const int i = (blockIdx.x / G.B) * blockDim.x + threadIdx.x;
    if (i >= G.N) return;
    const int N = G.N, nt = G.ntiles;
    const size_t bi = (size_t)b * N + i;
    const float m_i = mu[bi], s_i = sigma[bi];
    const float rs = W.rsig[bi], cinv = rs * fam_k_rt(hp.family);
    const float *wt = W.wts + (size_t)b * 4;
    const float w_dep = wt[0], w_res = wt[1], w_rec = wt[2];

    // resource term through the indicator changes of this op's type
    const int k = G.rtype[i];
    const int nt_k = W.ntrans[(size_t)b * G.K + k];
    const int *tr = W.trans + ((size_t)b * G.K + k) * G.D;
    // partial sums in fp64: an op can collect thousands of edge records
    // (e.g. a sink joined to every leaf)
    double rm = 0.0, rsg = 0.0;
    for (int q = 0; q < nt_k; ++q) {
        const int code = tr[q];
        const float sgn = code > 0 ? 1.0f : -1.0f;
        const int t = (code > 0 ? code : -code) - 1;
        const float z = ((float)t + 0.5f - m_i) * rs;
        const float Fm = -fam_h_rt(hp.family, z) * cinv;
        rm += (double)(sgn * Fm);
        rsg += (double)(sgn * (Fm * z));
    }

    // step-by-step records exist only in the tiles the op's spreads meet
    // (tile_prod_rec / tile_cons_rec, the op kernel's own tests)
    const float kZF = fam_zflush_rt(hp.family);
    unsigned cons_tiles = 0;   // bit t: tile t holds records of edges into this op (nt <= 32)
    if (nt <= 32)
        for (int tl = 0; tl < nt; ++tl) {
            const int t0 = tl * G.tile;
            cons_tiles |= tile_cons_rec(kZF, m_i, rs, t0, min(t0 + G.tile, G.D)) ? 1u << tl : 0u;
        }
    auto cons_tile = [&](int tl) {
        if (nt <= 32) return ((cons_tiles >> tl) & 1u) != 0;
        const int t0 = tl * G.tile;
        return tile_cons_rec(kZF, m_i, rs, t0, min(t0 + G.tile, G.D));
    };
    double dm = 0.0, ds = 0.0, cm = 0.0, cs = 0.0;
    const int dfl = W.dflag[bi];   // 1: op-kernel records per tile, 2: narrow kernel's single record
    if (dfl == 1 && !G.lap_on) {   // (Laplace: the producer terms are all in the closed-form record)
        const float *pp = W.ppart + bi * nt * kPP;
        const int lat_i = G.delay[i];
        for (int tl = 0; tl < nt; ++tl) {
            const int t0 = tl * G.tile;
            if (!tile_prod_rec(kZF, m_i, rs, lat_i, t0, min(t0 + G.tile, G.D))) continue;
            dm += pp[tl * kPP + 2]; ds += pp[tl * kPP + 3];
            cm += pp[tl * kPP + 4]; cs += pp[tl * kPP + 5];
        }
    }
    const bool poly_i = W.cls[bi] != 0;
    if (G.lap_on) {   // Laplace: the closed-form records of the out-edges
        for (int e = G.row_ptr[i]; e < G.row_ptr[i + 1]; ++e) {
            const float4 p4 = *reinterpret_cast<const float4 *>(W.pedge + ((size_t)b * G.E + e) * 4);
            dm += p4.x; ds += p4.y; cm += p4.z; cs += p4.w;
        }
    } else if (poly_i || dfl == 2) {   // single producer record (polynomial path, or the narrow kernel)
        const float *ppy = W.ppoly + bi * kPP;
        dm += ppy[2]; ds += ppy[3]; cm += ppy[4]; cs += ppy[5];
    }
    const int big = G.big_of[i];
    const double *bsum = big >= 0 ? W.bigsum + ((size_t)b * G.nbig + big) * 6 : nullptr;
    if (bsum) { dm += bsum[0]; ds += bsum[1]; cm += bsum[2]; cs += bsum[3]; }
    // in-edges four at a time: their ids, then the producers' flags and the
    // single records (loaded whether used or not), then the sums in edge order
    constexpr int kInB = 4;
    const int qa = bsum ? G.pred_ptr[i + 1] : G.pred_ptr[i], qb = G.pred_ptr[i + 1];
    for (int q0 = qa; q0 < qb; q0 += kInB) {
        int ev[kInB], sv[kInB];
#pragma unroll
        for (int k = 0; k < kInB; ++k) {
            const int q = min(q0 + k, qb - 1);
            ev[k] = G.pred_eid[q]; sv[k] = G.pred_src[q];
        }
        bool one[kInB];
        float4 r4[kInB];
#pragma unroll
        for (int k = 0; k < kInB; ++k) {
            const size_t bs = (size_t)b * N + sv[k];
            one[k] = (poly_i && W.cls[bs]) || W.dflag[bs] == 2 || G.lap_on;   // single record of the edge
            r4[k] = *reinterpret_cast<const float4 *>(W.cpoly + ((size_t)b * G.E + ev[k]) * kCP);
        }
#pragma unroll
        for (int k = 0; k < kInB; ++k) {
            if (q0 + k >= qb) break;
            if (one[k]) {
                dm += r4[k].x; ds += r4[k].y; cm += r4[k].z; cs += r4[k].w;
                continue;
            }
            const float *cp = W.cpart + (((size_t)b * G.E + ev[k]) * nt) * kCP;
            for (int tl = 0; tl < nt; ++tl) {
                if (!cons_tile(tl)) continue;
                dm += cp[tl * kCP + 0]; ds += cp[tl * kCP + 1];
                cm += cp[tl * kCP + 2]; cs += cp[tl * kCP + 3];
            }
        }
    }
    double qm = 0.0, qs = 0.0;
    for (int q = G.bout_ptr[i]; q < G.bout_ptr[i + 1]; ++q) {
        const float *bp = W.bpart + (((size_t)b * G.nb + G.bout[q]) * nt) * kBP;
        for (int tl = 0; tl < nt; ++tl) { qm += bp[tl * kBP + 1]; qs += bp[tl * kBP + 2]; }
    }
    for (int q = G.bin_ptr[i]; q < G.bin_ptr[i + 1]; ++q) {
        const float *bp = W.bpart + (((size_t)b * G.nb + G.bin[q]) * nt) * kBP;
        for (int tl = 0; tl < nt; ++tl) { qm += bp[tl * kBP + 3]; qs += bp[tl * kBP + 4]; }
    }
    float g_mu = combine_grad(w_res, (float)rm, w_dep, (float)dm, w_rec, (float)qm, hp.alpha, (float)cm);
    float g_sg = combine_grad(w_res, (float)rsg, w_dep, (float)ds, w_rec, (float)qs, hp.alpha, (float)cs);
    if (hp.beta != 0.0f) {   // smooth peak usage, already weighted by beta
        double lm = 0.0, ls = 0.0;
        if (poly_i) {
            lm = W.lpoly[bi * 2 + 0]; ls = W.lpoly[bi * 2 + 1];
        } else {
            const float *lp = W.lpart + bi * nt * 2;
            for (int tl = 0; tl < nt; ++tl) { lm += lp[tl * 2 + 0]; ls += lp[tl * 2 + 1]; }
        }
        g_mu = __fadd_rn(g_mu, (float)lm);
        g_sg = __fadd_rn(g_sg, (float)ls);
    }
    if (hp.gamma != 0.0f) {   // smooth peak storage, already weighted by gamma
        double om = 0.0, os = 0.0;
        if (W.mpoly[bi]) {   // holder on the polynomials
            om += W.mopoly[bi * 2 + 0]; os += W.mopoly[bi * 2 + 1];
        } else if (G.row_ptr[i + 1] > G.row_ptr[i]) {
            const float *op = W.mown + bi * nt * 2;
            for (int tl = 0; tl < nt; ++tl) { om += op[tl * 2 + 0]; os += op[tl * 2 + 1]; }
        }
        if (bsum) { om += bsum[4]; os += bsum[5]; }
        for (int q = bsum ? G.pred_ptr[i + 1] : G.pred_ptr[i]; q < G.pred_ptr[i + 1]; ++q) {
            const int e = G.pred_eid[q];
            if (W.mpoly[(size_t)b * N + G.pred_src[q]]) {
                om += W.mspoly[((size_t)b * G.E + e) * 2 + 0];
                os += W.mspoly[((size_t)b * G.E + e) * 2 + 1];
            } else {
                const float *sp = W.msucc + ((size_t)b * G.E + e) * nt * 2;
                for (int tl = 0; tl < nt; ++tl) { om += sp[tl * 2 + 0]; os += sp[tl * 2 + 1]; }
            }
        }
        g_mu = __fadd_rn(g_mu, (float)om);
        g_sg = __fadd_rn(g_sg, (float)os);
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

// The same with the schedule in LDS (chosen on the host when it fits:
// 16-bit entries for II = 0 with D < 2^15, where every value stays in
// [ASAP, ALAP]; 32-bit entries, with the pass snapshot beside them, for
// II > 0 when no value can leave the 32-bit range).  LDS holds the ready
// time r_v = s_v + Lat_v, so a predecessor costs one LDS read; each thread's
// op of the next level is loaded during the current level as one 32-byte
// item (op, delay, predecessor count, the first kLegPre predecessors), so the
// per-level barrier does not wait on dependent global loads.
constexpr int kLegLdsBS = 1024;
constexpr int kLegInitU = 4;    // ops per thread and round of the initial rounding (loads in flight)

// Work-group barrier for LDS-only communication: waits for this wave's LDS
// accesses (lgkmcnt 0), not for its global loads, so loads issued for later
// levels stay in flight across it (__syncthreads would also wait for them).
__device__ __forceinline__ void lds_barrier() {
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);   // vmcnt 63, expcnt 7, lgkmcnt 0
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
}

struct LegItem {
    int v, dv, n, p0;
    int u[kLegPre];
};

// Item q, clamped into [0, N) (the caller tests q against its level's end):
// the load is issued on every path, which keeps its wait count predictable.
__device__ __forceinline__ void leg_load(const Graph &G, int q, int q1, LegItem &it) {
    (void)q1;
    const size_t qc = (size_t)min(q, G.N - 1);
    const int4 a = reinterpret_cast<const int4 *>(G.leg_items)[2 * qc];
    const int4 c = reinterpret_cast<const int4 *>(G.leg_items)[2 * qc + 1];
    it.v = a.x; it.dv = a.y; it.n = a.z; it.p0 = a.w;
    it.u[0] = c.x; it.u[1] = c.y; it.u[2] = c.z; it.u[3] = c.w;
}

template <typename T>
__global__ __launch_bounds__(kLegLdsBS) void k_legalize_lds(Graph G, Work W, const float *__restrict__ mu,
                                                         int *sched) {
    extern __shared__ __align__(16) unsigned char sDynLeg[];
    const int nl = G.nlevels, nlp = (nl + 1 + 3) & ~3;
    int *lp = reinterpret_cast<int *>(sDynLeg);         // level bounds (lvl_ptr)
    T *rd = reinterpret_cast<T *>(lp + nlp);            // ready times s_v + Lat_v
    T *rp = rd + G.N;                                  // II > 0: their snapshot at the start of a pass
    __shared__ int changed, over;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = G.N, D = G.D;
    for (int l = tid; l <= nl; l += kLegLdsBS) lp[l] = G.lvl_ptr[l];
    for (int v0 = tid; v0 < N; v0 += kLegInitU * kLegLdsBS) {
        float m[kLegInitU];
        int lo[kLegInitU], hi[kLegInitU], dl[kLegInitU];
#pragma unroll
        for (int k = 0; k < kLegInitU; ++k) {
            const int v = v0 + k * kLegLdsBS;
            if (v < N) {
                m[k] = mu[(size_t)b * N + v];
                lo[k] = G.II == 0 ? G.asap[v] : 0;
                hi[k] = G.II == 0 ? G.alap[v] : D - 1;
                dl[k] = G.delay[v];
            }
        }
#pragma unroll
        for (int k = 0; k < kLegInitU; ++k) {
            const int v = v0 + k * kLegLdsBS;
            if (v < N) {
                long long r = round_half_up(m[k], D);
                r = r < lo[k] ? lo[k] : (r > hi[k] ? hi[k] : r);
                rd[v] = (T)(r + dl[k]);
            }
        }
    }
    __syncthreads();
    int st = 0;
    // levels l0.. of one sweep; each thread's first item of a level is loaded
    // two levels ahead into one of two buffers (A: levels l0, l0+2, ...; B:
    // l0+1, ...), reloaded right after its level is done, so no register
    // rotation makes the next level wait for the newest loads
    auto process = [&](const LegItem it, bool modulo) {
        const int v = it.v;
        long long req = modulo ? 0 : (long long)rd[v] - it.dv;
#pragma unroll
        for (int k = 0; k < kLegPre; ++k)
            if (k < it.n) req = max(req, (long long)rd[it.u[k]]);
        for (int k = kLegPre; k < it.n; ++k) req = max(req, (long long)rd[G.leg_over[it.p0 + k - kLegPre]]);
        if (modulo) {
            for (int r = G.bin_ptr[v]; r < G.bin_ptr[v + 1]; ++r) {
                const int e = G.bin[r], j = G.bsrc[e];
                req = max(req, (long long)rp[j] - (long long)G.bdist[e] * G.II);
            }
            if (req > (long long)rd[v] - it.dv) { rd[v] = (T)(req + it.dv); changed = 1; }
        } else {
            rd[v] = (T)(req + it.dv);
        }
    };
    auto level = [&](int l, LegItem cur, bool modulo) -> LegItem {
        const int qa = lp[l], qb = lp[l + 1];
        if (qa + tid < qb) process(cur, modulo);
        for (int q = qa + tid + kLegLdsBS; q < qb; q += kLegLdsBS) {   // levels wider than the work-group
            LegItem it;
            leg_load(G, q, qb, it);
            process(it, modulo);
        }
        const int l2 = min(l + 2, nl - 1);   // past the last level: a valid, unused item
        leg_load(G, lp[l2] + tid, lp[l2 + 1], cur);
        lds_barrier();
        return cur;
    };
    auto sweep = [&](int l0, bool modulo) {
        LegItem A{}, B{};
        leg_load(G, lp[l0] + tid, lp[l0 + 1], A);
        const int l1 = min(l0 + 1, nl - 1);
        leg_load(G, lp[l1] + tid, lp[l1 + 1], B);
        for (int l = l0; l < nl; l += 2) {
            A = level(l, A, modulo);
            if (l + 1 < nl) B = level(l + 1, B, modulo);
        }
    };
    if (G.II == 0) {
        if (G.nlevels > 1) sweep(1, false);
    } else {
        int converged = 0;
        for (int pass = 0; pass < (N > 0 ? N : 1); ++pass) {
            for (int v = tid; v < N; v += kLegLdsBS) rp[v] = rd[v];
            if (tid == 0) changed = 0;
            __syncthreads();
            if (G.nlevels > 0) sweep(0, true);
            const int ch = changed;
            __syncthreads();
            if (!ch) { converged = 1; break; }
        }
        if (!converged) {
            st = 4;  // GAUS_E_NOT_CONVERGED
        } else {
            if (tid == 0) over = 0;
            __syncthreads();
            for (int v = tid; v < N; v += kLegLdsBS)
                if ((long long)rd[v] - G.delay[v] > D - 1) over = 1;
            __syncthreads();
            st = over ? 5 : 0;  // GAUS_E_OVERFLOW
        }
    }
    for (int v = tid; v < N; v += kLegLdsBS) sched[(size_t)b * N + v] = (int)((long long)rd[v] - G.delay[v]);
    if (tid == 0) W.status[b] = st;
}

// Alg. 3 (II = 0) with the level items in a double-buffered LDS ring: the
// host cuts the items of levels 1 .. nlevels-1 (in level order) into batches
// whose items and predecessors past the first kLegPre fit one half of the
// ring (a wide level spans batches; its items are independent, and batches
// run in order); while batch k is processed from one half, the global loads
// of batch k+1 are in flight into registers and are written to the other
// half afterwards, so a level costs LDS reads and an LDS-only barrier.  Same
// arithmetic as k_legalize_lds, so the same schedules.
constexpr int kLegRingBS = 512;
constexpr int kLegRingV4 = 8;   // 16-byte loads staged per thread and batch (two per item)
constexpr int kLegRingOv = 4;   // overflow predecessors staged per thread and batch
constexpr int kLegRingU = 16;   // ops per thread and round of the rounding and the output (loads in flight)

template <typename T>
__global__ __launch_bounds__(kLegRingBS) void k_legalize_ring(Graph G, Work W, const float *__restrict__ mu,
                                                           int *sched) {
    extern __shared__ __align__(16) unsigned char sDynLeg[];
    const int nl = G.nlevels, nlp = (nl + 1 + 3) & ~3, nb = G.leg_nbatch, nbt = (3 * (nb + 1) + 3) & ~3;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = G.N, D = G.D;
    // LDS: level bounds, the batch table, ready times s_v + Lat_v, the ring.
    // Everything the level loop reads is in LDS, so its waits are LDS waits
    // and the staged global loads of the next batch stay in flight.
    int *lp = reinterpret_cast<int *>(sDynLeg);
    int *bt = lp + nlp;
    T *rd = reinterpret_cast<T *>(bt + nbt);
    const size_t rd_bytes = (sizeof(T) * (size_t)N + 15) & ~size_t(15);
    int4 *ring = reinterpret_cast<int4 *>(reinterpret_cast<unsigned char *>(rd) + rd_bytes);
    const int RI = G.leg_ring_items, RO = G.leg_ring_over;
    const int HS = 2 * RI + (RO + 3) / 4;               // int4 per ring half: items, then overflow
    for (int l = tid; l <= nl; l += kLegRingBS) lp[l] = G.lvl_ptr[l];
    for (int q = tid; q < 3 * (nb + 1); q += kLegRingBS) bt[q] = G.leg_batch[q];
    for (int v0 = tid; v0 < N; v0 += kLegRingU * kLegRingBS) {
        float m[kLegRingU];
        int lo[kLegRingU], hi[kLegRingU], dl[kLegRingU];
#pragma unroll
        for (int k = 0; k < kLegRingU; ++k) {
            const int v = v0 + k * kLegRingBS;
            if (v < N) { m[k] = mu[(size_t)b * N + v]; lo[k] = G.asap[v]; hi[k] = G.alap[v]; dl[k] = G.delay[v]; }
        }
#pragma unroll
        for (int k = 0; k < kLegRingU; ++k) {
            const int v = v0 + k * kLegRingBS;
            if (v < N) {
                long long r = round_half_up(m[k], D);
                r = r < lo[k] ? lo[k] : (r > hi[k] ? hi[k] : r);
                rd[v] = (T)(r + dl[k]);
            }
        }
    }
    __syncthreads();
    // staged data in native 4-vectors (plain registers)
    typedef int vi4 __attribute__((ext_vector_type(4)));
    const vi4 *items = reinterpret_cast<const vi4 *>(G.leg_items);
    vi4 *vring = reinterpret_cast<vi4 *>(ring);
    vi4 sv[kLegRingV4];
    int so[kLegRingOv];
    // batch 0 straight into half 0
    if (nb > 0) {
        const int q0 = bt[1], q1 = bt[4], o0 = bt[2], o1 = bt[5];
#pragma unroll
        for (int m = 0; m < kLegRingV4; ++m) {
            const int j = tid + m * kLegRingBS;
            sv[m] = items[j < 2 * (q1 - q0) ? 2 * (size_t)q0 + j : 0];
        }
#pragma unroll
        for (int m = 0; m < kLegRingOv; ++m) {
            const int j = tid + m * kLegRingBS;
            so[m] = G.leg_over[j < o1 - o0 ? o0 + j : 0];
        }
        int *ov = reinterpret_cast<int *>(ring + 2 * RI);
#pragma unroll
        for (int m = 0; m < kLegRingV4; ++m) {
            const int j = tid + m * kLegRingBS;
            if (j < 2 * (q1 - q0)) vring[j] = sv[m];
        }
#pragma unroll
        for (int m = 0; m < kLegRingOv; ++m) {
            const int j = tid + m * kLegRingBS;
            if (j < o1 - o0) ov[j] = so[m];
        }
    }
    __syncthreads();
    for (int k = 0; k < nb; ++k) {
        const int qb = bt[3 * k + 1], ob = bt[3 * k + 2], qe = bt[3 * k + 4], lb = bt[3 * k];
        const bool more = k + 1 < nb;
        const int nq0 = more ? bt[3 * k + 4] : 0, nq1 = more ? bt[3 * k + 7] : 0;
        const int no0 = more ? bt[3 * k + 5] : 0, no1 = more ? bt[3 * k + 8] : 0;
        // batch k+1 into registers: in flight while batch k is processed
        // (straight-line loads, each index clamped into its array, so that
        // no branch makes the compiler wait for the earlier ones)
#pragma unroll
        for (int m = 0; m < kLegRingV4; ++m) {
            const int j = tid + m * kLegRingBS;
            sv[m] = items[j < 2 * (nq1 - nq0) ? 2 * (size_t)nq0 + j : 0];
        }
#pragma unroll
        for (int m = 0; m < kLegRingOv; ++m) {
            const int j = tid + m * kLegRingBS;
            so[m] = G.leg_over[j < no1 - no0 ? no0 + j : 0];
        }
        const vi4 *base = vring + (size_t)(k & 1) * HS;
        const int *ov = reinterpret_cast<const int *>(base + 2 * RI);
        // one item: its ready time from its predecessors' (Alg. 3's raise)
        auto process = [&](const vi4 a, const vi4 c) __attribute__((always_inline)) {
            const int v = a.x, dv = a.y, n = a.z, p0 = a.w;
            // the first kLegPre predecessors read at once (absent ones read
            // v's own slot and count as 0: ready times are >= 0); values stay
            // below 2^31 (D + Lat < 2^31 for the LDS schedules)
            const int u[kLegPre] = {c.x, c.y, c.z, c.w};
            int x[kLegPre];
#pragma unroll
            for (int kk = 0; kk < kLegPre; ++kk) x[kk] = (int)rd[kk < n ? u[kk] : v];
            int req = (int)rd[v] - dv;
#pragma unroll
            for (int kk = 0; kk < kLegPre; ++kk) req = max(req, kk < n ? x[kk] : 0);
            // the rest four at a time: four independent index reads, then four
            // ready times (indices clamped into the overflow area; the values
            // past n are discarded)
            for (int kk = kLegPre; kk < n; kk += 4) {
                int w[4], y[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) w[j] = ov[min(p0 - ob + kk + j - kLegPre, RO - 1)];
#pragma unroll
                for (int j = 0; j < 4; ++j) y[j] = (int)rd[kk + j < n ? w[j] : v];
#pragma unroll
                for (int j = 0; j < 4; ++j) req = max(req, kk + j < n ? y[j] : 0);
            }
            rd[v] = (T)(req + dv);
        };
        // the levels this batch's items meet, one item per thread and level
        // (wider levels loop); the bounds and the item of the next level are
        // read before the barrier (they do not change during the batch), so
        // after it only the predecessors' ready times are waited for
        int l = lb;
        int qz = min(lp[l + 1], qe);
        int q = max(lp[l], qb) + tid;
        vi4 ia = {0, 0, 0, 0}, ic = {0, 0, 0, 0};
        if (q < qz) { ia = base[2 * (q - qb)]; ic = base[2 * (q - qb) + 1]; }
        while (true) {
            if (q < qz) process(ia, ic);
            for (int q2 = q + kLegRingBS; q2 < qz; q2 += kLegRingBS) process(base[2 * (q2 - qb)], base[2 * (q2 - qb) + 1]);
            const bool next = l + 1 < nl && lp[l + 1] < qe;
            if (next) {
                q = lp[l + 1] + tid;
                qz = min(lp[l + 2], qe);
                if (q < qz) { ia = base[2 * (q - qb)]; ic = base[2 * (q - qb) + 1]; }
            }
            lds_barrier();
            if (!next) break;
            ++l;
        }
        if (more) {   // the staged batch into the other half (its last readers finished batch k-1)
            vi4 *nbase = vring + (size_t)((k + 1) & 1) * HS;
            int *nov = reinterpret_cast<int *>(nbase + 2 * RI);
#pragma unroll
            for (int m = 0; m < kLegRingV4; ++m) {
                const int j = tid + m * kLegRingBS;
                if (j < 2 * (nq1 - nq0)) nbase[j] = sv[m];
            }
#pragma unroll
            for (int m = 0; m < kLegRingOv; ++m) {
                const int j = tid + m * kLegRingBS;
                if (j < no1 - no0) nov[j] = so[m];
            }
        }
        __syncthreads();
    }
    for (int v0 = tid; v0 < N; v0 += kLegRingU * kLegRingBS) {
        int dl[kLegRingU];
#pragma unroll
        for (int k = 0; k < kLegRingU; ++k) {
            const int v = v0 + k * kLegRingBS;
            dl[k] = v < N ? G.delay[v] : 0;
        }
#pragma unroll
        for (int k = 0; k < kLegRingU; ++k) {
            const int v = v0 + k * kLegRingBS;
            if (v < N) sched[(size_t)b * N + v] = (int)((long long)rd[v] - dl[k]);
        }
    }
    if (tid == 0) W.status[b] = 0;
}

size_t legalize_ring_lds(const Graph &g, int ready_bytes) {
    const size_t lvl = sizeof(int) * (size_t)((g.nlevels + 1 + 3) & ~3);
    const size_t bt = sizeof(int) * (size_t)((3 * (g.leg_nbatch + 1) + 3) & ~3);
    const size_t rd = ((size_t)ready_bytes * g.N + 15) & ~size_t(15);
    const size_t half = 16 * (2 * (size_t)g.leg_ring_items + (size_t)(g.leg_ring_over + 3) / 4);
    return lvl + bt + rd + 2 * half;
}

hipError_t launch_legalize(const Graph &g, const Work &w, const float *mu, int *sched, hipStream_t st) {
    const size_t lvl = sizeof(int) * (size_t)((g.nlevels + 1 + 3) & ~3);
    if (g.leg_ring && g.leg_mode == 1)
        hipLaunchKernelGGL(k_legalize_ring<short>, dim3(g.B), dim3(kLegRingBS), legalize_ring_lds(g, 2), st, g, w, mu,
                           sched);
    else if (g.leg_ring && g.leg_mode == 2)
        hipLaunchKernelGGL(k_legalize_ring<int>, dim3(g.B), dim3(kLegRingBS), legalize_ring_lds(g, 4), st, g, w, mu,
                           sched);
    else if (g.leg_mode == 1)
        hipLaunchKernelGGL(k_legalize_lds<short>, dim3(g.B), dim3(kLegLdsBS), lvl + sizeof(short) * (size_t)g.N, st,
                           g, w, mu, sched);
    else if (g.leg_mode == 2)
        hipLaunchKernelGGL(k_legalize_lds<int>, dim3(g.B), dim3(kLegLdsBS),
                           lvl + sizeof(int) * (size_t)g.N * (g.II > 0 ? 2 : 1), st, g, w, mu, sched);
    else
        hipLaunchKernelGGL(k_legalize, dim3(g.B), dim3(kLegBS), 0, st, g, w, mu, sched);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Discrete cost of integer schedules (Sec. 2.1): usage counts per (type,
// slot), storage held from s_i until the last successor starts (eq:mem) as a
// difference array in fixed point (integer sums are order-independent),
// sum of edge lengths, legality.  Then per restart: peaks, V_res, the cost
// alpha L_com + beta L_res + gamma L_mem.
// ---------------------------------------------------------------------------
constexpr double kMemFix = 1048576.0;   // storage units are counted in steps of 2^-20

__global__ void k_cost_clear(Graph G, Work W) {
    const int b = blockIdx.y;
    const size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t nh = (size_t)G.K * G.T, nd = (size_t)G.D + 1;
    if (x < nh) W.hist[(size_t)b * nh + x] = 0;
    if (x < nd) W.mdiff[(size_t)b * nd + x] = 0;
    if (x < (size_t)G.T) W.mprof[(size_t)b * G.T + x] = 0;
    if (x == 0) { W.lcom_acc[b] = 0; W.illegal[b] = 0; }
}

__global__ void k_cost_ops(Graph G, Work W, const int *__restrict__ sched) {
    const int b = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int N = G.N, D = G.D, T = G.T;
    const int *s = sched + (size_t)b * N;
    if (i < N) {
        const int si = s[i];
        bool bad = si < 0 || si > D - 1;
        if (!bad) atomicAdd(&W.hist[((size_t)b * G.K + G.rtype[i]) * T + si % T], 1);
        long long lc = 0;
        int last = -1;
        for (int e = G.row_ptr[i]; e < G.row_ptr[i + 1]; ++e) {
            const int sj = s[G.col[e]];
            if ((long long)sj < (long long)si + G.delay[i]) bad = true;
            if (sj > si) lc += (long long)sj - si;
            last = max(last, sj);
        }
        if (lc) atomicAdd(&W.lcom_acc[b], (unsigned long long)lc);
        const int lo = max(si, 0), hi = min(last, D);   // held at steps [s_i, last) inside the horizon
        if (lo < hi) {
            const long long v = llrint((double)G.bmem[i] * kMemFix);
            atomicAdd((unsigned long long *)&W.mdiff[(size_t)b * (D + 1) + lo], (unsigned long long)v);
            atomicAdd((unsigned long long *)&W.mdiff[(size_t)b * (D + 1) + hi], (unsigned long long)(-v));
        }
        if (bad) W.illegal[b] = 1;
    }
    if (i < G.nb) {   // back edge (producer j, consumer c, k): s_c + k II >= s_j + Lat_j
        const int j = G.bsrc[i], c = G.bdst[i];
        if ((long long)s[c] + (long long)G.bdist[i] * G.II < (long long)s[j] + G.delay[j]) W.illegal[b] = 1;
    }
}

constexpr int kCostBS = 1024;

// per restart: prefix sum of the storage differences, fold, peaks, V_res, cost
__global__ __launch_bounds__(kCostBS) void k_cost_final(Graph G, Work W, HP hp, double *cost) {
    __shared__ long long sScan[kCostBS];
    __shared__ double sRed[kCostBS / 64];
    __shared__ long long carry;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int D = G.D, T = G.T, K = G.K;
    const long long *md = W.mdiff + (size_t)b * (D + 1);
    long long *mp = W.mprof + (size_t)b * T;
    if (tid == 0) carry = 0;
    __syncthreads();
    for (int d0 = 0; d0 < D; d0 += kCostBS) {
        long long x = d0 + tid < D ? md[d0 + tid] : 0;
        sScan[tid] = x;
        __syncthreads();
        for (int off = 1; off < kCostBS; off <<= 1) {     // inclusive scan (Hillis-Steele)
            const long long y = tid >= off ? sScan[tid - off] : 0;
            __syncthreads();
            sScan[tid] += y;
            __syncthreads();
        }
        const long long held = carry + sScan[tid];
        if (d0 + tid < D) atomicAdd((unsigned long long *)&mp[(d0 + tid) % T], (unsigned long long)held);
        __syncthreads();
        if (tid == kCostBS - 1) carry = held;
        __syncthreads();
    }
    __threadfence();
    __syncthreads();
    // peaks and V_res (the profile is read back from L2, where the atomics landed)
    double lmem = 0.0, vres = 0.0, lres = 0.0;
    for (int t = tid; t < T; t += kCostBS)
        lmem = fmax(lmem, (double)__hip_atomic_load(&mp[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) / kMemFix);
    for (int k = 0; k < K; ++k) {
        double mx = 0.0;
        for (int t = tid; t < T; t += kCostBS) {
            const double u = (double)W.hist[((size_t)b * K + k) * T + t];
            mx = fmax(mx, u);
            if (u > (double)G.cap[k]) vres += u - (double)G.cap[k];
        }
        for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off, 64));
        if ((tid & 63) == 0) sRed[tid >> 6] = mx;
        __syncthreads();
        if (tid == 0) { double m2 = 0.0; for (int w = 0; w < kCostBS / 64; ++w) m2 = fmax(m2, sRed[w]); lres += m2; }
        __syncthreads();
    }
    for (int off = 32; off > 0; off >>= 1) {
        lmem = fmax(lmem, __shfl_xor(lmem, off, 64));
        vres += __shfl_xor(vres, off, 64);
    }
    __shared__ double sM[kCostBS / 64], sV[kCostBS / 64];
    if ((tid & 63) == 0) { sM[tid >> 6] = lmem; sV[tid >> 6] = vres; }
    __syncthreads();
    if (tid == 0) {
        double m2 = 0.0, v2 = 0.0;
        for (int w = 0; w < kCostBS / 64; ++w) { m2 = fmax(m2, sM[w]); v2 += sV[w]; }
        const double lcom = (double)W.lcom_acc[b];
        double *c = cost + (size_t)b * kCost;
        c[0] = (double)hp.alpha * lcom + (double)hp.beta * lres + (double)hp.gamma * m2;
        c[1] = lcom; c[2] = lres; c[3] = m2; c[4] = v2; c[5] = W.illegal[b] ? 0.0 : 1.0;
    }
}

hipError_t enqueue_schedule_cost(const Graph &g, const Work &w, const HP &hp, const int *sched, double *cost,
                                 hipStream_t st) {
    const size_t cells = std::max({(size_t)g.K * g.T, (size_t)g.D + 1, (size_t)g.T});
    hipLaunchKernelGGL(k_cost_clear, dim3((unsigned)((cells + 255) / 256), g.B), dim3(256), 0, st, g, w);
    hipLaunchKernelGGL(k_cost_ops, dim3((std::max(g.N, g.nb) + 255) / 256, g.B), dim3(256), 0, st, g, w, sched);
    hipLaunchKernelGGL(k_cost_final, dim3(g.B), dim3(kCostBS), 0, st, g, w, hp, cost);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Scratch of the allocation-free schedule cost: the usage counts, storage
// differences and profile, edge-length sums and legality flags of every
// restart (the buffers k_cost_* clear and fill) are carved from one
// file-scope device array instead of library allocations.  Each device holds
// its own copy until the process ends; host code takes its address on that
// device from hipGetSymbolAddress (cached per device) and never uses the
// array's name, which in host code is only a stand-in.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
}  // namespace

size_t cost_scratch_bytes(const Graph &g) {
    const size_t B = (size_t)g.B;
    return align256(sizeof(int) * B * g.K * g.T) + align256(sizeof(long long) * B * ((size_t)g.D + 1)) +
           align256(sizeof(long long) * B * g.T) + align256(sizeof(unsigned long long) * B) +
           align256(sizeof(int) * B);
}

hipError_t scratch_address(int device, void **out) {
    static std::mutex mu;
    static std::map<int, void *> by_device;
    std::lock_guard<std::mutex> lock(mu);
    auto it = by_device.find(device);
    if (it != by_device.end()) {
        *out = it->second;
        return hipSuccess;
    }
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // the current device's copy
    if (e != hipSuccess) return e;
    by_device[device] = p;
    *out = p;
    return hipSuccess;
}

hipError_t enqueue_schedule_cost_scratch(const Graph &g, const Work &w, const HP &hp, void *scratch_ptr,
                                         const int *sched, double *cost, hipStream_t st) {
    Work ws = w;   // the same kernels on buffers inside the scratch array
    unsigned char *q = static_cast<unsigned char *>(scratch_ptr);
    const size_t B = (size_t)g.B;
    ws.hist = reinterpret_cast<int *>(q);
    q += align256(sizeof(int) * B * g.K * g.T);
    ws.mdiff = reinterpret_cast<long long *>(q);
    q += align256(sizeof(long long) * B * ((size_t)g.D + 1));
    ws.mprof = reinterpret_cast<long long *>(q);
    q += align256(sizeof(long long) * B * g.T);
    ws.lcom_acc = reinterpret_cast<unsigned long long *>(q);
    q += align256(sizeof(unsigned long long) * B);
    ws.illegal = reinterpret_cast<int *>(q);
    return enqueue_schedule_cost(g, ws, hp, sched, cost, st);
}

// ---------------------------------------------------------------------------
// Alg. 1 driver check.  A schedule is feasible if legal and within the
// capacities (V_res = 0).  Order: feasible before infeasible; among feasible
// the lower cost; among infeasible legal before illegal, then the lower V_res,
// then the lower cost.
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool cost_better(const double *a, const double *b) {
    const bool fa = a[5] != 0.0 && a[4] == 0.0, fb = b[5] != 0.0 && b[4] == 0.0;
    if (fa != fb) return fa;
    if (fa) return a[0] < b[0];
    if (a[5] != b[5]) return a[5] != 0.0;
    if (a[4] != b[4]) return a[4] < b[4];
    return a[0] < b[0];
}

__global__ void k_best_init(int B, double *best_cost, Work W) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    double *c = best_cost + (size_t)b * kCost;
    c[0] = INFINITY; c[1] = INFINITY; c[2] = INFINITY; c[3] = INFINITY; c[4] = INFINITY; c[5] = 0.0;
    W.n_reinit[b] = 0;
    W.n_improve[b] = 0;
}

// was the rounding of mu already legal (legalization left it unchanged)?
__global__ __launch_bounds__(256) void k_round_cmp(Graph G, Work W, const float *__restrict__ mu) {
    const int b = blockIdx.x, tid = threadIdx.x;
    int diff = 0;
    for (int i = tid; i < G.N; i += 256)
        if (round_half_up(mu[(size_t)b * G.N + i], G.D) != (long long)W.cand[(size_t)b * G.N + i]) diff = 1;
    diff = __syncthreads_or(diff);
    if (tid == 0) W.round_bad[b] = diff;
}

__global__ __launch_bounds__(256) void k_best_update(Graph G, Work W, int *best_sched, double *best_cost) {
    __shared__ int improved;
    const int b = blockIdx.x, tid = threadIdx.x;
    if (tid == 0) {
        improved = cost_better(W.cand_cost + (size_t)b * kCost, best_cost + (size_t)b * kCost) ? 1 : 0;
        W.mode[b] = W.round_bad[b] ? (improved ? 1 : 2) : 0;
        W.n_reinit[b] += W.round_bad[b] ? 1 : 0;
        W.n_improve[b] += improved;
    }
    __syncthreads();
    if (!improved) return;
    for (int i = tid; i < G.N; i += 256) best_sched[(size_t)b * G.N + i] = W.cand[(size_t)b * G.N + i];
    if (tid < kCost) best_cost[(size_t)b * kCost + tid] = W.cand_cost[(size_t)b * kCost + tid];
}

// re-initialize the restarts marked by k_best_update: mu from the candidate
// (mode 1) or the best schedule so far (mode 2); Adam moments cleared;
// optionally sigma back to the paper's initial width
__global__ void k_reinit(Graph G, Work W, HP hp, const int *__restrict__ best_sched, float *mu, float *sigma,
                         float *m, float *v, int reinit_sigma) {
    const int b = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= G.N) return;
    const int md = W.mode[b];
    if (md == 0) return;
    const size_t bi = (size_t)b * G.N + i, half = (size_t)G.B * G.N;
    mu[bi] = (float)(md == 1 ? W.cand[bi] : best_sched[bi]);
    if (reinit_sigma) sigma[bi] = fmaxf(hp.kappa * (float)(G.alap[i] - G.asap[i]), hp.sigma_min);
    m[bi] = 0.0f; m[half + bi] = 0.0f;
    v[bi] = 0.0f; v[half + bi] = 0.0f;
}

hipError_t enqueue_best_init(const Graph &g, const Work &w, double *best_cost, hipStream_t st) {
    hipLaunchKernelGGL(k_best_init, dim3((g.B + 255) / 256), dim3(256), 0, st, g.B, best_cost, w);
    return hipGetLastError();
}

hipError_t enqueue_check(const Graph &g, const Work &w, const HP &hp, float *mu, float *sigma, float *m,
                         float *v, int *best_sched, double *best_cost, int reinit_sigma, hipStream_t st) {
    hipError_t e = launch_legalize(g, w, mu, w.cand, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_round_cmp, dim3(g.B), dim3(256), 0, st, g, w, mu);
    e = enqueue_schedule_cost(g, w, hp, w.cand, w.cand_cost, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_best_update, dim3(g.B), dim3(256), 0, st, g, w, best_sched, best_cost);
    hipLaunchKernelGGL(k_reinit, dim3((g.N + 255) / 256, g.B), dim3(256), 0, st, g, w, hp, best_sched, mu, sigma,
                       m, v, reinit_sigma);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Host-side enqueue helpers
// ---------------------------------------------------------------------------
hipError_t enqueue_iteration(const Graph &g, const Work &w, const HP &hp, const LaunchCfg &lc,
                             const PolyArgs &pa, const IterArgs &a, hipStream_t st) {
    hipLaunchKernelGGL(k_flags, dim3((g.N + 63) / 64, (g.B + kFlagPack - 1) / kFlagPack), dim3(64 * kFlagPack), 0, st,
                       g, pa, a.sigma, w, (hp.gamma != 0.0f && pa.enabled) ? 1 : 0);
    hipError_t e;
    if (a.ops_begin) (void)hipEventRecord(a.ops_begin, st);
    if ((e = launch_group(g, w, lc, a.mu, st)) != hipSuccess) return e;
    if ((e = launch_ops(g, w, lc, a.mu, a.sigma, st)) != hipSuccess) return e;
    if (g.lap_on && (e = launch_lap_edges(g, w, a.mu, a.sigma, st)) != hipSuccess) return e;
    if (a.ops_end) (void)hipEventRecord(a.ops_end, st);
    if (pa.enabled) {
        if (a.poly_begin) (void)hipEventRecord(a.poly_begin, st);
        if ((e = launch_poly(g, w, pa, a.mu, a.sigma, st)) != hipSuccess) return e;
        if (a.poly_end) (void)hipEventRecord(a.poly_end, st);
    }
    if (g.nb > 0 && (e = launch_back(g, w, lc, a.mu, a.sigma, st)) != hipSuccess) return e;
    if (pa.enabled) {
        int nent = 0;
        for (int gi = 0; gi < kGrids; ++gi)
            if (pa.gr[gi].on) nent = std::max(nent, pa.gr[gi].nc * kNC + pa.gr[gi].SP);
        hipLaunchKernelGGL(k_ucoef, dim3((nent + 63) / 64, g.K, g.B * kGrids), dim3(64 * kUcoefRows), 0, st,
                           g, pa, w);
    }
    // split work-groups of the op kernel: many step-by-step rows per slot
    if (g.parts > 1)
        hipLaunchKernelGGL(k_usage<4>, dim3((g.T + kUsageBS / 4 - 1) / (kUsageBS / 4), g.K, g.B), dim3(kUsageBS), 0,
                           st, g, pa, w);
    else
        hipLaunchKernelGGL(k_usage<1>, dim3((g.T + kUsageBS - 1) / kUsageBS, g.K, g.B), dim3(kUsageBS), 0, st, g,
                           pa, w);
    hipLaunchKernelGGL(k_vres, dim3(g.K, g.B), dim3(kTermsBS), 0, st, g, w, hp);
    if (hp.gamma != 0.0f) {   // expected storage units and their smooth peak
        if ((e = launch_mem_fwd(g, w, lc, a.mu, a.sigma, st)) != hipSuccess) return e;
        if (pa.enabled) {
            if ((e = launch_mem_poly_fwd(g, w, pa, a.mu, st)) != hipSuccess) return e;
            hipLaunchKernelGGL(k_mcoef, dim3((pa.nc * kNC + pa.SP + 63) / 64, g.B), dim3(64 * kUcoefRows), 0, st,
                               g, pa, w);
        }
        hipLaunchKernelGGL(k_mreg, dim3((g.T + 255) / 256, g.B), dim3(256), 0, st, g, pa, w);
        hipLaunchKernelGGL(k_mem_lse, dim3(g.B), dim3(kTermsBS), 0, st, g, w, hp);
    }
    hipLaunchKernelGGL(k_combine, dim3(g.B), dim3(kCombineBS), 0, st, g, pa, w, hp, a.lambda_in,
                       a.mode == 1 ? a.lambda_out : nullptr, a.mode == 1 ? a.adam_t : nullptr,
                       a.terms_out);
    if (hp.beta != 0.0f) {   // gradient of the smooth peak usage
        if ((e = launch_lse_ops(g, w, lc, a.mu, a.sigma, st)) != hipSuccess) return e;
        if (pa.enabled && (e = launch_lse_poly(g, w, pa, a.mu, a.sigma, st)) != hipSuccess) return e;
    }
    if (hp.gamma != 0.0f) {
        if ((e = launch_mem_bwd(g, w, lc, a.mu, a.sigma, st)) != hipSuccess) return e;
        if (pa.enabled && (e = launch_mem_poly_bwd(g, w, pa, a.mu, st)) != hipSuccess) return e;
    }
    if (g.nbig > 0) hipLaunchKernelGGL(k_gather_big, dim3(g.nbig, g.B), dim3(256), 0, st, g, w, hp, a.mu);
    {
        dim3 grid((unsigned)(((g.N + 255) / 256) * g.B));
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
    return launch_legalize(g, w, mu, sched, st);
}

}  // namespace gaus