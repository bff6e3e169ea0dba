"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and the CPU oracle on the same seeded inputs, and compare them."""
from __future__ import annotations

import sys

import numpy as np

from paper_2602_20427_amd import binding as bd

# fp32 GPU vs fp64 oracle: loss terms within 1e-5 of max(|x*|, 1), gradients
# within 1e-5 of the largest gradient entry (per restart and tensor), usage
# normwise, Adam elementwise from the same gradient.
TOL = 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def hparams(alpha=0.01, rho=1e-4, lr=1e-2, poly_chunk=0, beta=0.0, tau=1e-2):
    """poly_chunk: 0 = library's choice, < 0 = polynomial path off, else W;
    beta, tau: weight and temperature of the smooth peak usage term."""
    hp = bd.default_hparams()
    hp.alpha_com = alpha
    hp.rho = rho
    hp.lr = lr
    hp.poly_chunk = poly_chunk
    hp.beta_res = beta
    hp.tau = tau
    return hp


def gpu_loss_grad(prob, mu, sigma, lam, hp):
    import torch
    B, N = mu.shape
    ctx = bd.Context(prob, B, hp)
    say(f"  [ctx] poly {ctx.poly_config()}")
    dev = torch.device("cuda")
    m = torch.from_numpy(np.ascontiguousarray(mu, np.float32)).to(dev)
    s = torch.from_numpy(np.ascontiguousarray(sigma, np.float32)).to(dev)
    l = torch.from_numpy(np.ascontiguousarray(lam, np.float32)).to(dev)
    terms = torch.zeros(B, bd.N_TERMS, device=dev)
    gm = torch.zeros(B, N, device=dev)
    gs = torch.zeros(B, N, device=dev)
    ctx.loss_grad(m, s, l, terms, gm, gs)
    U = torch.zeros(B, ctx.K, ctx.T, device=dev)
    ctx.get_usage(U)
    ctx.sync()
    out = dict(terms=terms.cpu().numpy().astype(np.float64), gm=gm.cpu().numpy().astype(np.float64),
               gs=gs.cpu().numpy().astype(np.float64), U=U.cpu().numpy().astype(np.float64))
    ctx.close()
    return out


TIE_TOL = 1e-4        # usage cells within TIE_TOL * max(1, C) of their capacity are near ties
MAX_TIES_PER_TYPE = 10


def near_tie_branches(prob, mu_b, sg_b, lam_b, rho, o_terms, o_U):
    """Near-tie usage cells of one restart (|U* - C| < TIE_TOL max(1, C):
    fp32 rounding of U may put the ReLU indicator of eq:relu on either side)
    with, for each, the oracle's own indicator and the gradient the cell
    adds when its indicator is 1 (w_res dU/dtheta, from the oracle).
    Returns a list of (type, slot, indicator, d_mu [N], d_sigma [N])."""
    import oracle
    cap = np.asarray(prob.capacity, np.float64)
    ex = o_U - cap[:, None]
    cells = np.argwhere(np.abs(ex) < TIE_TOL * np.maximum(cap, 1.0)[:, None])
    if len(cells) == 0:
        return []
    w_res = float(np.float64(lam_b[1])) + float(rho) * float(o_terms[2])
    out = []
    for k, t in cells:
        dm, ds = oracle.usage_cell_grad(prob, mu_b, sg_b, int(k), int(t), w=w_res)
        out.append((int(k), int(t), int(ex[k, t] > 0.0), dm, ds))
    return out


def grad_errors(gm, gs, o_gm, o_gs, rtype, ties=()):
    """Normwise gradient errors max|g - g*| / max|g*| for mu and sigma.  At
    near-tie cells both indicator values are accepted: per resource type
    (only ops of that type see its cells) the branch combination with the
    smallest error is taken, the same for both tensors; the scale is that
    of the oracle's own branch."""
    sm, ss = np.abs(o_gm).max(), np.abs(o_gs).max()

    def err(a, b, sc):
        d = np.abs(a - b)
        if d.size == 0:
            return 0.0
        return float(d.max() / sc) if sc > 0 else float(np.abs(a).max())

    tied = sorted({k for k, *_ in ties})
    rtype = np.asarray(rtype)
    free = ~np.isin(rtype, tied)
    e_mu, e_sg = err(gm[free], o_gm[free], sm), err(gs[free], o_gs[free], ss)
    flips = 0
    for k in tied:
        cells = [c for c in ties if c[0] == k]
        assert len(cells) <= MAX_TIES_PER_TYPE, f"{len(cells)} near-tie cells of type {k}: reseed the case"
        ops = rtype == k
        best = None
        for mask in range(1 << len(cells)):
            am, as_ = o_gm[ops].copy(), o_gs[ops].copy()
            for j, (_, _, ind, dm, ds) in enumerate(cells):
                want = (mask >> j) & 1
                if want != ind:
                    sgn = 1.0 if want else -1.0
                    am += sgn * dm[ops]
                    as_ += sgn * ds[ops]
            cand = (err(gm[ops], am, sm), err(gs[ops], as_, ss))
            nflip = bin(mask ^ sum(c[2] << j for j, c in enumerate(cells))).count("1")
            if best is None or max(cand) < max(best[0]):
                best = (cand, nflip)
        e_mu, e_sg = max(e_mu, best[0][0]), max(e_sg, best[0][1])
        flips += best[1]
    return e_mu, e_sg, flips


def compare_restart(g, o_terms, o_U, o_gm, o_gs, b, what="", ties=(), rtype=None):
    """Assert the parity bar for restart b; returns the worst relative errors.
    ties: near_tie_branches() of the restart (either indicator accepted)."""
    t, ot = g["terms"][b], o_terms
    err_t = np.abs(t - ot) / np.maximum(np.abs(ot), 1.0)
    names = ["L", "V_dep", "V_res", "V_rec", "L_com", "L_res", "L_mem"]
    assert err_t.max() <= TOL, f"{what} b={b} terms {dict(zip(names, t))} vs {dict(zip(names, ot))} err {err_t}"
    eu = np.abs(g["U"][b] - o_U).max() / max(np.abs(o_U).max(), 1.0)
    assert eu <= TOL, f"{what} b={b} usage err {eu}"
    res = {"terms": float(err_t.max()), "U": float(eu)}
    if ties:
        assert rtype is not None
        e_mu, e_sg, flips = grad_errors(g["gm"][b], g["gs"][b], o_gm, o_gs, rtype, ties)
        res["ties"] = len(ties)
        res["flipped"] = flips
    else:
        e_mu, e_sg, _ = grad_errors(g["gm"][b], g["gs"][b], o_gm, o_gs, np.zeros(len(o_gm), np.int64))
    for name, e in (("g_mu", e_mu), ("g_sigma", e_sg)):
        assert e <= TOL, f"{what} b={b} {name} normwise err {e}"
        res[name] = float(e)
    return res


def oracle_compare(prob, g, b, mu, sg, lam, hp, what="", **okw):
    """Oracle of restart b (fp64, same seeded state) and the parity bar,
    accepting either indicator at near-tie usage cells.  okw go to
    oracle.loss_grad (beta, tau, gamma, mreg_out).  Returns (errors, oracle
    result: dict of terms, U, gm, gs)."""
    import oracle
    m64, s64 = mu[b].astype(np.float64), sg[b].astype(np.float64)
    lb = np.asarray(lam[b:b + 1], np.float64)
    ot, oU, ogm, ogs, _ = oracle.loss_grad(prob, m64[None], s64[None], lb, hp.alpha_com, hp.rho,
                                           tie_tol=TIE_TOL, **okw)
    ties = near_tie_branches(prob, m64, s64, lb[0], hp.rho, ot[0], oU[0])
    r = compare_restart(g, ot[0], oU[0], ogm[0], ogs[0], b, what, ties=ties, rtype=prob.rtype)
    return r, dict(terms=ot[0], U=oU[0], gm=ogm[0], gs=ogs[0])


# Tier bounds of the chunk-polynomial path (restated from the library's
# rule): the truncation bound of an op's series at degree d and
# rho = ((W-1)/2)/sigma, per family, and the sigma at which each degree
# starts (the bound equals the Gaussian degree-8 bound at rho = 1/4).
POLY_DEGREES = (8, 6, 5)


def poly_bound(family, d, rho):
    import math
    if family == "logistic":
        x = rho / math.sqrt(3.0)
        return 8.0 * (d + 1) / math.pi ** 2 * x ** d / (1.0 - x)
    if family == "cauchy":
        x = rho / math.sqrt(2.0 * math.log(2.0))
        return x ** d / (1.0 - x)
    return 1.09 * rho ** d / math.sqrt(math.factorial(d))


def poly_rho(family, d):
    target = poly_bound("gaussian", 8, 0.25)
    lo, hi = 0.0, 0.25
    for _ in range(200):
        m = 0.5 * (lo + hi)
        lo, hi = (m, hi) if poly_bound(family, d, m) <= target else (lo, m)
    return lo


def poly_sigma_thresholds(family, W):
    """{degree: smallest sigma that takes it} for chunk width W."""
    lam = (W - 1) / 2.0
    return {d: lam / poly_rho(family, d) for d in POLY_DEGREES}
