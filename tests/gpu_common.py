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


def compare_restart(g, o_terms, o_U, o_gm, o_gs, b, what=""):
    """Assert the parity bar for restart b; returns the worst relative errors."""
    t, ot = g["terms"][b], o_terms
    err_t = np.abs(t - ot) / np.maximum(np.abs(ot), 1.0)
    names = ["L", "V_dep", "V_res", "V_rec", "L_com", "L_res", "L_mem"]
    assert err_t.max() <= TOL, f"{what} b={b} terms {dict(zip(names, t))} vs {dict(zip(names, ot))} err {err_t}"
    eu = np.abs(g["U"][b] - o_U).max() / max(np.abs(o_U).max(), 1.0)
    assert eu <= TOL, f"{what} b={b} usage err {eu}"
    res = {"terms": float(err_t.max()), "U": float(eu)}
    for name, gg, oo in (("g_mu", g["gm"][b], o_gm), ("g_sigma", g["gs"][b], o_gs)):
        scale = np.abs(oo).max()
        e = np.abs(gg - oo).max() / scale if scale > 0 else np.abs(gg).max()
        assert e <= TOL, f"{what} b={b} {name} normwise err {e} (scale {scale})"
        res[name] = float(e)
    return res


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
