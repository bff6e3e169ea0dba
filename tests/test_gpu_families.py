"""Parity of the other start-time distributions (App. E: logistic, Laplace,
Cauchy, each with its scale matched to the Gaussian sigma): loss terms,
usage and gradients of the HIP path through the C ABI vs the fp64 oracle
with the same family, alone and with the smooth peak usage and storage
terms on."""
import numpy as np
import pytest

import oracle
from paper_2602_20427_amd import binding as bd
from paper_2602_20427_amd.workloads import (CONFIGS, Problem, make_problem, random_state, restart_uniforms,
                                            uniform_state, with_storage)
from tests.gpu_common import TOL, gpu_loss_grad, hparams, oracle_compare, poly_sigma_thresholds, say

pytestmark = pytest.mark.gpu

FAMS = ["logistic", "laplace", "cauchy"]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oracle.build(force=False)
    bd.load()
    yield
    oracle.set_family("gaussian")


def _hp(family, **kw):
    hp = hparams(**kw)
    hp.family = bd.FAMILIES[family]
    return hp


def _init_state(cfg, p, B):
    if CONFIGS[cfg].init == "uniform":
        return uniform_state(p.n_ops, p.D, B, seed=0, sigma0=CONFIGS[cfg].sigma0)
    mu, sg, rc = oracle.init_state(p, B, restart_uniforms(p.n_ops, B, seed=0))
    assert rc == 0
    return mu.astype(np.float32), sg.astype(np.float32)


def _compare(p, mu, sg, lam, hp, family, what, beta=0.0, tau=1e-2, gamma=0.0, restarts=None):
    g = gpu_loss_grad(p, mu, sg, lam, hp)
    B = mu.shape[0]
    oracle.set_family(family)
    try:
        for b in (sorted({0, B - 1}) if restarts is None else restarts):
            r, o = oracle_compare(p, g, b, mu, sg, lam, hp, what, beta=beta, tau=tau, gamma=gamma)
            dU = np.abs(g["U"][b] - o["U"]).max()
            say(f"  b={b}: dU={dU:.2e} (max U {np.abs(o['U']).max():.4g}, dU/tau {dU / tau:.1e}) "
                f"L={g['terms'][b][0]:.6g} (oracle {o['terms'][0]:.6g}) "
                + " ".join(f"{k}={v:.2e}" for k, v in r.items()))
    finally:
        oracle.set_family("gaussian")


@pytest.mark.parametrize("family", FAMS)
@pytest.mark.parametrize("cfg", ["tiny", "small", "pipelined"])
def test_family_loss_grad_random_state(family, cfg):
    """Random means and widths from 0.3 to 8 steps: narrow and wide laws, mass
    in the open end bins, heavy Cauchy tails across the whole horizon."""
    p = make_problem(cfg, seed=1)
    B = min(CONFIGS[cfg].B, 4)
    mu, sg = random_state(p.n_ops, p.D, B, seed=3)
    lam = np.random.default_rng(5).uniform(0.05, 1.0, size=(B, 3)).astype(np.float32)
    hp = _hp(family, alpha=0.05, rho=1e-3)
    say(f"[family] {family} {cfg} random: N={p.n_ops} D={p.D} II={p.II} B={B}")
    _compare(p, mu, sg, lam, hp, family, f"{cfg}/{family}")


@pytest.mark.parametrize("family", FAMS)
@pytest.mark.parametrize("cfg", ["small", "medium"])
def test_family_loss_grad_initial_state(family, cfg):
    """The initial state of Alg. 1 (means inside [ASAP, ALAP], widths kappa
    times the window), where the wide laws span most of the horizon."""
    p = make_problem(cfg, seed=0)
    B = min(CONFIGS[cfg].B, 4)
    mu, sg = _init_state(cfg, p, B)
    lam = np.full((B, 3), 0.2, np.float32)
    hp = _hp(family, alpha=0.01, rho=1e-4)
    say(f"[family] {family} {cfg} init: N={p.n_ops} D={p.D} B={B}")
    _compare(p, mu, sg, lam, hp, family, f"{cfg}-init/{family}")


@pytest.mark.parametrize("family", FAMS)
def test_family_polynomial_path_switch(family):
    """The logistic and Cauchy CDFs are analytic and take the chunk
    polynomials; the Laplace CDF has a kink at the median and takes its own
    closed forms instead."""
    p = make_problem("medium", seed=0)
    ctx = bd.Context(p, 1, _hp(family))
    try:
        cfg = ctx.poly_config()
    finally:
        ctx.close()
    assert cfg["enabled"] == (family != "laplace"), cfg


@pytest.mark.parametrize("beta", [0.0, 1.0])
@pytest.mark.parametrize("family", ["logistic", "cauchy"])
def test_family_polynomial_degree_tiers(family, beta):
    """Sigmas straddle the family's tier bounds (degree 8, 6, 5 and the
    step-by-step path below degree 8's), so edges join ops of different
    degrees and of both paths; delays 0..8; with the smooth peak usage on,
    its gradient takes each op's own degree."""
    from tests.test_gpu_parity import _ragged_problem
    p = _ragged_problem(177, N=1500, D=3000, big_delay=False)
    p.delay[:] = np.random.default_rng(178).integers(0, 9, size=p.n_ops).astype(np.int32)
    ctx = bd.Context(p, 1, _hp(family))
    W = ctx.poly_config()["W"]
    ctx.close()
    thr = poly_sigma_thresholds(family, W)
    B = 2
    rng = np.random.default_rng(179)
    centres = np.array([thr[8], thr[8], thr[6], thr[6], thr[5], thr[5], 3 * thr[5]])
    pick = rng.integers(0, len(centres), size=(B, p.n_ops))
    sg = (centres[pick] * rng.uniform(0.97, 1.03, size=(B, p.n_ops))).astype(np.float32)
    mu = rng.uniform(-100, p.D + 100, size=(B, p.n_ops)).astype(np.float32)
    for d, lo, hi in ((0, 0, thr[8]), (8, thr[8], thr[6]), (6, thr[6], thr[5]), (5, thr[5], np.inf)):
        share = np.mean((sg >= lo) & (sg < hi))
        say(f"  {family} W={W}: degree {d} for sigma in [{lo:.1f}, {hi:.1f}): {share:.2f} of the ops")
        assert share > 0.05
    lam = np.random.default_rng(180).uniform(0.05, 1.0, size=(B, 3)).astype(np.float32)
    hp = _hp(family, alpha=0.2, rho=0.01, beta=beta, tau=0.1)
    _compare(p, mu, sg, lam, hp, family, f"tiers/{family} beta={beta:g}", beta=beta, tau=0.1)


@pytest.mark.parametrize("family", ["gaussian"] + FAMS)
@pytest.mark.parametrize("cfg", ["small", "pipelined"])
def test_family_smooth_peak_usage(family, cfg):
    """Random state: with the modulo fold the slot usages lie close together,
    so the softmax weights are spread over many slots (the Gaussian runs on
    the polynomial path here)."""
    p = make_problem(cfg, seed=0)
    B = min(CONFIGS[cfg].B, 4)
    mu, sg = random_state(p.n_ops, p.D, B, seed=11)
    lam = np.random.default_rng(2).uniform(0.05, 1.0, size=(B, 3)).astype(np.float32)
    hp = _hp(family, alpha=0.01, rho=1e-3, beta=1.0, tau=0.1)
    say(f"[family] {family} {cfg} smooth peak usage tau=0.1")
    _compare(p, mu, sg, lam, hp, family, f"{cfg}-lse/{family}", beta=1.0, tau=0.1)


@pytest.mark.parametrize("family", FAMS)
@pytest.mark.parametrize("cfg", ["tiny", "small", "pipelined"])
def test_family_storage(family, cfg):
    p = with_storage(make_problem(cfg, seed=0), seed=4)
    B = min(CONFIGS[cfg].B, 4)
    mu, sg = random_state(p.n_ops, p.D, B, seed=13)
    lam = np.random.default_rng(3).uniform(0.05, 1.0, size=(B, 3)).astype(np.float32)
    hp = _hp(family, alpha=0.01, rho=1e-3, tau=1.0)
    hp.gamma_mem = 1.0
    say(f"[family] {family} {cfg} storage tau=1: N={p.n_ops} D={p.D} II={p.II}")
    _compare(p, mu, sg, lam, hp, family, f"{cfg}-mem/{family}", tau=1.0, gamma=1.0)


@pytest.mark.parametrize("family", ["logistic", "cauchy"])
def test_family_storage_initial_state(family):
    """Initial state of the 1k-op workload with storage units and a sink: the
    usage and edge terms of the wide ops run on the chunk polynomials, the
    storage term of the holders the rule admits too, the others step by
    step."""
    p = with_storage(make_problem("small", seed=0), seed=4)
    B = 4
    mu, sg = _init_state("small", p, B)
    lam = np.full((B, 3), 0.2, np.float32)
    hp = _hp(family, alpha=0.01, rho=1e-3, tau=1.0)
    hp.gamma_mem = 1.0
    say(f"[family] {family} small-init storage tau=1: N={p.n_ops} D={p.D}")
    _compare(p, mu, sg, lam, hp, family, f"small-init-mem/{family}", tau=1.0, gamma=1.0)


@pytest.mark.parametrize("tau", [1.0, 0.01])
@pytest.mark.parametrize("family", ["logistic", "cauchy"])
def test_family_storage_polynomial_holders(family, tau):
    """Storage holders on the chunk polynomials with the logistic and Cauchy
    laws (every successor polynomial, at most 4 of them, rho = ((W-1)/2)/sigma
    summed over the holder and its successors at most the family's degree-8
    rho, the Gaussian's 1/4 scaled as the tier bounds are) beside holders
    evaluated step by step: sigmas are drawn around those bounds on a
    1024-step horizon."""
    p = with_storage(make_problem("medium", seed=2), seed=3)
    B = 2
    hw = _hp(family)
    hw.gamma_mem = 1.0   # the chunk width chosen with the storage term on
    ctx = bd.Context(p, 1, hw)
    W = ctx.poly_config()["W"]
    ctx.close()
    lam_w = (W - 1) / 2.0
    thr = poly_sigma_thresholds(family, W)[8]   # the polynomial path's sigma threshold
    rho8 = lam_w / thr
    rng = np.random.default_rng(23)
    rho = np.exp(rng.uniform(np.log(0.08 * rho8), np.log(1.2 * rho8), size=(B, p.n_ops)))
    sg = (lam_w / rho).astype(np.float32)
    mu = rng.uniform(-50, p.D + 50, size=(B, p.n_ops)).astype(np.float32)
    # the holders the rule puts on the polynomials (a coverage check only)
    deg = np.diff(p.row_ptr)
    n_poly = []
    for b in range(B):
        poly = (sg[b] >= thr) & (p.delay <= 8)
        cnt = 0
        for i in range(p.n_ops):
            succ = p.col_idx[p.row_ptr[i]:p.row_ptr[i + 1]]
            if poly[i] and 1 <= deg[i] <= 4 and poly[succ].all() and \
                    lam_w * (1.0 / sg[b, i] + (1.0 / sg[b, succ]).sum()) <= rho8:
                cnt += 1
        n_poly.append(cnt)
    holders = int((deg > 0).sum())
    say(f"  {family} W={W} rho8={rho8:.4f}: polynomial holders {n_poly} of {holders}")
    assert min(n_poly) > 0.15 * holders and max(n_poly) < 0.85 * holders
    lam = np.random.default_rng(24).uniform(0.05, 1.0, size=(B, 3)).astype(np.float32)
    hp = _hp(family, alpha=0.01, rho=1e-3, tau=tau)
    hp.gamma_mem = 1.0
    _compare(p, mu, sg, lam, hp, family, f"poly holders tau={tau}/{family}", tau=tau, gamma=1.0,
             restarts=range(B))


@pytest.mark.parametrize("family", FAMS)
def test_family_large_full_size(family):
    """Each family on the 50k-op workload at full size (B=8, D=4096) in
    bench.py's launch configuration (logistic and Cauchy on the packed chunk
    polynomials; Laplace on its own path), restarts 0, 1, 2 (pack positions
    0..2) and 7."""
    cfg = CONFIGS["large"]
    p = make_problem(cfg, seed=0)
    B = cfg.B
    mu, sg = _init_state("large", p, B)
    hp = bd.default_hparams()
    hp.lr = cfg.lr
    hp.family = bd.FAMILIES[family]
    lam = np.full((B, 3), hp.lambda0, np.float32)
    say(f"[family] {family} large: N={p.n_ops} D={p.D} B={B}")
    _compare(p, mu, sg, lam, hp, family, f"large/{family}", restarts=(0, 1, 2, B - 1))


def _bipartite_problem(seed, N, D):
    """Producers 0..N/2-1 (sources) feeding consumers N/2..N-1 (sinks), so any
    producer delay up to D-1 fits the horizon: delays 0 and D-1, a few around
    D/2 and small ones."""
    rng = np.random.default_rng(seed)
    h = N // 2
    rows = [np.unique(rng.integers(h, N, size=1 + rng.poisson(2.0))) for _ in range(h)]
    rows += [np.zeros(0, np.int64)] * (N - h)
    row_ptr = np.zeros(N + 1, np.int32)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.concatenate(rows).astype(np.int32)
    delay = np.zeros(N, np.int32)
    delay[:h] = np.where(rng.random(h) < 0.5, rng.integers(0, 9, size=h), rng.integers(0, D, size=h))
    delay[:4] = [0, D - 1, D // 2, max(D - 2, 0)]
    rtype = rng.integers(0, 3, size=N).astype(np.int32)
    cap = np.array([3.0, 1.5, 0.7], np.float32)
    e = np.zeros(0, np.int32)
    return Problem(n_ops=N, row_ptr=row_ptr, col_idx=col, delay=delay, rtype=rtype, capacity=cap, D=D, II=0,
                   back_src=e, back_dst=e, back_dist=e)


@pytest.mark.parametrize("D", [50, 300, 1500])
def test_laplace_closed_form_extremes(D):
    """The Laplace edge sums in closed form at the ends of their ranges:
    widths from 0.02 to 5000 steps (log-uniform, so the ratio e^-lam of the
    geometric sums runs from 0 to within 3e-4 of 1 and the sums take their
    direct, expm1 and power-series forms), means on the horizon's ends, on
    half steps (a median exactly on a bin edge, where the cases change) and
    far outside it, and producer delays from 0 to D-1."""
    N = 400 if D > 100 else 120
    p = _bipartite_problem(60 + D, N, D)
    B = 3
    rng = np.random.default_rng(61 + D)
    ends = np.array([0.0, D - 1.0, D / 2.0])[rng.integers(0, 3, size=(B, N))] + rng.normal(0.0, 2.0, size=(B, N))
    half = rng.integers(-3, D + 3, size=(B, N)) + 0.5
    far = rng.uniform(-3.0 * D, 4.0 * D, size=(B, N))
    pick = rng.integers(0, 3, size=(B, N))
    mu = np.choose(pick, [ends, half, far]).astype(np.float32)
    sg = np.exp(rng.uniform(np.log(0.02), np.log(5000.0), size=(B, N))).astype(np.float32)
    lam = np.random.default_rng(62 + D).uniform(0.05, 1.0, size=(B, 3)).astype(np.float32)
    hp = _hp("laplace", alpha=0.3, rho=0.02)
    say(f"[family] laplace extremes: N={N} E={p.n_edges} D={D} B={B}")
    _compare(p, mu, sg, lam, hp, "laplace", f"extremes D={D}/laplace", restarts=range(B))


def test_laplace_tight_horizon_full_size():
    """Laplace on the 50k-op workload with the tight horizon (D = longest
    delay-weighted path + 8, one step tile) at full size from the paper's
    initialization, as bench.py --workload large-tight --family laplace times
    it: the producers' delays cut most runs near the horizon's end."""
    cfg = CONFIGS["large-tight"]
    p = make_problem(cfg, seed=0)
    B = cfg.B
    mu, sg, rc = oracle.init_state(p, B, restart_uniforms(p.n_ops, B, seed=0))
    assert rc == 0
    hp = bd.default_hparams()
    hp.lr = cfg.lr
    hp.family = bd.FAMILIES["laplace"]
    lam = np.full((B, 3), hp.lambda0, np.float32)
    say(f"[family] laplace large-tight: N={p.n_ops} D={p.D} B={B}")
    _compare(p, mu.astype(np.float32), sg.astype(np.float32), lam, hp, "laplace", "large-tight/laplace",
             restarts=(0, B - 1))
