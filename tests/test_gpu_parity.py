"""Parity of the gfx950 HIP path (through the C ABI) with the fp64 CPU oracle
on identical seeded inputs."""
import math

import numpy as np
import pytest

import oracle
from paper_2602_20427_amd import binding as bd
from paper_2602_20427_amd.workloads import (CONFIGS, Problem, make_problem, random_state,
                                            restart_uniforms, uniform_state)
from tests.gpu_common import TOL, gpu_loss_grad, hparams, oracle_compare, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oracle.build(force=False)
    bd.load()
    yield


def _check(prob, mu, sigma, lam, hp, restarts, what):
    say(f"[parity] {what}: N={prob.n_ops} E={prob.n_edges} nb={prob.n_back} D={prob.D} II={prob.II} B={mu.shape[0]}")
    g = gpu_loss_grad(prob, mu, sigma, lam, hp)
    for b in restarts:
        r, _ = oracle_compare(prob, g, b, mu, sigma, lam, hp, what, beta=hp.beta_res, tau=hp.tau)
        say(f"  b={b}: " + " ".join(f"{k}={v:.2e}" for k, v in r.items()))
    return g


def _lam(B, seed, lo=0.05, hi=1.0):
    return np.random.default_rng(seed).uniform(lo, hi, size=(B, 3)).astype(np.float32)


@pytest.mark.parametrize("cfg", ["tiny", "small"])
def test_loss_grad_random_state(cfg):
    """Narrow and mixed regimes: random mu (some outside the horizon), sigma in [0.3, 8]."""
    p = make_problem(cfg, seed=0)
    B = CONFIGS[cfg].B
    mu, sg = random_state(p.n_ops, p.D, B, seed=1)
    _check(p, mu, sg, _lam(B, 2), hparams(alpha=0.37, rho=0.05), range(B), f"{cfg}/random")


@pytest.mark.parametrize("poly", [0, -1])
@pytest.mark.parametrize("cfg", ["tiny", "small", "medium", "pipelined"])
def test_loss_grad_paper_init(cfg, poly):
    """Timing state: the paper's ASAP/ALAP initialization (dense regime)."""
    p = make_problem(cfg, seed=0)
    B = CONFIGS[cfg].B
    if CONFIGS[cfg].init == "uniform":
        mu, sg = uniform_state(p.n_ops, p.D, B, seed=0, sigma0=CONFIGS[cfg].sigma0)
    else:
        u = restart_uniforms(p.n_ops, B, seed=0)
        mu, sg, rc = oracle.init_state(p, B, u)
        assert rc == 0
        mu, sg = mu.astype(np.float32), sg.astype(np.float32)
    restarts = [0, B - 1] if B > 2 else range(B)
    _check(p, mu, sg, _lam(B, 3), hparams(alpha=0.01, rho=1e-3, poly_chunk=poly), restarts,
           f"{cfg}/init poly={poly}")


def test_loss_grad_large_full_size():
    """The 50k-op workload at its full size (B=8, D=4096) in the launch
    configuration bench.py times (library defaults: chunk-polynomial path with
    the automatic chunk width and restart packs of 4), from the paper's
    initialization; every restart against the oracle."""
    cfg = CONFIGS["large"]
    p = make_problem(cfg, seed=0)
    B = cfg.B
    u = restart_uniforms(p.n_ops, B, seed=0)
    mu, sg, rc = oracle.init_state(p, B, u)
    assert rc == 0
    mu, sg = mu.astype(np.float32), sg.astype(np.float32)
    hp = bd.default_hparams()
    hp.lr = cfg.lr
    _check(p, mu, sg, np.full((B, 3), hp.lambda0, np.float32), hp, range(B), "large/init bench config")


def test_loss_grad_large_after_steps():
    """The 50k-op workload after 20 fused steps on the GPU (moved means and
    widths, nonzero multipliers): the state is read back and the loss and
    gradient of that state are compared with the oracle."""
    import torch
    cfg = CONFIGS["large"]
    p = make_problem(cfg, seed=0)
    B = cfg.B
    hp = bd.default_hparams()
    hp.lr = 0.5                     # large steps: states far from the initialization
    hp.rho = 1e-2
    ctx = bd.Context(p, B, hp)
    dev = torch.device("cuda")
    mu = torch.zeros(B, p.n_ops, device=dev)
    sg = torch.zeros(B, p.n_ops, device=dev)
    ctx.init_state(mu, sg, restart_uniforms(p.n_ops, B, seed=0))
    lam = torch.full((B, 3), 0.5, device=dev)
    m = torch.zeros(2, B, p.n_ops, device=dev)
    v = torch.zeros(2, B, p.n_ops, device=dev)
    t = torch.zeros(1, dtype=torch.int32, device=dev)
    ctx.bind_state(mu, sg, m, v, lam, t)
    ctx.step(20)
    ctx.sync()
    say(f"  [large] after 20 steps: poly census {ctx.poly_census()}")
    mu_h, sg_h, lam_h = mu.cpu().numpy(), sg.cpu().numpy(), lam.cpu().numpy()
    ctx.close()
    _check(p, mu_h, sg_h, lam_h, hp, [0, 1, 2, B - 1], "large/after 20 steps")


def test_loss_grad_tight_horizon_full_size():
    """The 50k-op workload with the tight horizon (D = longest delay-weighted
    path + 8 = 793: one step tile) at full size from the paper's
    initialization, as bench.py --workload large-tight times it: a quarter of
    the (restart, op) pairs off the chunk polynomials, most of them wide
    (one wave per op, or the row path when the consumers span the tile),
    polynomial producers with such consumers, and the op kernel split over
    two work-groups per group."""
    cfg = CONFIGS["large-tight"]
    p = make_problem(cfg, seed=0)
    B = cfg.B
    u = restart_uniforms(p.n_ops, B, seed=0)
    mu, sg, rc = oracle.init_state(p, B, u)
    assert rc == 0
    mu, sg = mu.astype(np.float32), sg.astype(np.float32)
    hp = bd.default_hparams()
    hp.lr = cfg.lr
    _check(p, mu, sg, np.full((B, 3), hp.lambda0, np.float32), hp, [0, 3, B - 1], "large-tight/init")


@pytest.mark.parametrize("sigma,restarts", [(0.4, range(8)), (3.0, [0, 5])])
def test_loss_grad_large_sharpened(sigma, restarts):
    """The 50k-op workload at full size in a sharpened state (the paper's
    initial means, every sigma the same small value, as bench.py --sigma
    times it): at sigma = 0.4 every op and edge runs through the narrow
    kernel over the whole horizon, at sigma = 3 most do."""
    cfg = CONFIGS["large"]
    p = make_problem(cfg, seed=0)
    B = cfg.B
    u = restart_uniforms(p.n_ops, B, seed=0)
    mu, sg, rc = oracle.init_state(p, B, u)
    assert rc == 0
    mu = mu.astype(np.float32)
    sg = np.full(mu.shape, sigma, np.float32)
    hp = bd.default_hparams()
    hp.lr = cfg.lr
    _check(p, mu, sg, _lam(B, 7), hp, restarts, f"large/sigma={sigma}")


def test_loss_grad_pipelined_random():
    p = make_problem("pipelined", seed=0)
    B = 4
    mu, sg = random_state(p.n_ops, p.D, B, seed=5, sigma_range=(0.5, 40.0))
    _check(p, mu, sg, _lam(B, 6), hparams(alpha=0.2, rho=0.01), range(B), "pipelined/random")


def _ragged_problem(seed, N=700, D=1500, II=0, n_back=0, big_delay=True):
    """Several tiles with a ragged tail (D % 1024 != 0), type-group
    boundaries, sinks, and a few producer delays above the LDS halo."""
    rng = np.random.default_rng(seed)
    rows = []
    for i in range(N):
        k = rng.poisson(2.0)
        tg = np.unique(rng.integers(i + 1, min(N, i + 60), size=k)) if i < N - 1 else np.zeros(0, int)
        rows.append(tg)
    row_ptr = np.zeros(N + 1, np.int32)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.concatenate(rows).astype(np.int32)
    delay = rng.integers(0, 4, size=N).astype(np.int32)
    if big_delay:
        delay[rng.choice(N - 100, size=3, replace=False)] = [300, 257, 600]
    rtype = rng.integers(0, 3, size=N).astype(np.int32)
    cap = np.array([3.0, 1.5, 0.7], np.float32)
    bs, bd_, bk = [], [], []
    for _ in range(n_back):
        j = int(rng.integers(1, N)); i = int(rng.integers(0, j))
        bs.append(j); bd_.append(i); bk.append(int(rng.integers(1, 4)))
    return Problem(n_ops=N, row_ptr=row_ptr, col_idx=col, delay=delay, rtype=rtype, capacity=cap, D=D, II=II,
                   back_src=np.array(bs, np.int32), back_dst=np.array(bd_, np.int32),
                   back_dist=np.array(bk, np.int32))


@pytest.mark.parametrize("poly", [0, 32, -1])
@pytest.mark.parametrize("II,n_back", [(0, 0), (37, 25), (2000, 10)])
def test_loss_grad_ragged_tiles_and_big_delays(II, n_back, poly):
    """Mixed regimes: sigma from 0.2 to 300 puts ops on both the polynomial and
    the step-by-step path, and edges between them."""
    p = _ragged_problem(11 + II, II=II, n_back=n_back)
    B = 3
    rng = np.random.default_rng(12)
    mu = rng.uniform(-20, p.D + 20, size=(B, p.n_ops)).astype(np.float32)
    sg = np.exp(rng.uniform(np.log(0.2), np.log(300.0), size=(B, p.n_ops))).astype(np.float32)
    _check(p, mu, sg, _lam(B, 13), hparams(alpha=0.3, rho=0.02, poly_chunk=poly), range(B),
           f"ragged II={II} poly={poly}")


@pytest.mark.parametrize("poly", [0, -1])
@pytest.mark.parametrize("D,II", [(50, 0), (300, 0), (1500, 0), (1500, 37)])
def test_loss_grad_narrow_ops(D, II, poly):
    """Sharpened states (sigma from 0.03 to 8: most ops and edges on the
    narrow-op path of the step-by-step kernel), with means gathered at the
    horizon's ends and at the step-tile boundaries, mixed with uniform ones,
    and producer delays far beyond the ops' spreads."""
    p = _ragged_problem(31 + D + II, N=700 if D > 100 else 200, D=D, II=II, n_back=6 if II else 0,
                        big_delay=D > 1000)
    B = 3
    rng = np.random.default_rng(32 + D)
    centers = np.array([0.0, D - 1.0] + [t for t in (64.0, 256.0, 1024.0) if t < D], np.float64)
    near = centers[rng.integers(0, len(centers), size=(B, p.n_ops))] + rng.normal(0.0, 3.0, size=(B, p.n_ops))
    far = rng.uniform(-25, p.D + 25, size=(B, p.n_ops))
    mu = np.where(rng.random((B, p.n_ops)) < 0.5, near, far).astype(np.float32)
    sg = np.exp(rng.uniform(np.log(0.03), np.log(8.0), size=(B, p.n_ops))).astype(np.float32)
    _check(p, mu, sg, _lam(B, 33), hparams(alpha=0.3, rho=0.02, poly_chunk=poly), range(B),
           f"narrow D={D} II={II} poly={poly}")


def test_loss_grad_split_op_work_groups():
    """The 10k-op workload with 32 restarts has a single 1024-step tile and
    fewer than 4096 op-kernel work-groups over 320k (restart, op) pairs, so
    each (group, tile) is split over several work-groups; a mixed state
    (sigma 0.2 .. 40) puts ops on the constant, narrow, wide and polynomial
    paths of every split."""
    p = make_problem("medium", seed=1)
    B = CONFIGS["medium"].B
    mu, sg = random_state(p.n_ops, p.D, B, seed=41, sigma_range=(0.2, 40.0), mu_margin=10.0)
    _check(p, mu, sg, _lam(B, 42), hparams(alpha=0.25, rho=0.02), [0, 13, B - 1], "medium/split work-groups")


def test_loss_grad_split_op_work_groups_pipelined():
    """The pipelined workload (II > 0, back edges) with 80 restarts: two
    tiles and 3360 op-kernel work-groups, split three ways (a split that
    does not divide the group sizes)."""
    p = make_problem("pipelined", seed=2)
    B = 80
    mu, sg = random_state(p.n_ops, p.D, B, seed=43, sigma_range=(0.2, 40.0), mu_margin=10.0)
    _check(p, mu, sg, _lam(B, 44), hparams(alpha=0.25, rho=0.02), [0, 41, B - 1], "pipelined/split work-groups")


def test_usage_over_a_thousand_groups_of_one_type():
    """5000 ops of one resource type with one restart are cut into groups of
    4 ops: more than the 1024 groups the usage kernel lists in LDS, so it
    scans the group flags instead."""
    rng = np.random.default_rng(51)
    N, D = 5000, 300
    rows = [np.unique(rng.integers(i + 1, min(N, i + 40), size=rng.poisson(1.5))) if i < N - 1
            else np.zeros(0, int) for i in range(N)]
    row_ptr = np.zeros(N + 1, np.int32); row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.concatenate(rows).astype(np.int32)
    p = Problem(n_ops=N, row_ptr=row_ptr, col_idx=col, delay=rng.integers(0, 2, size=N).astype(np.int32),
                rtype=np.zeros(N, np.int32), capacity=np.array([40.0], np.float32), D=D)
    mu, sg = random_state(N, D, 1, seed=52, sigma_range=(0.3, 30.0))
    _check(p, mu, sg, _lam(1, 53), hparams(alpha=0.2, rho=0.01), [0], "one type, 1250 groups")


@pytest.mark.parametrize("W", [16, 32, 64, 128, 256])
def test_polynomial_path_chunk_widths(W):
    """Every chunk width on a wide-sigma state (all ops polynomial where the
    width allows), delays 0..8, means partly outside the horizon."""
    p = _ragged_problem(40 + W, N=400, D=min(3000, 60 * W + 10), big_delay=False)
    p.delay[:] = np.random.default_rng(W).integers(0, 9, size=p.n_ops).astype(np.int32)
    B = 2
    rng = np.random.default_rng(41)
    mu = rng.uniform(-200, p.D + 200, size=(B, p.n_ops)).astype(np.float32)
    sg = rng.uniform(2.0 * W, 1500.0, size=(B, p.n_ops)).astype(np.float32)
    _check(p, mu, sg, _lam(B, 42), hparams(alpha=0.2, rho=0.01, poly_chunk=W), range(B), f"chunk W={W}")


@pytest.mark.parametrize("beta", [0.0, 1.0])
def test_polynomial_degree_tiers(beta):
    """Wide ops take fewer series terms: degree 8 for rho = ((W-1)/2)/sigma up to
    1/4, degree 6 and degree 5 above the sigmas where their truncation error
    matches degree 8's at rho = 1/4.  Sigmas straddle every boundary, so edges
    join ops of different degrees (the producer's vectors then take the
    higher degree) and ops of both paths; with the smooth peak usage on, its
    gradient takes each op's own degree."""
    p = _ragged_problem(77, N=1500, D=3000, big_delay=False)
    p.delay[:] = np.random.default_rng(78).integers(0, 9, size=p.n_ops).astype(np.int32)
    ctx = bd.Context(p, 1, hparams())
    W = ctx.poly_config()["W"]
    ctx.close()
    lam_w = (W - 1) / 2.0
    f = math.factorial
    thr = {d: lam_w / (0.25 ** 8 * math.sqrt(f(d) / f(8))) ** (1.0 / d) for d in (8, 6, 5)}
    B = 2
    rng = np.random.default_rng(79)
    centres = np.array([thr[8], thr[8], thr[6], thr[6], thr[5], thr[5], 3 * thr[5]])
    pick = rng.integers(0, len(centres), size=(B, p.n_ops))
    sg = (centres[pick] * rng.uniform(0.97, 1.03, size=(B, p.n_ops))).astype(np.float32)
    mu = rng.uniform(-100, p.D + 100, size=(B, p.n_ops)).astype(np.float32)
    for d, lo, hi in ((8, thr[8], thr[6]), (6, thr[6], thr[5]), (5, thr[5], np.inf)):
        share = np.mean((sg >= lo) & (sg < hi))
        say(f"  W={W}: degree {d} for sigma in [{lo:.1f}, {hi:.1f}): {share:.2f} of the ops")
        assert share > 0.1
    _check(p, mu, sg, _lam(B, 80), hparams(alpha=0.2, rho=0.01, beta=beta, tau=0.1), range(B),
           f"degree tiers, smooth peak weight {beta:g}")


def _grid_census(p, mu, sg, hp):
    """Grid census of one loss+gradient evaluation (and the grids' layout)."""
    import torch
    B = mu.shape[0]
    ctx = bd.Context(p, B, hp)
    dev = torch.device("cuda")
    m = torch.from_numpy(mu).to(dev)
    s = torch.from_numpy(sg).to(dev)
    l = torch.full((B, 3), 0.1, device=dev)
    terms = torch.zeros(B, bd.N_TERMS, device=dev)
    gm = torch.zeros(B, p.n_ops, device=dev)
    gs = torch.zeros(B, p.n_ops, device=dev)
    ctx.loss_grad(m, s, l, terms, gm, gs)
    out = ctx.poly_grid_census(), ctx.poly_grids()
    ctx.close()
    return out


@pytest.mark.parametrize("beta", [0.0, 1.0])
def test_packed_grids(beta):
    """Restart packing: ops whose pack (2 or 4 restarts sharing a wave) and
    consumers all reach a packed grid's degree-8 bound take it; mixed packs,
    narrower consumers and delays above 8 fall back to grid 0 or to the
    step-by-step path.  B = 7 leaves partial packs (4 + 3, 2+2+2+1).  Every
    restart matches the oracle; the packed evaluation matches the unpacked
    one (poly_pack = -1) to fp32 rounding."""
    p = _ragged_problem(301, N=1500, D=3000, big_delay=False)
    rng = np.random.default_rng(302)
    p.delay[:] = rng.integers(0, 11, size=p.n_ops).astype(np.int32)
    B = 7
    hp0 = hparams(alpha=0.2, rho=0.01, beta=beta, tau=0.1)
    ctx = bd.Context(p, B, hp0)
    grids = ctx.poly_grids()
    ctx.close()
    say(f"  grids {grids}")
    assert all(g["on"] for g in grids)
    lam = [(g["W"] - 1) / 2.0 for g in grids]
    # width classes: step by step, grid 0, grid 1, grid 2 (degree 8), grid 2 (low degree)
    cls_sigma = np.array([0.5 * lam[0] / 0.25, 1.3 * lam[0] / 0.25, 1.3 * lam[1] / 0.25,
                          1.3 * lam[2] / 0.25, 6.0 * lam[2] / 0.25])
    prob = np.array([0.1, 0.15, 0.15, 0.3, 0.3])
    base = rng.choice(len(cls_sigma), size=p.n_ops, p=prob)
    pick = np.repeat(base[None, :], B, axis=0)
    flip = rng.random((B, p.n_ops)) < 0.08
    pick[flip] = rng.choice(len(cls_sigma), size=int(flip.sum()), p=prob)
    sg = (cls_sigma[pick] * rng.uniform(0.97, 1.03, size=(B, p.n_ops))).astype(np.float32)
    mu = rng.uniform(-100, p.D + 100, size=(B, p.n_ops)).astype(np.float32)
    census, _ = _grid_census(p, mu, sg, hp0)
    say(f"  (restart, op) pairs per grid: {census}")
    assert min(census) > 0.03 * B * p.n_ops, census
    lamb = _lam(B, 303)
    g = _check(p, mu, sg, lamb, hp0, range(B), f"packed grids beta={beta:g}")
    hp1 = hparams(alpha=0.2, rho=0.01, beta=beta, tau=0.1)
    hp1.poly_pack = -1
    g1 = gpu_loss_grad(p, mu, sg, lamb, hp1)
    for b in range(B):
        dt = np.abs(g["terms"][b] - g1["terms"][b]) / np.maximum(np.abs(g1["terms"][b]), 1.0)
        assert dt.max() <= 1e-6, (b, g["terms"][b], g1["terms"][b])
        for k in ("gm", "gs"):
            e = np.abs(g[k][b] - g1[k][b]).max() / np.abs(g1[k][b]).max()
            assert e <= 1e-6, (b, k, e)


def test_packed_grids_explicit_chunk_width():
    """An explicit grid-0 chunk width (W = 200) with packing on: the packed
    grid of 2 restarts (W = 127) then has the lower sigma threshold, and ops
    or consumers between the two thresholds must stay step by step in every
    restart (never on a pack while grid 0 leaves them to the op kernel).
    50k-op workload, B = 8, sigmas drawn around the three thresholds; four
    restarts against the oracle and every restart against the unpacked
    evaluation."""
    cfg = CONFIGS["large"]
    p = make_problem(cfg, seed=0)
    B = cfg.B
    hp0 = hparams(alpha=0.2, rho=0.01)
    hp0.poly_chunk = 200
    hp0.poly_pack = 1
    ctx = bd.Context(p, B, hp0)
    grids = ctx.poly_grids()
    ctx.close()
    say(f"  grids {grids}")
    assert all(g["on"] for g in grids) and grids[0]["W"] == 200
    thr = [4.0 * (g["W"] - 1) / 2.0 for g in grids]   # degree-8 bound rho = 1/4
    assert thr[1] < thr[0] < thr[2], thr
    rng = np.random.default_rng(401)
    cls_sigma = np.array([0.8 * thr[1], 0.5 * (thr[1] + thr[0]), 0.5 * (thr[0] + thr[2]), 1.4 * thr[2]])
    base = rng.choice(4, size=p.n_ops, p=[0.1, 0.3, 0.3, 0.3])
    pick = np.repeat(base[None, :], B, axis=0)
    flip = rng.random((B, p.n_ops)) < 0.05
    pick[flip] = rng.choice(4, size=int(flip.sum()))
    sg = (cls_sigma[pick] * rng.uniform(0.98, 1.02, size=(B, p.n_ops))).astype(np.float32)
    u = restart_uniforms(p.n_ops, B, seed=0)
    mu, _, rc = oracle.init_state(p, B, u)
    assert rc == 0
    mu = mu.astype(np.float32)
    census, _ = _grid_census(p, mu, sg, hp0)
    say(f"  (restart, op) pairs per grid: {census}")
    assert min(census) > 0.02 * B * p.n_ops, census
    lamb = _lam(B, 402)
    g = _check(p, mu, sg, lamb, hp0, [0, 1, 2, B - 1], "explicit W=200 with packs")
    hp1 = hparams(alpha=0.2, rho=0.01)
    hp1.poly_chunk = 200
    hp1.poly_pack = -1
    g1 = gpu_loss_grad(p, mu, sg, lamb, hp1)
    for b in range(B):
        dt = np.abs(g["terms"][b] - g1["terms"][b]) / np.maximum(np.abs(g1["terms"][b]), 1.0)
        assert dt.max() <= 1e-6, (b, g["terms"][b], g1["terms"][b])
        for k in ("gm", "gs"):
            e = np.abs(g[k][b] - g1[k][b]).max() / np.abs(g1[k][b]).max()
            assert e <= 1e-6, (b, k, e)


@pytest.mark.parametrize("II,n_back", [(0, 0), (3001, 3)])
def test_maximum_horizon(II, n_back):
    """D = 2^22, the largest horizon the library takes: 4096 tiles of the
    step-by-step kernel, no polynomial path (no chunk width leaves a strip of
    at most 320 steps), sigmas from 0.5 to 2e5 (sharp ops leave most tiles
    to the exact far-tail shortcut, wide ones span the horizon), delays up
    to 70000 steps."""
    p = _ragged_problem(91 + II, N=40, D=1 << 22, II=II, n_back=n_back, big_delay=False)
    p.delay[[5, 17]] = [300, 70000]
    B = 2
    rng = np.random.default_rng(92)
    mu = rng.uniform(-100, p.D + 100, size=(B, p.n_ops)).astype(np.float32)
    sg = np.exp(rng.uniform(np.log(0.5), np.log(2e5), size=(B, p.n_ops))).astype(np.float32)
    _check(p, mu, sg, _lam(B, 93), hparams(alpha=0.2, rho=0.01), range(B), f"D=2^22 II={II}")


def test_small_edge_cases():
    """D = 1 (one bin holds all mass), a single op, no edges."""
    for D, N, with_edges in ((1, 5, True), (2, 1, False), (3, 4, False), (64, 1, False)):
        rows = [[j for j in range(i + 1, N) if (i + j) % 2] if with_edges else [] for i in range(N)]
        row_ptr = np.zeros(N + 1, np.int32); row_ptr[1:] = np.cumsum([len(r) for r in rows])
        col = np.array([j for r in rows for j in r], np.int32)
        p = Problem(n_ops=N, row_ptr=row_ptr, col_idx=col, delay=np.zeros(N, np.int32),
                    rtype=np.zeros(N, np.int32), capacity=np.array([0.5], np.float32), D=D)
        mu, sg = random_state(N, D, 2, seed=D + N)
        _check(p, mu, sg, _lam(2, 4), hparams(alpha=0.5, rho=0.1), range(2), f"edge D={D} N={N}")


@pytest.mark.parametrize("D", [200, 3000])
def test_sigma_to_zero_usage_bit_exact(D):
    """sigma -> 0: usage is the integer histogram of the rounded schedule,
    bit for bit; the violation and edge-length terms are exact counts (one
    op-kernel tile at D = 200; at D = 3000 the narrow kernel takes every op
    over the whole horizon)."""
    for II in (0, 5):
        p = _ragged_problem(21, N=300, D=D, II=II, n_back=8 if II else 0, big_delay=False)
        rng = np.random.default_rng(22)
        s_int = rng.integers(-3, D + 5, size=(2, p.n_ops))
        mu = (s_int + rng.uniform(-0.4, 0.4, size=s_int.shape)).astype(np.float32)
        sg = np.full(mu.shape, 1e-5, np.float32)
        g = gpu_loss_grad(p, mu, sg, np.zeros((2, 3), np.float32), hparams(alpha=0.0, rho=0.0))
        for b in range(2):
            ot, oU, *_ = oracle.loss_grad(p, mu[b:b + 1].astype(np.float64), sg[b:b + 1].astype(np.float64),
                                          [0, 0, 0], 0.0, 0.0, grad=False)
            assert np.array_equal(g["U"][b], oU[0])
            # V_dep, V_rec, L_com are integer counts; V_res = sum (U - C)^+ has
            # non-integer capacities and is compared within the float tolerance
            for c in (1, 3, 4):
                assert g["terms"][b][c] == ot[0][c], (c, g["terms"][b], ot[0])
            assert abs(g["terms"][b][2] - ot[0][2]) <= TOL * max(ot[0][2], 1.0)
            assert np.all(g["gm"][b] == 0) and np.all(g["gs"][b] == 0)


def test_deterministic_bitwise():
    p = make_problem("small", seed=3)
    mu, sg = random_state(p.n_ops, p.D, 4, seed=3, sigma_range=(0.5, 60))
    lam = _lam(4, 3)
    a = gpu_loss_grad(p, mu, sg, lam, hparams())
    b = gpu_loss_grad(p, mu, sg, lam, hparams())
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("cfg,sig", [("medium", (0.05, 6.0)), ("large", (0.2, 4.0))])
def test_deterministic_bitwise_narrow_and_split(cfg, sig):
    """Repeat runs agree bit for bit where ops of a wave share LDS usage rows
    (four-op lane groups), constant ops add integer counts with LDS atomics
    and the op kernel's work-groups are split (the 10k-op workload with 32
    restarts)."""
    p = make_problem(cfg, seed=5)
    B = CONFIGS[cfg].B
    mu, sg = random_state(p.n_ops, p.D, B, seed=5, sigma_range=sig)
    lam = _lam(B, 5)
    a = gpu_loss_grad(p, mu, sg, lam, hparams())
    b = gpu_loss_grad(p, mu, sg, lam, hparams())
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def _state(ctx, mu, sg, lam):
    import torch
    dev = torch.device("cuda")
    B, N = mu.shape
    st = dict(mu=torch.from_numpy(mu).to(dev), sigma=torch.from_numpy(sg).to(dev),
              m=torch.zeros(2, B, N, device=dev), v=torch.zeros(2, B, N, device=dev),
              lam=torch.from_numpy(lam).to(dev), t=torch.zeros(1, dtype=torch.int32, device=dev))
    ctx.bind_state(st["mu"], st["sigma"], st["m"], st["v"], st["lam"], st["t"])
    return st


def test_adam_from_grad_matches_oracle():
    """Adam (Kingma & Ba) + sigma clamp + lambda update, fed the GPU's own
    gradient, against the fp64 oracle's Adam on the same gradient."""
    import torch
    p = make_problem("small", seed=4)
    B = 4
    hp = hparams(alpha=0.1, rho=0.01, lr=0.05)
    mu, sg = random_state(p.n_ops, p.D, B, seed=4, sigma_range=(0.04, 30))
    lam = _lam(B, 5)
    ctx = bd.Context(p, B, hp)
    st = _state(ctx, mu.copy(), sg.copy(), lam.copy())
    dev = torch.device("cuda")
    terms = torch.zeros(B, bd.N_TERMS, device=dev)
    gm = torch.zeros(B, p.n_ops, device=dev); gs = torch.zeros(B, p.n_ops, device=dev)
    m_o = np.zeros((2, B, p.n_ops)); v_o = np.zeros((2, B, p.n_ops))
    th_mu, th_sg, lam_o = mu.astype(np.float64), sg.astype(np.float64), lam.astype(np.float64)
    for it in range(1, 4):
        ctx.loss_grad(st["mu"], st["sigma"], st["lam"], terms, gm, gs)
        ctx.adam_from_grad(gm, gs, terms)
        ctx.sync()
        g1 = gm.cpu().numpy().astype(np.float64); g2 = gs.cpu().numpy().astype(np.float64)
        tt = terms.cpu().numpy().astype(np.float64)
        # oracle Adam from the GPU gradient, starting from the GPU's pre-step state
        for b in range(B):
            th_mu[b], m_o[0, b], v_o[0, b] = oracle.adam(th_mu[b], m_o[0, b], v_o[0, b], g1[b], it, hp.lr)
            th_sg[b], m_o[1, b], v_o[1, b] = oracle.adam(th_sg[b], m_o[1, b], v_o[1, b], g2[b], it, hp.lr)
        th_sg = np.maximum(th_sg, float(np.float32(hp.sigma_min)))
        lam_o = lam_o + float(np.float32(hp.rho)) * tt[:, 1:4]
        gmu_ = st["mu"].cpu().numpy(); gsg_ = st["sigma"].cpu().numpy()
        assert np.all(np.abs(gmu_ - th_mu) <= TOL * np.maximum(np.abs(th_mu), 1.0))
        assert np.all(np.abs(gsg_ - th_sg) <= TOL * np.maximum(np.abs(th_sg), 1.0))
        assert np.allclose(st["lam"].cpu().numpy(), lam_o, rtol=1e-6, atol=1e-7)
        assert int(st["t"].item()) == it
        # continue from the GPU state so that rounding does not accumulate
        th_mu, th_sg = gmu_.astype(np.float64), gsg_.astype(np.float64)
        m_o = st["m"].cpu().numpy().astype(np.float64); v_o = st["v"].cpu().numpy().astype(np.float64)
    ctx.close()


def test_step_equals_loss_grad_plus_adam_bitwise():
    """gaus_step fuses exactly loss_grad + adam_from_grad (same kernels)."""
    import torch
    p = make_problem("pipelined", seed=1, n_ops=800)
    B = 3
    hp = hparams(alpha=0.05, rho=0.01, lr=0.02)
    mu, sg = random_state(p.n_ops, p.D, B, seed=8, sigma_range=(0.3, 50))
    lam = _lam(B, 9)
    ca = bd.Context(p, B, hp); sa = _state(ca, mu.copy(), sg.copy(), lam.copy())
    cb = bd.Context(p, B, hp); sb = _state(cb, mu.copy(), sg.copy(), lam.copy())
    dev = torch.device("cuda")
    terms_a = torch.zeros(B, bd.N_TERMS, device=dev)
    ca.step(5, terms_a)
    terms = torch.zeros(B, bd.N_TERMS, device=dev)
    gm = torch.zeros(B, p.n_ops, device=dev); gs = torch.zeros(B, p.n_ops, device=dev)
    for _ in range(5):
        cb.loss_grad(sb["mu"], sb["sigma"], sb["lam"], terms, gm, gs)
        cb.adam_from_grad(gm, gs, terms)
    ca.sync(); cb.sync()
    for k in ("mu", "sigma", "m", "v", "lam", "t"):
        assert torch.equal(sa[k], sb[k]), k
    assert torch.equal(terms_a, terms)
    ca.close(); cb.close()


@pytest.mark.parametrize("cfg,II,D", [("small", 0, 0), ("medium", 0, 0), ("pipelined", 64, 0), ("large", 0, 0),
                                      ("large", 0, 40000)])
def test_legalize_bit_exact(cfg, II, D):
    """Alg. 3 / Alg. 4 bit for bit against the oracle, with the schedule in
    LDS as 16-bit ready times (II = 0, D < 2^15), as 32-bit ones with the
    pass snapshot (modulo), and in HBM (50k ops at D = 40000: neither fits)."""
    import dataclasses
    import torch
    p = make_problem(cfg, seed=2)
    if D:
        p = dataclasses.replace(p, D=D)
    B = 4
    rng = np.random.default_rng(30)
    mu = rng.uniform(-3, p.D + 3, size=(B, p.n_ops)).astype(np.float32)
    mu[0, :50] = np.floor(mu[0, :50]) + 0.5           # exact ties round up
    mu[1, :5] = [np.nan, np.inf, -np.inf, 0.49999997, -0.5]
    if B > 2:                                          # a nearly legal restart
        a, l, _ = oracle.asap_alap(p)
        mu[2] = ((a + l) / 2).astype(np.float32)
    say(f"[legalize] {cfg} N={p.n_ops} nb={p.n_back} II={p.II}")
    ctx = bd.Context(p, B, hparams())
    dev = torch.device("cuda")
    sched = torch.zeros(B, p.n_ops, dtype=torch.int32, device=dev)
    st = ctx.legalize(torch.from_numpy(mu).to(dev), sched)
    s_o, st_o = oracle.legalize(p, mu)
    assert np.array_equal(st, st_o), (st, st_o)
    for b in range(B):
        if st_o[b] in (0, 5):   # converged: the least fixed point is unique
            assert np.array_equal(sched[b].cpu().numpy().astype(np.int64), s_o[b]), b
    ctx.close()


def test_legalize_infeasible_recurrence():
    """A recurrence that no II-periodic schedule satisfies never converges."""
    import torch
    p = Problem(n_ops=3, row_ptr=np.array([0, 1, 2, 2], np.int32), col_idx=np.array([1, 2], np.int32),
                delay=np.array([5, 1, 1], np.int32), rtype=np.zeros(3, np.int32),
                capacity=np.array([1.0], np.float32), D=40, II=2, back_src=np.array([1], np.int32),
                back_dst=np.array([0], np.int32), back_dist=np.array([1], np.int32))
    ctx = bd.Context(p, 1, hparams())
    sched = torch.zeros(1, 3, dtype=torch.int32, device="cuda")
    st = ctx.legalize(torch.tensor([[0.0, 6.0, 8.0]], device="cuda"), sched)
    _, st_o = oracle.legalize(p, np.array([[0.0, 6.0, 8.0]], np.float32))
    assert st[0] == st_o[0] == bd.E_NOT_CONVERGED
    ctx.close()


def test_init_state_matches_oracle():
    import torch
    p = make_problem("medium", seed=0)
    B = 3
    u = restart_uniforms(p.n_ops, B, seed=0)
    ctx = bd.Context(p, B, hparams())
    mu = torch.zeros(B, p.n_ops, device="cuda"); sg = torch.zeros(B, p.n_ops, device="cuda")
    ctx.init_state(mu, sg, u)
    hp = hparams()
    mo, so, rc = oracle.init_state(p, B, u, kappa=float(np.float32(hp.kappa)),
                                   sigma_min=float(np.float32(hp.sigma_min)))
    assert rc == 0
    assert np.array_equal(mu.cpu().numpy(), mo.astype(np.float32))
    assert np.array_equal(sg.cpu().numpy(), so.astype(np.float32))
    a, l = ctx.asap_alap()
    ao, lo, _ = oracle.asap_alap(p)
    assert np.array_equal(a, ao) and np.array_equal(l, lo)
    ctx.close()
