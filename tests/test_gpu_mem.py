"""Parity of the storage term (expected storage units of eq:active, folded
like the usage, and its smooth peak L_mem = tau log sum_t exp(MReg(t)/tau))
and its gradient: HIP path through the C ABI vs the fp64 oracle."""
import numpy as np
import pytest

import oracle
from paper_2602_20427_amd import binding as bd
from paper_2602_20427_amd.workloads import CONFIGS, make_problem, random_state, with_storage
from tests.gpu_common import TOL, hparams, oracle_compare, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oracle.build(force=False)
    bd.load()
    yield


def _run(p, mu, sg, lam, hp):
    """loss_grad on the GPU; returns terms, gradients, usage and storage."""
    import torch
    B, N = mu.shape
    ctx = bd.Context(p, B, hp)
    dev = torch.device("cuda")
    m, s, l = (torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(dev) for x in (mu, sg, lam))
    terms = torch.zeros(B, bd.N_TERMS, device=dev)
    gm = torch.zeros(B, N, device=dev)
    gs = torch.zeros(B, N, device=dev)
    ctx.loss_grad(m, s, l, terms, gm, gs)
    U = torch.zeros(B, ctx.K, ctx.T, device=dev)
    M = torch.zeros(B, ctx.T, device=dev)
    ctx.get_usage(U)
    ctx.get_storage(M)
    ctx.sync()
    say(f"  [ctx] poly {ctx.poly_config()}")
    out = dict(terms=terms.cpu().numpy().astype(np.float64), gm=gm.cpu().numpy().astype(np.float64),
               gs=gs.cpu().numpy().astype(np.float64), U=U.cpu().numpy().astype(np.float64),
               M=M.cpu().numpy().astype(np.float64))
    ctx.close()
    return out


def _storage_bar(dM, tau, x, gamma, p, sigma, g_all):
    """Gradient error bound derived from the arithmetic (reported with each
    comparison; the tests hold the plain bar).

    The storage gradient of op i is sum_t c(t) dMReg(t)/dtheta_i with
    c = gamma softmax(MReg/tau).  If the fp32 profile is off by at most dM
    per slot (measured: the error of this very evaluation), each perturbed
    weight of a slot t other than the peak t* obeys
    |c'(t) - c(t)| <= min(exp((x_t - x_t* + 2 dM)/tau), c(t) (exp(2 dM/tau) - 1)),
    and the peak's change is at most their sum, so
    |dc|_1 <= 2 gamma sum_{t != t*} min(...).  With
    |dMReg(t)/dtheta_i| <= n_fold (b_i + sum over predecessors b_h) phi(0)/sigma_i
    (|z phi(z)| <= phi(0) as well), the gradient moves by at most
    |dc|_1 max_i of that bound; the rest of the path keeps the plain bar."""
    x = np.asarray(x, np.float64)
    T = x.shape[0]
    ts = int(x.argmax())
    c = np.exp((x - x.max()) / tau)
    c /= c.sum()
    others = np.delete(np.arange(T), ts)
    dc = 2.0 * gamma * np.minimum(np.exp((x[others] - x[ts] + 2 * dM) / tau),
                                  c[others] * np.expm1(2 * dM / tau)).sum()
    bmem = np.asarray(p.mem_units, np.float64)
    hold = np.where(np.diff(p.row_ptr) > 0, bmem, 0.0)
    pred_b = np.zeros(p.n_ops)
    src = np.repeat(np.arange(p.n_ops), np.diff(p.row_ptr))
    np.add.at(pred_b, p.col_idx, bmem[src])
    n_fold = -(-p.D // T)
    deriv = n_fold * (hold + pred_b) * 0.3989422804014327 / np.asarray(sigma, np.float64)
    return TOL + dc * deriv.max() / max(np.abs(g_all).max(), 1e-30)


def _check_storage(p, mu, sg, lam, hp, what):
    tau = hp.tau
    say(f"[mem] {what}: N={p.n_ops} E={p.n_edges} D={p.D} II={p.II} B={mu.shape[0]} tau={tau}")
    g = _run(p, mu, sg, lam, hp)
    for b in range(mu.shape[0]):
        _compare_storage(p, g, b, mu, sg, lam, hp, what)


def _compare_storage(p, g, b, mu, sg, lam, hp, what):
    """Storage profile, terms, usage and gradients of restart b against the
    oracle, all at the plain bar (either indicator at near-tie usage
    cells); the derived bound on how far the softmax could amplify the
    profile's rounding error is printed beside each gradient error."""
    mr = np.zeros((1, g["M"].shape[1]))
    r, o = oracle_compare(p, g, b, mu, sg, lam, hp, what, tau=hp.tau, gamma=hp.gamma_mem, mreg_out=mr)
    dM = np.abs(g["M"][b] - mr[0]).max()
    em = dM / max(np.abs(mr[0]).max(), 1.0)
    assert em <= TOL, f"{what} b={b} storage err {em}"
    for name, key in (("g_mu", "gm"), ("g_sigma", "gs")):
        bar = _storage_bar(dM, hp.tau, mr[0], hp.gamma_mem, p, sg[b], o[key])
        say(f"  b={b} {name}: err {r[name]:.2e} (derived bound {bar:.2e}, dM {dM:.2e}, max MReg "
            f"{mr[0].max():.6g}, L_mem {g['terms'][b][6]:.8g} vs {o['terms'][6]:.8g})")
    return r


@pytest.mark.parametrize("tau", [100.0, 1.0, 0.01])
@pytest.mark.parametrize("cfg", ["tiny", "small", "medium", "pipelined"])
def test_storage_loss_grad(cfg, tau):
    """Storage units drawn from {1, 8, 16, 32} bits plus a sink; random
    states (some means outside the horizon, sigma from 0.5 to 12% of D)."""
    p = with_storage(make_problem(cfg, seed=0), seed=1)
    B = 2
    mu, sg = random_state(p.n_ops, p.D, B, seed=3, sigma_range=(0.5, 0.12 * p.D))
    lam = np.random.default_rng(4).uniform(0.05, 1.0, size=(B, 3)).astype(np.float32)
    hp = hparams(alpha=0.01, rho=1e-3, tau=tau)
    hp.gamma_mem = 1.0
    _check_storage(p, mu, sg, lam, hp, cfg)


@pytest.mark.parametrize("tau", [1.0, 0.01])
def test_storage_polynomial_holders(tau):
    """Holders whose storage term is taken on the chunk polynomials (every
    successor polynomial, at most 4 of them, rho = ((W-1)/2)/sigma summed over
    the holder and its successors at most 1/4) beside holders evaluated step
    by step (more successors, a narrow successor, too large a summed rho):
    sigmas are drawn around those bounds on a 1024-step horizon."""
    p = with_storage(make_problem("medium", seed=2), seed=3)
    B = 2
    hw = hparams()
    hw.gamma_mem = 1.0   # the chunk width chosen with the storage term on
    ctx = bd.Context(p, 1, hw)
    W = ctx.poly_config()["W"]
    ctx.close()
    lam_w = (W - 1) / 2.0
    rng = np.random.default_rng(21)
    rho = np.exp(rng.uniform(np.log(0.02), np.log(0.3), size=(B, p.n_ops)))
    sg = (lam_w / rho).astype(np.float32)
    mu = rng.uniform(-50, p.D + 50, size=(B, p.n_ops)).astype(np.float32)
    # the holders the rule puts on the polynomials (a coverage check only)
    deg = np.diff(p.row_ptr)
    thr = lam_w / 0.25   # the degree-8 bound rho <= 1/4
    n_poly = []
    for b in range(B):
        poly = (sg[b] >= thr) & (p.delay <= 8)
        cnt = 0
        for i in range(p.n_ops):
            succ = p.col_idx[p.row_ptr[i]:p.row_ptr[i + 1]]
            if poly[i] and 1 <= deg[i] <= 4 and poly[succ].all() and \
                    lam_w * (1.0 / sg[b, i] + (1.0 / sg[b, succ]).sum()) <= 0.25:
                cnt += 1
        n_poly.append(cnt)
    holders = int((deg > 0).sum())
    say(f"  W={W}: polynomial holders {n_poly} of {holders}")
    assert min(n_poly) > 0.15 * holders and max(n_poly) < 0.85 * holders
    lam = np.random.default_rng(22).uniform(0.05, 1.0, size=(B, 3)).astype(np.float32)
    hp = hparams(alpha=0.01, rho=1e-3, tau=tau)
    hp.gamma_mem = 1.0
    _check_storage(p, mu, sg, lam, hp, f"polynomial holders tau={tau}")


def test_storage_large_full_size():
    """The 50k-op workload with storage units and a sink at full size (B=8,
    D=4096) in bench.py's launch configuration, from the paper's
    initialization; restarts 0 and 7 against the oracle."""
    from paper_2602_20427_amd.workloads import restart_uniforms
    cfg = CONFIGS["large"]
    p = with_storage(make_problem(cfg, seed=0), seed=1)
    B = cfg.B
    mu, sg, rc = oracle.init_state(p, B, restart_uniforms(p.n_ops, B, seed=0))
    assert rc == 0
    mu, sg = mu.astype(np.float32), sg.astype(np.float32)
    hp = bd.default_hparams()
    hp.lr = cfg.lr
    hp.gamma_mem = 1.0
    lam = np.full((B, 3), hp.lambda0, np.float32)
    g = _run(p, mu, sg, lam, hp)
    for b in (0, B - 1):
        _compare_storage(p, g, b, mu, sg, lam, hp, "large/mem")


def test_storage_unit_bits_plain_bar():
    """One storage unit per op and a temperature far above the storage
    profile's rounding error: the plain 1e-5 bar holds without derivation."""
    p = with_storage(make_problem("small", seed=0), seed=1, bits=(1,))
    B = 2
    mu, sg = random_state(p.n_ops, p.D, B, seed=9, sigma_range=(0.5, 30.0))
    hp = hparams(alpha=0.01, rho=1e-3, tau=10.0)
    hp.gamma_mem = 1.0
    g = _run(p, mu, sg, np.full((B, 3), 0.3, np.float32), hp)
    for b in range(B):
        r = _compare_storage(p, g, b, mu, sg, np.full((B, 3), 0.3, np.float32), hp, "small/mem unit bits")
        say(f"  b={b}: " + " ".join(f"{k}={v:.2e}" for k, v in r.items()))


def test_storage_sigma_to_zero_bit_exact():
    """sigma -> 0 with integer storage units: MReg is the integer storage
    profile of the rounded schedule, bit for bit."""
    for II in (0, 7):
        base = make_problem("small", seed=5, n_ops=300)
        base.II = II
        p = with_storage(base, seed=6)
        rng = np.random.default_rng(7)
        s_int = rng.integers(-2, p.D + 2, size=(2, p.n_ops))
        mu = (s_int + rng.uniform(-0.4, 0.4, size=s_int.shape)).astype(np.float32)
        sg = np.full(mu.shape, 1e-5, np.float32)
        hp = hparams(alpha=0.0, rho=0.0, tau=1.0)
        hp.gamma_mem = 1.0
        g = _run(p, mu, sg, np.zeros((2, 3), np.float32), hp)
        for b in range(2):
            mr = np.zeros((1, g["M"].shape[1]))
            oracle.loss_grad(p, mu[b:b + 1].astype(np.float64), sg[b:b + 1].astype(np.float64), [0, 0, 0],
                             0.0, 0.0, grad=False, tau=1.0, gamma=1.0, mreg_out=mr)
            assert np.array_equal(g["M"][b], mr[0]), (II, b)


def test_storage_step_equals_loss_grad_plus_adam():
    """With the storage term on, the fused step equals loss_grad followed by
    adam_from_grad bit for bit."""
    import torch
    p = with_storage(make_problem("small", seed=0), seed=1)
    B = 2
    mu, sg = random_state(p.n_ops, p.D, B, seed=8, sigma_range=(0.5, 30.0))
    hp = hparams(alpha=0.01, rho=1e-3, lr=0.05, tau=0.05)
    hp.gamma_mem = 1.0
    dev = torch.device("cuda")

    def mk():
        st = dict(mu=torch.from_numpy(mu).to(dev), sigma=torch.from_numpy(sg).to(dev),
                  lam=torch.full((B, 3), 0.2, device=dev), m=torch.zeros(2, B, p.n_ops, device=dev),
                  v=torch.zeros(2, B, p.n_ops, device=dev), t=torch.zeros(1, dtype=torch.int32, device=dev))
        c = bd.Context(p, B, hp)
        c.bind_state(st["mu"], st["sigma"], st["m"], st["v"], st["lam"], st["t"])
        return c, st
    ca, sa = mk()
    cb, sb = mk()
    ta = torch.zeros(B, bd.N_TERMS, device=dev)
    ca.step(3, ta)
    tb = torch.zeros(B, bd.N_TERMS, device=dev)
    gm = torch.zeros(B, p.n_ops, device=dev)
    gs = torch.zeros(B, p.n_ops, device=dev)
    for _ in range(3):
        cb.loss_grad(sb["mu"], sb["sigma"], sb["lam"], tb, gm, gs)
        cb.adam_from_grad(gm, gs, tb)
    ca.sync(); cb.sync()
    assert torch.equal(sa["mu"], sb["mu"]) and torch.equal(sa["sigma"], sb["sigma"])
    assert torch.equal(ta, tb)
    ca.close(); cb.close()
