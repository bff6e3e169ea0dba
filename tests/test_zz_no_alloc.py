"""The allocation-free discrete schedule cost (gaus_schedule_cost_noalloc,
scratch in the library's fixed device array) against gaus_schedule_cost on
the same schedules: two calls in a row, the second with a smaller input (its
scratch still holds the first call's counts), and the size limit."""
import numpy as np
import pytest

import oracle
from paper_2602_20427_amd import binding as bd
from paper_2602_20427_amd.workloads import Problem, make_problem, random_state, with_storage
from tests.gpu_common import hparams, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oracle.build(force=False)
    bd.load()
    yield


def _schedules(p, B, seed):
    """Legalized roundings, a random (illegal) row, a plain rounding and a row
    with steps outside the horizon."""
    rng = np.random.default_rng(seed)
    mu, _ = random_state(p.n_ops, p.D, B, seed=seed + 1)
    sched, _ = oracle.legalize(p, mu)
    sched[B - 1] = rng.integers(0, p.D, size=p.n_ops)
    if B > 2:
        sched[1] = np.floor(mu[1] + 0.5).astype(np.int64)
        sched[2, :7] = -1
    return sched.astype(np.int32)


def test_noalloc_schedule_cost_equals_allocating_entry_point():
    import torch
    dev = torch.device("cuda")
    for cfg, B in (("medium", 8), ("small", 3)):   # the second input is smaller in N, B, D and T
        p = with_storage(make_problem(cfg, seed=0), seed=2)
        hp = hparams(alpha=0.37)
        hp.beta_res, hp.gamma_mem = 1.5, 0.25
        ctx = bd.Context(p, B, hp)
        s = torch.from_numpy(_schedules(p, B, 40 + B)).to(dev)
        ref = torch.zeros(B, bd.N_COST, dtype=torch.float64, device=dev)
        got = torch.full((B, bd.N_COST), float("nan"), dtype=torch.float64, device=dev)
        ctx.schedule_cost(s, ref)
        ctx.schedule_cost_noalloc(s, got)
        ctx.sync()
        say(f"[noalloc] {cfg} B={B} N={p.n_ops} D={p.D}: legal {got[:, 5].tolist()}")
        assert torch.equal(ref, got), (ref, got)
        o = oracle.schedule_cost(p, s.cpu().numpy().astype(np.int64), alpha=hp.alpha_com, beta=hp.beta_res,
                                 gamma=hp.gamma_mem)
        g = got.cpu().numpy()
        assert np.array_equal(g[:, [1, 2, 5]], o[:, [1, 2, 5]])
        assert np.allclose(g[:, [0, 3, 4]], o[:, [0, 3, 4]], rtol=1e-12, atol=0)
        ctx.close()


def test_noalloc_schedule_cost_rejects_oversized_inputs():
    """More scratch than the fixed array holds: INVALID_ARG, nothing launched."""
    import torch
    N, B, D = 4, 8, 1 << 18   # usage counts alone: 8 * 2^18 * 4 B = 8 MiB, plus the storage rows
    p = Problem(n_ops=N, row_ptr=np.array([0, 1, 2, 3, 3], np.int32), col_idx=np.array([1, 2, 3], np.int32),
                delay=np.ones(N, np.int32), rtype=np.zeros(N, np.int32), capacity=np.array([1.0], np.float32), D=D)
    ctx = bd.Context(p, B, hparams(poly_chunk=-1))
    s = torch.zeros(B, N, dtype=torch.int32, device="cuda")
    c = torch.zeros(B, bd.N_COST, dtype=torch.float64, device="cuda")
    with pytest.raises(bd.GausError) as ei:
        ctx.schedule_cost_noalloc(s, c)
    assert ei.value.status == bd.E_INVALID_ARG and "scratch" in str(ei.value)
    ctx.close()
