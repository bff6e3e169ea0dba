"""Seeded synthetic scheduling problems.

This module only draws inputs: random layered DAGs with per-op resource types,
integer delays, capacities, horizon D, initiation interval II and (for
pipelined problems) loop-carried back edges, plus random (mu, sigma) states.
It holds none of the scheduling method's arithmetic (no masses, usages,
penalties, gradients or legalization) so that both the GPU library and the
CPU oracle can be fed from it without sharing any of the method.

The shapes follow the paper's workloads (Section 4.1.2 and the benchmark
statistics table in Appendix C): random-workload graphs of about 1k and 10k
operators, EPFL-sized graphs up to ~57k operators, and a modulo-scheduling
variant with recurrence (back) edges added in proportion to the graph size.
The EPFL and RW suites themselves are not available; these graphs stand in
for them.

Draw order (fixed, from numpy PCG64(seed)): types, delays, forward edges (ops
in id order), back edges.
"""
from __future__ import annotations

from dataclasses import dataclass, field
import numpy as np

# Resource-type mix used for the HLS-like configurations: ALU, MUL, MEM, DIV.
HLS_TYPE_PROBS = (0.60, 0.25, 0.10, 0.05)
HLS_TYPE_DELAYS = (1, 1, 3, 8)


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    n_ops: int
    n_layers: int
    out_degree: float          # Poisson mean of forward out-degree
    type_probs: tuple          # probabilities of each resource type
    delays: object             # tuple per type, or ("uniform", lo, hi) per op
    capacities: tuple
    D: int
    II: int = 0
    back_edge_frac: float = 0.0
    back_dist: tuple = (1, 3)
    B: int = 1
    iters: int = 1000
    lr: float = 1e-2
    init: str = "asap_alap"     # "asap_alap" (paper init) or "uniform" (mu~U[0,D), sigma=sigma0)
    sigma0: float = 1.0
    tight_slack: int = 0        # > 0: D = (longest delay-weighted path to a start) + tight_slack


def _zipf_probs(k: int, s: float) -> tuple:
    w = np.arange(1, k + 1, dtype=np.float64) ** (-s)
    return tuple((w / w.sum()).tolist())


CONFIGS = {
    "tiny": WorkloadConfig("tiny", 64, 8, 2.0, (0.5, 0.5), ("uniform", 1, 3), (2.0, 2.0),
                           D=32, B=1, iters=200, lr=0.05, init="uniform", sigma0=1.0),
    "small": WorkloadConfig("small", 1000, 40, 2.0, HLS_TYPE_PROBS, HLS_TYPE_DELAYS,
                            (8.0, 4.0, 2.0, 1.0), D=256, B=16, iters=1000),
    "medium": WorkloadConfig("medium", 10000, 200, 2.5, HLS_TYPE_PROBS, HLS_TYPE_DELAYS,
                             (32.0, 16.0, 8.0, 2.0), D=1024, B=32, iters=2000),
    "large": WorkloadConfig("large", 50000, 500, 2.0, _zipf_probs(8, 1.2), ("uniform", 1, 4),
                            (64.0,) * 8, D=4096, B=8, iters=2000),
    "pipelined": WorkloadConfig("pipelined", 5000, 100, 2.0, HLS_TYPE_PROBS, HLS_TYPE_DELAYS,
                                (16.0, 8.0, 4.0, 1.0), D=2048, II=64, back_edge_frac=0.02,
                                B=32, iters=2000),
    # the 50k-op graph with the horizon cut to its critical path + 8 steps (the
    # paper sizes horizons by graph depth): narrow start-time laws
    "large-tight": WorkloadConfig("large-tight", 50000, 500, 2.0, _zipf_probs(8, 1.2), ("uniform", 1, 4),
                                  (64.0,) * 8, D=0, B=8, iters=2000, tight_slack=8),
}


@dataclass
class Problem:
    """A scheduling problem in the layout the C ABI takes (CSR by producer)."""
    n_ops: int
    row_ptr: np.ndarray        # int32 [N+1]
    col_idx: np.ndarray        # int32 [E], consumers, sorted within a row
    delay: np.ndarray          # int32 [N]
    rtype: np.ndarray          # int32 [N]
    capacity: np.ndarray       # float32 [K]
    D: int
    II: int = 0
    back_src: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    back_dst: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    back_dist: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    layer: np.ndarray | None = None
    name: str = ""
    mem_units: np.ndarray | None = None   # float32 [N] storage units b_i (None: 1 each)

    @property
    def n_edges(self) -> int:
        return int(self.row_ptr[-1])

    @property
    def n_types(self) -> int:
        return int(self.capacity.shape[0])

    @property
    def n_back(self) -> int:
        return int(self.back_src.shape[0])

    def edges(self):
        """(src, dst) int32 arrays of the forward edges in CSR order."""
        src = np.repeat(np.arange(self.n_ops, dtype=np.int32), np.diff(self.row_ptr))
        return src, self.col_idx.copy()


def _longest_from(src: int, n: int, row_ptr, col_idx, delay) -> np.ndarray:
    """Delay-weighted longest path lengths from `src` along forward edges
    (ids are a topological order).  -1 marks unreachable ops."""
    dist = np.full(n, -1, dtype=np.int64)
    dist[src] = 0
    for u in range(src, n):
        du = dist[u]
        if du < 0:
            continue
        for e in range(row_ptr[u], row_ptr[u + 1]):
            v = col_idx[e]
            cand = du + delay[u]
            if cand > dist[v]:
                dist[v] = cand
    return dist


def make_problem(cfg: WorkloadConfig | str, seed: int = 0, n_ops: int | None = None) -> Problem:
    """Draw one problem.  `n_ops` overrides the size (layers scale with it)."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    rng = np.random.Generator(np.random.PCG64(seed))
    N = cfg.n_ops if n_ops is None else int(n_ops)
    L = cfg.n_layers if n_ops is None else max(2, min(N, round(cfg.n_layers * N / cfg.n_ops)))
    layer = (np.arange(N, dtype=np.int64) * L) // N
    layer_start = np.searchsorted(layer, np.arange(L + 1))

    K = len(cfg.type_probs)
    rtype = rng.choice(K, size=N, p=np.asarray(cfg.type_probs)).astype(np.int32)
    if isinstance(cfg.delays, tuple) and len(cfg.delays) == 3 and cfg.delays[0] == "uniform":
        lo, hi = cfg.delays[1], cfg.delays[2]
        delay = rng.integers(lo, hi + 1, size=N).astype(np.int32)
    else:
        delay = np.asarray(cfg.delays, dtype=np.int32)[rtype]

    rows = []
    for i in range(N):
        l = layer[i]
        if l >= L - 1:
            rows.append(np.zeros(0, np.int64))
            continue
        n = rng.poisson(cfg.out_degree)
        tg = []
        for _ in range(n):
            if l + 2 > L - 1 or rng.random() < 0.5:
                tl = l + 1
            else:
                tl = rng.integers(l + 2, L)
            a, b = layer_start[tl], layer_start[tl + 1]
            tg.append(rng.integers(a, b))
        rows.append(np.unique(np.asarray(tg, dtype=np.int64)))
    row_ptr = np.zeros(N + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col_idx = np.concatenate(rows).astype(np.int32) if row_ptr[-1] else np.zeros(0, np.int32)
    row_ptr = row_ptr.astype(np.int32)

    bsrc, bdst, bdist = [], [], []
    if cfg.II > 0 and cfg.back_edge_frac > 0:
        nb = int(round(cfg.back_edge_frac * int(row_ptr[-1])))
        first_l1 = layer_start[1]
        tries = 0
        while len(bsrc) < nb and tries < 100 * max(nb, 1):
            tries += 1
            j = int(rng.integers(first_l1, N))             # producer (layer >= 1)
            i = int(rng.integers(0, layer_start[layer[j]]))  # consumer in an earlier layer
            k = int(rng.integers(cfg.back_dist[0], cfg.back_dist[1] + 1))
            dist = _longest_from(i, N, row_ptr, col_idx, delay)
            if dist[j] >= 0 and dist[j] + delay[j] > k * cfg.II:
                continue  # recurrence i ~> j -> i could not fit k*II
            bsrc.append(j); bdst.append(i); bdist.append(k)
    D = cfg.D
    if cfg.tight_slack > 0:   # longest delay-weighted path to any op's start (ids are topological)
        start = np.zeros(N, dtype=np.int64)
        for u in range(N):
            for e in range(row_ptr[u], row_ptr[u + 1]):
                v = col_idx[e]
                start[v] = max(start[v], start[u] + delay[u])
        D = int(start.max()) + cfg.tight_slack
    return Problem(
        n_ops=N, row_ptr=row_ptr, col_idx=col_idx, delay=delay, rtype=rtype,
        capacity=np.asarray(cfg.capacities, dtype=np.float32), D=D, II=cfg.II,
        back_src=np.asarray(bsrc, np.int32), back_dst=np.asarray(bdst, np.int32),
        back_dist=np.asarray(bdist, np.int32), layer=layer.astype(np.int32), name=cfg.name)


def random_state(n_ops: int, D: int, B: int, seed: int, sigma_range=(0.3, 8.0),
                 mu_margin: float = 2.0):
    """Random (mu, sigma) float32 [B][N] used as a common test input.

    mu ~ U[-mu_margin, D-1+mu_margin] (some mass outside the horizon on
    purpose), log(sigma) ~ U[log lo, log hi]."""
    rng = np.random.Generator(np.random.PCG64(seed + 7919))
    mu = rng.uniform(-mu_margin, D - 1 + mu_margin, size=(B, n_ops)).astype(np.float32)
    lo, hi = sigma_range
    sigma = np.exp(rng.uniform(np.log(lo), np.log(hi), size=(B, n_ops))).astype(np.float32)
    return mu, sigma


def uniform_state(n_ops: int, D: int, B: int, seed: int, sigma0: float = 1.0):
    """The 'uniform' initial state: mu ~ U[0, D), sigma = sigma0."""
    rng = np.random.Generator(np.random.PCG64(seed + 104729))
    mu = rng.uniform(0.0, float(D), size=(B, n_ops)).astype(np.float32)
    sigma = np.full((B, n_ops), sigma0, dtype=np.float32)
    return mu, sigma


def restart_uniforms(n_ops: int, B: int, seed: int) -> np.ndarray:
    """U[0,1) draws, float64 [B][N], used to place restarts b>=1 inside their
    [ASAP, ALAP] window (the library and the oracle both take these as input)."""
    rng = np.random.Generator(np.random.PCG64(seed + 15485863))
    return rng.random((B, n_ops))


def with_storage(prob: Problem, seed: int, bits=(1, 8, 16, 32)) -> Problem:
    """The same graph prepared for the storage (memory-footprint) objective of
    Formulations B and C: every op's output gets a bit width drawn from `bits`
    as its storage units, and one sink op is appended as a successor of every
    op without successors, so that their outputs are held until the end
    (the footnote to the memory-footprint definition, Sec. 2.1).  The sink has
    storage 0, delay 0 and a resource type of its own that never binds."""
    rng = np.random.default_rng(seed)
    n = prob.n_ops
    mem = rng.choice(np.asarray(bits, np.float32), size=n).astype(np.float32)
    leaves = [i for i in range(n) if prob.row_ptr[i + 1] == prob.row_ptr[i]]
    rows = [list(prob.col_idx[prob.row_ptr[i]:prob.row_ptr[i + 1]]) for i in range(n)]
    for i in leaves:
        rows[i].append(n)
    rows.append([])
    row_ptr = np.zeros(n + 2, np.int32)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([j for r in rows for j in r], np.int32)
    K = prob.n_types
    return Problem(n_ops=n + 1, row_ptr=row_ptr, col_idx=col,
                   delay=np.append(prob.delay, 0).astype(np.int32),
                   rtype=np.append(prob.rtype, K).astype(np.int32),
                   capacity=np.append(prob.capacity, np.float32(n + 1)).astype(np.float32),
                   D=prob.D, II=prob.II, back_src=prob.back_src, back_dst=prob.back_dst,
                   back_dist=prob.back_dist, layer=None, name=prob.name + "+sink",
                   mem_units=np.append(mem, np.float32(0.0)).astype(np.float32))
