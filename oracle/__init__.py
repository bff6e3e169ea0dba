"""CPU oracle for the Gaussian-relaxed scheduling objective (fp64).

TEST INFRASTRUCTURE ONLY: only `tests/`, `__graft_entry__.smoke()` and the
CPU-baseline leg of `bench.py` may import this package.  It shares no code with
the GPU library (`paper_2602_20427_amd`), and the library never imports it.

`gaus_oracle.c` holds the arithmetic; this module builds it with gcc, loads it
with ctypes and converts numpy arrays.  `brute.py` enumerates all schedules of
tiny instances for the pins.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gaus_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, E_INVALID, E_CYCLE, E_HORIZON, E_NOT_CONVERGED, E_OVERFLOW, E_NOMEM = 0, 1, 2, 3, 4, 5, 7


def build(force: bool = True) -> str:
    """Compile the oracle (plain C, fp64, OpenMP) into oracle/liboracle.so."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-D_GNU_SOURCE",
               "-Wall", "-Wextra", "-Wno-unused-parameter", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Problem(C.Structure):
    _fields_ = [("n", C.c_int32), ("e", C.c_int32),
                ("row_ptr", C.c_void_p), ("col", C.c_void_p), ("delay", C.c_void_p),
                ("rtype", C.c_void_p), ("K", C.c_int32), ("cap", C.c_void_p),
                ("D", C.c_int32), ("II", C.c_int32), ("nb", C.c_int32),
                ("bsrc", C.c_void_p), ("bdst", C.c_void_p), ("bdist", C.c_void_p),
                ("bmem", C.c_void_p)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = C.CDLL(_LIB)
        P = C.POINTER(_Problem)
        vp, i32, i64, dbl = C.c_void_p, C.c_int32, C.c_int64, C.c_double
        lib.orc_loss_grad.argtypes = [P, vp, vp, vp, dbl, dbl, dbl, dbl, dbl, dbl, vp, vp, vp, vp, vp, vp]
        lib.orc_loss_grad.restype = C.c_int
        lib.orc_edge_terms_double_sum.argtypes = [P, vp, vp, vp]
        lib.orc_edge_terms_double_sum.restype = None
        lib.orc_adam.argtypes = [i64, vp, vp, vp, vp, i32, dbl, dbl, dbl, dbl]
        lib.orc_adam.restype = None
        lib.orc_schedule_cost.argtypes = [P, vp, dbl, dbl, dbl, vp]
        lib.orc_schedule_cost.restype = C.c_int
        lib.orc_legalize.argtypes = [P, vp, vp]
        lib.orc_legalize.restype = C.c_int
        lib.orc_asap_alap.argtypes = [P, vp, vp]
        lib.orc_asap_alap.restype = C.c_int
        lib.orc_topo.argtypes = [P, vp, vp]
        lib.orc_topo.restype = C.c_int
        lib.orc_init_state.argtypes = [P, i32, vp, dbl, dbl, vp, vp]
        lib.orc_init_state.restype = C.c_int
        lib.orc_set_family.argtypes = [i32]
        lib.orc_set_family.restype = None
        lib.orc_mass.argtypes = [dbl, dbl, i32, i32]
        lib.orc_mass.restype = dbl
        lib.orc_check.argtypes = [P, vp, vp, vp, vp, vp, vp, dbl, dbl, dbl, i32, C.c_float, C.c_float,
                                  vp, vp, vp, vp]
        lib.orc_check.restype = C.c_int
        lib.orc_usage_cell_grad.argtypes = [P, vp, vp, i32, i32, dbl, vp, vp]
        lib.orc_usage_cell_grad.restype = C.c_int
        lib.orc_set_num_threads.argtypes = [i32]
        lib.orc_set_num_threads.restype = None
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = C.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


class OracleProblem:
    """Holds contiguous copies of a problem's arrays for the C oracle."""

    def __init__(self, prob):
        self.n = int(prob.n_ops)
        self.D = int(prob.D)
        self.II = int(prob.II)
        self.K = int(prob.n_types)
        self.row_ptr = np.ascontiguousarray(prob.row_ptr, np.int32)
        self.col = np.ascontiguousarray(prob.col_idx, np.int32)
        self.delay = np.ascontiguousarray(prob.delay, np.int32)
        self.rtype = np.ascontiguousarray(prob.rtype, np.int32)
        self.cap = np.ascontiguousarray(prob.capacity, np.float64)
        self.bsrc = np.ascontiguousarray(prob.back_src, np.int32)
        self.bdst = np.ascontiguousarray(prob.back_dst, np.int32)
        self.bdist = np.ascontiguousarray(prob.back_dist, np.int32)
        mem = getattr(prob, "mem_units", None)
        self.bmem = np.ascontiguousarray(np.ones(self.n) if mem is None else mem, np.float64)
        self.s = _Problem(self.n, int(self.row_ptr[-1]), _ptr(self.row_ptr), _ptr(self.col),
                          _ptr(self.delay), _ptr(self.rtype), self.K, _ptr(self.cap),
                          self.D, self.II, int(self.bsrc.shape[0]), _ptr(self.bsrc),
                          _ptr(self.bdst), _ptr(self.bdist), _ptr(self.bmem))

    @property
    def T(self) -> int:
        return self.II if self.II > 0 else self.D


def _op(prob):
    return prob if isinstance(prob, OracleProblem) else OracleProblem(prob)


def num_threads() -> int:
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads of the oracle's loops from now on."""
    _load().orc_set_num_threads(int(n))


FAMILIES = {"gaussian": 0, "logistic": 1, "laplace": 2, "cauchy": 3}


def set_family(family) -> None:
    """Distribution family of the relaxed start times (App. E) for the calls
    that follow: "gaussian", "logistic", "laplace", "cauchy" (or 0..3)."""
    _load().orc_set_family(int(FAMILIES.get(family, family)))


def loss_grad(prob, mu, sigma, lam, alpha, rho, grad=True, tie_tol=1e-4, beta=0.0, tau=1e-2, gamma=0.0,
              mreg_out=None):
    """Per restart b: terms [B,7] = (L, V_dep, V_res, V_rec, L_com, L_res, L_mem),
    U [B,K,T], g_mu, g_sigma [B,N] (fp64), ties [B] (count of near-tie usage
    cells).  beta weights the smooth peak usage L_res, gamma the smooth peak
    storage L_mem (both temperature tau) in L.  mreg_out [B,T], if given,
    receives the expected (folded) storage units per slot."""
    lib, op = _load(), _op(prob)
    mu = np.atleast_2d(np.asarray(mu, np.float64))
    sigma = np.atleast_2d(np.asarray(sigma, np.float64))
    lam = np.atleast_2d(np.asarray(lam, np.float64))
    B = mu.shape[0]
    terms = np.zeros((B, 7)); U = np.zeros((B, op.K, op.T))
    gm = np.zeros((B, op.n)); gs = np.zeros((B, op.n)); ties = np.zeros(B, np.int64)
    for b in range(B):
        m = np.ascontiguousarray(mu[b]); s = np.ascontiguousarray(sigma[b])
        l = np.ascontiguousarray(lam[b if lam.shape[0] > 1 else 0])
        t = np.zeros(7); u = np.zeros((op.K, op.T)); nt = np.zeros(1, np.int64)
        mr = np.zeros(op.T) if mreg_out is not None else None
        g1 = np.zeros(op.n); g2 = np.zeros(op.n)
        rc = lib.orc_loss_grad(C.byref(op.s), _ptr(m), _ptr(s), _ptr(l), float(alpha), float(rho),
                               float(beta), float(tau), float(gamma), float(tie_tol), _ptr(t), _ptr(u),
                               _ptr(mr) if mr is not None else None,
                               _ptr(g1) if grad else None, _ptr(g2) if grad else None, _ptr(nt))
        if rc != OK:
            raise RuntimeError(f"oracle loss_grad failed: {rc}")
        terms[b] = t; U[b] = u; gm[b] = g1; gs[b] = g2; ties[b] = nt[0]
        if mr is not None:
            mreg_out[b] = mr
    return terms, U, gm, gs, ties


def usage_cell_grad(prob, mu, sigma, k, s, w=1.0):
    """w * dU_k(s)/dmu_i and w * dU_k(s)/dsigma_i for every op i (fp64 [N]
    each) of one restart: the gradient the ReLU indicator of cell (k, s) adds
    when it is 1 (App. B.2 eq:relu, folded as in App. B.3)."""
    lib, op = _load(), _op(prob)
    m = np.ascontiguousarray(mu, np.float64); sg = np.ascontiguousarray(sigma, np.float64)
    gm = np.zeros(op.n); gs = np.zeros(op.n)
    rc = lib.orc_usage_cell_grad(C.byref(op.s), _ptr(m), _ptr(sg), int(k), int(s), float(w), _ptr(gm), _ptr(gs))
    if rc != OK:
        raise RuntimeError(f"oracle usage_cell_grad failed: {rc}")
    return gm, gs


def edge_terms_double_sum(prob, mu, sigma):
    """(V_dep, L_com, V_rec) from the paper's literal double sums (tiny only)."""
    lib, op = _load(), _op(prob)
    m = np.ascontiguousarray(mu, np.float64); s = np.ascontiguousarray(sigma, np.float64)
    out = np.zeros(3)
    lib.orc_edge_terms_double_sum(C.byref(op.s), _ptr(m), _ptr(s), _ptr(out))
    return out


def adam(theta, m, v, g, t, lr, b1=0.9, b2=0.999, eps=1e-8):
    """One Adam step in fp64; returns new (theta, m, v)."""
    lib = _load()
    th = np.ascontiguousarray(theta, np.float64).copy()
    mm = np.ascontiguousarray(m, np.float64).copy()
    vv = np.ascontiguousarray(v, np.float64).copy()
    gg = np.ascontiguousarray(g, np.float64)
    lib.orc_adam(th.size, _ptr(th), _ptr(mm), _ptr(vv), _ptr(gg), int(t), float(lr), float(b1),
                 float(b2), float(eps))
    return th, mm, vv


def legalize(prob, mu):
    """Legalize each restart of mu [B,N] float32: (sched int64 [B,N], status [B])."""
    lib, op = _load(), _op(prob)
    mu = np.atleast_2d(np.asarray(mu, np.float32))
    out = np.zeros(mu.shape, np.int64); st = np.zeros(mu.shape[0], np.int32)
    for b in range(mu.shape[0]):
        m = np.ascontiguousarray(mu[b]); s = np.zeros(op.n, np.int64)
        st[b] = lib.orc_legalize(C.byref(op.s), _ptr(m), _ptr(s))
        out[b] = s
    return out, st


NO_BEST = (np.inf, np.inf, np.inf, np.inf, np.inf, 0.0)   # a best-cost row holding no schedule yet


def check(prob, mu, sigma, m, v, best_s, best_c, alpha=0.0, beta=0.0, gamma=0.0, reinit_sigma=0,
          kappa=1.0 / 6.0, sigma_min=0.05):
    """One check of the Alg. 1 driver for every restart (orc_check): mu,
    sigma [B,N] float32, m, v [2,B,N] float32 (moments of mu, then sigma),
    best_s [B,N] int64, best_c [B,6]; returns new copies of all six and
    (cand [B,N] int64, cand_c [B,6], mode [B], improved [B])."""
    lib, op = _load(), _op(prob)
    mu = np.array(mu, np.float32, copy=True); sigma = np.array(sigma, np.float32, copy=True)
    m = np.array(m, np.float32, copy=True); v = np.array(v, np.float32, copy=True)
    best_s = np.array(best_s, np.int64, copy=True); best_c = np.array(best_c, np.float64, copy=True)
    B = mu.shape[0]
    cand = np.zeros((B, op.n), np.int64); cand_c = np.zeros((B, 6))
    mode = np.zeros(B, np.int32); imp = np.zeros(B, np.int32)
    for b in range(B):
        mb, sb = np.ascontiguousarray(mu[b]), np.ascontiguousarray(sigma[b])
        m2, v2 = np.ascontiguousarray(m[:, b]), np.ascontiguousarray(v[:, b])
        bs, bc = np.ascontiguousarray(best_s[b]), np.ascontiguousarray(best_c[b])
        cs, cc = np.zeros(op.n, np.int64), np.zeros(6)
        md, im = np.zeros(1, np.int32), np.zeros(1, np.int32)
        rc = lib.orc_check(C.byref(op.s), _ptr(mb), _ptr(sb), _ptr(m2), _ptr(v2), _ptr(bs), _ptr(bc),
                           float(alpha), float(beta), float(gamma), int(reinit_sigma), float(kappa),
                           float(sigma_min), _ptr(cs), _ptr(cc), _ptr(md), _ptr(im))
        if rc != OK:
            raise RuntimeError(f"oracle check failed: {rc}")
        mu[b], sigma[b], m[:, b], v[:, b], best_s[b], best_c[b] = mb, sb, m2, v2, bs, bc
        cand[b], cand_c[b], mode[b], imp[b] = cs, cc, md[0], im[0]
    return mu, sigma, m, v, best_s, best_c, cand, cand_c, mode, imp


def schedule_cost(prob, sched, alpha=0.0, beta=0.0, gamma=0.0):
    """Discrete cost of integer schedules sched [B,N]: [B,6] = (cost, L_com,
    L_res, L_mem, V_res, legal)."""
    lib, op = _load(), _op(prob)
    sched = np.atleast_2d(np.asarray(sched, np.int64))
    out = np.zeros((sched.shape[0], 6))
    for b in range(sched.shape[0]):
        sb = np.ascontiguousarray(sched[b]); o = np.zeros(6)
        rc = lib.orc_schedule_cost(C.byref(op.s), _ptr(sb), float(alpha), float(beta), float(gamma), _ptr(o))
        if rc != OK:
            raise RuntimeError(f"oracle schedule_cost failed: {rc}")
        out[b] = o
    return out


def asap_alap(prob):
    lib, op = _load(), _op(prob)
    a = np.zeros(op.n, np.int64); l = np.zeros(op.n, np.int64)
    rc = lib.orc_asap_alap(C.byref(op.s), _ptr(a), _ptr(l))
    return a, l, rc


def topo(prob):
    lib, op = _load(), _op(prob)
    lev = np.zeros(op.n, np.int32); order = np.zeros(op.n, np.int32)
    rc = lib.orc_topo(C.byref(op.s), _ptr(lev), _ptr(order))
    return lev, order, rc


def init_state(prob, B, u, kappa=1.0 / 6.0, sigma_min=0.05):
    lib, op = _load(), _op(prob)
    uu = np.ascontiguousarray(np.broadcast_to(u, (B, op.n)), np.float64)
    mu = np.zeros((B, op.n)); sg = np.zeros((B, op.n))
    rc = lib.orc_init_state(C.byref(op.s), int(B), _ptr(uu), float(kappa), float(sigma_min),
                            _ptr(mu), _ptr(sg))
    return mu, sg, rc


def mass(mu, sigma, d, D):
    return float(_load().orc_mass(float(mu), float(sigma), int(d), int(D)))
