"""Thin ctypes binding of libgaus (include/gaus.h).

Argument marshalling only: every step of the scheduling hot path runs in the
gfx950 kernels of libgaus.so.  Device buffers are torch tensors on the current
HIP device; their data pointers and the current HIP stream are handed to the
library.  If the library has not been built this module raises on first use:
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgaus.so")

OK, E_INVALID_ARG, E_CYCLE, E_HORIZON, E_NOT_CONVERGED, E_OVERFLOW, E_DEVICE, E_NOMEM = range(8)

# symbols declared in include/gaus.h
EXPORTS = ("gaus_default_hparams", "gaus_init", "gaus_bind_state", "gaus_loss_grad", "gaus_step",
           "gaus_adam_from_grad", "gaus_legalize", "gaus_schedule_cost", "gaus_schedule_cost_noalloc",
           "gaus_solve", "gaus_solve_check",
           "gaus_init_state",
           "gaus_asap_alap",
           "gaus_get_usage", "gaus_get_storage", "gaus_kernel_timing", "gaus_kernel_timing_read", "gaus_sync",
           "gaus_get_dims", "gaus_get_poly_config", "gaus_poly_census", "gaus_get_poly_grids",
           "gaus_poly_grid_census", "gaus_poly_tier_census", "gaus_last_error", "gaus_status_string",
           "gaus_destroy")


class GausError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_status_name(status)}: {msg}")
        self.status = status


class _Problem(C.Structure):
    _fields_ = [("n_ops", C.c_int32), ("n_edges", C.c_int32), ("row_ptr", C.c_void_p),
                ("col_idx", C.c_void_p), ("delay", C.c_void_p), ("rtype", C.c_void_p),
                ("n_types", C.c_int32), ("capacity", C.c_void_p), ("D", C.c_int32), ("II", C.c_int32),
                ("n_back", C.c_int32), ("back_src", C.c_void_p), ("back_dst", C.c_void_p),
                ("back_dist", C.c_void_p), ("mem_units", C.c_void_p)]


class SolveParams(C.Structure):
    _fields_ = [("max_iters", C.c_int32), ("check_every", C.c_int32), ("time_limit_s", C.c_double),
                ("reinit_sigma", C.c_int32)]


class SolveStats(C.Structure):
    _fields_ = [("iters", C.c_int32), ("checks", C.c_int32), ("reinits", C.c_int32),
                ("improvements", C.c_int32), ("best_restart", C.c_int32), ("seconds", C.c_double)]


N_COST = 6    # cost, L_com, L_res, L_mem, V_res, legal


class HParams(C.Structure):
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("rho", C.c_float), ("lambda0", C.c_float), ("alpha_com", C.c_float),
                ("sigma_min", C.c_float), ("kappa", C.c_float), ("poly_chunk", C.c_int32),
                ("beta_res", C.c_float), ("tau", C.c_float), ("gamma_mem", C.c_float),
                ("family", C.c_int32), ("poly_pack", C.c_int32)]

# CDF family of the relaxed start times (App. E), the values of HParams.family
FAMILIES = {"gaussian": 0, "logistic": 1, "laplace": 2, "cauchy": 3}

N_TERMS = 7   # L, V_dep, V_res, V_rec, L_com, L_res, L_mem


_lib = None


def load():
    """Load libgaus.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (HIP runtime and device memory come from torch)
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(hipcc --offload-arch=gfx950); there is no CPU fallback")
    lib = C.CDLL(LIB_PATH)
    vp, i32 = C.c_void_p, C.c_int32
    sig = {
        "gaus_default_hparams": ([C.POINTER(HParams)], None),
        "gaus_init": ([C.POINTER(_Problem), C.POINTER(HParams), i32, vp, C.POINTER(vp)], C.c_int),
        "gaus_bind_state": ([vp] * 7, C.c_int),
        "gaus_loss_grad": ([vp] * 7, C.c_int),
        "gaus_step": ([vp, i32, vp], C.c_int),
        "gaus_adam_from_grad": ([vp] * 4, C.c_int),
        "gaus_legalize": ([vp] * 4, C.c_int),
        "gaus_schedule_cost": ([vp] * 3, C.c_int),
        "gaus_schedule_cost_noalloc": ([vp] * 3, C.c_int),
        "gaus_solve": ([vp] * 5, C.c_int),
        "gaus_solve_check": ([vp, vp, vp, i32, vp], C.c_int),
        "gaus_init_state": ([vp] * 4, C.c_int),
        "gaus_asap_alap": ([vp] * 3, C.c_int),
        "gaus_get_usage": ([vp] * 2, C.c_int),
        "gaus_get_storage": ([vp] * 2, C.c_int),
        "gaus_kernel_timing": ([vp, i32], C.c_int),
        "gaus_kernel_timing_read": ([vp, vp, vp], C.c_int),
        "gaus_sync": ([vp], C.c_int),
        "gaus_get_dims": ([vp, vp], C.c_int),
        "gaus_get_poly_config": ([vp, vp], C.c_int),
        "gaus_poly_census": ([vp, vp], C.c_int),
        "gaus_get_poly_grids": ([vp, vp], C.c_int),
        "gaus_poly_grid_census": ([vp, vp], C.c_int),
        "gaus_poly_tier_census": ([vp, vp], C.c_int),
        "gaus_last_error": ([vp], C.c_char_p),
        "gaus_status_string": ([C.c_int], C.c_char_p),
        "gaus_destroy": ([vp], None),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def _status_name(s: int) -> str:
    try:
        return load().gaus_status_string(int(s)).decode()
    except Exception:
        return str(s)


def default_hparams() -> HParams:
    hp = HParams()
    load().gaus_default_hparams(C.byref(hp))
    return hp


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def _dptr(t, dtype, shape, name):
    import torch
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name}: expected a device tensor")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")
    return C.c_void_p(t.data_ptr())


class Context:
    """One gaus_ctx: a validated problem on the current device for B restarts."""

    def __init__(self, problem, B: int, hparams: HParams | None = None, stream=None):
        import torch
        lib = load()
        self._arrays = [np.ascontiguousarray(problem.row_ptr, np.int32),
                        np.ascontiguousarray(problem.col_idx, np.int32),
                        np.ascontiguousarray(problem.delay, np.int32),
                        np.ascontiguousarray(problem.rtype, np.int32),
                        np.ascontiguousarray(problem.capacity, np.float32),
                        np.ascontiguousarray(problem.back_src, np.int32),
                        np.ascontiguousarray(problem.back_dst, np.int32),
                        np.ascontiguousarray(problem.back_dist, np.int32)]
        rp, col, dl, rt, cap, bs, bd, bk = self._arrays
        mem = getattr(problem, "mem_units", None)
        if mem is not None:
            mem = np.ascontiguousarray(mem, np.float32)
            self._arrays.append(mem)
        self._p = _Problem(int(problem.n_ops), int(rp[-1]), _np_ptr(rp), _np_ptr(col), _np_ptr(dl),
                           _np_ptr(rt), int(cap.shape[0]), _np_ptr(cap), int(problem.D), int(problem.II),
                           int(bs.shape[0]), _np_ptr(bs), _np_ptr(bd), _np_ptr(bk),
                           None if mem is None else _np_ptr(mem))
        self.hp = hparams if hparams is not None else default_hparams()
        self.B = int(B)
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        h = C.c_void_p()
        st = lib.gaus_init(C.byref(self._p), C.byref(self.hp), self.B, C.c_void_p(stream.cuda_stream),
                           C.byref(h))
        if st != OK:
            raise GausError(st, lib.gaus_last_error(None).decode())
        self._h = h
        dims = np.zeros(8, np.int32)
        self._check(lib.gaus_get_dims(self._h, _np_ptr(dims)))
        self.N, self.E, self.K, self.D, self.II, self.T, self.n_back, _ = (int(x) for x in dims)

    def _check(self, st):
        if st != OK:
            raise GausError(st, load().gaus_last_error(self._h).decode())

    def close(self):
        if getattr(self, "_h", None):
            load().gaus_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # --- entry points (same names as the C ABI, without the prefix) ---
    def bind_state(self, mu, sigma, adam_m, adam_v, lam, adam_t):
        import torch
        B, N = self.B, self.N
        f = torch.float32
        self._bound = (mu, sigma, adam_m, adam_v, lam, adam_t)
        self._check(load().gaus_bind_state(
            self._h, _dptr(mu, f, (B, N), "mu"), _dptr(sigma, f, (B, N), "sigma"),
            _dptr(adam_m, f, (2, B, N), "adam_m"), _dptr(adam_v, f, (2, B, N), "adam_v"),
            _dptr(lam, f, (B, 3), "lambda"), _dptr(adam_t, torch.int32, (1,), "adam_t")))

    def loss_grad(self, mu, sigma, lam, terms, grad_mu, grad_sigma):
        import torch
        B, N = self.B, self.N
        f = torch.float32
        self._check(load().gaus_loss_grad(
            self._h, _dptr(mu, f, (B, N), "mu"), _dptr(sigma, f, (B, N), "sigma"),
            _dptr(lam, f, (B, 3), "lambda"), _dptr(terms, f, (B, N_TERMS), "terms"),
            _dptr(grad_mu, f, (B, N), "grad_mu"), _dptr(grad_sigma, f, (B, N), "grad_sigma")))

    def step(self, n_iters: int, terms_last=None):
        import torch
        tp = None if terms_last is None else _dptr(terms_last, torch.float32, (self.B, N_TERMS), "terms_last")
        self._check(load().gaus_step(self._h, int(n_iters), tp))

    def adam_from_grad(self, g_mu, g_sigma, terms):
        import torch
        B, N = self.B, self.N
        f = torch.float32
        self._check(load().gaus_adam_from_grad(
            self._h, _dptr(g_mu, f, (B, N), "g_mu"), _dptr(g_sigma, f, (B, N), "g_sigma"),
            _dptr(terms, f, (B, N_TERMS), "terms")))

    def legalize(self, mu, sched):
        """Returns the per-restart status array (host)."""
        import torch
        status = np.zeros(self.B, np.int32)
        self._check(load().gaus_legalize(self._h, _dptr(mu, torch.float32, (self.B, self.N), "mu"),
                                         _dptr(sched, torch.int32, (self.B, self.N), "sched"),
                                         _np_ptr(status)))
        return status

    def schedule_cost(self, sched, cost):
        """Discrete cost of device schedules sched [B,N] int32 into cost [B,6] float64."""
        import torch
        self._check(load().gaus_schedule_cost(self._h, _dptr(sched, torch.int32, (self.B, self.N), "sched"),
                                              _dptr(cost, torch.float64, (self.B, N_COST), "cost")))

    def schedule_cost_noalloc(self, sched, cost):
        """gaus_schedule_cost with its scratch in the library's fixed device
        array (the call allocates nothing)."""
        import torch
        self._check(load().gaus_schedule_cost_noalloc(
            self._h, _dptr(sched, torch.int32, (self.B, self.N), "sched"),
            _dptr(cost, torch.float64, (self.B, N_COST), "cost")))

    def solve(self, best_sched, best_cost, max_iters: int, check_every: int, time_limit_s: float = 0.0,
              reinit_sigma: bool = False) -> dict:
        """Alg. 1 driver on the bound state; returns the stats as a dict."""
        import torch
        prm = SolveParams(int(max_iters), int(check_every), float(time_limit_s), 1 if reinit_sigma else 0)
        st = SolveStats()
        self._check(load().gaus_solve(self._h, C.byref(prm),
                                      _dptr(best_sched, torch.int32, (self.B, self.N), "best_sched"),
                                      _dptr(best_cost, torch.float64, (self.B, N_COST), "best_cost"),
                                      C.byref(st)))
        return {f: getattr(st, f) for f, _ in SolveStats._fields_}

    def solve_check(self, best_sched, best_cost, reinit_sigma: bool = False) -> np.ndarray:
        """One check of the Alg. 1 driver on the bound state; returns the
        per-restart re-initialization mode (0 kept, 1 candidate, 2 prior best)."""
        import torch
        mode = np.zeros(self.B, np.int32)
        self._check(load().gaus_solve_check(self._h, _dptr(best_sched, torch.int32, (self.B, self.N), "best_sched"),
                                            _dptr(best_cost, torch.float64, (self.B, N_COST), "best_cost"),
                                            1 if reinit_sigma else 0, _np_ptr(mode)))
        return mode

    def init_state(self, mu, sigma, u=None):
        import torch
        B, N = self.B, self.N
        uu = None
        if u is not None:
            uu = np.ascontiguousarray(np.broadcast_to(u, (B, N)), np.float64)
        self._check(load().gaus_init_state(self._h, None if uu is None else _np_ptr(uu),
                                           _dptr(mu, torch.float32, (B, N), "mu"),
                                           _dptr(sigma, torch.float32, (B, N), "sigma")))

    def asap_alap(self):
        a = np.zeros(self.N, np.int32)
        l = np.zeros(self.N, np.int32)
        self._check(load().gaus_asap_alap(self._h, _np_ptr(a), _np_ptr(l)))
        return a, l

    def get_usage(self, U):
        import torch
        self._check(load().gaus_get_usage(self._h, _dptr(U, torch.float32, (self.B, self.K, self.T), "U")))

    def get_storage(self, M):
        import torch
        self._check(load().gaus_get_storage(self._h, _dptr(M, torch.float32, (self.B, self.T), "M")))

    def kernel_timing(self, enable):
        """False/0: off; True/1: bracket the op and polynomial kernels of every
        iteration with HIP events; n > 1: of every n-th iteration."""
        self._check(load().gaus_kernel_timing(self._h, int(enable)))

    def kernel_timing_read(self):
        """{kernel: (total milliseconds, launches)} for the step-by-step op
        kernel ("ops") and the chunk-polynomial kernel ("poly")."""
        ms = (C.c_double * 2)()
        n = (C.c_int32 * 2)()
        self._check(load().gaus_kernel_timing_read(self._h, ms, n))
        return {"ops": (ms[0], n[0]), "poly": (ms[1], n[1])}

    def poly_config(self):
        cfg = np.zeros(4, np.int32)
        self._check(load().gaus_get_poly_config(self._h, _np_ptr(cfg)))
        return {"enabled": bool(cfg[0]), "W": int(cfg[1]), "chunks": int(cfg[2]), "L0": int(cfg[3])}

    def poly_census(self):
        """(restart, op) and (restart, edge) pairs evaluated by the chunk-
        polynomial kernel in the last iteration."""
        c = np.zeros(2, np.int64)
        self._check(load().gaus_poly_census(self._h, _np_ptr(c)))
        return {"ops": int(c[0]), "edges": int(c[1])}

    def poly_grids(self):
        """Chunk grids: [{on, P (restarts per wave), W, chunks, L0}] for grids 0, 1, 2."""
        cfg = np.zeros(15, np.int32)
        self._check(load().gaus_get_poly_grids(self._h, _np_ptr(cfg)))
        return [{"on": bool(cfg[5 * g]), "P": int(cfg[5 * g + 1]), "W": int(cfg[5 * g + 2]),
                 "chunks": int(cfg[5 * g + 3]), "L0": int(cfg[5 * g + 4])} for g in range(3)]

    def poly_grid_census(self):
        """(restart, op) pairs evaluated on each chunk grid in the last iteration."""
        c = np.zeros(3, np.int64)
        self._check(load().gaus_poly_grid_census(self._h, _np_ptr(c)))
        return [int(x) for x in c]

    def poly_tier_census(self):
        """[grid][tier][0: (restart, op) pairs, 1: their polynomial out-edges] of
        the last iteration (tier 1..3 = degree 8, 6, 5; tier 0 unused)."""
        c = np.zeros((3, 4, 2), np.int64)
        self._check(load().gaus_poly_tier_census(self._h, _np_ptr(c)))
        return c

    def sync(self):
        self._check(load().gaus_sync(self._h))


def init_error() -> str:
    return load().gaus_last_error(None).decode()
