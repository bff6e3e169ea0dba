"""C-ABI contract checks that need no GPU: the library loads, exports every
symbol include/gaus.h declares, carries the paper's default hyper-parameters,
and rejects invalid problems before touching the device."""
import ctypes as C
import json
import os
import re

import numpy as np
import pytest

from paper_2602_20427_amd import binding as bd
from paper_2602_20427_amd.workloads import Problem

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return bd.load()


def test_exports_every_declared_symbol(lib):
    with open(os.path.join(ROOT, "include", "gaus.h")) as f:
        hdr = f.read()
    declared = set(re.findall(r"\b(gaus_[a-z_]+)\s*\(", hdr))
    assert declared == set(bd.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_default_hparams_match_paper():
    """App. C.1 (lr, rho, kappa) and Sec. 3.3 (lambda0) values."""
    with open(os.path.join(ROOT, "tests", "golden", "hyperparameters.json")) as f:
        g = json.load(f)
    hp = bd.default_hparams()
    assert hp.lr == pytest.approx(g["lr"], rel=1e-7)
    assert hp.rho == pytest.approx(g["rho"], rel=1e-7)
    assert hp.kappa == pytest.approx(g["kappa"], rel=1e-7)
    assert hp.lambda0 == pytest.approx(g["lambda0"], rel=1e-7)
    assert (hp.beta1, hp.beta2) == (pytest.approx(0.9), pytest.approx(0.999))


def _init(lib, p, B=1, hp=None):
    arrs = [np.ascontiguousarray(x) for x in (p.row_ptr, p.col_idx, p.delay, p.rtype, p.capacity,
                                              p.back_src, p.back_dst, p.back_dist)]
    ptr = lambda a: a.ctypes.data_as(C.c_void_p)
    mem = None if p.mem_units is None else np.ascontiguousarray(p.mem_units, np.float32)
    prob = bd._Problem(p.n_ops, int(p.row_ptr[-1]) if len(p.row_ptr) else 0, ptr(arrs[0]), ptr(arrs[1]),
                       ptr(arrs[2]), ptr(arrs[3]), len(p.capacity), ptr(arrs[4]), p.D, p.II,
                       len(p.back_src), ptr(arrs[5]), ptr(arrs[6]), ptr(arrs[7]),
                       None if mem is None else ptr(mem))
    h = C.c_void_p(12345)
    st = lib.gaus_init(C.byref(prob), None if hp is None else C.byref(hp), B, None, C.byref(h))
    return st, h.value, lib.gaus_last_error(None).decode()


def _chain(**kw):
    d = dict(n_ops=3, row_ptr=np.array([0, 1, 2, 2], np.int32), col_idx=np.array([1, 2], np.int32),
             delay=np.ones(3, np.int32), rtype=np.zeros(3, np.int32), capacity=np.array([1.0], np.float32), D=10)
    d.update(kw)
    return Problem(**d)


@pytest.mark.parametrize("mutate,status,needle", [
    (dict(col_idx=np.array([1, 3], np.int32)), bd.E_INVALID_ARG, "col_idx"),
    (dict(row_ptr=np.array([0, 2, 1, 2], np.int32)), bd.E_INVALID_ARG, "row_ptr"),
    (dict(row_ptr=np.array([1, 1, 2, 2], np.int32)), bd.E_INVALID_ARG, "row_ptr"),
    (dict(rtype=np.array([0, 1, 0], np.int32)), bd.E_INVALID_ARG, "rtype"),
    (dict(delay=np.array([1, -1, 1], np.int32)), bd.E_INVALID_ARG, "delay"),
    (dict(capacity=np.array([np.nan], np.float32)), bd.E_INVALID_ARG, "capacity"),
    (dict(D=0), bd.E_INVALID_ARG, "D must"),
    (dict(row_ptr=np.array([0, 2, 3, 3], np.int32), col_idx=np.array([1, 1, 2], np.int32)),
     bd.E_INVALID_ARG, "duplicate edge"),
    (dict(mem_units=np.array([1.0, -1.0, 1.0], np.float32)), bd.E_INVALID_ARG, "mem_units"),
    (dict(mem_units=np.array([1.0, np.inf, 1.0], np.float32)), bd.E_INVALID_ARG, "mem_units"),
    (dict(D=2), bd.E_HORIZON, "horizon"),
    (dict(row_ptr=np.array([0, 1, 2, 3], np.int32), col_idx=np.array([1, 2, 0], np.int32)), bd.E_CYCLE, "cycle"),
    (dict(II=0, back_src=np.array([2], np.int32), back_dst=np.array([0], np.int32),
          back_dist=np.array([1], np.int32)), bd.E_INVALID_ARG, "II > 0"),
    (dict(II=4, back_src=np.array([2], np.int32), back_dst=np.array([2], np.int32),
          back_dist=np.array([1], np.int32)), bd.E_INVALID_ARG, "self loop"),
    (dict(II=4, back_src=np.array([2], np.int32), back_dst=np.array([0], np.int32),
          back_dist=np.array([0], np.int32)), bd.E_INVALID_ARG, "k*II"),
])
def test_init_rejects_invalid_problems(lib, mutate, status, needle):
    st, h, msg = _init(lib, _chain(**mutate))
    assert st == status, msg
    assert h is None, "out must be NULL on failure"
    assert needle in msg


@pytest.mark.parametrize("field,value,needle", [
    ("family", 4, "family"), ("family", -1, "family"),
    ("tau", 0.0, "tau"), ("tau", float("nan"), "tau"),
    ("beta_res", -1.0, "beta_res"), ("gamma_mem", float("inf"), "gamma_mem"),
    ("poly_chunk", 8, "poly_chunk"), ("poly_chunk", 512, "poly_chunk"),
])
def test_init_rejects_invalid_hparams(lib, field, value, needle):
    hp = bd.default_hparams()
    setattr(hp, field, value)
    st, h, msg = _init(lib, _chain(), hp=hp)
    assert st == bd.E_INVALID_ARG and h is None, msg
    assert needle in msg


def test_init_rejects_bad_restart_count(lib):
    st, h, msg = _init(lib, _chain(), B=0)
    assert st == bd.E_INVALID_ARG and h is None and "B must" in msg


def test_null_context_entry_points(lib):
    assert lib.gaus_loss_grad(None, None, None, None, None, None, None) == bd.E_INVALID_ARG
    assert lib.gaus_step(None, 1, None) == bd.E_INVALID_ARG
    assert lib.gaus_legalize(None, None, None, None) == bd.E_INVALID_ARG
    assert lib.gaus_sync(None) == bd.E_INVALID_ARG
    lib.gaus_destroy(None)
    assert lib.gaus_status_string(bd.E_HORIZON).decode() == "GAUS_E_HORIZON"
