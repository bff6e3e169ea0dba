"""Brute-force enumeration over every integer schedule of a tiny instance.

TEST INFRASTRUCTURE ONLY.  Independent of both the GPU library and the C
oracle: it evaluates the *discrete* definitions of the paper (dependency,
resource usage, edge length, recurrence; Sec. 2.1) on each of the D^N
schedules and weights them by the product of the independent per-op masses
(Sec. 3.1: the operators' start steps are independent).  The per-op mass
vector is supplied by the caller, so the enumeration checks the expectation
formulas without re-deriving the masses.
"""
from __future__ import annotations

import itertools
import numpy as np


def expectations(prob, P):
    """P: [N][D] per-op masses.  Returns a dict of exact expectations:
    V_dep, L_com, V_rec, U [K][T] (usage folded mod II when II > 0)."""
    N, D = P.shape
    src, dst = prob.edges()
    K = prob.n_types
    T = prob.II if prob.II > 0 else D
    vdep = lcom = vrec = 0.0
    U = np.zeros((K, T))
    for s in itertools.product(range(D), repeat=N):
        w = 1.0
        for i in range(N):
            w *= P[i, s[i]]
        if w == 0.0:
            continue
        for a, b in zip(src, dst):
            if s[b] < s[a] + prob.delay[a]:        # Dep violated (producer delay)
                vdep += w
            lcom += w * max(s[b] - s[a], 0)        # edge length, App. B.1
        for j, i, k in zip(prob.back_src, prob.back_dst, prob.back_dist):
            if s[j] + prob.delay[j] > s[i] + k * prob.II:   # Rec violated
                vrec += w
        for i in range(N):
            U[prob.rtype[i], s[i] % T] += w
    return {"V_dep": vdep, "L_com": lcom, "V_rec": vrec, "U": U}


def feasible(prob, s, lo=None, hi=None):
    """Is the integer schedule s feasible for Dep (and Rec when II > 0)?"""
    src, dst = prob.edges()
    for a, b in zip(src, dst):
        if s[b] < s[a] + prob.delay[a]:
            return False
    for j, i, k in zip(prob.back_src, prob.back_dst, prob.back_dist):
        if s[j] + prob.delay[j] > s[i] + k * prob.II:
            return False
    if lo is not None and np.any(np.asarray(s) < lo):
        return False
    if hi is not None and np.any(np.asarray(s) > hi):
        return False
    return True


def least_feasible_above(prob, s0, upper):
    """Componentwise least feasible schedule s >= s0 with s <= upper, found by
    enumerating every candidate in the box [s0, upper].  None if none exists."""
    s0 = np.asarray(s0, np.int64)
    upper = np.asarray(upper, np.int64)
    if np.any(s0 > upper):
        return None
    ranges = [range(int(a), int(b) + 1) for a, b in zip(s0, upper)]
    best = None
    for s in itertools.product(*ranges):
        if feasible(prob, s):
            s = np.asarray(s, np.int64)
            if best is None:
                best = s
            else:
                # the least element exists because feasible sets of difference
                # constraints are closed under componentwise min
                best = np.minimum(best, s)
    if best is not None and not feasible(prob, best):
        raise AssertionError("componentwise min of feasible schedules is infeasible")
    return best
