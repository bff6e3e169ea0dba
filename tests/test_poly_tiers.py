"""Host-side rule of the chunk-polynomial path: the Taylor recursions of each
family's CDF (Gaussian: Hermite; logistic: S' = S(1 - S); Cauchy: geometric
series of 1/(u - i)) against the exact functions, and each family's
truncation bound against the measured truncation error at the tier bounds
the library uses (degree 8, 6, 5).  fp64, CPU only."""
import math

import numpy as np
import pytest
from scipy.special import expit, ndtr

from tests.gpu_common import POLY_DEGREES, poly_bound, poly_rho

C = {"gaussian": 1.0, "logistic": math.sqrt(3.0) / math.pi, "cauchy": math.sqrt(2.0 * math.log(2.0))}


def cdf(family, u):
    if family == "gaussian":
        return ndtr(u)
    if family == "logistic":
        return expit(u)
    return 0.5 + np.arctan(u) / math.pi


def density(family, u):
    if family == "gaussian":
        return np.exp(-u * u / 2) / math.sqrt(2 * math.pi)
    if family == "logistic":
        e = np.exp(-np.abs(u))
        return e / (1 + e) ** 2
    return 1.0 / (math.pi * (1 + u * u))


def cdf_taylor(family, u0, n):
    """Coefficients s_0..s_n of F(u0 + h) in h (u units)."""
    s = np.zeros(n + 1)
    s[0] = cdf(family, u0)
    if family == "gaussian":
        he = [1.0, u0]   # probabilists' Hermite polynomials
        for k in range(1, n):
            he.append(u0 * he[k] - k * he[k - 1])
        phi = math.exp(-u0 * u0 / 2) / math.sqrt(2 * math.pi)
        for m in range(1, n + 1):   # F^(m) = (-1)^(m-1) He_(m-1) phi
            s[m] = (-1) ** (m - 1) * he[m - 1] * phi / math.factorial(m)
    elif family == "logistic":
        t0 = 1.0 - s[0]
        s[1] = s[0] * t0
        for m in range(1, n):
            acc = s[m] * (t0 - s[0]) - sum(s[k] * s[m - k] for k in range(1, m))
            s[m + 1] = acc / (m + 1)
    else:
        w = -1.0 / complex(u0, -1.0)
        p = 1.0 + 0j
        for m in range(1, n + 1):
            p *= w
            s[m] = -p.imag / (math.pi * m)
    return s


@pytest.mark.parametrize("family", ["gaussian", "logistic", "cauchy"])
def test_taylor_recursions_match_the_cdf(family):
    """A degree-12 expansion reproduces the CDF to 1e-13 near its centre."""
    for u0 in (-7.0, -2.3, -0.4, 0.0, 0.9, 3.1, 9.0):
        s = cdf_taylor(family, u0, 12)
        h = np.linspace(-0.05, 0.05, 21)
        approx = np.polyval(s[::-1], h)
        assert np.abs(approx - cdf(family, u0 + h)).max() < 1e-13, (family, u0)


def truncation_error(family, d, rho):
    """Largest error of the density series truncated after degree d-1 over a
    chunk of half-width rho (sigma units), relative to the peak density."""
    ru = rho / C[family]
    h = np.linspace(-ru, ru, 201)
    worst = 0.0
    for u0 in np.linspace(0.0, 14.0, 281):
        s = cdf_taylor(family, u0, d + 1)
        f = np.array([(k + 1) * s[k + 1] for k in range(d)])
        err = np.abs(np.polyval(f[::-1], h) - density(family, u0 + h)).max()
        worst = max(worst, err)
    return worst / density(family, 0.0)


@pytest.mark.parametrize("family", ["gaussian", "logistic", "cauchy"])
@pytest.mark.parametrize("d", POLY_DEGREES)
def test_tier_bound_holds_at_its_threshold(family, d):
    """At each tier's rho bound the measured truncation error stays below the
    common target (the Gaussian degree-8 bound at rho = 1/4, 8.3e-8) and
    within a factor 4 of it (the bounds are not loose)."""
    target = poly_bound("gaussian", 8, 0.25)
    rho = poly_rho(family, d)
    err = truncation_error(family, d, rho)
    assert err <= target, (family, d, rho, err, target)
    assert err >= target / 4, (family, d, rho, err, target)
