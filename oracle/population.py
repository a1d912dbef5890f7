"""Population distortion of scalar codebooks (Sec. 3), float64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).  These functions are
not on the GPU path; they pin the oracle's level function to numbers and
closed forms the paper prints.

Covers
  * the affine basis r_i, u_i, v_i and levels y_i = s (r_i + a u_i + b v_i)
    (eq. cubic-basis, eq. affine-cubic-level) and the midpoint boundaries
    (eq. affine-cubic-boundary);
  * the cell-moment form of the distortion (eq. cell-moment-risk,
    eq. explicit-cubic-risk) with the closed-form half-line moments of the
    unit-variance Uniform, Gaussian and Laplace laws (eq. reference-cell-moments);
  * D_INT = min_s D(s, 1, 0), D_C = min over s and admissible (a, b), the
    Lloyd-Max fixed point (eq. lloyd-max) and the finite floating-point
    reference (eq. finite-fp-levels .. eq. fp-reference);
  * the Monte Carlo estimate used in Sec. 3.4 to check the analytic values.
"""
from __future__ import annotations

import math

import numpy as np
from scipy import optimize, special

from .format import max_code, shape_margin

SQRT3 = math.sqrt(3.0)
BETA = 1.0 / math.sqrt(2.0)


# ---------------------------------------------------------------- half-line cell moments


def moments(dist: str, lo, hi):
    """(mu0, mu1, mu2) of x^r f(x) over [lo, hi] on the positive half-line.

    hi may be +inf (the last cell); the upper-endpoint terms then vanish.
    """
    lo = np.asarray(lo, dtype=np.float64)
    hi = np.asarray(hi, dtype=np.float64)
    if dist == "uniform":
        a = SQRT3
        l = np.clip(lo, 0.0, a)
        u = np.clip(hi, 0.0, a)
        return tuple((u ** (r + 1) - l ** (r + 1)) / (2.0 * a * (r + 1)) for r in range(3))
    if dist == "gaussian":
        finite = np.isfinite(hi)
        hu = np.where(finite, hi, 0.0)
        phi_l = np.exp(-0.5 * lo * lo) / math.sqrt(2.0 * math.pi)
        phi_u = np.where(finite, np.exp(-0.5 * hu * hu) / math.sqrt(2.0 * math.pi), 0.0)
        cdf_u = np.where(finite, special.ndtr(hu), 1.0)
        mu0 = cdf_u - special.ndtr(lo)
        mu1 = phi_l - phi_u
        mu2 = mu0 + lo * phi_l - np.where(finite, hu * phi_u, 0.0)
        return mu0, mu1, mu2
    if dist == "laplace":
        finite = np.isfinite(hi)
        hu = np.where(finite, hi, 0.0)
        el = np.exp(-lo / BETA)
        eu = np.where(finite, np.exp(-hu / BETA), 0.0)
        mu0 = 0.5 * (el - eu)
        mu1 = 0.5 * ((lo + BETA) * el - np.where(finite, (hu + BETA) * eu, 0.0))
        mu2 = 0.5 * ((lo * lo + 2 * BETA * lo + 2 * BETA * BETA) * el
                     - np.where(finite, (hu * hu + 2 * BETA * hu + 2 * BETA * BETA) * eu, 0.0))
        return mu0, mu1, mu2
    raise ValueError(dist)


def distortion_levels(dist: str, y) -> float:
    """D for a symmetric codebook {0, +-y_1, ..., +-y_M} (y_0 = 0, increasing).

    D = 2 sum_i [mu2 - 2 y_i mu1 + y_i^2 mu0] over (h_{i-1}, h_i) with
    h_{-1} = 0, h_i = (y_i + y_{i+1}) / 2 and h_M = inf (eq. cell-moment-risk).
    """
    y = np.asarray(y, dtype=np.float64)
    h = np.concatenate([[0.0], 0.5 * (y[:-1] + y[1:]), [np.inf]])
    mu0, mu1, mu2 = moments(dist, h[:-1], h[1:])
    return float(2.0 * np.sum(mu2 - 2.0 * y * mu1 + y * y * mu0))


# ---------------------------------------------------------------- Cubic family (Sec. 3.1)


def basis(bits: int):
    """r_i = t^3, u_i = t - t^3, v_i = t^2 - t^3 at t_i = i/M (eq. cubic-basis)."""
    m = max_code(bits)
    t = np.arange(m + 1, dtype=np.float64) / m
    return t ** 3, t - t ** 3, t * t - t ** 3


def cubic_levels(bits: int, s: float, a: float, b: float) -> np.ndarray:
    """y_i = s (r_i + a u_i + b v_i) (eq. affine-cubic-level)."""
    r, u, v = basis(bits)
    return s * (r + a * u + b * v)


def cubic_distortion(dist: str, bits: int, s: float, a: float, b: float) -> float:
    """D_B(s, a, b) (eq. explicit-cubic-risk)."""
    return distortion_levels(dist, cubic_levels(bits, s, a, b))


def best_scale(fun, lo=1e-3, hi=40.0, grid=400) -> tuple[float, float]:
    """Minimise a 1-D function of the scale: grid bracket then bounded refine."""
    ss = np.geomspace(lo, hi, grid)
    vals = np.array([fun(s) for s in ss])
    i = int(np.argmin(vals))
    a = ss[max(i - 1, 0)]
    b = ss[min(i + 1, grid - 1)]
    res = optimize.minimize_scalar(fun, bounds=(a, b), method="bounded",
                                   options={"xatol": 1e-12, "maxiter": 500})
    if res.fun <= vals[i]:
        return float(res.x), float(res.fun)
    return float(ss[i]), float(vals[i])


def d_int(dist: str, bits: int) -> tuple[float, float]:
    """D_INT(B) = min_s D(s, 1, 0); returns (s*, D)."""
    return best_scale(lambda s: cubic_distortion(dist, bits, s, 1.0, 0.0))


def d_cubic_at(dist: str, bits: int, a: float, b: float) -> tuple[float, float]:
    """min_s D(s, a, b) at a fixed shape; returns (s*, D)."""
    return best_scale(lambda s: cubic_distortion(dist, bits, s, a, b))


def d_cubic(dist: str, bits: int, start=(1.0, 0.0)) -> tuple[float, float, float, float]:
    """D_C(B) = min over s > 0 and (a, b) with m(a, b) >= 0; returns (s, a, b, D).

    Nelder-Mead over (a, b) with the scale optimised inside; infeasible shapes
    are rejected with an infinite objective.
    """
    def obj(p):
        a, b = p
        if shape_margin(a, b) < 0:
            return np.inf
        return d_cubic_at(dist, bits, a, b)[1]

    res = optimize.minimize(obj, np.asarray(start, dtype=np.float64), method="Nelder-Mead",
                            options={"xatol": 1e-7, "fatol": 1e-14, "maxiter": 4000})
    a, b = res.x
    s, d = d_cubic_at(dist, bits, a, b)
    return s, float(a), float(b), d


# ---------------------------------------------------------------- Lloyd-Max (Sec. 3.2)


def lloyd_max(dist: str, bits: int, iters: int = 20000, tol: float = 1e-15) -> tuple[np.ndarray, float]:
    """Free symmetric codebook with an exact zero: alternate the midpoint and
    centroid conditions (eq. lloyd-max).  Returns (levels y_0..y_M, D_LM)."""
    m = max_code(bits)
    # start from the high-resolution companding point density f^(1/3), which
    # only speeds up convergence; the fixed point is the same
    p = (m + np.arange(m + 1) + 0.5) / (2 * m + 1)
    if dist == "uniform":
        y = SQRT3 * (2 * p - 1)
    elif dist == "gaussian":
        y = math.sqrt(3.0) * special.ndtri(p)
    else:
        y = -3.0 * BETA * np.log(2.0 * (1.0 - p))
    y[0] = 0.0
    for _ in range(iters):
        h = np.concatenate([[0.0], 0.5 * (y[:-1] + y[1:]), [np.inf]])
        mu0, mu1, _ = moments(dist, h[:-1], h[1:])
        ynew = y.copy()
        filled = mu0[1:] > 0
        ynew[1:] = np.where(filled, mu1[1:] / np.where(filled, mu0[1:], 1.0), y[1:])
        if np.max(np.abs(ynew - y)) < tol:
            y = ynew
            break
        y = ynew
    return y, distortion_levels(dist, y)


def gap_closed(d_int_v: float, d_c: float, d_lm: float) -> float:
    """eta_B = (D_INT - D_C) / (D_INT - D_LM) (eq. gap-closed)."""
    return (d_int_v - d_c) / (d_int_v - d_lm)


def w3_shape_from_levels(y1: float, y2: float, y3: float) -> tuple[float, float]:
    """Recover (a, b) of a W3 codebook 0 < y1 < y2 < y3 (eq. w3-shape-solution).

    Solves 27 p1 = 1 + 8a + 2b, 27 p2 = 8 + 10a + 4b with p = y / y3.
    """
    p1, p2 = y1 / y3, y2 / y3
    mat = np.array([[8.0, 2.0], [10.0, 4.0]])
    rhs = np.array([27.0 * p1 - 1.0, 27.0 * p2 - 8.0])
    a, b = np.linalg.solve(mat, rhs)
    return float(a), float(b)


# ---------------------------------------------------------------- finite FP (Sec. 3.2)


def fp_levels(e: int, m: int) -> np.ndarray:
    """Normalised non-negative levels of an all-finite EeMm format.

    E = 0: J 2^-m 2^(1-gamma); E > 0: (1 + J 2^-m) 2^(E-gamma), with
    gamma = 2^(e-1) - 1 (eq. finite-fp-levels); sorted, divided by the max.
    """
    gamma = 2 ** (e - 1) - 1
    vals = set()
    for E in range(2 ** e):
        for J in range(2 ** m):
            if E == 0:
                v = J * 2.0 ** (-m) * 2.0 ** (1 - gamma)
            else:
                v = (1.0 + J * 2.0 ** (-m)) * 2.0 ** (E - gamma)
            vals.add(v)
    z = np.array(sorted(vals))
    return z / z[-1]


def d_fp(dist: str, bits: int) -> tuple[str, float, float]:
    """D_FP(B) = min over splits e + m = B - 1 of min_s D_{e,m}(s) (eq. fp-reference).

    Returns (split name, s*, D).
    """
    best = ("", 0.0, np.inf)
    for e in range(1, bits):
        m = bits - 1 - e
        z = fp_levels(e, m)
        s, d = best_scale(lambda s: distortion_levels(dist, s * z))
        if d < best[2]:
            best = (f"E{e}M{m}", s, d)
    return best


# ---------------------------------------------------------------- Monte Carlo (Sec. 3.4)


def sample(dist: str, n: int, rng: np.random.Generator) -> np.ndarray:
    """Zero-mean unit-variance samples of the reference laws."""
    if dist == "uniform":
        return rng.uniform(-SQRT3, SQRT3, n)
    if dist == "gaussian":
        return rng.standard_normal(n)
    if dist == "laplace":
        return rng.laplace(0.0, BETA, n)
    raise ValueError(dist)


def mc_distortion(dist: str, y, n: int, rng: np.random.Generator) -> tuple[float, float]:
    """Monte Carlo estimate of D for the symmetric codebook with non-negative
    levels y (nearest level), and its standard error."""
    y = np.asarray(y, dtype=np.float64)
    x = sample(dist, n, rng)
    ax = np.abs(x)
    mids = 0.5 * (y[:-1] + y[1:])
    idx = np.searchsorted(mids, ax, side="left")
    err = (ax - y[idx]) ** 2
    return float(err.mean()), float(err.std(ddof=1) / math.sqrt(n))
