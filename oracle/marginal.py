"""Law of one coordinate of a randomly rotated unit vector (oracle; test use only).

Section II-B, steps 2-3: once an L2-normalised vector has been rotated by the
random orthogonal matrix, each of its coordinates follows the marginal that
the paper names as Beta, approaching N(0, 1/d).  For a vector uniform on the
unit sphere of R^d that law is exact: X has density

    f_d(x) = C_d (1 - x^2)^((d-3)/2)  on [-1, 1],
    C_d    = Gamma(d/2) / (sqrt(pi) Gamma((d-1)/2)),

equivalently X^2 ~ Beta(1/2, (d-1)/2) with a symmetric sign, and it tends to
N(0, 1/d) as d grows.  The oracle uses this exact (sphere / Beta) reading.

Cell integrals used by Lloyd-Max are evaluated with library primitives --
scipy's complemented regularised incomplete beta function for the tail mass,
mpmath for C_d = 1 / B(1/2, (d-1)/2) -- and the closed form of the first
moment:
    int_a^b x f_d(x) dx = C_d [(1-a^2)^((d-1)/2) - (1-b^2)^((d-1)/2)] / (d-1).
The tail is taken as (1/2) * (1 - I_{x^2}(1/2, (d-1)/2)) through the
complemented function, whose argument x^2 carries one rounding only; the
equivalent form I_{1-x^2}((d-1)/2, 1/2) loses ~1e-11 relative precision near
x = 0 because 1 - x^2 is rounded.
"""
from __future__ import annotations

import numpy as np
import functools

import mpmath
from scipy.special import betainc, betaincc


@functools.lru_cache(maxsize=None)
def norm_const(d: int) -> float:
    """C_d = 1 / B(1/2, (d-1)/2), evaluated with 40 significant digits."""
    with mpmath.workdps(40):
        return float(1 / mpmath.beta(mpmath.mpf(1) / 2, mpmath.mpf(d - 1) / 2))


def log_norm_const(d: int) -> float:
    """log C_d of the sphere-coordinate density (section II-B, step 2)."""
    return float(np.log(norm_const(d)))


def density(x, d: int):
    """f_d(x): density of one coordinate of a uniform unit vector in R^d."""
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    inside = np.abs(x) < 1.0
    out[inside] = np.exp(log_norm_const(d)
                         + 0.5 * (d - 3) * np.log1p(-x[inside] ** 2))
    return out


def tail_prob(x, d: int):
    """P(X > x) for x >= 0:  (1/2) (1 - I_{x^2}(1/2, (d-1)/2))."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(x < 0):
        raise ValueError("tail_prob expects x >= 0")
    return 0.5 * betaincc(0.5, (d - 1) / 2.0, x * x)


def _central_prob(x, d: int):
    """P(|X| <= x) = I_{x^2}(1/2, (d-1)/2) for x >= 0 (small and exact near 0)."""
    return betainc(0.5, (d - 1) / 2.0, x * x)


def cell_mass(a, b, d: int):
    """P(a < X <= b).  For 0 <= a < b the two CDF values are differenced in the
    better-conditioned form: through the upper tails tail(a) - tail(b) when
    tail(a) < 1/4 (outer cells), else through the central probabilities
    (I_{b^2} - I_{a^2}) / 2 (inner cells, where those are the small numbers)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    aa, bb = np.broadcast_arrays(a, b)
    out = np.empty(aa.shape, dtype=np.float64)

    def pos_mass(lo, hi):
        ta = tail_prob(lo, d)
        outer = ta < 0.25
        res = np.empty(lo.shape, dtype=np.float64)
        res[outer] = ta[outer] - tail_prob(hi[outer], d)
        inner = ~outer
        res[inner] = 0.5 * (_central_prob(hi[inner], d) - _central_prob(lo[inner], d))
        return res

    pos = aa >= 0
    neg = bb <= 0
    mid = ~(pos | neg)
    if np.any(pos):
        out[pos] = pos_mass(aa[pos], bb[pos])
    if np.any(neg):
        out[neg] = pos_mass(-bb[neg], -aa[neg])
    if np.any(mid):
        out[mid] = 0.5 * (_central_prob(-aa[mid], d) + _central_prob(bb[mid], d))
    return out


def cell_first_moment(a, b, d: int):
    """int_a^b x f_d(x) dx in closed form (antiderivative of x(1-x^2)^((d-3)/2)):
    C_d [(1-a^2)^e - (1-b^2)^e] / (d-1), e = (d-1)/2.  For |a| <= |b| the
    difference is evaluated without cancellation as
        (1-b^2)^e * expm1(e * log1p((b-a)(b+a) / (1-b^2)))
    (and symmetrically), since (1-a^2)/(1-b^2) = 1 + (b-a)(b+a)/(1-b^2)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    a, b = np.broadcast_arrays(a, b)
    e = 0.5 * (d - 1)
    out = np.empty(a.shape, dtype=np.float64)
    swap = np.abs(a) > np.abs(b)          # always factor out the smaller power
    lo = np.where(swap, b, a)             # |lo| <= |hi|
    hi = np.where(swap, a, b)
    sign = np.where(swap, -1.0, 1.0)
    edge = np.abs(hi) >= 1.0
    with np.errstate(divide="ignore", invalid="ignore"):
        ghi = np.exp(e * np.log1p(-hi * hi))
        ratio = (hi - lo) * (hi + lo) / ((1.0 - hi) * (1.0 + hi))
        diff = ghi * np.expm1(e * np.log1p(ratio))
        glo = np.exp(e * np.log1p(-lo * lo))
    out = np.where(edge, glo, diff) * sign
    return norm_const(d) * out / (d - 1)


def cell_second_moment(a, b, d: int):
    """int_a^b x^2 f_d(x) dx.  X^2 weighted by its own law is Beta(3/2,(d-1)/2)
    scaled by E[X^2] = 1/d, so for 0 <= a < b the integral is
    (1/(2d)) [J(a) - J(b)] with J(x) = 1 - I_{x^2}(3/2, (d-1)/2)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)

    def upper(x):  # int_x^1 t^2 f(t) dt for x >= 0
        return 0.5 / d * betaincc(1.5, (d - 1) / 2.0, x * x)

    aa, bb = np.broadcast_arrays(a, b)
    out = np.empty(aa.shape, dtype=np.float64)
    pos = aa >= 0
    neg = bb <= 0
    mid = ~(pos | neg)
    out[pos] = upper(aa[pos]) - upper(bb[pos])
    out[neg] = upper(-bb[neg]) - upper(-aa[neg])
    out[mid] = (0.5 / d - upper(-aa[mid])) + (0.5 / d - upper(bb[mid]))
    return out


def mse_per_coord(bounds, cents, d: int) -> float:
    """E[(X - Q(X))^2] for the scalar quantiser with the given boundaries and
    reconstruction levels, X following f_d (section II-B, step 3)."""
    bounds = np.asarray(bounds, dtype=np.float64)
    cents = np.asarray(cents, dtype=np.float64)
    edges = np.concatenate(([-1.0], bounds, [1.0]))
    lo, hi = edges[:-1], edges[1:]
    m0 = cell_mass(lo, hi, d)
    m1 = cell_first_moment(lo, hi, d)
    m2 = cell_second_moment(lo, hi, d)
    return float(np.sum(m2 - 2.0 * cents * m1 + cents * cents * m0))
