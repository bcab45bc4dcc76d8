"""Pins of the oracle's Lloyd-Max codebook (section II-B step 3) against facts
that do not come from the oracle's own code: a published table (Max 1960),
closed forms, an independent quadrature, Monte Carlo on the sphere and the
high-rate (Panter-Dite) asymptote."""
import math
import os

import mpmath
import numpy as np
import pytest
from scipy import integrate

import oracle
from oracle.marginal import cell_mass, density, mse_per_coord, tail_prob


def _max1960(golden_dir):
    rows = {}
    with open(os.path.join(golden_dir, "max1960_gaussian_lloyd_max.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            p = line.split()
            rows[(int(p[0]), p[1])] = np.array([float(v) for v in p[2:]])
    return rows


@pytest.mark.parametrize("d", [64, 300, 1536])
@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
def test_symmetric_monotone_converged(d, bits):
    cb = oracle.lloyd_max(d, bits)
    L = 1 << bits
    assert cb.converged
    assert cb.bounds.shape == (L - 1,) and cb.cents.shape == (L,)
    assert np.all(np.diff(cb.cents) > 0) and np.all(np.diff(cb.bounds) > 0)
    # antisymmetry, middle boundary exactly 0
    assert np.array_equal(cb.cents, -cb.cents[::-1])
    assert np.array_equal(cb.bounds, -cb.bounds[::-1])
    assert cb.bounds[L // 2 - 1] == 0.0
    # boundaries interleave the levels: c_i < t_i < c_{i+1}
    assert np.all(cb.cents[:-1] < cb.bounds) and np.all(cb.bounds < cb.cents[1:])


@pytest.mark.parametrize("d,bits", [(1536, 2), (1536, 4), (128, 3), (1536, 8), (128, 8)])
def test_stationarity_by_independent_quadrature(d, bits):
    """Every level is the conditional mean of its cell, with the cell integrals
    done by adaptive quadrature of the density (no incomplete beta, no closed
    form) -- and every boundary is the midpoint of its neighbours.  At b = 8
    Lloyd's iteration contracts at a rate close to 1, so a solve stopped
    short leaves residuals far above this bound."""
    cb = oracle.lloyd_max(d, bits)
    assert np.allclose(cb.bounds, 0.5 * (cb.cents[:-1] + cb.cents[1:]), rtol=0, atol=0)
    e = 0.5 * (d - 3)
    g = lambda x: math.exp(e * math.log1p(-x * x))        # unnormalised density
    edges = np.concatenate(([0.0], cb.bounds[cb.bounds >= 0][1:], [1.0]))
    sigma = 1 / math.sqrt(d)
    pos = cb.cents[cb.cents > 0]
    for i, c in enumerate(pos):
        a, b = edges[i], edges[i + 1]
        b_eff = min(b, a + 40 * sigma)          # density is ~0 beyond 40 sigma
        num = integrate.quad(lambda x: x * g(x), a, b_eff, epsabs=0, epsrel=1e-13, limit=200)[0]
        den = integrate.quad(g, a, b_eff, epsabs=0, epsrel=1e-13, limit=200)[0]
        assert abs(num / den - c) <= 1e-12 * c, (i, num / den, c)


def _quadrature_mse(d, cb):
    """E[(X - Q(X))^2] by adaptive quadrature of (x - c)^2 times the
    unnormalised density over every cell, divided by the quadrature of the
    density itself (no incomplete beta, no closed-form moment)."""
    e = 0.5 * (d - 3)
    g = lambda x: math.exp(e * math.log1p(-x * x))
    sigma = 1 / math.sqrt(d)
    top = min(1.0, 40 * sigma)
    Z = 2 * integrate.quad(g, 0, top, epsabs=0, epsrel=1e-13, limit=400)[0]
    edges = np.concatenate(([0.0], cb.bounds[cb.bounds >= 0][1:], [1.0]))
    tot = 0.0
    for i, c in enumerate(cb.cents[cb.cents > 0]):
        a, b = edges[i], min(edges[i + 1], edges[i] + 40 * sigma)
        tot += integrate.quad(lambda x: (x - c) ** 2 * g(x), a, b, epsabs=0, epsrel=1e-13,
                              limit=200)[0]
    return 2 * tot / Z


@pytest.mark.parametrize("bits,dmse", [(1, 0.363173), (2, 0.117358), (3, 0.034499),
                                       (4, 0.0094854)])
def test_dmse_table_at_1536_by_quadrature(bits, dmse):
    """d * MSE at d = 1536 for b = 1..4 (0.363173, 0.117358, 0.034499,
    0.0094854): the oracle's value equals an independent quadrature of the
    squared error to 1e-12 relative, and both round to the tabulated digits."""
    d = 1536
    cb = oracle.lloyd_max(d, bits)
    q = d * _quadrature_mse(d, cb)
    assert abs(d * cb.mse() - q) <= 1e-12 * q
    digits = len(repr(dmse).split(".")[1])
    assert round(q, digits) == dmse, (q, dmse)


def test_dmse_8bit_by_quadrature():
    """b = 8: the quadrature of the squared error over all 256 cells agrees
    with the oracle's moment-based distortion (the Panter-Dite test below
    only brackets it within 3%)."""
    for d in (128, 1536):
        cb = oracle.lloyd_max(d, 8)
        q = _quadrature_mse(d, cb)
        assert abs(cb.mse() - q) <= 1e-10 * q


def test_one_bit_closed_form():
    """b=1: levels +-E|X| with E|X| = Gamma(d/2) / (sqrt(pi) Gamma((d+1)/2)), and
    d*MSE = 1 - d (E|X|)^2 (= 0.363173 at d=1536)."""
    for d in (16, 64, 1536, 4096):
        cb = oracle.lloyd_max(d, 1)
        with mpmath.workdps(40):
            ea = float(mpmath.gamma(mpmath.mpf(d) / 2)
                       / (mpmath.sqrt(mpmath.pi) * mpmath.gamma(mpmath.mpf(d + 1) / 2)))
        assert abs(cb.cents[1] - ea) <= 1e-15 * ea
        assert abs(d * cb.mse() - (1 - d * ea * ea)) < 1e-12
    assert abs(1536 * oracle.lloyd_max(1536, 1).mse() - 0.363173) < 5e-7


def test_gaussian_limit_matches_max1960(golden_dir):
    """sqrt(d) * tables tend to Max's Gaussian Lloyd-Max tables as d grows."""
    ref = _max1960(golden_dir)
    d = 1_000_000
    for bits in (1, 2, 3, 4):
        L = 1 << bits
        cb = oracle.lloyd_max(d, bits)
        s = math.sqrt(d)
        lev = s * cb.cents[L // 2:]
        bnd = s * cb.bounds[L // 2 - 1:]
        # table values carry 4 significant digits
        np.testing.assert_allclose(lev, ref[(L, "level")], rtol=6e-4, atol=6e-5)
        np.testing.assert_allclose(bnd, ref[(L, "bound")], rtol=6e-4, atol=6e-5)
        assert abs(d * cb.mse() - ref[(L, "mse")][0]) <= 6e-4 * ref[(L, "mse")][0]


def test_dmse_approaches_gaussian_from_below(golden_dir):
    """At finite d the sphere marginal has lighter tails than N(0,1/d): d*MSE is
    below the Gaussian value and the gap shrinks as d grows."""
    ref = _max1960(golden_dir)
    for bits in (1, 2, 3, 4):
        g = ref[(1 << bits, "mse")][0]
        gaps = [g - d * oracle.lloyd_max(d, bits).mse() for d in (256, 1536, 16384)]
        assert gaps[0] > gaps[1] > gaps[2] > -1e-4
        assert abs(gaps[1]) < 2e-3 * g + 1e-4


def test_monte_carlo_distortion_on_the_sphere():
    """Quantise coordinates of uniform unit vectors (normalised Gaussians) with
    numpy's searchsorted and compare the empirical MSE with the quadrature MSE."""
    d, bits = 1536, 4
    cb = oracle.lloyd_max(d, bits)
    rng = np.random.default_rng(7)
    per_vec = []
    for _ in range(8):
        g = rng.standard_normal((500, d))
        x = g / np.linalg.norm(g, axis=1, keepdims=True)
        q = cb.cents[np.searchsorted(cb.bounds, x, side="right")]
        per_vec.append(np.sum((x - q) ** 2, axis=1))
    per_vec = np.concatenate(per_vec)
    se = per_vec.std(ddof=1) / math.sqrt(per_vec.size)
    assert abs(per_vec.mean() - d * cb.mse()) < 5 * se


def test_high_rate_panter_dite_8bit():
    """b=8 is in the high-rate regime: d*MSE ~ (sqrt(3) pi / 2) 4^-8."""
    cb = oracle.lloyd_max(1536, 8)
    assert cb.converged
    pd = math.sqrt(3) * math.pi / 2 * 4.0 ** -8
    dm = 1536 * cb.mse()
    assert 0.97 * pd < dm < 1.0 * pd
    assert np.array_equal(cb.cents, -cb.cents[::-1]) and cb.bounds[127] == 0.0


def test_marginal_is_a_probability_law():
    """The density integrates to 1, the tail matches quadrature, E[X^2] = 1/d."""
    for d in (64, 1536):
        tot = 2 * integrate.quad(lambda x: density(np.array([x]), d)[0], 0, 1,
                                 epsabs=0, epsrel=1e-13, limit=400, points=[3 / math.sqrt(d)])[0]
        assert abs(tot - 1) < 1e-11
        for x in (0.3 / math.sqrt(d), 1 / math.sqrt(d), 2.5 / math.sqrt(d)):
            q = integrate.quad(lambda t: density(np.array([t]), d)[0], x, 1,
                               epsabs=0, epsrel=1e-13, limit=400)[0]
            assert abs(tail_prob(x, d) - q) < 1e-12 * q
        # mse of the trivial quantiser (single level 0) is E[X^2] = 1/d
        assert abs(mse_per_coord([], [0.0], d) - 1 / d) < 1e-15
        assert abs(cell_mass(-1.0, 1.0, d) - 1) < 1e-15


def test_codebook_is_data_independent():
    """Section VI-A: the codebook depends on (d, b) only -- the API takes no data
    and repeated calls return identical tables."""
    a, b = oracle.lloyd_max(1536, 4), oracle.lloyd_max.__wrapped__(1536, 4)
    assert np.array_equal(a.cents, b.cents) and np.array_equal(a.bounds, b.bounds)
