"""Analytic Lloyd-Max codebook (oracle; test use only).

Section II-B, step 3: the scalar quantiser's boundaries and reconstruction
levels are precomputed from the known post-rotation coordinate law, with no
data-dependent training (the codebook is a function of (d, b) alone; section
VI-A notes it is identical across corpora).

A Lloyd-Max quantiser with L = 2^b levels satisfies two conditions:
  (i)  every boundary is the midpoint of the two levels beside it;
  (ii) every level is the conditional mean of X over its cell.
Writing F for one Lloyd step (apply (i), then (ii)), the levels are a fixed
point p = F(p).  The oracle finds it in three plain phases:
  1. Lloyd's iteration p <- F(p), 300 steps from Gaussian quantiles
     Phi^-1((i + 1/2)/L) / sqrt(d) (it converges monotonically but slowly:
     its rate tends to 1 as L grows);
  2. Newton's method on G(p) = F(p) - p with a forward-difference Jacobian,
     until max|G| is at the rounding level (4 ulp of the largest level) or
     stops shrinking; the iterate with the smallest max|G| is returned.
The law is symmetric, so the positive half is solved and mirrored; this
makes the middle boundary exactly 0 and the tables exactly antisymmetric.
"""
from __future__ import annotations

import functools
from dataclasses import dataclass

import numpy as np
from scipy.stats import norm

from .marginal import cell_first_moment, cell_mass, mse_per_coord


@dataclass(frozen=True)
class Codebook:
    d: int
    bits: int
    bounds: np.ndarray      # float64 [L-1], strictly increasing, bounds[L/2-1] == 0
    cents: np.ndarray       # float64 [L],   strictly increasing
    iterations: int
    converged: bool

    @property
    def levels(self) -> int:
        return 1 << self.bits

    def mse(self) -> float:
        """Per-coordinate distortion E[(X - Q(X))^2]."""
        return mse_per_coord(self.bounds, self.cents, self.d)


@functools.lru_cache(maxsize=None)
def lloyd_max(d: int, bits: int) -> Codebook:
    """Lloyd-Max boundaries and centroids for the d-dimensional sphere marginal."""
    if d < 3:
        raise ValueError("d must be >= 3")
    if bits < 1 or bits > 8:
        raise ValueError("bits must be in 1..8")
    L = 1 << bits
    h = L // 2
    # positive-half levels p_0 < ... < p_{h-1}
    p = norm.ppf((np.arange(h) + h + 0.5) / L) / np.sqrt(d)

    def lloyd_step(p):
        # condition (i): cell edges of the positive half, 0 and 1 at the ends
        edges = np.concatenate(([0.0], 0.5 * (p[:-1] + p[1:]), [1.0]))
        # condition (ii): level = E[X | X in cell]
        return cell_first_moment(edges[:-1], edges[1:], d) / cell_mass(edges[:-1], edges[1:], d)

    it = 0
    # phase 1: plain Lloyd iteration
    for _ in range(300):
        p = lloyd_step(p)
        it += 1
    # phase 2: Newton on G(p) = F(p) - p
    tiny = 4 * np.finfo(np.float64).eps * np.max(p)
    best_p, best_r = p, np.inf
    converged = False
    for _ in range(40):
        g = lloyd_step(p) - p
        it += 1
        r = float(np.max(np.abs(g)))
        if r < best_r:
            best_p, best_r = p, r
        if r <= tiny:
            converged = True
            break
        if r > 0.5 * best_r and best_r < 1e-13 * np.max(p):
            converged = True        # at the rounding floor: no further progress
            break
        J = np.empty((h, h))
        for j in range(h):
            step = 1e-8 * p[j]
            q = p.copy()
            q[j] += step
            J[:, j] = ((lloyd_step(q) - q) - g) / step
        p = p - np.linalg.solve(J, g)
        if np.any(np.diff(p) <= 0) or p[0] <= 0 or p[-1] >= 1:
            raise RuntimeError("Newton step left the feasible region")
    p = best_p
    inner = 0.5 * (p[:-1] + p[1:])
    cents = np.concatenate((-p[::-1], p))
    bounds = np.concatenate((-inner[::-1], [0.0], inner))
    cents.setflags(write=False)
    bounds.setflags(write=False)
    return Codebook(d=d, bits=bits, bounds=bounds, cents=cents,
                    iterations=it, converged=converged)
