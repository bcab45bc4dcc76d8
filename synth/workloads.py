"""Synthetic stand-ins for the paper's embedding workloads.

The paper measures on pre-computed d=1536 L2-normalised text embeddings
(section IV-A: 100K / 500K / 999K corpus sizes, 1,000 held-out queries).
Those vectors are not available here; these seeded generators produce inputs
of the same dimension, normalisation, scale and clustered structure.  No item
of any public dataset is reproduced.

Recipes (numpy Generator over SFC64 keyed by SeedSequence; every chunk of CHUNK rows has its own seed so any
row range can be regenerated alone and chunks are generated in parallel):

* small      -- N=10,000, d=1536.  100 centres mu_k ~ N(0, I_d); row =
                mu_z + 0.3 eps (z uniform, eps ~ N(0, I_d)), L2-normalised.
                64 queries: distinct corpus rows + N(0, 0.05^2) per coordinate,
                renormalised.  Corpus seed 42, query seed 43.
* powerlaw   -- d=1536.  1,000 centres; axis-aligned covariance diag(lambda),
                lambda_i proportional to i^-0.8 scaled to mean 1;
                mu_k = lambda^(1/2) g_k, row = mu_z + 0.3 lambda^(1/2) eps,
                L2-normalised.  One stream of rows (seed 42):
                  100K corpus: rows [0, 100000), queries rows [100000, 101000)
                  999K corpus: rows [0, 999000), queries rows [999000, 1000000)
                  1M corpus:   999K corpus + rows [1000000, 1001000), same queries
* shifted    -- the small recipe plus one offset shared by every row:
                row = shift g + mu_z + 0.3 eps, g ~ N(0, I_d), L2-normalised
                (rows then lie in a cone around g, as text embeddings with a
                common component do; the rotated coordinates have non-zero
                means).  Corpus seed 46, queries as for 'small' (seed 47).
* tenants    -- Zipf(s=1.1) over T tenants, i.i.d. per vector by inverse CDF
                (random positions), seed 44.  Equal uniform partitions are also
                available (T equal-size contiguous-id groups, shuffled).
* allowlists -- per query, either one tenant drawn uniformly ("selective") or
                ceil(T/10) distinct tenants ("broad"), seed 45; encoded as a
                bitmap of ceil(T/64) 64-bit words, tenant t = bit (t & 63) of
                word (t >> 6).
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNK = 65536
_TAG_CENTRES = 0
_TAG_ROWS = 1


def _rng(*key) -> np.random.Generator:
    """SFC64 stream keyed by integers (about 3x faster than PCG64 for normals)."""
    return np.random.Generator(np.random.SFC64(np.random.SeedSequence(list(key))))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _normalise_rows_into(out: np.ndarray, rows32: np.ndarray) -> None:
    """out[i] = rows32[i] / ||rows32[i]|| (norm in float64, result float32)."""
    sub = 8192
    for s in range(0, rows32.shape[0], sub):
        r = rows32[s:s + sub].astype(np.float64)
        nrm = np.sqrt(np.einsum("ij,ij->i", r, r))
        nrm[nrm == 0] = 1.0
        out[s:s + sub] = (r / nrm[:, None]).astype(np.float32)


# ---------------------------------------------------------------- small case
def isotropic_mixture(n: int = 10_000, d: int = 1536, n_clusters: int = 100,
                      sigma: float = 0.3, seed: int = 42) -> np.ndarray:
    rng = _rng(seed, _TAG_CENTRES)
    centres = rng.standard_normal((n_clusters, d), dtype=np.float32)
    out = np.empty((n, d), dtype=np.float32)
    for c0 in range(0, n, CHUNK):
        c1 = min(n, c0 + CHUNK)
        r = _rng(seed, _TAG_ROWS, c0 // CHUNK)
        z = r.integers(0, n_clusters, size=c1 - c0)
        eps = r.standard_normal((c1 - c0, d), dtype=np.float32)
        _normalise_rows_into(out[c0:c1], centres[z] + np.float32(sigma) * eps)
    return out


def shifted_mixture(n: int = 10_000, d: int = 1536, shift: float = 1.5, n_clusters: int = 100,
                    sigma: float = 0.3, seed: int = 46) -> np.ndarray:
    rng = _rng(seed, _TAG_CENTRES)
    centres = rng.standard_normal((n_clusters, d), dtype=np.float32)
    g = rng.standard_normal(d, dtype=np.float32) * np.float32(shift)
    out = np.empty((n, d), dtype=np.float32)
    for c0 in range(0, n, CHUNK):
        c1 = min(n, c0 + CHUNK)
        r = _rng(seed, _TAG_ROWS, c0 // CHUNK)
        z = r.integers(0, n_clusters, size=c1 - c0)
        eps = r.standard_normal((c1 - c0, d), dtype=np.float32)
        _normalise_rows_into(out[c0:c1], g[None, :] + centres[z] + np.float32(sigma) * eps)
    return out


def isotropic_queries(X: np.ndarray, nq: int = 64, noise: float = 0.05,
                      seed: int = 43) -> np.ndarray:
    rng = _rng(seed)
    rows = rng.choice(X.shape[0], size=nq, replace=False)
    q = X[rows].astype(np.float32) + np.float32(noise) * rng.standard_normal(
        (nq, X.shape[1]), dtype=np.float32)
    out = np.empty_like(q)
    _normalise_rows_into(out, q)
    return out


# ------------------------------------------------------------ power-law case
def _powerlaw_params(d: int, n_clusters: int, alpha: float, seed: int):
    lam = np.arange(1, d + 1, dtype=np.float64) ** (-alpha)
    lam *= d / lam.sum()
    sq = np.sqrt(lam).astype(np.float32)
    rng = _rng(seed, _TAG_CENTRES)
    centres = rng.standard_normal((n_clusters, d), dtype=np.float32) * sq[None, :]
    return sq, centres


def powerlaw_mixture_rows(start: int, stop: int, d: int = 1536,
                          n_clusters: int = 1000, alpha: float = 0.8,
                          sigma: float = 0.3, seed: int = 42,
                          out: np.ndarray | None = None) -> np.ndarray:
    """Rows [start, stop) of the power-law mixture stream."""
    n = stop - start
    if out is None:
        out = np.empty((n, d), dtype=np.float32)
    if out.shape != (n, d) or out.dtype != np.float32:
        raise ValueError("bad output buffer")
    sq, centres = _powerlaw_params(d, n_clusters, alpha, seed)
    first, last = start // CHUNK, (stop - 1) // CHUNK if n > 0 else -1

    def one(c):
        r = _rng(seed, _TAG_ROWS, c)
        z = r.integers(0, n_clusters, size=CHUNK)
        lo = max(start, c * CHUNK)
        hi = min(stop, (c + 1) * CHUNK)
        # draw the whole chunk's noise so a row never depends on the range asked
        sub = 16384
        for s in range(0, CHUNK, sub):
            g0, g1 = c * CHUNK + s, c * CHUNK + s + sub
            if g0 >= hi:
                break           # later sub-chunks are never needed for this range
            eps = r.standard_normal((sub, d), dtype=np.float32)
            a, b = max(lo, g0), min(hi, g1)
            if a >= b:
                continue
            rows = centres[z[a - c * CHUNK:b - c * CHUNK]] + \
                np.float32(sigma) * eps[a - g0:b - g0] * sq[None, :]
            _normalise_rows_into(out[a - start:b - start], rows)

    chunks = list(range(first, last + 1))
    if len(chunks) <= 1:
        for c in chunks:
            one(c)
    else:
        with ThreadPoolExecutor(min(_threads(), len(chunks))) as ex:
            list(ex.map(one, chunks))
    return out


# ------------------------------------------------------- tenants / allowlists
def zipf_tenants(n: int, T: int, s: float = 1.1, seed: int = 44) -> np.ndarray:
    """i.i.d. Zipf(s) tenant ids in [0, T), uint16."""
    if not (1 <= T <= 65535):
        raise ValueError("T must be in 1..65535")
    p = np.arange(1, T + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(p / p.sum())
    cdf[-1] = 1.0
    u = _rng(seed).random(n)
    return np.minimum(np.searchsorted(cdf, u, side="right"), T - 1).astype(np.uint16)


def uniform_partition_tenants(n: int, T: int, seed: int = 44) -> np.ndarray:
    """T equal-size tenant groups (sizes differ by at most one) at random positions."""
    t = (np.arange(n, dtype=np.int64) * T // n).astype(np.uint16)
    _rng(seed).shuffle(t)
    return t


def allowlists(nq: int, T: int, mode: str = "selective", seed: int = 45):
    """List of allowed-tenant arrays, one per query."""
    rng = _rng(seed)
    out = []
    for _ in range(nq):
        if mode == "selective":
            out.append(np.array([rng.integers(0, T)], dtype=np.int64))
        elif mode == "broad":
            out.append(np.sort(rng.choice(T, size=math.ceil(T / 10), replace=False)))
        else:
            raise ValueError(mode)
    return out


def allowlist_bitmap(allowed, T: int) -> np.ndarray:
    """Allowed-tenant lists -> bitmap [nq, ceil(T/64)] of uint64 words."""
    W = (T + 63) // 64
    bm = np.zeros((len(allowed), W), dtype=np.uint64)
    for q, ts in enumerate(allowed):
        for t in np.asarray(ts, dtype=np.int64):
            bm[q, t >> 6] |= np.uint64(1) << np.uint64(t & 63)
    return bm


# ------------------------------------------------------------------ workloads
def workload(name: str, d: int = 1536, out: np.ndarray | None = None):
    """(corpus float32 [N, d], queries float32 [nq, d]) for a named workload:
    'small' (10K), 'powerlaw100k', 'powerlaw999k', 'powerlaw1m'."""
    if name == "small":
        X = isotropic_mixture(10_000, d)
        return X, isotropic_queries(X)
    if name == "powerlaw100k":
        return (powerlaw_mixture_rows(0, 100_000, d, out=out),
                powerlaw_mixture_rows(100_000, 101_000, d))
    if name == "powerlaw999k":
        return (powerlaw_mixture_rows(0, 999_000, d, out=out),
                powerlaw_mixture_rows(999_000, 1_000_000, d))
    if name == "powerlaw1m":
        if out is None:
            out = np.empty((1_000_000, d), dtype=np.float32)
        powerlaw_mixture_rows(0, 999_000, d, out=out[:999_000])
        powerlaw_mixture_rows(1_000_000, 1_001_000, d, out=out[999_000:])
        return out, powerlaw_mixture_rows(999_000, 1_000_000, d)
    raise ValueError(name)
