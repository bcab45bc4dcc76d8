"""Seeded random orthogonal rotation (oracle; test use only).

Section II-B, step 2: every vector is multiplied by one orthogonal matrix R,
drawn at random once and then kept.  The paper does not fix the law, the generator or the seed; the
reading taken here (shared with the library, which implements it separately):

* Random numbers: SplitMix64 in its counter form, z_i = mix(seed + (i+1)*gamma)
  with gamma = 0x9E3779B97F4A7C15 and the published finaliser
  (Steele, Lea & Flood, OOPSLA 2014):
      z ^= z >> 30; z *= 0xBF58476D1CE4E5B9
      z ^= z >> 27; z *= 0x94D049BB133111EB
      z ^= z >> 31
* Uniforms on (0, 1): u = ((z >> 11) + 1/2) * 2^-53  (never 0 or 1).
* Normals: Box-Muller on consecutive pairs (u_{2p}, u_{2p+1}):
      g_{2p}   = sqrt(-2 ln u_{2p}) cos(2 pi u_{2p+1})
      g_{2p+1} = sqrt(-2 ln u_{2p}) sin(2 pi u_{2p+1})
  filling the d x d matrix G row-major.
* Haar orthogonal: G = Q T (Householder QR), R = Q diag(sign(diag T)), the sign
  fix that makes R Haar-distributed (Mezzadri, Notices AMS 2007).
* The GPU uses R rounded to float32; y = R x, i.e. y_j = sum_k R[j,k] x_k.
"""
from __future__ import annotations

import functools

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix64(seed: int, count: int, start: int = 0) -> np.ndarray:
    """Outputs start .. start+count-1 of the SplitMix64 stream for `seed`."""
    with np.errstate(over="ignore"):
        i = np.arange(start + 1, start + count + 1, dtype=np.uint64)
        z = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) + i * _GAMMA
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        z = z ^ (z >> np.uint64(31))
    return z


def uniforms53(seed: int, count: int, start: int = 0) -> np.ndarray:
    """Uniform doubles on (0, 1) from the top 53 bits of each output."""
    z = splitmix64(seed, count, start)
    return ((z >> np.uint64(11)).astype(np.float64) + 0.5) * (2.0 ** -53)


def gaussians(seed: int, count: int) -> np.ndarray:
    """`count` (even) standard normals by Box-Muller on consecutive uniforms."""
    if count % 2:
        raise ValueError("count must be even")
    u = uniforms53(seed, count)
    u1, u2 = u[0::2], u[1::2]
    r = np.sqrt(-2.0 * np.log(u1))
    g = np.empty(count, dtype=np.float64)
    g[0::2] = r * np.cos(2.0 * np.pi * u2)
    g[1::2] = r * np.sin(2.0 * np.pi * u2)
    return g


@functools.lru_cache(maxsize=4)
def haar_rotation(d: int, seed: int = 42):
    """(R64, R32): the Haar orthogonal matrix for (d, seed) and its float32 copy."""
    G = gaussians(seed, d * d).reshape(d, d)
    Q, T = np.linalg.qr(G)
    s = np.sign(np.diag(T))
    s[s == 0] = 1.0
    R64 = Q * s[None, :]
    R32 = R64.astype(np.float32)
    R64.setflags(write=False)
    R32.setflags(write=False)
    return R64, R32
