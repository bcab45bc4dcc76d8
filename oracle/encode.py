"""TurboQuant encode and bit packing (oracle; test use only).

Section II-B, steps 1-5.  The arithmetic of steps 1-3 and 5 is the plain C in
csrc/tq_oracle.c (sequential float64, exact products, no fused multiply-add);
this module marshals arguments and does step 4, bit packing.

Bit packing (step 4; a 1536-d vector takes 768 bytes at 4 bits): the codes of
a row form one little-endian bitstream, coordinate j occupying bits
[b*j, b*j + b) least-significant bit first.  At b = 4 coordinate 2m is the low
nibble and 2m+1 the high nibble of byte m.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build
from .codebook import Codebook

_lib = None


def _load():
    global _lib
    if _lib is None:
        # TQ_ORACLE_LIBRARY: another build of tq_oracle.c (the sanitizer build)
        path = os.environ.get("TQ_ORACLE_LIBRARY") or _build.LIB
        if not os.environ.get("TQ_ORACLE_LIBRARY") and (
                not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC)):
            path = _build.build(force=True)
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        lib.tqo_encode.argtypes = [P, ctypes.c_int64, ctypes.c_int32, P, P,
                                   ctypes.c_int32, P, P, P, P]
        lib.tqo_encode.restype = ctypes.c_int
        lib.tqo_scales.argtypes = [P, P, ctypes.c_int64, ctypes.c_int32, P,
                                   ctypes.c_int32, P]
        lib.tqo_scales.restype = ctypes.c_int
        lib.tqo_quantise.argtypes = [P, P, ctypes.c_int64, ctypes.c_int32, P, ctypes.c_int32, P]
        lib.tqo_quantise.restype = ctypes.c_int
        lib.tqo_encode_plus.argtypes = [P, ctypes.c_int64, ctypes.c_int32, P, P, ctypes.c_int32,
                                        P, P, P, P]
        lib.tqo_encode_plus.restype = ctypes.c_int
        lib.tqo_scales_plus.argtypes = [P, P, ctypes.c_int64, ctypes.c_int32, P, ctypes.c_int32,
                                        P, P, P]
        lib.tqo_scales_plus.restype = ctypes.c_int
        _lib = lib
    return _lib


def code_bytes_per_vector(d: int, bits: int) -> int:
    """Packed size of one vector: d*b/8 bytes (768 at d=1536, b=4)."""
    if (d * bits) % 8:
        raise ValueError("d*bits must be a multiple of 8")
    return d * bits // 8


def encode(X: np.ndarray, R32: np.ndarray, cb: Codebook, return_rotated: bool = False):
    """Encode float32 rows X [n, d] with rotation R32 [d, d] and codebook cb.

    Returns (codes uint8 [n, d] unpacked, norms float64 [n], scales float32 [n])
    and, with return_rotated, also the rotated values S float64 [n, d].
    Raises ValueError on a non-finite row.
    """
    X = np.ascontiguousarray(X, dtype=np.float32)
    R32 = np.ascontiguousarray(R32, dtype=np.float32)
    n, d = X.shape
    if R32.shape != (d, d) or cb.d != d:
        raise ValueError("shape mismatch")
    L = cb.levels
    bounds = np.ascontiguousarray(cb.bounds, dtype=np.float64)
    cents = np.ascontiguousarray(cb.cents, dtype=np.float64)
    codes = np.empty((n, d), dtype=np.uint8)
    norms = np.empty(n, dtype=np.float64)
    scales = np.empty(n, dtype=np.float32)
    rot = np.empty((n, d), dtype=np.float64) if return_rotated else None
    bad = ctypes.c_int64(-1)
    lib = _load()
    st = lib.tqo_encode(X.ctypes.data, n, d, R32.ctypes.data, bounds.ctypes.data,
                        L, codes.ctypes.data, norms.ctypes.data,
                        rot.ctypes.data if rot is not None else None, ctypes.byref(bad))
    if st == -2:
        raise ValueError("non-finite input in row %d" % bad.value)
    if st != 0:
        raise RuntimeError("tqo_encode failed (%d)" % st)
    st = lib.tqo_scales(codes.ctypes.data, norms.ctypes.data, n, d,
                        cents.ctypes.data, L, scales.ctypes.data)
    if st != 0:
        raise RuntimeError("tqo_scales failed (%d)" % st)
    if return_rotated:
        return codes, norms, scales, rot
    return codes, norms, scales


def quantise_rotated(S: np.ndarray, norms: np.ndarray, cb: Codebook):
    """Steps 3 and 5 for rows already rotated by encode(..., return_rotated=True):
    S float64 [n, d] and norms float64 [n] as it returned them, coded with the
    codebook cb (so one rotation serves several bit widths).  Returns (codes
    uint8 [n, d] unpacked, scales float32 [n]), equal to what encode returns
    for the same rows with cb."""
    S = np.ascontiguousarray(S, dtype=np.float64)
    norms = np.ascontiguousarray(norms, dtype=np.float64)
    n, d = S.shape
    if norms.shape != (n,) or cb.d != d:
        raise ValueError("shape mismatch")
    L = cb.levels
    bounds = np.ascontiguousarray(cb.bounds, dtype=np.float64)
    cents = np.ascontiguousarray(cb.cents, dtype=np.float64)
    codes = np.empty((n, d), dtype=np.uint8)
    scales = np.empty(n, dtype=np.float32)
    lib = _load()
    st = lib.tqo_quantise(S.ctypes.data, norms.ctypes.data, n, d, bounds.ctypes.data, L,
                          codes.ctypes.data)
    if st != 0:
        raise RuntimeError("tqo_quantise failed (%d)" % st)
    st = lib.tqo_scales(codes.ctypes.data, norms.ctypes.data, n, d, cents.ctypes.data, L,
                        scales.ctypes.data)
    if st != 0:
        raise RuntimeError("tqo_scales failed (%d)" % st)
    return codes, scales


def tqplus_fit(X: np.ndarray, R32: np.ndarray):
    """TQ+ calibration (section II-B): per-coordinate first and second
    moments of the rotated, L2-normalised rows of the first batch X.  Returns
    (mu, kappa) in float64: mu_j the mean of y_j = (R x / ||x||)_j and
    kappa_j = sigma_j sqrt(d), sigma_j the population standard deviation --
    the map z_j = (y_j - mu_j) / kappa_j gives the batch mean 0 and variance
    1/d per coordinate, the first two moments of the canonical marginal."""
    X = np.asarray(X, dtype=np.float32).astype(np.float64)
    R = np.asarray(R32, dtype=np.float32).astype(np.float64)
    d = X.shape[1]
    Y = (X @ R.T) / np.linalg.norm(X, axis=1, keepdims=True)
    mu = Y.mean(axis=0)
    sigma = np.sqrt(((Y - mu) ** 2).mean(axis=0))
    return mu, sigma * np.sqrt(d)


def encode_tqplus(X: np.ndarray, R32: np.ndarray, cb: Codebook, mu32: np.ndarray,
                  kappa32: np.ndarray):
    """Encode with TQ+ calibration (section II-B) given as float32 mu, kappa
    (as an index stores them): thresholds a_jt = mu_j + kappa_j t_t per
    coordinate, reconstruction yhat_j = mu_j + kappa_j c[code_j] for the
    scale.  Returns (codes uint8 [n, d], norms float64 [n], scales float32 [n])."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    R32 = np.ascontiguousarray(R32, dtype=np.float32)
    n, d = X.shape
    mu = np.ascontiguousarray(mu32, dtype=np.float32)
    kappa = np.ascontiguousarray(kappa32, dtype=np.float32)
    if R32.shape != (d, d) or cb.d != d or mu.shape != (d,) or kappa.shape != (d,):
        raise ValueError("shape mismatch")
    L = cb.levels
    bounds = np.ascontiguousarray(cb.bounds, dtype=np.float64)
    cents = np.ascontiguousarray(cb.cents, dtype=np.float64)
    codes = np.empty((n, d), dtype=np.uint8)
    norms = np.empty(n, dtype=np.float64)
    scales = np.empty(n, dtype=np.float32)
    lib = _load()
    st = lib.tqo_encode_plus(X.ctypes.data, n, d, R32.ctypes.data, bounds.ctypes.data, L,
                             mu.ctypes.data, kappa.ctypes.data, codes.ctypes.data, norms.ctypes.data)
    if st == -2:
        raise ValueError("non-finite input")
    if st != 0:
        raise RuntimeError("tqo_encode_plus failed (%d)" % st)
    st = lib.tqo_scales_plus(codes.ctypes.data, norms.ctypes.data, n, d, cents.ctypes.data, L,
                             mu.ctypes.data, kappa.ctypes.data, scales.ctypes.data)
    if st != 0:
        raise RuntimeError("tqo_scales_plus failed (%d)" % st)
    return codes, norms, scales


def pack_codes(codes: np.ndarray, bits: int) -> np.ndarray:
    """Unpacked codes [n, d] -> canonical LSB-first bitstream rows [n, d*b/8]."""
    codes = np.asarray(codes, dtype=np.uint8)
    n, d = codes.shape
    nbytes = code_bytes_per_vector(d, bits)
    if np.any(codes >> bits):
        raise ValueError("code out of range for %d bits" % bits)
    bitplanes = (codes[:, :, None] >> np.arange(bits, dtype=np.uint8)) & 1
    flat = bitplanes.reshape(n, d * bits)
    return np.packbits(flat, axis=1, bitorder="little")[:, :nbytes]


def unpack_codes(packed: np.ndarray, d: int, bits: int) -> np.ndarray:
    """Canonical packed rows [n, d*b/8] -> unpacked codes [n, d]."""
    packed = np.asarray(packed, dtype=np.uint8)
    n = packed.shape[0]
    flat = np.unpackbits(packed, axis=1, bitorder="little")[:, : d * bits]
    planes = flat.reshape(n, d, bits).astype(np.uint8)
    return np.sum(planes << np.arange(bits, dtype=np.uint8), axis=2, dtype=np.uint8)
