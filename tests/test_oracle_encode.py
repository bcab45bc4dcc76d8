"""Pins of the oracle's encode (section II-B steps 1-5): special rotations that
reduce it to numpy's searchsorted, hand-placed boundary ties, zero rows,
exact scale invariance, sign symmetry, the packed layout and the paper's
printed sizes, and the distortion / scale statistics predicted by the
codebook's quadrature MSE."""
import math
import os

import numpy as np
import pytest

import oracle
from oracle.codebook import Codebook


def _cb_custom(d, bounds, cents):
    b = int(round(math.log2(len(cents))))
    return Codebook(d=d, bits=b, bounds=np.array(bounds, dtype=np.float64),
                    cents=np.array(cents, dtype=np.float64), iterations=0, converged=True)


@pytest.mark.parametrize("d,bits", [(64, 4), (1536, 4), (128, 2), (256, 3), (128, 8)])
def test_identity_rotation_is_searchsorted(d, bits):
    cb = oracle.lloyd_max(d, bits)
    rng = np.random.default_rng(d + bits)
    X = rng.standard_normal((40, d)).astype(np.float32)
    codes, norms, scales = oracle.encode(X, np.eye(d, dtype=np.float32), cb)
    X64 = X.astype(np.float64)
    ref = np.searchsorted(cb.bounds, X64 / np.linalg.norm(X64, axis=1, keepdims=True), side="right")
    assert np.array_equal(codes, ref)
    np.testing.assert_allclose(norms, np.linalg.norm(X64, axis=1), rtol=1e-13)


def test_permutation_rotation_applies_rows_of_R():
    """R = cyclic shift P (P[j, (j+1) % d] = 1): y_j = x_{j+1}.  Using R^T
    instead of R would shift the other way."""
    d = 64
    cb = oracle.lloyd_max(d, 4)
    P = np.zeros((d, d), dtype=np.float32)
    P[np.arange(d), (np.arange(d) + 1) % d] = 1
    X = np.random.default_rng(1).standard_normal((20, d)).astype(np.float32)
    codes, _, _ = oracle.encode(X, P, cb)
    y = np.roll(X.astype(np.float64), -1, axis=1)
    ref = np.searchsorted(cb.bounds, y / np.linalg.norm(y, axis=1, keepdims=True), side="right")
    assert np.array_equal(codes, ref)


def test_ties_go_to_the_upper_cell():
    d = 64
    # exact zeros sit on the middle boundary t = 0 -> code L/2, never L/2 - 1
    cb = oracle.lloyd_max(d, 4)
    x = np.zeros((1, d), dtype=np.float32)
    x[0, 5] = 3.0
    x[0, 9] = -0.0
    codes, norms, _ = oracle.encode(x, np.eye(d, dtype=np.float32), cb)
    assert norms[0] == 3.0
    assert codes[0, 5] == 15
    assert np.all(np.delete(codes[0], 5) == 8)
    # custom codebook with float32-exact boundaries; ||x|| = 1 exactly
    cbc = _cb_custom(d, [-0.5, 0.0, 0.5], [-0.75, -0.25, 0.25, 0.75])
    x = np.zeros((1, d), dtype=np.float32)
    x[0, :4] = [0.5, -0.5, 0.5, -0.5]
    codes, norms, _ = oracle.encode(x, np.eye(d, dtype=np.float32), cbc)
    assert norms[0] == 1.0
    assert list(codes[0, :4]) == [3, 1, 3, 1]
    assert np.all(codes[0, 4:] == 2)


def test_zero_row_and_nonfinite():
    d = 64
    cb = oracle.lloyd_max(d, 4)
    R = oracle.haar_rotation(d, 3)[1]
    codes, norms, scales = oracle.encode(np.zeros((2, d), dtype=np.float32), R, cb)
    assert np.all(codes == 8) and np.all(norms == 0) and np.all(scales == 0)
    bad = np.ones((3, d), dtype=np.float32)
    bad[1, 7] = np.nan
    with pytest.raises(ValueError, match="row 1"):
        oracle.encode(bad, R, cb)


def test_power_of_two_scaling_is_exact():
    d = 256
    cb = oracle.lloyd_max(d, 4)
    R = oracle.haar_rotation(d, 11)[1]
    X = np.random.default_rng(2).standard_normal((30, d)).astype(np.float32)
    c1, n1, s1 = oracle.encode(X, R, cb)
    c2, n2, s2 = oracle.encode(X * np.float32(8.0), R, cb)
    assert np.array_equal(c1, c2)
    assert np.array_equal(n2, n1 * 8) and np.array_equal(s2, s1 * np.float32(8))


def test_sign_symmetry():
    d = 256
    cb = oracle.lloyd_max(d, 4)
    R = oracle.haar_rotation(d, 12)[1]
    X = np.random.default_rng(3).standard_normal((30, d)).astype(np.float32)
    c1, _, s1 = oracle.encode(X, R, cb)
    c2, _, s2 = oracle.encode(-X, R, cb)
    assert np.array_equal(c2, 15 - c1)
    assert np.array_equal(s1, s2)


def test_pack_layout_and_round_trip():
    assert oracle.pack_codes(np.array([[1, 2, 3, 4]], np.uint8), 4).tolist() == [[0x21, 0x43]]
    assert oracle.pack_codes(np.array([[1, 2, 3, 0]], np.uint8), 2).tolist() == [[0x39]]
    assert oracle.pack_codes(np.array([[5, 3, 7, 0, 0, 0, 0, 0]], np.uint8), 3).tolist() == [[0xDD, 0x01, 0x00]]
    assert oracle.pack_codes(np.array([[200]], np.uint8), 8).tolist() == [[200]]
    rng = np.random.default_rng(4)
    for bits in (1, 2, 3, 4, 8):
        c = rng.integers(0, 1 << bits, size=(7, 1536)).astype(np.uint8)
        p = oracle.pack_codes(c, bits)
        assert p.shape == (7, 1536 * bits // 8)
        assert np.array_equal(oracle.unpack_codes(p, 1536, bits), c)


def test_sizes_printed_in_the_paper(golden_dir):
    with open(os.path.join(golden_dir, "paper_sizes.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            kind, d, bits, n, val = line.split()
            d, bits, n = int(d), int(bits), int(n)
            total = n * oracle.code_bytes_per_vector(d, bits)
            if kind == "bytes_per_vector":
                assert total == int(val)
            else:
                decimals = len(val.split(".")[1]) if "." in val else 0
                assert round(total / 1e6, decimals) == float(val)


def test_distortion_and_scale_match_the_codebook():
    """Uniform unit vectors through a Haar rotation: the reconstruction
    R^T xhat misses x by d*MSE in squared norm on average, and the
    length-renormalisation scalar averages 1/sqrt(1 - d*MSE)."""
    d, bits = 1536, 4
    cb = oracle.lloyd_max(d, bits)
    R64, R32 = oracle.haar_rotation(d, 42)
    g = np.random.default_rng(5).standard_normal((600, d))
    X = (g / np.linalg.norm(g, axis=1, keepdims=True)).astype(np.float32)
    codes, norms, scales = oracle.encode(X, R32, cb)
    xhat = cb.cents[codes]
    recon = xhat @ R32.astype(np.float64)            # R^T xhat, as rows
    X64 = X.astype(np.float64) / norms[:, None]
    err = np.sum((X64 - recon) ** 2, axis=1)
    dm = d * cb.mse()
    assert abs(err.mean() - dm) < 5 * err.std(ddof=1) / math.sqrt(err.size)
    s = scales.astype(np.float64) / norms
    # the scaled reconstruction has exactly the original length
    np.testing.assert_allclose(np.linalg.norm(xhat, axis=1) * s, 1.0, rtol=1e-7)
    assert abs(s.mean() - 1 / math.sqrt(1 - dm)) < 5 * s.std(ddof=1) / math.sqrt(s.size) + 1e-6


def test_quantise_rotated_is_searchsorted_of_the_rotated_rows():
    """Step 3 on rows already rotated: with the identity rotation the rotated
    values are the rows themselves, so the codes are numpy's searchsorted of
    x/||x|| against the boundaries (ties upper); a zero row gets L/2; and the
    codes and scales equal encode's at every bit width."""
    d = 128
    rng = np.random.default_rng(11)
    X = rng.standard_normal((50, d)).astype(np.float32)
    X[3] = 0
    R = oracle.haar_rotation(d, 3)[1]
    _, norms, _, S = oracle.encode(X, R, oracle.lloyd_max(d, 4), return_rotated=True)
    for bits in (1, 2, 3, 4, 8):
        cb = oracle.lloyd_max(d, bits)
        codes, scales = oracle.quantise_rotated(S, norms, cb)
        c2, _, s2 = oracle.encode(X, R, cb)
        assert np.array_equal(codes, c2) and np.array_equal(scales, s2)
        assert np.all(codes[3] == (1 << bits) // 2) and scales[3] == 0
        X64 = X.astype(np.float64)
        Y = X64 / np.maximum(np.linalg.norm(X64, axis=1, keepdims=True), 1e-300)
        ci, _ = oracle.quantise_rotated(X64, np.linalg.norm(X64, axis=1), cb)
        ref = np.searchsorted(cb.bounds, Y, side="right")
        ref[3] = (1 << bits) // 2
        # X64 / n and fl64(t n) <= x agree except within one rounding of a
        # boundary; random normal rows have none there
        assert np.array_equal(ci, ref)
