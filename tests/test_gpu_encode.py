"""GPU parity of the rotation and the quantiser (section II-B, steps 1-5):
query rotation within float32 rounding of the oracle's float64 product, and
codes equal to the oracle's bit for bit (canonical layout), scales to the
float32 rounding of the oracle's float64 value.

The oracle's encode runs with the parameters the kernels use -- the
library's float32 rotation (Rotation.matrix()) and its exported boundaries
and centroids (tests.parity.oracle_tables) -- so every code must be equal,
at every bit width, dimension and on rows built to sit on thresholds.  The
agreement of those parameters with the oracle's own factorisation and
Lloyd-Max solve is tested on the host (tests/test_lib_host.py)."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available
from tests.parity import assert_codes_equal, assert_scales_close, oracle_tables

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402

D = 1536


@pytest.fixture(scope="module")
def small():
    X, Q = synth.workload("small")
    return X[:3000].copy(), Q


@pytest.fixture(scope="module")
def rot_pair():
    rot = tq.Rotation(D, 42)
    return rot, rot.matrix()


def test_query_rotation(small, rot_pair):
    _, Q = small
    rot, R32 = rot_pair
    print("query rotation nq=%d" % Q.shape[0], flush=True)
    out = tq.rotate_queries(rot, torch.from_numpy(Q).cuda()).cpu().numpy().astype(np.float64)
    ref = oracle.rotate_queries(R32, Q)
    err = np.abs(out - ref).max(axis=1) / np.linalg.norm(Q.astype(np.float64), axis=1)
    assert err.max() < 2e-6, err.max()
    # single query and a ragged batch
    out1 = tq.rotate_queries(rot, torch.from_numpy(Q[5:6]).cuda()).cpu().numpy()
    assert np.abs(out1[0] - ref[5]).max() < 2e-6


@pytest.mark.parametrize("d", [1536, 64, 192, 2048])
def test_query_rotation_does_not_depend_on_the_batch(d):
    """Short batches (up to 64 rows) take their own kernel; every row must
    rotate to the same bits as in a long batch."""
    print("query rotation batches d=%d" % d, flush=True)
    rot = tq.Rotation(d, 9)
    rng = np.random.default_rng(d)
    Q = torch.from_numpy(rng.standard_normal((300, d)).astype(np.float32)).cuda()
    full = tq.rotate_queries(rot, Q)
    for a, b in [(0, 1), (5, 6), (0, 16), (17, 81), (250, 300), (64, 127)]:
        part = tq.rotate_queries(rot, Q[a:b].contiguous())
        assert torch.equal(part, full[a:b]), (a, b)


@pytest.mark.parametrize("bits", [4, 2, 8, 3, 1])
def test_codes_bit_exact(small, rot_pair, bits):
    X, _ = small
    rot, R32 = rot_pair
    print("rotate_quantize bits=%d n=%d" % (bits, X.shape[0]), flush=True)
    cb = tq.Codebook(D, bits)
    codes, scales = tq.rotate_quantize(cb, rot, torch.from_numpy(X).cuda())
    c_or, n_or, s_or = oracle.encode(X, R32, oracle_tables(cb))
    assert_codes_equal(codes.cpu().numpy(), c_or, bits)
    assert_scales_close(scales.cpu().numpy(), s_or)


@pytest.mark.parametrize("d,bits", [(64, 4), (192, 2), (2048, 4), (2048, 8), (128, 3),
                                    (64, 8), (192, 8)])
def test_codes_bit_exact_other_dimensions(d, bits):
    """Rotation tiles of 128 output columns clipped (d = 64) or ragged
    (d = 192), the largest d, and 3-bit packing at its smallest d; the 8-bit
    cases take the tiled recomputation of flagged coordinates, here with
    clipped and ragged column tiles and a ragged last row tile."""
    print("rotate_quantize d=%d bits=%d" % (d, bits), flush=True)
    rng = np.random.default_rng(d * 10 + bits)
    X = rng.standard_normal((1000, d)).astype(np.float32)
    X[7] *= np.float32(1e-20)
    rot = tq.Rotation(d, 5)
    R32 = rot.matrix()
    cb = tq.Codebook(d, bits)
    codes, scales = tq.rotate_quantize(cb, rot, torch.from_numpy(X).cuda())
    c_or, n_or, s_or = oracle.encode(X, R32, oracle_tables(cb))
    assert_codes_equal(codes.cpu().numpy(), c_or, bits)
    assert_scales_close(scales.cpu().numpy(), s_or)


def test_codes_special_rows(rot_pair):
    """Zero rows, tiny and huge norms, exact-zero coordinates, a ragged count."""
    rot, R32 = rot_pair
    rng = np.random.default_rng(3)
    X = rng.standard_normal((131, D)).astype(np.float32)
    X[0] = 0
    X[1] *= np.float32(1e-30)
    X[2] *= np.float32(1e30)
    X[3, :] = 0
    X[3, 7] = 1.0
    X[4] = X[5]
    cb = tq.Codebook(D, 4)
    codes, scales = tq.rotate_quantize(cb, rot, torch.from_numpy(X).cuda())
    c_or, n_or, s_or = oracle.encode(X, R32, oracle_tables(cb))
    assert_codes_equal(codes.cpu().numpy(), c_or, 4)
    c_gpu = oracle.unpack_codes(codes.cpu().numpy(), D, 4)
    assert np.all(c_gpu[0] == 8) and scales[0].item() == 0.0
    assert_scales_close(scales.cpu().numpy(), s_or)


def test_nonfinite_input_is_rejected(rot_pair):
    rot, _ = rot_pair
    X = np.ones((70, D), dtype=np.float32)
    X[65, 3] = np.inf
    cb = tq.Codebook(D, 4)
    with pytest.raises(tq.TQError, match="TQ_EINVAL"):
        tq.rotate_quantize(cb, rot, torch.from_numpy(X).cuda())


def test_gemm_error_is_far_inside_the_proven_band(small, rot_pair):
    """The fix-up band assumes |y - S| <= 4e-6 ||x|| for the MFMA product.
    Measured errors must be orders of magnitude smaller (float32 products,
    float64 accumulation every 32 terms)."""
    X, _ = small
    rot, R32 = rot_pair
    Y = tq.rotate_queries(rot, torch.from_numpy(X[:512]).cuda()).cpu().numpy().astype(np.float64)
    ref = X[:512].astype(np.float64) @ R32.astype(np.float64).T
    rel = np.abs(Y - ref).max(axis=1) / np.linalg.norm(X[:512].astype(np.float64), axis=1)
    print("max |y - S| / ||x|| = %.3e" % rel.max())
    assert rel.max() < 4e-7


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_codes_of_rows_built_on_thresholds(rot_pair, bits):
    """Rows whose rotated coordinates sit on thresholds to float32 rounding:
    90% of the coordinates of a random unit vector are moved to their nearest
    threshold and the others rescaled to keep the norm at one.  Nearly every
    coordinate then falls inside the proven band, each 128 x 128 output tile
    carries about 15,000 flags (about 29 rounds of the 8-bit tile
    recomputation), and the codes are decided by the exact sums."""
    rot, R32 = rot_pair
    print("rotate_quantize on thresholds bits=%d" % bits, flush=True)
    cb = tq.Codebook(D, bits)
    ocb = oracle_tables(cb)
    t = np.asarray(ocb.bounds, dtype=np.float64)
    rng = np.random.default_rng(17 + bits)
    n = 300
    Y = rng.standard_normal((n, D))
    Y /= np.linalg.norm(Y, axis=1, keepdims=True)
    snap = rng.random((n, D)) < 0.9
    pos = np.clip(np.searchsorted(t, Y), 1, len(t) - 1)
    lo, hi = t[pos - 1], t[pos]
    nearest = np.where(np.abs(Y - lo) <= np.abs(Y - hi), lo, hi)
    Y = np.where(snap, nearest, Y)
    on = np.where(snap, Y, 0.0)
    free = np.where(snap, 0.0, Y)
    rest = 1.0 - (on * on).sum(axis=1)
    assert np.all(rest > 0)
    Y = on + free * np.sqrt(rest / (free * free).sum(axis=1))[:, None]
    nrm = rng.uniform(0.5, 2.0, n)
    X = np.ascontiguousarray(((Y * nrm[:, None]) @ R32.astype(np.float64)).astype(np.float32))
    codes, scales = tq.rotate_quantize(cb, rot, torch.from_numpy(X).cuda())
    c_or, n_or, s_or, S = oracle.encode(X, R32, ocb, return_rotated=True)
    u = S / n_or[:, None]
    p2 = np.clip(np.searchsorted(t, u), 1, len(t) - 1)
    gap = np.minimum(np.abs(u - t[p2 - 1]), np.abs(u - t[p2]))
    print("coordinates inside the band: %.3f" % (gap <= 4e-6).mean(), flush=True)
    assert (gap <= 4e-6).mean() > 0.85
    # coordinates within one float64 rounding of a threshold: there the tie
    # rule and the exact sums decide the code
    print("coordinates within 1e-15 of a threshold: %d" % int((gap <= 1e-15).sum()), flush=True)
    assert_codes_equal(codes.cpu().numpy(), c_or, bits)
    assert_scales_close(scales.cpu().numpy(), s_or)
