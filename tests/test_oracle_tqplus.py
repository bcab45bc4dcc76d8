"""Pins of the oracle's TQ+ calibration (section II-B): per-coordinate shift
and spread fitted on a first batch, applied before quantisation and in the
reconstruction.  Checked against what the method fixes: the identity
calibration is plain TurboQuant bit for bit; the fitted map gives the batch
the first two moments of the canonical marginal (mean 0, variance 1/d);
isotropic data needs no calibration; and on data whose rotated coordinates
are shifted, calibrated codes reconstruct the vectors more closely."""
import numpy as np

import oracle

D = 256


def _setup(seed):
    cb = oracle.lloyd_max(D, 4)
    R = oracle.haar_rotation(D, seed)[1]
    return cb, R


def test_identity_calibration_is_plain_turboquant():
    cb, R = _setup(5)
    X = np.random.default_rng(1).standard_normal((300, D)).astype(np.float32)
    c0, n0, s0 = oracle.encode(X, R, cb)
    c1, n1, s1 = oracle.encode_tqplus(X, R, cb, np.zeros(D, np.float32), np.ones(D, np.float32))
    assert np.array_equal(c0, c1) and np.array_equal(n0, n1) and np.array_equal(s0, s1)
    Q = np.random.default_rng(2).standard_normal((4, D)).astype(np.float32)
    a = oracle.search(c0, s0, cb.cents, R, Q, 7)
    b = oracle.search(c0, s0, cb.cents, R, Q, 7, calib=(np.zeros(D), np.ones(D)))
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_fit_gives_the_canonical_moments():
    _, R = _setup(6)
    rng = np.random.default_rng(3)
    X = (rng.standard_normal((2000, D)) * rng.uniform(0.2, 3.0, D) + rng.standard_normal(D)).astype(np.float32)
    mu, kappa = oracle.tqplus_fit(X, R)
    Y = (X.astype(np.float64) @ R.astype(np.float64).T)
    Y /= np.linalg.norm(X.astype(np.float64), axis=1, keepdims=True)
    Z = (Y - mu) / kappa
    assert np.max(np.abs(Z.mean(axis=0))) < 1e-12
    assert np.allclose(Z.var(axis=0), 1.0 / D, rtol=1e-9)


def test_isotropic_data_needs_no_calibration():
    _, R = _setup(7)
    X = np.random.default_rng(4).standard_normal((8000, D)).astype(np.float32)   # uniform directions
    mu, kappa = oracle.tqplus_fit(X, R)
    # sampling error of a mean of 8000 values of spread 1/sqrt(d), of a spread estimate
    assert np.max(np.abs(mu)) < 5 / np.sqrt(8000 * D)
    assert np.max(np.abs(kappa - 1.0)) < 0.06


def test_calibration_lowers_distortion_on_shifted_data():
    cb, R = _setup(8)
    rng = np.random.default_rng(5)
    offset = rng.standard_normal(D)
    X = (rng.standard_normal((3000, D)) * 0.6 + 2.0 * offset).astype(np.float32)
    mu, kappa = oracle.tqplus_fit(X[:1000], R)
    mu32, kappa32 = mu.astype(np.float32), kappa.astype(np.float32)
    Y = X.astype(np.float64) @ R.astype(np.float64).T
    Y /= np.linalg.norm(X.astype(np.float64), axis=1, keepdims=True)
    c0, _, _ = oracle.encode(X, R, cb)
    c1, _, _ = oracle.encode_tqplus(X, R, cb, mu32, kappa32)
    err0 = np.mean(np.sum((Y - cb.cents[c0]) ** 2, axis=1))
    yhat = mu32.astype(np.float64) + kappa32.astype(np.float64) * cb.cents[c1]
    err1 = np.mean(np.sum((Y - yhat) ** 2, axis=1))
    assert err1 < 0.5 * err0, (err0, err1)
    # the exact top 10 is found better with calibrated codes
    Q = (rng.standard_normal((20, D)) + 2.0 * offset).astype(np.float32)
    ex, _ = oracle.exact_search(X, Q, 10)
    _, _, s0 = oracle.encode(X, R, cb)
    _, _, s1 = oracle.encode_tqplus(X, R, cb, mu32, kappa32)
    i0, _ = oracle.search(c0, s0, cb.cents, R, Q, 10)
    i1, _ = oracle.search(c1, s1, cb.cents, R, Q, 10, calib=(mu32, kappa32))
    assert oracle.recall_at_k(i1, ex, 10) > oracle.recall_at_k(i0, ex, 10)


def test_fit_hand_worked():
    """Two unit rows under the identity rotation: per coordinate the mean is
    (1/2, 1/2, 0, 0) and the population standard deviation (1/2, 1/2, 0, 0),
    so kappa = sigma * sqrt(4) = (1, 1, 0, 0)."""
    X = np.array([[2.0, 0, 0, 0], [0, 3.0, 0, 0]], dtype=np.float32)   # norms removed by the fit
    mu, kappa = oracle.tqplus_fit(X, np.eye(4, dtype=np.float32))
    assert np.allclose(mu, [0.5, 0.5, 0, 0], atol=1e-15)
    assert np.allclose(kappa, [1, 1, 0, 0], atol=1e-15)


def test_encode_hand_worked():
    """d = 4, 1 bit (threshold 0, centroids -+4/(3 pi), the closed form of
    E|X| for a coordinate of a uniform unit vector in R^4), identity
    rotation, x = (3, 4, 0, 0): y = (0.6, 0.8, 0, 0).  With mu = (0.7, 0.5,
    -0.1, 0.1) and kappa = (1, 2, 1, 0.5) the thresholds mu + kappa * 0 are
    (0.7, 0.5, -0.1, 0.1): codes (0, 1, 1, 0), where plain TurboQuant gives
    (1, 1, 1, 1).  Reconstruction mu + kappa c_code, scale 5 / ||yhat||, and
    the score of q = e_0 is scale * yhat_0."""
    cb = oracle.lloyd_max(4, 1)
    R = np.eye(4, dtype=np.float32)
    X = np.array([[3.0, 4.0, 0.0, 0.0]], dtype=np.float32)
    mu = np.array([0.7, 0.5, -0.1, 0.1], dtype=np.float32)
    kappa = np.array([1.0, 2.0, 1.0, 0.5], dtype=np.float32)
    codes, norms, scales = oracle.encode_tqplus(X, R, cb, mu, kappa)
    assert codes.tolist() == [[0, 1, 1, 0]]
    assert oracle.encode(X, R, cb)[0].tolist() == [[1, 1, 1, 1]]
    c = 4.0 / (3.0 * np.pi)
    yhat = mu.astype(np.float64) + kappa.astype(np.float64) * np.array([-c, c, c, -c])
    s = 5.0 / np.sqrt(np.sum(yhat ** 2))
    assert norms[0] == 5.0
    assert abs(scales[0] - s) <= 1e-6 * s
    score = oracle.scores_for_ids(codes, scales, cb.cents, np.array([1.0, 0, 0, 0]), [0],
                                  calib=(mu, kappa))
    assert abs(score[0] - scales[0] * yhat[0]) <= 1e-12
