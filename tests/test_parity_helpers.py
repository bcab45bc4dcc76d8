"""The parity checkers catch planted mistakes (CPU only: the "GPU" lists here
are the oracle's own results, then corrupted)."""
import numpy as np
import pytest

import oracle
from tests.parity import check_topk, check_topk_sampled

D = 256


@pytest.fixture(scope="module")
def small():
    rng = np.random.default_rng(11)
    X = rng.standard_normal((3000, D)).astype(np.float32)
    X[:300] += 3 * rng.standard_normal((1, D)).astype(np.float32)   # a dense cluster
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    Q = (X[:6] + 0.05 * rng.standard_normal((6, D))).astype(np.float32)
    R32 = oracle.haar_rotation(D, 42)[1]
    cb = oracle.lloyd_max(D, 4)
    codes, _, scales = oracle.encode(X, R32, cb)
    ids, sc = oracle.search(codes, scales, cb.cents, R32, Q, 10)
    return X, Q, R32, cb, codes, scales, ids, sc


def test_oracle_lists_pass(small):
    X, Q, R32, cb, codes, scales, ids, sc = small
    qrot = oracle.rotate_queries(R32, Q)
    qn = np.linalg.norm(Q.astype(np.float64), axis=1)
    assert check_topk(ids, sc, codes, scales, cb.cents, qrot, qn, 10, ids, sc) == 0
    check_topk_sampled(ids, sc, X, R32, cb, Q, 10, np.arange(X.shape[0]))


@pytest.mark.parametrize("mistake", ["worse_id", "wrong_score", "duplicate", "unordered"])
def test_planted_mistakes_fail(small, mistake):
    X, Q, R32, cb, codes, scales, ids, sc = small
    qrot = oracle.rotate_queries(R32, Q)
    qn = np.linalg.norm(Q.astype(np.float64), axis=1)
    bad_i, bad_s = ids.copy(), sc.copy()
    if mistake == "worse_id":
        # replace the last entry by a vector far down the ranking, with its true score
        full_i, full_s = oracle.search(codes, scales, cb.cents, R32, Q[:1], 500)
        bad_i[0, 9], bad_s[0, 9] = full_i[0, 499], full_s[0, 499]
    elif mistake == "wrong_score":
        bad_s[0, 0] *= 1.001
    elif mistake == "duplicate":
        bad_i[0, 1] = bad_i[0, 0]
    else:
        bad_i[0, [0, 5]] = bad_i[0, [5, 0]]
        bad_s[0, [0, 5]] = bad_s[0, [5, 0]]
    with pytest.raises(AssertionError):
        check_topk(bad_i, bad_s, codes, scales, cb.cents, qrot, qn, 10, ids, sc)
    with pytest.raises(AssertionError):
        check_topk_sampled(bad_i, bad_s, X, R32, cb, Q, 10, np.arange(X.shape[0]))
