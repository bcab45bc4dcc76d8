"""Pins of the oracle's search (section II-B step 5, section III-B filtering,
section IV-A ground truth): scores equal inner products with the scaled
reconstruction computed without rotating the query; filtering equals search
on the subset; padding, ties and exact-match cases."""
import numpy as np

import oracle
import synth


def _index(n=300, d=128, bits=4, seed=0):
    cb = oracle.lloyd_max(d, bits)
    R64, R32 = oracle.haar_rotation(d, 42)
    X = np.random.default_rng(seed).standard_normal((n, d)).astype(np.float32)
    codes, norms, scales = oracle.encode(X, R32, cb)
    return cb, R32, X, codes, scales


def test_score_is_inner_product_with_reconstruction():
    """score_i = <q, s_i R^T xhat_i> in the original space.  Rotating the query
    with R^T instead of R, or dropping the scale, breaks this."""
    cb, R32, X, codes, scales = _index()
    Q = np.random.default_rng(9).standard_normal((5, X.shape[1])).astype(np.float32)
    recon = scales[:, None].astype(np.float64) * (cb.cents[codes] @ R32.astype(np.float64))
    ids, sc = oracle.search(codes, scales, cb.cents, R32, Q, k=X.shape[0])
    for b in range(Q.shape[0]):
        direct = recon @ Q[b].astype(np.float64)
        np.testing.assert_allclose(sc[b], direct[ids[b]], rtol=1e-12, atol=1e-12)
        assert np.all(np.diff(sc[b]) <= 0)
        assert sorted(ids[b].tolist()) == list(range(X.shape[0]))
    qr = oracle.rotate_queries(R32, Q[:1])[0]
    np.testing.assert_allclose(oracle.scores_for_ids(codes, scales, cb.cents, qr, ids[0, :7]),
                               sc[0, :7], rtol=1e-13)


def test_scores_estimate_the_true_inner_product():
    cb, R32, X, codes, scales = _index(n=400, d=1536)
    Q = np.random.default_rng(10).standard_normal((4, 1536)).astype(np.float32)
    ids, sc = oracle.search(codes, scales, cb.cents, R32, Q, k=400)
    exact = Q.astype(np.float64) @ X.astype(np.float64).T
    for b in range(4):
        rel = np.abs(sc[b] - exact[b, ids[b]]) / (np.linalg.norm(Q[b]) * np.linalg.norm(X[ids[b]], axis=1))
        assert rel.max() < 0.02


def test_filter_equals_subset_search():
    cb, R32, X, codes, scales = _index(n=500)
    T = 7
    tenants = synth.zipf_tenants(500, T, seed=3)
    allowed = [np.array([0, 3]), np.array([5]), np.array([1, 2, 4, 6])]
    bm = synth.allowlist_bitmap(allowed, T)
    Q = np.random.default_rng(11).standard_normal((3, 128)).astype(np.float32)
    ids, sc = oracle.search(codes, scales, cb.cents, R32, Q, k=10, tenants=tenants, allow=bm)
    for b in range(3):
        sub = np.flatnonzero(np.isin(tenants, allowed[b]))
        i2, s2 = oracle.search(codes[sub], scales[sub], cb.cents, R32, Q[b:b + 1], k=10)
        valid = i2[0] >= 0
        assert np.array_equal(ids[b][valid], sub[i2[0][valid]])
        np.testing.assert_allclose(sc[b], s2[0], rtol=1e-13)


def test_padding_empty_allowlist_and_large_k():
    cb, R32, X, codes, scales = _index(n=20)
    Q = np.random.default_rng(12).standard_normal((2, 128)).astype(np.float32)
    tenants = np.zeros(20, dtype=np.uint16)
    empty = np.zeros((2, 1), dtype=np.uint64)
    ids, sc = oracle.search(codes, scales, cb.cents, R32, Q, k=5, tenants=tenants, allow=empty)
    assert np.all(ids == -1) and np.all(np.isneginf(sc))
    ids, sc = oracle.search(codes, scales, cb.cents, R32, Q, k=25)
    assert np.all(ids[:, 20:] == -1) and np.all(np.isneginf(sc[:, 20:]))
    assert np.all(ids[:, :20] >= 0)


def test_ties_order_by_id():
    cb, R32, X, codes, scales = _index(n=10)
    codes = np.concatenate([codes, codes[[3, 3, 7]]])
    scales = np.concatenate([scales, scales[[3, 3, 7]]])
    Q = X[3:4]
    ids, sc = oracle.search(codes, scales, cb.cents, R32, Q, k=13)
    pos = {int(i): p for p, i in enumerate(ids[0])}
    assert pos[3] < pos[10] < pos[11]
    assert sc[0][pos[3]] == sc[0][pos[10]] == sc[0][pos[11]]
    assert pos[7] < pos[12]


def test_exact_search_and_recall():
    X = np.random.default_rng(13).standard_normal((200, 64)).astype(np.float32)
    ids, sc = oracle.exact_search(X, X[[5, 17]], k=3)
    assert ids[0, 0] == 5 and ids[1, 0] == 17
    assert sc[0, 0] == np.dot(X[5].astype(np.float64), X[5].astype(np.float64))
    assert oracle.recall_at_k(ids, ids, 3) == 1.0
    assert oracle.recall_at_k(np.array([[5, -1, -1]]), np.array([[5, 9, 2]]), 3) == 1 / 3


def test_hit_and_mrr_hand_worked():
    """Hit@k and MRR@k (section IV-E) on lists worked out by hand."""
    approx = np.array([[5, 3, 1], [2, 9, 7], [4, 6, 8], [1, 2, 3]])
    exact = np.array([[3], [7], [0], [-1]])          # last query: nothing eligible
    assert oracle.hit_at_k(approx, exact, 1) == 0.0
    assert oracle.hit_at_k(approx, exact, 2) == 1 / 3
    assert oracle.hit_at_k(approx, exact, 3) == 2 / 3
    assert abs(oracle.mrr_at_k(approx, exact, 3) - (1 / 2 + 1 / 3 + 0) / 3) < 1e-15
    assert abs(oracle.mrr_at_k(approx, exact, 2) - (1 / 2) / 3) < 1e-15


def test_hit_and_mrr_properties():
    X = np.random.default_rng(21).standard_normal((300, 32)).astype(np.float32)
    Q = np.random.default_rng(22).standard_normal((40, 32)).astype(np.float32)
    ex, _ = oracle.exact_search(X, Q, k=20)
    # exact search scores perfectly against itself
    assert oracle.hit_at_k(ex, ex, 1) == 1.0 and oracle.mrr_at_k(ex, ex, 20) == 1.0
    # a perturbed ranking: Hit@1 <= MRR@k <= Hit@k, and Hit@k grows with k
    rng = np.random.default_rng(23)
    approx = np.array([rng.permutation(row) for row in ex])
    h = [oracle.hit_at_k(approx, ex, k) for k in (1, 3, 5, 10, 20)]
    assert all(a <= b for a, b in zip(h, h[1:])) and h[-1] == 1.0
    m = oracle.mrr_at_k(approx, ex, 20)
    assert h[0] <= m <= h[-1]
    # the top-1 moved to rank r everywhere gives MRR exactly 1/r
    shifted = np.concatenate([ex[:, 1:4], ex[:, :1], ex[:, 4:]], axis=1)
    assert abs(oracle.mrr_at_k(shifted, ex, 20) - 1 / 4) < 1e-15
    assert oracle.hit_at_k(shifted, ex, 3) == 0.0 and oracle.hit_at_k(shifted, ex, 4) == 1.0


def test_search_masks_equal_subset_search():
    """A per-query position mask (deleted vectors, slot allowlists) gives the
    search over the masked subset, with ids mapped back."""
    rng = np.random.default_rng(31)
    d = 64
    cb = oracle.lloyd_max(d, 4)
    R = oracle.haar_rotation(d, 3)[1]
    X = rng.standard_normal((500, d)).astype(np.float32)
    codes, _, scales = oracle.encode(X, R, cb)
    Q = rng.standard_normal((3, d)).astype(np.float32)
    masks = [rng.random(500) < p for p in (0.5, 0.05, 0.0)]
    ids, sc = oracle.search(codes, scales, cb.cents, R, Q, 8, masks=masks)
    for b in range(3):
        sub = np.nonzero(masks[b])[0]
        si, ss = oracle.search(codes[sub], scales[sub], cb.cents, R, Q[b:b + 1], 8)
        valid = si[0] >= 0
        assert np.array_equal(ids[b][valid], sub[si[0][valid]])
        assert np.array_equal(ids[b][~valid], si[0][~valid])
        # the subset's matrix product may sum in another order: last-bit differences
        assert np.allclose(sc[b], ss[0], rtol=1e-12, atol=0)
    assert np.all(ids[2] == -1)


def test_postfilter_baseline():
    """The over-fetch post-filter of section V-C: with every tenant allowed
    it is the plain search; on a hand-made case it keeps, in rank order, the
    allowed vectors of the over-fetched list only."""
    rng = np.random.default_rng(41)
    d = 64
    cb = oracle.lloyd_max(d, 4)
    R = oracle.haar_rotation(d, 3)[1]
    X = rng.standard_normal((400, d)).astype(np.float32)
    codes, _, scales = oracle.encode(X, R, cb)
    Q = rng.standard_normal((4, d)).astype(np.float32)
    ten = (np.arange(400) % 4).astype(np.uint16)
    everyone = np.full((4, 1), 0b1111, dtype=np.uint64)
    a_i, a_s = oracle.postfilter_search(codes, scales, cb.cents, R, Q, 5, 3, ten, everyone)
    b_i, b_s = oracle.search(codes, scales, cb.cents, R, Q, 5)
    assert np.array_equal(a_i, b_i) and np.array_equal(a_s, b_s)
    # tenant 2 only, over-fetch 3: the tenant-2 members of the top 15, first 5
    only2 = np.full((4, 1), 0b0100, dtype=np.uint64)
    p_i, _ = oracle.postfilter_search(codes, scales, cb.cents, R, Q, 5, 3, ten, only2)
    top15, _ = oracle.search(codes, scales, cb.cents, R, Q, 15)
    for b in range(4):
        want = [i for i in top15[b] if ten[i] == 2][:5]
        assert list(p_i[b][:len(want)]) == want and np.all(p_i[b][len(want):] == -1)
    # an over-fetch that covers the corpus gives the filtered search
    f_i, _ = oracle.postfilter_search(codes, scales, cb.cents, R, Q, 5, 80, ten, only2)
    g_i, _ = oracle.search(codes, scales, cb.cents, R, Q, 5, ten, only2)
    assert np.array_equal(f_i, g_i)


def test_topk_from_scores_brute_force_with_ties():
    """Selection on score rows full of ties (small integers) equals Python's
    sort by (score desc, id asc) over the eligible ids, for k below, at and
    above the number of eligible vectors."""
    rng = np.random.default_rng(5)
    sc = rng.integers(0, 6, (7, 40)).astype(np.float64)
    masks = [None] + [rng.random(40) < p for p in (0.9, 0.5, 0.2, 0.05, 0.0, 1.0)]
    for k in (1, 3, 8, 40, 50):
        ids, out = oracle.topk_from_scores(sc, k, masks=masks)
        for b in range(7):
            elig = [i for i in range(40) if masks[b] is None or masks[b][i]]
            ref = sorted(elig, key=lambda i: (-sc[b, i], i))[:k]
            n = len(ref)
            assert ids[b, :n].tolist() == ref
            assert np.array_equal(out[b, :n], sc[b, ref])
            assert np.all(ids[b, n:] == -1) and np.all(np.isneginf(out[b, n:]))
