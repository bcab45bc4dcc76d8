"""Comparison helpers shared by the GPU parity tests (no method arithmetic:
scores and rankings come from the oracle)."""
from __future__ import annotations

import numpy as np

import oracle

SCORE_RTOL = 1e-4          # relative tolerance on scores
SCORE_ATOL_Q = 1e-6        # absolute floor, times ||q||


def oracle_tables(cb) -> "oracle.Codebook":
    """The library's exported boundaries and centroids (tq.Codebook) as an
    oracle Codebook.  The encode definition (section II-B steps 1-4) takes
    the rotation and the tables as parameters: parity tests give the oracle
    exactly the parameters the kernels use (the library's float32 R from
    Rotation.matrix() and these tables), so the codes must agree bit for bit.
    That the library's tables and rotation agree with the oracle's own solve
    and factorisation is a separate host test (tests/test_lib_host.py)."""
    bounds = np.array(cb.bounds, dtype=np.float64)
    cents = np.array(cb.cents, dtype=np.float64)
    bounds.setflags(write=False)
    cents.setflags(write=False)
    return oracle.Codebook(d=cb.d, bits=cb.bits, bounds=bounds, cents=cents, iterations=0,
                           converged=True)


def assert_codes_equal(codes_gpu_packed, codes_or, bits):
    """Packed GPU codes equal to the oracle's unpacked codes, bit for bit;
    on failure the message names the first differing (row, coordinate)."""
    d = codes_or.shape[1]
    got = oracle.unpack_codes(np.asarray(codes_gpu_packed), d, bits)
    bad = np.argwhere(got != codes_or)
    assert bad.size == 0, ("code mismatches", len(bad), bad[:5].tolist())
    assert np.array_equal(np.asarray(codes_gpu_packed), oracle.pack_codes(codes_or, bits))


def assert_scales_close(scales_gpu, scales_or, max_ulp=1):
    """float32 scales within max_ulp units in the last place of the oracle's
    float64 value rounded to float32 (the library sums the squared levels in
    another order)."""
    a = np.asarray(scales_gpu, dtype=np.float32).view(np.int32).astype(np.int64)
    b = np.asarray(scales_or, dtype=np.float32).view(np.int32).astype(np.int64)
    if a.size:
        assert np.abs(a - b).max() <= max_ulp, int(np.abs(a - b).max())


def score_tol(ref, qnorm):
    return np.maximum(SCORE_RTOL * np.abs(ref), SCORE_ATOL_Q * qnorm)


def check_topk(gpu_ids, gpu_scores, codes, scales, cents, qrot, qnorms, k,
               ref_ids, ref_scores, allowed=None, n=None, calib=None):
    """Validity of GPU top-k lists against the oracle (see module docstring of
    tests/test_gpu_search.py).  `allowed` is a list of boolean masks (or None);
    `ref_*` are the oracle's own lists.  Returns the number of id lists that
    differ from the oracle's (ties within tolerance)."""
    gpu_ids = np.asarray(gpu_ids)
    gpu_scores = np.asarray(gpu_scores, dtype=np.float64)
    n = codes.shape[0] if n is None else n
    differ = 0
    for b in range(gpu_ids.shape[0]):
        ids = gpu_ids[b]
        valid = ids >= 0
        nv = int(valid.sum())
        n_allowed = n if allowed is None or allowed[b] is None else int(allowed[b].sum())
        assert nv == min(k, n_allowed), (b, nv, min(k, n_allowed))
        assert np.all(valid[:nv]) and not np.any(valid[nv:]), "padding must be at the end"
        assert np.all(np.isneginf(gpu_scores[b][nv:]))
        v = ids[:nv]
        assert len(set(v.tolist())) == nv, "duplicate ids"
        assert np.all(v < n)
        if allowed is not None and allowed[b] is not None:
            assert np.all(allowed[b][v]), "disallowed id returned"
        if nv == 0:
            continue
        ref = oracle.scores_for_ids(codes, scales, cents, qrot[b], v, calib=calib)
        tol = score_tol(ref, qnorms[b])
        err = np.abs(gpu_scores[b][:nv] - ref)
        assert np.all(err <= tol), (b, float((err / tol).max()))
        # ordered (within tolerance)
        assert np.all(np.diff(ref) <= 2 * tol[1:] + 1e-12), "not ordered"
        # nothing better was missed: the worst returned is at least the
        # oracle's nv-th best, within tolerance
        kth = ref_scores[b][nv - 1]
        assert ref.min() >= kth - score_tol(np.array([kth]), qnorms[b])[0]
        if not np.array_equal(v, ref_ids[b][:nv]):
            differ += 1
    return differ


def check_topk_sampled(gpu_ids, gpu_scores, X, R32, cb, Q, k, sample, allowed=None):
    """Validity of GPU top-k lists over a corpus too large for the oracle's
    full search.  The oracle encodes the returned vectors and a random sample
    of the corpus from the float rows X; then every returned score must match
    the oracle's score for its id, the lists must be ordered, distinct,
    allowed and full, and no sampled vector outside a list may beat its worst
    entry by more than the tolerance.  `allowed`: boolean mask over the
    corpus per query, or None."""
    gpu_ids = np.asarray(gpu_ids)
    gpu_scores = np.asarray(gpu_scores, dtype=np.float64)
    n = X.shape[0]
    rows = np.unique(np.concatenate([gpu_ids[gpu_ids >= 0].ravel(), np.asarray(sample)]))
    codes, _, scales = oracle.encode(np.ascontiguousarray(X[rows]), R32, cb)
    pos = {int(r): i for i, r in enumerate(rows)}
    qrot = oracle.rotate_queries(R32, Q)
    qn = np.linalg.norm(Q.astype(np.float64), axis=1)
    for b in range(gpu_ids.shape[0]):
        ids = gpu_ids[b]
        mask = None if allowed is None else allowed[b]
        n_allowed = n if mask is None else int(mask.sum())
        nv = int((ids >= 0).sum())
        assert nv == min(k, n_allowed), (b, nv)
        assert np.all(ids[:nv] >= 0) and np.all(ids[nv:] == -1)
        v = ids[:nv]
        assert len(set(v.tolist())) == nv, "duplicate ids"
        if mask is not None:
            assert np.all(mask[v]), "disallowed id returned"
        ref = oracle.scores_for_ids(codes, scales, cb.cents, qrot[b], [pos[int(i)] for i in v])
        tol = score_tol(ref, qn[b])
        assert np.all(np.abs(gpu_scores[b][:nv] - ref) <= tol), (b, float((np.abs(gpu_scores[b][:nv] - ref) / tol).max()))
        assert np.all(np.diff(ref) <= 2 * tol[1:] + 1e-12), "not ordered"
        s = np.setdiff1d(np.asarray(sample), v)
        if mask is not None:
            s = s[mask[s]]
        if s.size and nv == k:
            others = oracle.scores_for_ids(codes, scales, cb.cents, qrot[b], [pos[int(i)] for i in s])
            worst = ref.min()
            assert others.max() <= worst + score_tol(np.array([worst]), qn[b])[0], \
                (b, float(others.max()), float(worst))
