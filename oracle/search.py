"""Query rotation, scoring, allowlist filter, top-k and recall (oracle; test use only).

* Query (section II-B step 2): q' = R32 q in float64.  The query is not
  normalised -- ranking does not depend on its length and the score then
  estimates <q, x>.
* Score (section II-B step 5, length-renormalised scoring):
      score_i = s_i * sum_j c[code_ij] * q'_j            (float64)
* Filter (section III-B): a vector is eligible for query q iff the bit of its
  tenant is set in q's allowlist bitmap (tenant t is bit t & 63 of 64-bit word
  t >> 6).  Only eligible vectors are scored; the GPU's per-block summaries are
  an optimisation with no counterpart here.
* Top-k (section III-B, heap insert): eligible vectors ordered by
  (score descending, id ascending), the first min(k, #eligible) kept, the rest
  of the k slots padded with id -1 and score -inf.
* Exact ground truth (section IV-A): the same ordering of <q, x_i> computed in
  float64 on the original float32 vectors; Recall@k = |approx & exact| /
  min(k, #eligible), averaged over queries.
"""
from __future__ import annotations

import numpy as np


def rotate_queries(R32: np.ndarray, Q: np.ndarray) -> np.ndarray:
    """q'_b = R32 q_b for every row of Q, float64."""
    R = np.asarray(R32, dtype=np.float32).astype(np.float64)
    Q = np.atleast_2d(np.asarray(Q, dtype=np.float32)).astype(np.float64)
    return Q @ R.T


def allowed_mask(tenants, allow_row) -> np.ndarray:
    """Eligibility of every vector for one query's allowlist (None -> all)."""
    if allow_row is None or tenants is None:
        return None
    t = np.asarray(tenants, dtype=np.int64)
    words = np.asarray(allow_row, dtype=np.uint64)
    w = t >> 6
    if np.any(w >= words.shape[0]):
        raise ValueError("tenant id beyond the allowlist")
    return ((words[w] >> (t & 63).astype(np.uint64)) & np.uint64(1)).astype(bool)


def _reconstruct(codes, cents, calib):
    """Rotated-domain reconstruction of coded rows: c[code_j], or with TQ+
    calibration (mu, kappa) (section II-B) mu_j + kappa_j c[code_j]."""
    xhat = np.asarray(cents, dtype=np.float64)[codes]
    if calib is not None:
        mu = np.asarray(calib[0], dtype=np.float32).astype(np.float64)
        kappa = np.asarray(calib[1], dtype=np.float32).astype(np.float64)
        xhat = mu + kappa * xhat
    return xhat


def scores_for_ids(codes: np.ndarray, scales: np.ndarray, cents: np.ndarray,
                   qrot: np.ndarray, ids, calib=None) -> np.ndarray:
    """score_i for the given vector ids against one rotated query (float64);
    calib: TQ+ (mu, kappa) or None."""
    ids = np.asarray(ids, dtype=np.int64)
    xhat = _reconstruct(codes[ids], cents, calib)
    return np.asarray(scales, dtype=np.float64)[ids] * (xhat @ qrot)


def _order(scores: np.ndarray, ids: np.ndarray, k: int):
    """(score desc, id asc) ordering, first k."""
    o = np.lexsort((ids, -scores))[:k]
    return ids[o], scores[o]


def _pad(ids, sc, k):
    out_i = np.full(k, -1, dtype=np.int64)
    out_s = np.full(k, -np.inf, dtype=np.float64)
    out_i[: len(ids)] = ids
    out_s[: len(sc)] = sc
    return out_i, out_s


def score_all(codes: np.ndarray, scales: np.ndarray, cents: np.ndarray, qrot: np.ndarray,
              chunk: int = 65536, calib=None) -> np.ndarray:
    """score_i of every vector against every rotated query (section II-B step
    5), float64 [nq, n]; qrot float64 [nq, d] from rotate_queries.  The rows
    are dequantised a chunk at a time; calib: TQ+ (mu, kappa) or None."""
    qrot = np.atleast_2d(np.asarray(qrot, dtype=np.float64))
    nq = qrot.shape[0]
    n = codes.shape[0]
    cents = np.asarray(cents, dtype=np.float64)
    sc_all = np.empty((nq, n), dtype=np.float64)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        xhat = _reconstruct(codes[s:e], cents, calib)    # [m, d]
        sc_all[:, s:e] = (xhat @ qrot.T).T * np.asarray(scales[s:e], dtype=np.float64)[None, :]
    return sc_all


def topk_from_scores(sc_all: np.ndarray, k: int, tenants=None, allow=None, masks=None):
    """Top-k of every query's row of scores (section III-B): the eligible
    vectors ordered by (score descending, id ascending), the first
    min(k, #eligible) kept and the rest padded with (-1, -inf).  A vector is
    eligible for query b when its tenant's bit is set in allow[b] (if given)
    and masks[b][i] is true (if given)."""
    if k <= 0:
        raise ValueError("k must be positive")
    nq, n = sc_all.shape
    ids_out = np.empty((nq, k), dtype=np.int64)
    sc_out = np.empty((nq, k), dtype=np.float64)
    all_ids = np.arange(n, dtype=np.int64)
    for b in range(nq):
        m = allowed_mask(tenants, None if allow is None else allow[b])
        if masks is not None and masks[b] is not None:
            mb = np.asarray(masks[b], dtype=bool)
            m = mb if m is None else (m & mb)
        ids = all_ids if m is None else all_ids[m]
        sc = sc_all[b] if m is None else sc_all[b][m]
        if sc.shape[0] > k:
            # only vectors scoring at least the k-th largest score can be
            # among the first k (ties at that score included); the order
            # below then decides among them
            kth = np.partition(sc, sc.shape[0] - k)[sc.shape[0] - k]
            keep = sc >= kth
            ids, sc = ids[keep], sc[keep]
        i, s_ = _order(sc, ids, k)
        ids_out[b], sc_out[b] = _pad(i, s_, k)
    return ids_out, sc_out


def search(codes: np.ndarray, scales: np.ndarray, cents: np.ndarray,
           R32: np.ndarray, Q: np.ndarray, k: int, tenants=None, allow=None,
           chunk: int = 65536, masks=None, calib=None):
    """Top-k over TurboQuant codes for every query.  Returns (ids int64 [nq,k],
    scores float64 [nq,k]).  The eligible vectors of query b are those whose
    tenant the allowlist row allow[b] admits (section III-B) and, when masks
    is given, those with masks[b][i] true: a per-query set of allowed
    positions (slot-level allowlists, and the vectors of an id-map index not
    deleted, section III-A).  calib: TQ+ calibration (mu, kappa), section
    II-B, or None."""
    if k <= 0:
        raise ValueError("k must be positive")
    sc_all = score_all(codes, scales, cents, rotate_queries(R32, Q), chunk=chunk, calib=calib)
    return topk_from_scores(sc_all, k, tenants, allow, masks)


def exact_search(X: np.ndarray, Q: np.ndarray, k: int, tenants=None, allow=None,
                 chunk: int = 65536):
    """Brute-force exact inner-product top-k (float64 on float32 inputs)."""
    Q64 = np.atleast_2d(np.asarray(Q, dtype=np.float32)).astype(np.float64)
    n = X.shape[0]
    nq = Q64.shape[0]
    sc_all = np.empty((nq, n), dtype=np.float64)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        sc_all[:, s:e] = Q64 @ np.asarray(X[s:e], dtype=np.float32).astype(np.float64).T
    ids_out = np.empty((nq, k), dtype=np.int64)
    sc_out = np.empty((nq, k), dtype=np.float64)
    all_ids = np.arange(n, dtype=np.int64)
    for b in range(nq):
        m = allowed_mask(tenants, None if allow is None else allow[b])
        ids = all_ids if m is None else all_ids[m]
        sc = sc_all[b] if m is None else sc_all[b][m]
        i, s_ = _order(sc, ids, k)
        ids_out[b], sc_out[b] = _pad(i, s_, k)
    return ids_out, sc_out


def recall_at_k(approx_ids: np.ndarray, exact_ids: np.ndarray, k: int) -> float:
    """Mean over queries of |approx & exact| / min(k, #eligible) (section IV-A;
    #eligible is read off the exact list's padding)."""
    approx_ids = np.atleast_2d(approx_ids)[:, :k]
    exact_ids = np.atleast_2d(exact_ids)[:, :k]
    vals = []
    for a, e in zip(approx_ids, exact_ids):
        e_set = set(int(v) for v in e if v >= 0)
        if not e_set:
            continue
        a_set = set(int(v) for v in a if v >= 0)
        vals.append(len(a_set & e_set) / len(e_set))
    return float(np.mean(vals)) if vals else float("nan")


def _rank_of_top1(approx_row, top1, k):
    """1-based position of top1 among the first k approximate ids, or 0."""
    for r, v in enumerate(approx_row[:k]):
        if int(v) == int(top1):
            return r + 1
    return 0


def hit_at_k(approx_ids: np.ndarray, exact_ids: np.ndarray, k: int) -> float:
    """Hit@k of section IV-E: the fraction of queries whose exact top-1 id is
    among the first k approximate ids.  exact_ids: [nq, >=1], column 0 the
    exact best (queries with no eligible vector, id -1, are skipped)."""
    approx_ids = np.atleast_2d(approx_ids)
    exact_ids = np.atleast_2d(exact_ids)
    vals = [1.0 if _rank_of_top1(a, e[0], k) > 0 else 0.0
            for a, e in zip(approx_ids, exact_ids) if e[0] >= 0]
    return float(np.mean(vals)) if vals else float("nan")


def mrr_at_k(approx_ids: np.ndarray, exact_ids: np.ndarray, k: int = 20) -> float:
    """MRR@k of section IV-E: the mean over queries of 1 / rank of the exact
    top-1 id in the approximate list, counting 0 when it is not among the
    first k (the paper reports k = 20)."""
    approx_ids = np.atleast_2d(approx_ids)
    exact_ids = np.atleast_2d(exact_ids)
    vals = []
    for a, e in zip(approx_ids, exact_ids):
        if e[0] < 0:
            continue
        r = _rank_of_top1(a, e[0], k)
        vals.append(1.0 / r if r else 0.0)
    return float(np.mean(vals)) if vals else float("nan")


def postfilter_search(codes: np.ndarray, scales: np.ndarray, cents: np.ndarray,
                      R32: np.ndarray, Q: np.ndarray, k: int, overfetch: int, tenants,
                      allow, masks=None, calib=None):
    """The over-fetch post-filter baseline of section V-C: the unfiltered top
    k * overfetch of each query (over the vectors in masks, if given), then,
    in that order, the first k whose tenant the query's allowlist admits.
    Returns (ids int64 [nq,k], scores float64 [nq,k]), padded with (-1, -inf)."""
    ids, sc = search(codes, scales, cents, R32, Q, k * overfetch, masks=masks, calib=calib)
    out_i = np.full((ids.shape[0], k), -1, dtype=np.int64)
    out_s = np.full((ids.shape[0], k), -np.inf, dtype=np.float64)
    for b in range(ids.shape[0]):
        m = allowed_mask(tenants, allow[b])
        kept = [(i, v) for i, v in zip(ids[b], sc[b]) if i >= 0 and m[i]][:k]
        for r, (i, v) in enumerate(kept):
            out_i[b, r], out_s[b, r] = i, v
    return out_i, out_s
