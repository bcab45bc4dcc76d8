"""GPU parity of the batched matrix-core path in passes of 65 to 256 queries
(one pass over the code store per pass, no score matrix: a pilot launch
scores every vector of some tiles, the KC-th best allowed pilot score per
query is its threshold, the main launch keeps only vectors that reach it,
then the KC best candidates are rescored exactly and certified).

Against the oracle's brute force over the whole corpus (section II-B step 5
scores, section IV-A ground truth) and against the single-query path's
scores for the same ids:

* the 10,000-row workload, where every tile is a pilot tile, in passes of
  65, 100, 200 and 300 (a pass of 256, then 44 queries in tiles of 32) at
  k = 10 and 100;
* a 70,037-row corpus (274 tiles: pilot and main launches both work, the
  last block is partial) in passes of 65, 128 and 256 queries, k = 10 and
  100, and filtered by Zipf tenants (section V-C), selective and broad;
* forced failures (all scores tied) in a pass of 64 queries, re-run on the
  single-query path."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available
from tests.parity import check_topk, oracle_tables

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402

D = 1536


def same_as_lut(idx, Q, k, mi, ms, allow=None):
    """Every id the batched path returns carries the single-query path's
    score for it, and both lists agree up to swaps of equal scores."""
    li, ls = idx.search(Q, k, allow=allow, path="lut")
    li, ls, mi, ms = (t.cpu().numpy() for t in (li, ls, mi, ms))
    for b in range(Q.shape[0]):
        assert np.array_equal(np.sort(ls[b]), np.sort(ms[b])), b
        tied = np.isin(ms[b], ms[b][np.isin(mi[b], li[b], invert=True)])
        assert np.all(np.isin(mi[b], li[b]) | tied), b


class Corpus:
    pass


def _corpus(X, Q, rot, cb):
    c = Corpus()
    c.X, c.Q, c.cb, c.rot = X, Q, cb, rot
    c.R32 = rot.matrix()
    c.ocb = oracle_tables(cb)
    c.codes, _, c.scales = oracle.encode(X, c.R32, c.ocb)
    c.qrot = oracle.rotate_queries(c.R32, Q)
    c.qn = np.linalg.norm(Q.astype(np.float64), axis=1)
    c.scores = oracle.score_all(c.codes, c.scales, c.ocb.cents, c.qrot)
    c.idx = tq.Index(cb, rot, n_tenants=1)
    c.idx.add(torch.from_numpy(X).cuda())
    c.Qd = torch.from_numpy(Q).cuda()
    return c


@pytest.fixture(scope="module")
def small(small_env):
    e = small_env
    Q = synth.isotropic_queries(e.X, 300, seed=61)
    return _corpus(e.X, Q, e.rot, e.cb)


@pytest.fixture(scope="module")
def mid(small_env):
    X = synth.isotropic_mixture(70_037, D, seed=62)
    Q = synth.isotropic_queries(X, 256, seed=63)
    return _corpus(X, Q, small_env.rot, small_env.cb)


def _check(c, nq, k, ids, sc, tenants=None, bm=None):
    ref_i, ref_s = oracle.topk_from_scores(c.scores[:nq], k, tenants=tenants, allow=bm)
    masks = None if bm is None else [oracle.allowed_mask(tenants, bm[b]) for b in range(nq)]
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), c.codes, c.scales, c.ocb.cents, c.qrot[:nq],
               c.qn[:nq], k, ref_i, ref_s, allowed=masks)


@pytest.mark.parametrize("nq,k", [(65, 10), (100, 100), (200, 10), (300, 100), (300, 10)])
def test_all_pilot_passes(small, nq, k):
    print("wide small nq=%d k=%d" % (nq, k), flush=True)
    Q = small.Qd[:nq].contiguous()
    ids, sc = small.idx.search(Q, k, path="mfma")
    print("fallbacks %d" % tq.last_search_fallbacks(), flush=True)
    _check(small, nq, k, ids, sc)
    same_as_lut(small.idx, Q, k, ids, sc)


@pytest.mark.parametrize("nq,k", [(65, 10), (128, 10), (256, 10), (256, 100), (128, 100)])
def test_pilot_and_main_passes(mid, nq, k):
    print("wide mid nq=%d k=%d" % (nq, k), flush=True)
    Q = mid.Qd[:nq].contiguous()
    ids, sc = mid.idx.search(Q, k, path="mfma")
    fb = tq.last_search_fallbacks()
    print("fallbacks %d" % fb, flush=True)
    _check(mid, nq, k, ids, sc)
    same_as_lut(mid.idx, Q, k, ids, sc)
    assert fb <= nq // 8


@pytest.mark.parametrize("mode", ["selective", "broad"])
def test_filtered_pass(mid, mode):
    T, nq = 100, 96
    n = mid.X.shape[0]
    tenants = synth.zipf_tenants(n, T, seed=44)
    bm = synth.allowlist_bitmap(synth.allowlists(nq, T, mode, seed=45), T)
    idx = tq.Index(mid.cb, mid.rot, n_tenants=T)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(mid.codes, 4)).cuda(),
                  torch.from_numpy(mid.scales).cuda(), torch.from_numpy(tenants.view(np.int16)).cuda())
    allow_d = torch.from_numpy(bm.view(np.int64)).cuda()
    Q = mid.Qd[:nq].contiguous()
    for k in (10, 100):
        print("wide filtered %s k=%d" % (mode, k), flush=True)
        ids, sc = idx.search(Q, k, allow=allow_d, path="mfma")
        print("fallbacks %d" % tq.last_search_fallbacks(), flush=True)
        _check(mid, nq, k, ids, sc, tenants=tenants, bm=bm)
        same_as_lut(idx, Q, k, ids, sc, allow=allow_d)


def test_tied_scores_fall_back(small_env):
    """200,000 copies of one vector: every score ties, the pilot keeps more
    tied vectors than its candidate room and the main launch overflows its
    lists, so every query of the pass is re-run on the single-query path
    (ties resolved by the lowest ids)."""
    e = small_env
    n = 200_000
    one = oracle.pack_codes(e.codes[:1], 4)
    idx = tq.Index(e.cb, e.rot, n_tenants=1)
    idx.add_codes(torch.from_numpy(one).cuda().expand(n, -1).contiguous(),
                  torch.from_numpy(e.scales[:1]).cuda().expand(n).contiguous())
    Q = torch.cat([e.Qd, e.Qd[:16]]).contiguous()   # 80 queries: one wide pass
    ids, sc = idx.search(Q, 10, path="mfma")
    assert tq.last_search_fallbacks() == 80
    li, ls = idx.search(Q, 10, path="lut")
    assert torch.equal(ids, li) and torch.equal(sc, ls)
    assert np.array_equal(ids.cpu().numpy()[0], np.arange(10))


def test_few_vectors_every_one_a_candidate(small_env):
    """100 vectors and 80 queries at k = 10: fewer vectors than candidate
    slots, so every vector is a candidate and the result is certified
    without a threshold."""
    e = small_env
    idx = tq.Index(e.cb, e.rot, n_tenants=1)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(e.codes[:100], 4)).cuda(),
                  torch.from_numpy(e.scales[:100]).cuda())
    Q = np.concatenate([e.Q, e.Q[:16]])
    ids, sc = idx.search(torch.from_numpy(Q).cuda(), 10, path="mfma")
    assert tq.last_search_fallbacks() == 0
    ref_i, ref_s = oracle.search(e.codes[:100], e.scales[:100], e.ocb.cents, e.R32, Q, 10)
    qrot = oracle.rotate_queries(e.R32, Q)
    qn = np.linalg.norm(Q.astype(np.float64), axis=1)
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), e.codes[:100], e.scales[:100], e.ocb.cents,
               qrot, qn, 10, ref_i, ref_s, n=100)
