"""GPU parity of the batched matrix-core search path (TQ_PATH_MFMA) against
the oracle and against the single-query path on the small workload.

The batched path selects 256 candidates per query (512 for k > 64) from
float16 matrix-core scores -- through per-block score maxima when there is
no filter -- and rescores them with the single-query path's integer tables,
so a returned (id, score) pair carries exactly the score the single-query
path gives that id; a certificate proves the exact top k is among the
candidates, and queries without one are re-run on the single-query path."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available
from tests.parity import check_topk, check_topk_sampled, oracle_tables

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402

D = 1536


@pytest.fixture(scope="module")
def env(small_env):
    return small_env


def same_as_lut(idx, Q, k, mi, ms, allow=None):
    """Every id the batched path returns carries the single-query path's
    score for it, and both lists agree up to swaps of equal scores."""
    li, ls = idx.search(Q, k, allow=allow, path="lut")
    li, ls, mi, ms = (t.cpu().numpy() for t in (li, ls, mi, ms))
    for b in range(Q.shape[0]):
        assert np.array_equal(np.sort(ls[b]), np.sort(ms[b])), b
        tied = np.isin(ms[b], ms[b][np.isin(mi[b], li[b], invert=True)])
        assert np.all(np.isin(mi[b], li[b]) | tied), b


@pytest.mark.parametrize("k", [10, 1, 64, 100, 256])
def test_batched_matches_oracle_and_lut(env, k):
    print("mfma k=%d" % k, flush=True)
    ids, sc = env.idx.search(env.Qd, k, path="mfma")
    fb = tq.last_search_fallbacks()
    ref_i, ref_s = oracle.search(env.codes, env.scales, env.ocb.cents, env.R32, env.Q, k)
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents,
               env.qrot, env.qn, k, ref_i, ref_s)
    same_as_lut(env.idx, env.Qd, k, ids, sc)
    print("fallbacks %d of %d" % (fb, env.Q.shape[0]), flush=True)
    if k == 10:
        # the certificate should hold for nearly every query of this workload
        assert fb <= env.Q.shape[0] // 4


@pytest.mark.parametrize("nq", [1, 15, 45])
def test_ragged_query_counts(env, nq):
    Q = env.Qd[:nq].contiguous()
    ids, sc = env.idx.search(Q, 10, path="mfma")
    ref_i, ref_s = oracle.search(env.codes, env.scales, env.ocb.cents, env.R32, env.Q[:nq], 10)
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents,
               env.qrot[:nq], env.qn[:nq], 10, ref_i, ref_s)


def test_ragged_index_and_filter(env):
    """n not a multiple of 64 (or of 512), with a selective tenant filter."""
    n = 5000 + 37
    T = 100
    tenants = synth.zipf_tenants(n, T, seed=44)
    allowed = synth.allowlists(env.Q.shape[0], T, "broad", seed=45)
    bm = synth.allowlist_bitmap(allowed, T)
    idx = tq.Index(env.cb, env.rot, n_tenants=T)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(env.codes[:n], 4)).cuda(),
                  torch.from_numpy(env.scales[:n]).cuda(),
                  torch.from_numpy(tenants.view(np.int16)).cuda())
    allow_d = torch.from_numpy(bm.view(np.int64)).cuda()
    ids, sc = idx.search(env.Qd, 10, allow=allow_d, path="mfma")
    ref_i, ref_s = oracle.search(env.codes[:n], env.scales[:n], env.ocb.cents, env.R32, env.Q, 10,
                                 tenants, bm)
    masks = [oracle.allowed_mask(tenants, bm[b]) for b in range(env.Q.shape[0])]
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes[:n], env.scales[:n],
               env.ocb.cents, env.qrot, env.qn, 10, ref_i, ref_s, allowed=masks, n=n)
    same_as_lut(idx, env.Qd, 10, ids, sc, allow=allow_d)


def test_ragged_index_unfiltered(env):
    """Block-maximum selection with a partial last block (n = 5037)."""
    n = 5000 + 37
    idx = tq.Index(env.cb, env.rot, n_tenants=1)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(env.codes[:n], 4)).cuda(),
                  torch.from_numpy(env.scales[:n]).cuda())
    for k in (10, 100):
        ids, sc = idx.search(env.Qd, k, path="mfma")
        ref_i, ref_s = oracle.search(env.codes[:n], env.scales[:n], env.ocb.cents, env.R32, env.Q, k)
        check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes[:n], env.scales[:n],
                   env.ocb.cents, env.qrot, env.qn, k, ref_i, ref_s, n=n)
        same_as_lut(idx, env.Qd, k, ids, sc)


@pytest.mark.parametrize("k", [10, 100])
def test_more_blocks_than_candidates(env, k):
    """40,037 vectors (626 blocks): more blocks than the 256 or 512
    candidates, so the selection goes through the block-maximum threshold."""
    print("mfma n=40037 k=%d" % k, flush=True)
    X = synth.isotropic_mixture(40_037, D, seed=48)
    idx = tq.Index(env.cb, env.rot, n_tenants=1)
    idx.add(torch.from_numpy(X).cuda())
    Q = env.Q[:32].copy()
    Qd = torch.from_numpy(Q).cuda()
    ids, sc = idx.search(Qd, k, path="mfma")
    print("fallbacks %d of 32" % tq.last_search_fallbacks(), flush=True)
    same_as_lut(idx, Qd, k, ids, sc)
    # every vector of the corpus is scored by the oracle (the "sample" is all rows)
    check_topk_sampled(ids.cpu().numpy(), sc.cpu().numpy(), X, env.R32, env.ocb, Q, k,
                       np.arange(X.shape[0]))


def test_filtered_large_k(env):
    """k = 100 with a tenant filter: 512 candidates from the filtered selection."""
    T = 10
    n = env.X.shape[0]
    tenants = synth.zipf_tenants(n, T, seed=44)
    bm = synth.allowlist_bitmap(synth.allowlists(env.Q.shape[0], T, "selective", seed=45), T)
    idx = tq.Index(env.cb, env.rot, n_tenants=T)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(env.codes, 4)).cuda(),
                  torch.from_numpy(env.scales).cuda(), torch.from_numpy(tenants.view(np.int16)).cuda())
    allow_d = torch.from_numpy(bm.view(np.int64)).cuda()
    ids, sc = idx.search(env.Qd, 100, allow=allow_d, path="mfma")
    ref_i, ref_s = oracle.search(env.codes, env.scales, env.ocb.cents, env.R32, env.Q, 100, tenants, bm)
    masks = [oracle.allowed_mask(tenants, bm[b]) for b in range(env.Q.shape[0])]
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents,
               env.qrot, env.qn, 100, ref_i, ref_s, allowed=masks)
    same_as_lut(idx, env.Qd, 100, ids, sc, allow=allow_d)


def test_many_tied_blocks_fall_back(env):
    """600,000 copies of one vector: every block maximum ties, more blocks
    reach the threshold than a query's selection lists, and every query is
    re-run on the single-query path (ties resolved by the lowest ids)."""
    n = 600_000
    one = oracle.pack_codes(env.codes[:1], 4)
    idx = tq.Index(env.cb, env.rot, n_tenants=1)
    idx.add_codes(torch.from_numpy(one).cuda().expand(n, -1).contiguous(),
                  torch.from_numpy(env.scales[:1]).cuda().expand(n).contiguous())
    Q = env.Qd[:4].contiguous()
    ids, sc = idx.search(Q, 10, path="mfma")
    assert tq.last_search_fallbacks() == 4
    li, ls = idx.search(Q, 10, path="lut")
    assert torch.equal(ids, li) and torch.equal(sc, ls)
    assert np.array_equal(ids.cpu().numpy()[0], np.arange(10))


def test_certificate_failure_falls_back(env):
    """400 copies of one vector (more than the 256 candidates) tie every
    score: no certificate can hold, so every query is re-run on the
    single-query path."""
    n = 400
    pk = torch.from_numpy(oracle.pack_codes(np.repeat(env.codes[:1], n, axis=0), 4)).cuda()
    sc0 = torch.from_numpy(np.repeat(env.scales[:1], n)).cuda()
    idx = tq.Index(env.cb, env.rot, n_tenants=1)
    idx.add_codes(pk, sc0)
    Q = env.Qd[:8].contiguous()
    ids, sc = idx.search(Q, 10, path="mfma")
    assert tq.last_search_fallbacks() == 8
    li, ls = idx.search(Q, 10, path="lut")
    assert torch.equal(ids, li) and torch.equal(sc, ls)
    assert np.array_equal(ids.cpu().numpy()[0], np.arange(10))   # ties: lowest ids


def test_largest_dimension():
    """d = 1792, the largest dimension whose query tile fits in LDS, against
    the single-query path and the oracle."""
    d = 1792
    X = synth.isotropic_mixture(3000, d, seed=50)
    Q = synth.isotropic_queries(X, 16, seed=51)
    cb, rot = tq.Codebook(d, 4), tq.Rotation(d, 7)
    idx = tq.Index(cb, rot, n_tenants=1)
    idx.add(torch.from_numpy(X).cuda())
    Qd = torch.from_numpy(Q).cuda()
    ids, sc = idx.search(Qd, 10, path="mfma")
    same_as_lut(idx, Qd, 10, ids, sc)
    check_topk_sampled(ids.cpu().numpy(), sc.cpu().numpy(), X, rot.matrix(), oracle_tables(cb),
                       Q, 10, np.arange(X.shape[0]))


def test_unsupported_shapes_rejected(env):
    with pytest.raises(tq.TQError, match="TQ_EUNSUPPORTED"):
        env.idx.search(env.Qd, 257, path="mfma")
    many = tq.Index(env.cb, env.rot, n_tenants=4097)   # 65 allowlist words
    many.add_codes(torch.from_numpy(oracle.pack_codes(env.codes[:100], 4)).cuda(),
                   torch.from_numpy(env.scales[:100]).cuda())
    with pytest.raises(tq.TQError, match="TQ_EUNSUPPORTED"):
        many.search(env.Qd, 10, path="mfma")
    cb2 = tq.Codebook(D, 2)
    idx = tq.Index(cb2, env.rot, n_tenants=1)
    idx.add(env.Xd[:100].contiguous())
    with pytest.raises(tq.TQError, match="TQ_EUNSUPPORTED"):
        idx.search(env.Qd, 10, path="mfma")
