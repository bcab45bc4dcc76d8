"""GPU parity of the search path (section II-B step 5, section III-B) against
the oracle on the small workload (10,000 x 1536 isotropic mixture, 64 noisy
queries).

A GPU top-k list is valid when (1) its ids are distinct, allowed and padded
with -1 only after min(k, #allowed) entries; (2) every returned score is
within 1e-4 relative (floor 1e-6 ||q||) of the oracle's score for that id;
(3) the list is ordered; (4) no returned vector scores below the oracle's
k-th best minus the tolerance.  Ids may differ from the oracle's list only by
swaps between scores tied within the tolerance."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available
from tests.parity import (assert_codes_equal, assert_scales_close, check_topk,
                          oracle_tables)

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402

D = 1536


@pytest.fixture(scope="module")
def env(small_env):
    return small_env


def oracle_topk(s, k, tenants=None, allow=None, n=None):
    codes = s.codes if n is None else s.codes[:n]
    scales = s.scales if n is None else s.scales[:n]
    return oracle.search(codes, scales, s.ocb.cents, s.R32, s.Q, k, tenants, allow)


def test_index_holds_the_oracle_codes(env):
    codes, scales, tenants = env.idx.export()
    assert_codes_equal(codes.cpu().numpy(), env.codes, 4)
    assert_scales_close(scales.cpu().numpy(), env.scales)
    assert np.all(tenants.cpu().numpy() == 0)


@pytest.mark.parametrize("k", [10, 1, 5, 64, 100, 256])
def test_search_matches_oracle(env, k):
    print("search k=%d" % k, flush=True)
    ids, sc = env.idx.search(env.Qd, k)
    ref_i, ref_s = oracle_topk(env, k)
    differ = check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents,
                        env.qrot, env.qn, k, ref_i, ref_s)
    assert differ <= env.Q.shape[0] // 8


def test_search_deterministic_and_single_query(env):
    a_i, a_s = env.idx.search(env.Qd, 10)
    b_i, b_s = env.idx.search(env.Qd, 10)
    assert torch.equal(a_i, b_i) and torch.equal(a_s, b_s)
    c_i, c_s = env.idx.search(env.Qd[7:8].contiguous(), 10)
    assert torch.equal(c_i[0], a_i[7]) and torch.equal(c_s[0], a_s[7])
    d_i, d_s = env.idx.search_alloc(env.Qd, 10)
    assert torch.equal(d_i, a_i) and torch.equal(d_s, a_s)


def test_add_codes_path_and_ragged_sizes(env):
    """Index built from oracle codes (decoupled from the GPU encode), with a
    count that is not a multiple of 64 and k above it."""
    n = 1000 + 37
    idx = tq.Index(env.cb, env.rot, n_tenants=1)
    pk = torch.from_numpy(oracle.pack_codes(env.codes[:n], 4)).cuda()
    idx.add_codes(pk[:600].contiguous(), torch.from_numpy(env.scales[:600]).cuda())
    idx.add_codes(pk[600:].contiguous(), torch.from_numpy(env.scales[600:n]).cuda())
    assert len(idx) == n
    for k in (10, 256):
        ids, sc = idx.search(env.Qd, k)
        ref_i, ref_s = oracle_topk(env, k, n=n)
        check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes[:n], env.scales[:n],
                   env.ocb.cents, env.qrot, env.qn, k, ref_i, ref_s, n=n)
    tiny = tq.Index(env.cb, env.rot, n_tenants=1)
    tiny.add_codes(pk[:3].contiguous(), torch.from_numpy(env.scales[:3]).cuda())
    ids, sc = tiny.search(env.Qd[:2].contiguous(), 5)
    ids = ids.cpu().numpy()
    assert np.all(ids[:, 3:] == -1) and np.all(ids[:, :3] >= 0)
    empty = tq.Index(env.cb, env.rot, n_tenants=1)
    ids, sc = empty.search(env.Qd[:2].contiguous(), 4)
    assert np.all(ids.cpu().numpy() == -1) and torch.all(torch.isinf(sc))


@pytest.mark.parametrize("T,mode", [(10, "selective"), (100, "selective"), (1000, "selective"),
                                    (100, "broad"), (65535, "broad")])
def test_filtered_search(env, T, mode):
    print("filtered T=%d %s" % (T, mode), flush=True)
    n = env.X.shape[0]
    tenants = synth.zipf_tenants(n, T, seed=44)
    allowed = synth.allowlists(env.Q.shape[0], T, mode, seed=45)
    bm = synth.allowlist_bitmap(allowed, T)
    idx = tq.Index(env.cb, env.rot, n_tenants=T)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(env.codes, 4)).cuda(),
                  torch.from_numpy(env.scales).cuda(),
                  torch.from_numpy(tenants.view(np.int16)).cuda())
    allow_d = torch.from_numpy(bm.view(np.int64)).cuda()
    ids, sc = idx.search(env.Qd, 10, allow=allow_d)
    ref_i, ref_s = oracle_topk(env, 10, tenants, bm)
    masks = [oracle.allowed_mask(tenants, bm[b]) for b in range(env.Q.shape[0])]
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents,
               env.qrot, env.qn, 10, ref_i, ref_s, allowed=masks)
    # block skipping never changes results: an all-ones allowlist equals no filter
    ones = torch.full((env.Q.shape[0], idx.words), -1, dtype=torch.int64, device="cuda")
    a_i, a_s = idx.search(env.Qd, 10, allow=ones)
    b_i, b_s = idx.search(env.Qd, 10)
    assert torch.equal(a_i, b_i) and torch.equal(a_s, b_s)
    # an empty allowlist returns only padding
    zeros = torch.zeros((env.Q.shape[0], idx.words), dtype=torch.int64, device="cuda")
    z_i, _ = idx.search(env.Qd, 10, allow=zeros)
    assert torch.all(z_i == -1)


def test_bad_tenant_rejected(env):
    idx = tq.Index(env.cb, env.rot, n_tenants=5)
    t = torch.tensor([0, 1, 7], dtype=torch.int16, device="cuda")
    pk = torch.from_numpy(oracle.pack_codes(env.codes[:3], 4)).cuda()
    with pytest.raises(tq.TQError, match="TQ_EINVAL"):
        idx.add_codes(pk, torch.from_numpy(env.scales[:3]).cuda(), t)
    assert len(idx) == 0


@pytest.mark.parametrize("bits", [2, 8, 3, 1])
def test_other_bit_widths(env, bits):
    print("bits=%d search" % bits, flush=True)
    n = 2000
    cb = tq.Codebook(D, bits)
    ocb = oracle_tables(cb)
    codes, norms, scales = oracle.encode(env.X[:n], env.R32, ocb)
    idx = tq.Index(cb, env.rot, n_tenants=1)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(codes, bits)).cuda(),
                  torch.from_numpy(scales).cuda())
    ids, sc = idx.search(env.Qd, 10)
    ref_i, ref_s = oracle.search(codes, scales, ocb.cents, env.R32, env.Q, 10)
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), codes, scales, ocb.cents, env.qrot, env.qn,
               10, ref_i, ref_s)
    # the index built by the GPU encode holds the same codes
    idx2 = tq.Index(cb, env.rot, n_tenants=1)
    idx2.add(env.Xd[:n].contiguous())
    c2, s2, _ = idx2.export()
    assert_codes_equal(c2.cpu().numpy(), codes, bits)
    assert_scales_close(s2.cpu().numpy(), scales)
