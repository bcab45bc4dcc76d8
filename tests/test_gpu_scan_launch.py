"""GPU parity of the single-query scan (section II-B step 5, section III-B)
across launch shapes: many queries in one launch (the scan keeps per-query
state across its query loop), results that must not depend on the other
queries of a launch, dimensions from 64 to 2048 at every bit width, with 1
to 6 eight-chunk groups per vector or chunk counts outside that scheme,
unfiltered and tenant-filtered, and exact agreement between the top-64 lists
of k = 64 and k = 65 (wave lists of one and of two 64-entry slots; both sum
the same integer table entries)."""
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


@pytest.fixture(scope="module")
def env(small_env):
    return small_env


def test_many_queries_per_launch(env):
    print("scan: 300 queries in one launch", flush=True)
    rng = np.random.default_rng(51)
    noisy = [env.Q + np.float32(0.01) * rng.standard_normal(env.Q.shape).astype(np.float32)
             for _ in range(4)]
    Q = np.ascontiguousarray(np.concatenate([env.Q] + noisy)[:300])
    Qd = torch.from_numpy(Q).cuda()
    ids, sc = env.idx.search(Qd, 10)
    ref_i, ref_s = oracle.search(env.codes, env.scales, env.ocb.cents, env.R32, Q, 10)
    qrot = oracle.rotate_queries(env.R32, Q)
    qn = np.linalg.norm(Q.astype(np.float64), axis=1)
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents, qrot,
               qn, 10, ref_i, ref_s)
    # a query's result does not depend on the other queries of its launch
    for lo, hi in [(0, 1), (0, 2), (1, 4), (150, 153), (299, 300)]:
        a_i, a_s = env.idx.search(Qd[lo:hi].contiguous(), 10)
        assert torch.equal(a_i, ids[lo:hi]) and torch.equal(a_s, sc[lo:hi]), (lo, hi)


def test_top64_of_k64_and_k65_agree(env):
    a_i, a_s = env.idx.search(env.Qd, 64)
    b_i, b_s = env.idx.search(env.Qd, 65)
    assert torch.equal(a_i, b_i[:, :64]) and torch.equal(a_s, b_s[:, :64])


# (d, b): code chunks per vector d*b/128, eight-chunk groups chunks/8.  The
# edges: the smallest d (64); chunk counts that are not a multiple of 8
# (d = 192 at b = 4, d = 64 at b = 2 and 8); the largest d (2048), whose
# 4-bit table no longer fits beside the split scan's other LDS regions.
# 3-bit codes (ten per word, chunks rounded up to a multiple of 4): d = 128
# (4 chunks) and 2048 (52 chunks, 2080 table rows) take the block-per-wave
# scan, d = 256 (8 chunks) and 1792 (48) the split scans.
@pytest.mark.parametrize("d,bits", [(256, 4), (1024, 4), (1280, 4), (512, 2), (1024, 1),
                                    (64, 4), (192, 4), (2048, 4), (2048, 8), (128, 3),
                                    (64, 2), (64, 8), (2048, 1), (256, 3), (1792, 3),
                                    (2048, 3)])
def test_other_dimensions(d, bits):
    print("scan d=%d b=%d" % (d, bits), flush=True)
    rng = np.random.default_rng(d + bits)
    n, nq = 3013, 24
    X = rng.standard_normal((n, d)).astype(np.float32)
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    Q = (X[:nq] + np.float32(0.05) * rng.standard_normal((nq, d)).astype(np.float32))
    Q = np.ascontiguousarray(Q.astype(np.float32))
    rot = tq.Rotation(d, 11)
    R32 = rot.matrix()
    cb = tq.Codebook(d, bits)
    ocb = oracle_tables(cb)
    codes, _, scales = oracle.encode(X, R32, ocb)
    tenants = rng.integers(0, 5, n).astype(np.uint16)
    idx = tq.Index(cb, rot, n_tenants=5)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(codes, bits)).cuda(),
                  torch.from_numpy(scales).cuda(),
                  torch.from_numpy(tenants.view(np.int16)).cuda())
    Qd = torch.from_numpy(Q).cuda()
    qrot = oracle.rotate_queries(R32, Q)
    qn = np.linalg.norm(Q.astype(np.float64), axis=1)
    for k in (10, 64):
        ids, sc = idx.search(Qd, k)
        ref_i, ref_s = oracle.search(codes, scales, ocb.cents, R32, Q, k)
        check_topk(ids.cpu().numpy(), sc.cpu().numpy(), codes, scales, ocb.cents, qrot, qn, k,
                   ref_i, ref_s)
    a_i, a_s = idx.search(Qd, 64)
    b_i, b_s = idx.search(Qd, 65)
    assert torch.equal(a_i, b_i[:, :64]) and torch.equal(a_s, b_s[:, :64])
    # one tenant of five per query
    bm = np.zeros((nq, 1), dtype=np.uint64)
    bm[:, 0] = np.left_shift(np.uint64(1), (np.arange(nq) % 5).astype(np.uint64))
    ids, sc = idx.search(Qd, 10, allow=torch.from_numpy(bm.view(np.int64)).cuda())
    ref_i, ref_s = oracle.search(codes, scales, ocb.cents, R32, Q, 10, tenants, bm)
    masks = [oracle.allowed_mask(tenants, bm[b]) for b in range(nq)]
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), codes, scales, ocb.cents, qrot, qn, 10,
               ref_i, ref_s, allowed=masks)


@pytest.mark.parametrize("grid", [1, 2])
def test_one_workgroup_share_spans_list_windows(monkeypatch, grid):
    """With one or two workgroups, each covers more than 4,096 blocks: the
    filtered scan lists its blocks in several windows and the unfiltered split
    scan runs over 64 passes per query.  Codes and scales are random (the scan
    does not depend on how they were made); d = 256, b = 4 takes the split
    scans (8 chunks per vector)."""
    d, bits, T, nq = 256, 4, 100, 6
    n = 2 * 4096 * 64 + 3 * 64 + 17
    print("scan grid=%d n=%d" % (grid, n), flush=True)
    rng = np.random.default_rng(77)
    codes = rng.integers(0, 16, size=(n, d), dtype=np.uint8)
    scales = rng.uniform(0.5, 1.5, n).astype(np.float32)
    tenants = synth.zipf_tenants(n, T, seed=78)
    rot = tq.Rotation(d, 5)
    R32 = rot.matrix()
    cb = tq.Codebook(d, bits)
    ocb = oracle_tables(cb)
    Q = rng.standard_normal((nq, d)).astype(np.float32)
    idx = tq.Index(cb, rot, n_tenants=T)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(codes, bits)).cuda(),
                  torch.from_numpy(scales).cuda(),
                  torch.from_numpy(tenants.view(np.int16)).cuda())
    Qd = torch.from_numpy(Q).cuda()
    qrot = oracle.rotate_queries(R32, Q)
    qn = np.linalg.norm(Q.astype(np.float64), axis=1)
    monkeypatch.setenv("TQ_SCAN_GRID", str(grid))
    for k in (10, 100):
        ids, sc = idx.search(Qd, k)
        ref_i, ref_s = oracle.search(codes, scales, ocb.cents, R32, Q, k)
        check_topk(ids.cpu().numpy(), sc.cpu().numpy(), codes, scales, ocb.cents, qrot, qn, k,
                   ref_i, ref_s)
    for mode in ("selective", "broad"):
        bm = synth.allowlist_bitmap(synth.allowlists(nq, T, mode, seed=79), T)
        ids, sc = idx.search(Qd, 10, allow=torch.from_numpy(bm.view(np.int64)).cuda())
        ref_i, ref_s = oracle.search(codes, scales, ocb.cents, R32, Q, 10, tenants, bm)
        masks = [oracle.allowed_mask(tenants, bm[b]) for b in range(nq)]
        check_topk(ids.cpu().numpy(), sc.cpu().numpy(), codes, scales, ocb.cents, qrot, qn, 10,
                   ref_i, ref_s, allowed=masks)
    monkeypatch.delenv("TQ_SCAN_GRID")
    # the default launch returns the same lists
    ids1, sc1 = idx.search(Qd, 100)
    monkeypatch.setenv("TQ_SCAN_GRID", str(grid))
    ids2, sc2 = idx.search(Qd, 100)
    assert torch.equal(ids1, ids2) and torch.equal(sc1, sc2)
