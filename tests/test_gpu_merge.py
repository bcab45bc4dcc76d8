"""The final merge of the workgroup lists (section III-B top-k) when many list
entries tie: an index where every 5th vector is a copy of one code row and
scale, searched with a query for which those copies score best.  Every
workgroup's list then holds k copies with the same score, every entry
reaches the merge's bound, and the result must be the k copies with the
smallest ids (ties are broken by id everywhere).  At k = 1 and 10 the
256 x k entries exceed one wave's 64 and are folded in sorted runs; at
k = 64 the 16,384 entries exceed the gathering capacity and take the full
pairwise merge.  The oracle ranks the same codes for the expected list."""
import numpy as np
import pytest

import oracle
from tests.conftest import gpu_available

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402

N = 60_000
EVERY = 5


@pytest.fixture(scope="module")
def tied(small_env):
    s = small_env
    rng = np.random.default_rng(7)
    rows = rng.integers(0, s.codes.shape[0], N)
    codes = s.codes[rows].copy()
    scales = s.scales[rows].copy()
    src = 123
    dup = np.arange(0, N, EVERY)
    codes[dup] = s.codes[src]
    scales[dup] = s.scales[src]
    idx = tq.Index(s.cb, s.rot, n_tenants=1)
    idx.add_codes(torch.from_numpy(oracle.pack_codes(codes, 4)).cuda(), torch.from_numpy(scales).cuda())
    # the query: the copied row's own reconstruction direction, so that the
    # copies (identical codes and scale, identical scores) come first
    recon = s.ocb.cents[s.codes[src]].astype(np.float64)
    q = (s.R32.astype(np.float64).T @ recon).astype(np.float32)
    q /= np.linalg.norm(q)
    return s, idx, codes, scales, dup, q


@pytest.mark.parametrize("k", [1, 10, 64])
def test_tied_lists_merge_to_the_smallest_ids(tied, k):
    s, idx, codes, scales, dup, q = tied
    print("tied merge k=%d" % k, flush=True)
    qd = torch.from_numpy(q[None, :]).cuda()
    ids, sc = idx.search(qd, k, path="lut")
    ids = ids.cpu().numpy()[0]
    sc = sc.cpu().numpy()[0]
    ref_i, ref_s = oracle.search(codes, scales, s.ocb.cents, s.R32, q[None, :], k)
    # the oracle puts the copies first and breaks their tie by id
    assert np.array_equal(ref_i[0], dup[:k])
    assert np.array_equal(ids, dup[:k]), (ids[:12], dup[:12])
    assert np.all(sc == sc[0])
    assert abs(float(sc[0]) - float(ref_s[0][0])) <= 1e-4 * abs(float(ref_s[0][0])) + 1e-6


def test_tied_lists_in_a_batch(tied):
    """The same query among others: its list is unchanged by the batch."""
    s, idx, codes, scales, dup, q = tied
    Q = np.concatenate([s.Q[:7], q[None, :]], axis=0).astype(np.float32)
    ids, sc = idx.search(torch.from_numpy(Q).cuda(), 10, path="lut")
    assert np.array_equal(ids.cpu().numpy()[7], dup[:10])
