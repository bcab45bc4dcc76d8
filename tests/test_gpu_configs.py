"""GPU parity on the power-law workloads other than the 1M headline corpus.

* 100,000 x 1536, 1,000 queries from the same mixture: k = 5 and 10 on the
  single-query scan and on the batched path in calls of 64 queries.
* 999,000 x 1536 (the 1M corpus without its last 1,000 rows): calls of 1,
  32 and 256 queries on the batched path at k = 10 and 100.

The oracle scores returned ids one by one and a random sample of the corpus
(tests.parity.check_topk_sampled); the batched path must also return the
single-query path's scores."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available
from tests.parity import check_topk_sampled

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402

D = 1536


class Env:
    pass


def _env(name, n_check):
    e = Env()
    print("generating %s" % name, flush=True)
    e.X, Q = synth.workload(name, d=D)
    e.Q = np.ascontiguousarray(Q)
    e.R32 = oracle.haar_rotation(D, 42)[1]
    e.ocb = oracle.lloyd_max(D, 4)
    cb, rot = tq.Codebook(D, 4), tq.Rotation(D, 42)
    e.idx = tq.Index(cb, rot, n_tenants=1)
    e.idx.reserve(e.X.shape[0])
    e.idx.add(torch.from_numpy(e.X).cuda())
    e.Qd = torch.from_numpy(e.Q).cuda()
    torch.cuda.synchronize()
    e.sample = np.random.default_rng(61).choice(e.X.shape[0], n_check, replace=False)
    return e


@pytest.fixture(scope="module")
def c100k():
    return _env("powerlaw100k", 20_000)


def _same_scores(a, b):
    a, b = a.cpu().numpy(), b.cpu().numpy()
    assert np.array_equal(np.sort(a, axis=1), np.sort(b, axis=1))


@pytest.mark.parametrize("k", [5, 10])
def test_100k_single_query_and_batch_of_64(c100k, k):
    e = c100k
    print("100K k=%d" % k, flush=True)
    li, ls = e.idx.search(e.Qd, k, path="lut")
    for q0 in range(0, 1000, 64):
        q = e.Qd[q0:q0 + 64].contiguous()
        mi, ms = e.idx.search(q, k, path="mfma")
        _same_scores(ms, ls[q0:q0 + 64])
    # the oracle on 32 of the queries
    check_topk_sampled(li[:32].cpu().numpy(), ls[:32].cpu().numpy(), e.X, e.R32, e.ocb, e.Q[:32],
                       k, e.sample)


@pytest.fixture(scope="module")
def c999k():
    return _env("powerlaw999k", 20_000)


@pytest.mark.parametrize("k", [10, 100])
def test_999k_batches_of_1_32_256(c999k, k):
    e = c999k
    print("999K k=%d" % k, flush=True)
    q = e.Qd[:256].contiguous()
    li, ls = e.idx.search(q, k, path="lut")
    for b in (1, 32, 256):
        mi, ms = e.idx.search(q[:b].contiguous(), k, path="mfma")
        print("batch %d fallbacks %d" % (b, tq.last_search_fallbacks()), flush=True)
        _same_scores(ms, ls[:b])
        if b == 32:
            check_topk_sampled(mi[:8].cpu().numpy(), ms[:8].cpu().numpy(), e.X, e.R32, e.ocb,
                               e.Q[:8], k, e.sample)
