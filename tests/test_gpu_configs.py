"""GPU parity on the 100,000 x 1536 power-law workload (1,000 queries from
the same mixture) against the oracle's brute force over the whole corpus:
k = 5 and 10 on the single-query scan, and on the batched path in calls of
64 queries, which must also return the single-query path's scores.

The 999,000-row and 1,000,000-row workloads are in tests/test_gpu_fullsize.py."""
import numpy as np
import pytest

from tests.conftest import gpu_available
from tests.parity import check_topk

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402
from tests.fullsize import PowerlawCorpus, assert_index_codes_equal  # noqa: E402

D, NQ = 1536, 32


class Env:
    pass


@pytest.fixture(scope="module")
def c100k():
    e = Env()
    e.c = PowerlawCorpus("powerlaw100k", nq=NQ, bits=(4,))
    e.idx = tq.Index(e.c.cb[4], e.c.rot, n_tenants=1)
    e.idx.reserve(e.c.n)
    e.idx.add(torch.from_numpy(e.c.X).cuda())
    e.Qd = torch.from_numpy(e.c.Qall).cuda()
    torch.cuda.synchronize()
    return e


def _same_scores(a, b):
    a, b = a.cpu().numpy(), b.cpu().numpy()
    assert np.array_equal(np.sort(a, axis=1), np.sort(b, axis=1))


def _check(c, ids, sc, k):
    ref_i, ref_s = c.topk(4, k)
    check_topk(ids[:NQ].cpu().numpy(), sc[:NQ].cpu().numpy(), c.codes[4], c.scales[4],
               c.ocb[4].cents, c.qrot, c.qn, k, ref_i, ref_s)


def test_100k_codes(c100k):
    assert_index_codes_equal(c100k.idx, c100k.c.codes[4], 4)


@pytest.mark.parametrize("k", [5, 10])
def test_100k_single_query_and_batch_of_64(c100k, k):
    e = c100k
    print("100K k=%d" % k, flush=True)
    li, ls = e.idx.search(e.Qd, k, path="lut")
    _check(e.c, li, ls, k)
    for q0 in range(0, 1000, 64):
        q = e.Qd[q0:q0 + 64].contiguous()
        mi, ms = e.idx.search(q, k, path="mfma")
        _same_scores(ms, ls[q0:q0 + 64])
        if q0 == 0:
            _check(e.c, mi, ms, k)
