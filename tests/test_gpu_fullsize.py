"""GPU parity at the full benchmark size against the oracle's brute force over
the whole corpus (section IV-A ground truth; section II-B for the codes and
scores).

The 1,000,000 x 1536 power-law corpus is coded by the oracle in full at
b = 2, 3, 4 and 8 and scored against 32 queries (tests/fullsize.py).  Then:

* the index's codes equal the oracle's for every one of the 10^6 rows, at
  every bit width;
* every top-k list -- the single-query scan at k = 10 and 100, the batched
  matrix-core path at k = 10 and 100, tenant-filtered searches at
  T in {10, 100, 1000} with selective and broad allowlists (section V-C), and
  the 2-, 3- and 8-bit scans -- is checked by tests.parity.check_topk against
  the oracle's top-k over all 10^6 vectors;
* the 999,000-row corpus (the first 999,000 rows, same queries) on the
  single-query scan at k = 10 and 100 and in batched calls of 1, 32 and 256
  queries.

Searches run in bench.py's launch configuration: queries rotated first,
then the scan with the rotation step skipped."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available
from tests.parity import check_topk

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402
from tests.fullsize import PowerlawCorpus, assert_index_codes_equal  # noqa: E402

D, N, NQ = 1536, 1_000_000, 32
N999 = 999_000


class Big:
    pass


@pytest.fixture(scope="module")
def big():
    b = Big()
    b.c = PowerlawCorpus("powerlaw1m", nq=NQ, bits=(4, 2, 3, 8))
    b.Xd = torch.from_numpy(b.c.X).cuda()
    b.idx = tq.Index(b.c.cb[4], b.c.rot, n_tenants=1)
    b.idx.reserve(N)
    print("index add n=%d" % N, flush=True)
    b.idx.add(b.Xd)
    b.Qall = torch.from_numpy(b.c.Qall).cuda()
    b.Qrot = tq.rotate_queries(b.c.rot, b.Qall[:NQ].contiguous())
    torch.cuda.synchronize()
    yield b
    del b.Xd
    torch.cuda.empty_cache()


def _check(big, bits, ids, sc, k, n=None, tenants=None, allow=None, masks=None):
    c = big.c
    n = N if n is None else n
    ref_i, ref_s = c.topk(bits, k, n=n, tenants=tenants, allow=allow)
    check_topk(ids[:NQ].cpu().numpy(), sc[:NQ].cpu().numpy(), c.codes[bits][:n],
               c.scales[bits][:n], c.ocb[bits].cents, c.qrot, c.qn, k, ref_i, ref_s,
               allowed=masks, n=n)


def test_codes_of_every_row(big):
    print("codes of %d rows, b=4" % N, flush=True)
    assert_index_codes_equal(big.idx, big.c.codes[4], 4)


@pytest.mark.parametrize("path,k", [("lut", 10), ("lut", 100), ("mfma", 10), ("mfma", 100)])
def test_search_full_size(big, path, k):
    print("search N=%d path=%s k=%d" % (N, path, k), flush=True)
    ids, sc = big.idx.search(big.Qrot, k, path=path, prerotated=True)
    _check(big, 4, ids, sc, k)
    if path == "mfma":
        li, ls = big.idx.search(big.Qrot, k, path="lut", prerotated=True)
        assert torch.equal(torch.sort(sc, 1).values, torch.sort(ls, 1).values)


def test_top64_of_k64_and_k65_agree_full_size(big):
    """k = 64 keeps one 64-entry slot per wave list, k = 65 two; both sum the
    same integer table entries, so the leading 64 entries agree exactly."""
    print("search N=%d k=64 and k=65" % N, flush=True)
    a_i, a_s = big.idx.search(big.Qrot, 64, path="lut", prerotated=True)
    b_i, b_s = big.idx.search(big.Qrot, 65, path="lut", prerotated=True)
    assert torch.equal(a_i, b_i[:, :64]) and torch.equal(a_s, b_s[:, :64])


@pytest.mark.parametrize("T", [10, 100, 1000])
def test_filtered_full_size(big, T):
    """Zipf(1.1) tenants at random positions; one tenant per query
    (selective) or ceil(T/10) tenants (broad); blocks skipped by summary."""
    ten = synth.zipf_tenants(N, T, seed=44)
    idx = tq.Index(big.c.cb[4], big.c.rot, n_tenants=T)
    idx.reserve(N)
    idx.add(big.Xd, torch.from_numpy(ten.view(np.int16)).cuda())
    for mode in ("selective", "broad"):
        print("filtered N=%d T=%d %s" % (N, T, mode), flush=True)
        bm = synth.allowlist_bitmap(synth.allowlists(NQ, T, mode, seed=45), T)
        ids, sc = idx.search(big.Qrot, 10, allow=torch.from_numpy(bm.view(np.int64)).cuda(),
                             prerotated=True)
        masks = [oracle.allowed_mask(ten, bm[b]) for b in range(NQ)]
        _check(big, 4, ids, sc, 10, tenants=ten, allow=bm, masks=masks)
    del idx
    torch.cuda.empty_cache()


@pytest.mark.parametrize("bits", [2, 3, 8])
def test_other_bit_widths_full_size(big, bits):
    """The bit-width sweep's corpus: the GPU encode of all 10^6 rows equals
    the oracle's codes, and the single-query scan's top-10 the oracle's."""
    print("encode and search N=%d b=%d" % (N, bits), flush=True)
    idx = tq.Index(big.c.cb[bits], big.c.rot, n_tenants=1)
    idx.reserve(N)
    idx.add(big.Xd)
    assert_index_codes_equal(idx, big.c.codes[bits], bits)
    ids, sc = idx.search(big.Qrot, 10, prerotated=True)
    _check(big, bits, ids, sc, 10)
    del idx
    torch.cuda.empty_cache()


@pytest.mark.parametrize("k", [10, 100])
def test_999k_single_query_and_batches_of_1_32_256(big, k):
    """The 999K corpus: the single-query scan against the oracle's brute
    force, and the batched path in calls of 1, 32 and 256 queries returning
    the single-query path's scores (the first 32 queries also against the
    oracle)."""
    print("999K k=%d" % k, flush=True)
    idx = tq.Index(big.c.cb[4], big.c.rot, n_tenants=1)
    idx.reserve(N999)
    idx.add(big.Xd[:N999])
    q = big.Qall[:256].contiguous()
    li, ls = idx.search(q, k, path="lut")
    _check(big, 4, li, ls, k, n=N999)
    for b in (1, 32, 256):
        mi, ms = idx.search(q[:b].contiguous(), k, path="mfma")
        print("batch %d fallbacks %d" % (b, tq.last_search_fallbacks()), flush=True)
        assert np.array_equal(np.sort(ms.cpu().numpy(), axis=1), np.sort(ls[:b].cpu().numpy(), axis=1))
        if b >= NQ:
            _check(big, 4, mi, ms, k, n=N999)
    del idx
    torch.cuda.empty_cache()
