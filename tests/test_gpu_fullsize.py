"""GPU parity at the full benchmark size: the 1,000,000 x 1536 power-law
mixture corpus, 4-bit codes, k=10, in the launch configuration of bench.py
(queries rotated first, then the scan with the rotation step skipped).

The oracle cannot search 10^6 vectors per query here, so every check is on
outputs it can compute one by one: codes of sampled rows (bit-exact), the
score of every returned id, and the property that no sampled vector beats a
returned list's worst entry (see tests.parity.check_topk_sampled)."""
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

D, N, K, NQ = 1536, 1_000_000, 10, 16


class Big:
    pass


@pytest.fixture(scope="module")
def big():
    b = Big()
    print("generating the 1M corpus", flush=True)
    b.X, Q = synth.workload("powerlaw1m", d=D)
    b.Q = np.ascontiguousarray(Q[:NQ])
    b.R32 = oracle.haar_rotation(D, 42)[1]
    b.ocb = oracle.lloyd_max(D, 4)
    b.cb, b.rot = tq.Codebook(D, 4), tq.Rotation(D, 42)
    b.Xd = torch.from_numpy(b.X).cuda()
    b.idx = tq.Index(b.cb, b.rot, n_tenants=1)
    b.idx.reserve(N)
    print("index add n=%d" % N, flush=True)
    b.idx.add(b.Xd)
    b.Qrot = tq.rotate_queries(b.rot, torch.from_numpy(b.Q).cuda())
    torch.cuda.synchronize()
    b.sample = np.random.default_rng(7).choice(N, 20000, replace=False)
    yield b
    del b.Xd
    torch.cuda.empty_cache()


def test_codes_of_sampled_rows(big):
    rows = np.sort(np.random.default_rng(3).choice(N, 2000, replace=False))
    codes, _, _ = big.idx.export()
    got = codes[torch.from_numpy(rows).cuda()].cpu().numpy()
    ref, _, _ = oracle.encode(np.ascontiguousarray(big.X[rows]), big.R32, big.ocb)
    assert np.array_equal(got, oracle.pack_codes(ref, 4))
    del codes


@pytest.mark.parametrize("path", ["lut", "mfma"])
def test_search_full_size(big, path):
    print("search N=%d path=%s" % (N, path), flush=True)
    ids, sc = big.idx.search(big.Qrot, K, path=path, prerotated=True)
    check_topk_sampled(ids.cpu().numpy(), sc.cpu().numpy(), big.X, big.R32, big.ocb, big.Q, K,
                       big.sample)
    if path == "mfma":
        li, ls = big.idx.search(big.Qrot, K, path="lut", prerotated=True)
        assert torch.equal(torch.sort(sc, 1).values, torch.sort(ls, 1).values)


def test_top64_of_k64_and_k65_agree_full_size(big):
    """k = 64 keeps one 64-entry slot per wave list, k = 65 two; both sum the
    same integer table entries, so the leading 64 entries agree exactly."""
    print("search N=%d k=64 and k=65" % N, flush=True)
    a_i, a_s = big.idx.search(big.Qrot, 64, path="lut", prerotated=True)
    b_i, b_s = big.idx.search(big.Qrot, 65, path="lut", prerotated=True)
    assert torch.equal(a_i, b_i[:, :64]) and torch.equal(a_s, b_s[:, :64])


def test_filtered_full_size(big):
    T = 100
    ten = synth.zipf_tenants(N, T, seed=44)
    idx = tq.Index(big.cb, big.rot, n_tenants=T)
    idx.reserve(N)
    idx.add(big.Xd, torch.from_numpy(ten.view(np.int16)).cuda())
    for mode in ("selective", "broad"):
        print("filtered N=%d T=%d %s" % (N, T, mode), flush=True)
        bm = synth.allowlist_bitmap(synth.allowlists(NQ, T, mode, seed=45), T)
        ids, sc = idx.search(big.Qrot, K, allow=torch.from_numpy(bm.view(np.int64)).cuda(),
                             prerotated=True)
        masks = [oracle.allowed_mask(ten, bm[b]) for b in range(NQ)]
        check_topk_sampled(ids.cpu().numpy(), sc.cpu().numpy(), big.X, big.R32, big.ocb, big.Q, K,
                           big.sample, allowed=masks)
    del idx
    torch.cuda.empty_cache()
