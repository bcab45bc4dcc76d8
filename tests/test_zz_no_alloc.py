"""The allocation-free search (tq_search_noalloc) against tq_search, the
entry point it is a variant of: the same single-query scan kernels, with the
workspace in the library's device scratch array instead of a per-call
allocation, so ids and scores must be identical.  Consecutive calls share the
array; each case runs calls of decreasing size in a row."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402
from paper_2607_16973_amd import _lib  # noqa: E402

D, T = 1536, 5


class Env:
    pass


@pytest.fixture(scope="module")
def env():
    e = Env()
    e.X = synth.isotropic_mixture(5003, D, seed=60)
    e.Q = synth.isotropic_queries(e.X, 200, seed=61)
    e.cb, e.rot = tq.Codebook(D, 4), tq.Rotation(D, 42)
    e.tenants = (np.arange(e.X.shape[0]) % T).astype(np.uint16)
    e.idx = tq.Index(e.cb, e.rot, n_tenants=T)
    e.idx.add(torch.from_numpy(e.X).cuda(), torch.from_numpy(e.tenants.view(np.int16)).cuda())
    e.Qd = torch.from_numpy(e.Q).cuda()
    torch.cuda.synchronize()
    return e


def _same(a, b):
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_equal_to_tq_search_on_two_calls_the_second_smaller(env):
    print("noalloc: 64 queries k=100, then 7 queries k=10", flush=True)
    _same(env.idx.search_noalloc(env.Qd[:64].contiguous(), 100),
          env.idx.search_alloc(env.Qd[:64].contiguous(), 100))
    _same(env.idx.search_noalloc(env.Qd[:7].contiguous(), 10),
          env.idx.search_alloc(env.Qd[:7].contiguous(), 10))


def test_filtered_equal_to_tq_search(env):
    print("noalloc: filtered", flush=True)
    allowed = [[q % T] for q in range(64)]
    bm = torch.from_numpy(synth.allowlist_bitmap(allowed, T).view(np.int64)).cuda()
    _same(env.idx.search_noalloc(env.Qd[:64].contiguous(), 10, allow=bm),
          env.idx.search_alloc(env.Qd[:64].contiguous(), 10, allow=bm))
    _same(env.idx.search_noalloc(env.Qd[:3].contiguous(), 10, allow=bm[:3].contiguous()),
          env.idx.search_alloc(env.Qd[:3].contiguous(), 10, allow=bm[:3].contiguous()))


def test_queries_split_over_several_launches(env):
    """At k = 256 one query's candidate lists take about 0.5 MB, so 200
    queries go through the array in several launches."""
    print("noalloc: 200 queries k=256", flush=True)
    _same(env.idx.search_noalloc(env.Qd, 256), env.idx.search(env.Qd, 256, path="lut"))
    _same(env.idx.search_noalloc(env.Qd[:50].contiguous(), 256),
          env.idx.search(env.Qd[:50].contiguous(), 256, path="lut"))


def test_large_k_path(env):
    print("noalloc: k=1000", flush=True)
    _same(env.idx.search_noalloc(env.Qd[:9].contiguous(), 1000),
          env.idx.search(env.Qd[:9].contiguous(), 1000, path="lut"))
    _same(env.idx.search_noalloc(env.Qd[:2].contiguous(), 300),
          env.idx.search(env.Qd[:2].contiguous(), 300, path="lut"))


def test_empty_index_gives_padding(env):
    idx = tq.Index(env.cb, env.rot, n_tenants=1)
    ids, sc = idx.search_noalloc(env.Qd[:4].contiguous(), 10)
    assert torch.all(ids == -1) and torch.all(torch.isneginf(sc))


def test_rotation_must_be_resident_first(env):
    """An index filled from codes has not put its rotation on the device:
    the call refuses; after one allocating search it matches tq_search."""
    rot = tq.Rotation(D, 42)
    idx = tq.Index(env.cb, rot, n_tenants=1)
    codes, _, scales = oracle.encode(env.X[:500], rot.matrix(), oracle.Codebook(
        d=D, bits=4, bounds=env.cb.bounds, cents=env.cb.cents, iterations=0, converged=True))
    idx.add_codes(torch.from_numpy(oracle.pack_codes(codes, 4)).cuda(),
                  torch.from_numpy(scales).cuda())
    with pytest.raises(tq.TQError, match="TQ_EINVAL"):
        idx.search_noalloc(env.Qd[:4].contiguous(), 10)
    ref = idx.search_alloc(env.Qd[:4].contiguous(), 10)
    _same(idx.search_noalloc(env.Qd[:4].contiguous(), 10), ref)


def test_reserve_makes_the_rotation_resident(env):
    """tq_index_reserve uploads the index's rotation, so an index filled from
    codes after a reserve takes the no-alloc search at once."""
    rot = tq.Rotation(D, 42)
    idx = tq.Index(env.cb, rot, n_tenants=1)
    idx.reserve(500)
    codes, _, scales = oracle.encode(env.X[:500], rot.matrix(), oracle.Codebook(
        d=D, bits=4, bounds=env.cb.bounds, cents=env.cb.cents, iterations=0, converged=True))
    idx.add_codes(torch.from_numpy(oracle.pack_codes(codes, 4)).cuda(),
                  torch.from_numpy(scales).cuda())
    got = idx.search_noalloc(env.Qd[:4].contiguous(), 10)
    _same(got, idx.search_alloc(env.Qd[:4].contiguous(), 10))


def test_argument_errors(env):
    L = _lib.lib
    import ctypes
    null = ctypes.c_void_p(0)
    assert L.tq_search_noalloc(env.idx._h, null, 1, 0, None, null, null, None) == _lib.TQ_EINVAL
    assert L.tq_search_noalloc(env.idx._h, null, 1, 5000, None, null, null, None) == _lib.TQ_EINVAL
    assert L.tq_search_noalloc(None, null, 1, 10, None, null, null, None) == _lib.TQ_EINVAL
    assert L.tq_search_noalloc(env.idx._h, null, 0, 10, None, null, null, None) == _lib.TQ_OK
