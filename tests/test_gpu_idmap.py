"""GPU parity of the id-map index (section III-A: external uint64 ids, O(1)
deletion, access control by id) and of slot-level allowlists (section
III-B).  Vectors come from the oracle's codes of the small workload; every
search is checked against the oracle over exactly the eligible vectors --
not deleted, and allowed by the query's tenant or slot allowlist -- after
mapping the returned external ids back to positions."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available
from tests.parity import check_topk

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402

T = 100


class IdEnv:
    pass


@pytest.fixture(scope="module")
def ienv(small_env):
    s = small_env
    e = IdEnv()
    e.s = s
    n = s.X.shape[0]
    rng = np.random.default_rng(61)
    # distinct ids spread over the whole uint64 range (top bit set for half)
    e.ids = np.unique(rng.integers(0, 2**64 - 2, size=2 * n, dtype=np.uint64))[:n]
    rng.shuffle(e.ids)
    e.pos_of = {int(v): i for i, v in enumerate(e.ids)}
    e.ten = synth.zipf_tenants(n, T, seed=44)
    e.idx = tq.IdMapIndex(s.cb, s.rot, n_tenants=T)
    pk = torch.from_numpy(oracle.pack_codes(s.codes, 4)).cuda()
    sc = torch.from_numpy(s.scales).cuda()
    td = torch.from_numpy(e.ten.view(np.int16)).cuda()
    print("id-map add n=%d" % n, flush=True)
    e.idx.add_codes(pk[:6000].contiguous(), sc[:6000].contiguous(), e.ids[:6000], td[:6000].contiguous())
    e.idx.add_codes(pk[6000:].contiguous(), sc[6000:].contiguous(), e.ids[6000:], td[6000:].contiguous())
    e.live = np.ones(n, dtype=bool)
    return e


def to_pos(e, ids):
    """External ids (int64 bit patterns) -> positions; -1 stays -1."""
    u = ids.cpu().numpy().view(np.uint64)
    out = np.full(u.shape, -1, dtype=np.int64)
    for idx in np.ndindex(u.shape):
        v = int(u[idx])
        if v != 2**64 - 1:
            out[idx] = e.pos_of[v]
    return out


def check(e, got_i, got_s, k, masks, tenants=None, bm=None):
    s = e.s
    ref_i, ref_s = oracle.search(s.codes, s.scales, s.ocb.cents, s.R32, s.Q, k, tenants, bm,
                                 masks=masks)
    allowed = [m if bm is None else (m & oracle.allowed_mask(tenants, bm[b]))
               for b, m in enumerate(masks)]
    check_topk(to_pos(e, got_i), got_s.cpu().numpy(), s.codes, s.scales, s.ocb.cents, s.qrot,
               s.qn, k, ref_i, ref_s, allowed=allowed)


def test_ids_returned_and_searches_match(ienv):
    e = ienv
    print("id-map search", flush=True)
    i, sc = e.idx.search(e.s.Qd, 10)
    check(e, i, sc, 10, [e.live] * e.s.Q.shape[0])
    assert np.array_equal(e.idx.slots(e.ids[[0, 5999, 6000, 9999]]), [0, 5999, 6000, 9999])
    assert e.idx.slots(np.array([12345], dtype=np.uint64))[0] == -1 or 12345 in e.pos_of


def test_deletions(ienv):
    e = ienv
    n = e.s.X.shape[0]
    rng = np.random.default_rng(62)
    # a random 30% plus every vector of blocks 3, 4 and 100 (dead blocks)
    kill = np.unique(np.concatenate([rng.choice(n, 3000, replace=False),
                                     np.arange(192, 320), np.arange(6400, 6464)]))
    # the oracle's best answers are deleted too, so results must change
    top, _ = e.idx.search(e.s.Qd[:8].contiguous(), 1)
    kill = np.unique(np.concatenate([kill, to_pos(e, top).ravel()]))
    print("delete %d" % kill.size, flush=True)
    assert e.idx.remove(e.ids[kill]) == kill.size
    assert e.idx.remove(e.ids[kill[:10]]) == 0            # already gone
    e.live[kill] = False
    assert len(e.idx) == n - kill.size and e.idx.n_slots == n
    assert np.all(e.idx.slots(e.ids[kill]) == -1)
    for k in (10, 64, 100):
        i, sc = e.idx.search(e.s.Qd, k)
        check(e, i, sc, k, [e.live] * e.s.Q.shape[0])
    # with tenant allowlists too
    bm = synth.allowlist_bitmap(synth.allowlists(e.s.Q.shape[0], T, "selective", seed=45), T)
    i, sc = e.idx.search(e.s.Qd, 10, allow=torch.from_numpy(bm.view(np.int64)).cuda())
    check(e, i, sc, 10, [e.live] * e.s.Q.shape[0], e.ten, bm)
    # the matrix-core path does not take deletions
    with pytest.raises(tq.TQError, match="TQ_EUNSUPPORTED"):
        e.idx.search(e.s.Qd, 10, path="mfma")


def test_slot_allowlists(ienv):
    e = ienv
    n, nq = e.s.X.shape[0], e.s.Q.shape[0]
    rng = np.random.default_rng(63)
    lists, masks = [], []
    for b in range(nq):
        m = rng.random(n) < (0.3 if b % 2 else 0.02)
        lst = list(e.ids[m]) + [np.uint64(2**64 - 3)]        # an id not in the index
        lists.append(np.array(lst, dtype=np.uint64))
        masks.append(m & e.live)
    sa = e.idx.slot_allowlist(lists)
    print("slot allowlists", flush=True)
    i, sc = e.idx.search(e.s.Qd, 10, slot_allow=sa)
    check(e, i, sc, 10, masks)
    # the same on a positional index, ids being positions
    pidx = tq.Index(e.s.cb, e.s.rot, n_tenants=1)
    pidx.add_codes(torch.from_numpy(oracle.pack_codes(e.s.codes, 4)).cuda(),
                   torch.from_numpy(e.s.scales).cuda())
    plists = [np.nonzero(m)[0].astype(np.uint64) for m in masks]
    pi, ps = pidx.search(e.s.Qd, 10, slot_allow=pidx.slot_allowlist(plists))
    ref_i, ref_s = oracle.search(e.s.codes, e.s.scales, e.s.ocb.cents, e.s.R32, e.s.Q, 10, masks=masks)
    check_topk(pi.cpu().numpy(), ps.cpu().numpy(), e.s.codes, e.s.scales, e.s.ocb.cents, e.s.qrot,
               e.s.qn, 10, ref_i, ref_s, allowed=masks)


def test_readd_and_bad_batches(ienv):
    e = ienv
    s = e.s
    dead = np.nonzero(~e.live)[0][:5]
    pk = torch.from_numpy(oracle.pack_codes(s.codes[dead], 4)).cuda()
    scl = torch.from_numpy(s.scales[dead]).cuda()
    before = len(e.idx)
    with pytest.raises(tq.TQError, match="TQ_EINVAL"):      # repeated id in the batch
        e.idx.add_codes(pk[:2].contiguous(), scl[:2].contiguous(), e.ids[dead[[0, 0]]])
    live_id = e.ids[np.nonzero(e.live)[0][0]]
    with pytest.raises(tq.TQError, match="TQ_EINVAL"):      # id already present
        e.idx.add_codes(pk[:1].contiguous(), scl[:1].contiguous(), np.array([live_id], dtype=np.uint64))
    with pytest.raises(tq.TQError, match="TQ_EINVAL"):      # positional add on an id-map index
        tq.Index.add_codes(e.idx, pk, scl)
    assert len(e.idx) == before
    # deleted ids come back in new slots; searches see them again
    e.idx.add_codes(pk, scl, e.ids[dead], torch.from_numpy(e.ten[dead].view(np.int16)).cuda())
    slots = e.idx.slots(e.ids[dead])
    assert np.all(slots >= s.X.shape[0])
    e.live[dead] = True
    i, sc = e.idx.search(s.Qd, 10)
    check(e, i, sc, 10, [e.live] * s.Q.shape[0])


def test_idmap_file_round_trip(ienv, tmp_path):
    e = ienv
    path = tmp_path / "idmap.tq"
    e.idx.save(path)
    back = tq.Index.load(e.s.cb, e.s.rot, path)
    assert isinstance(back, tq.IdMapIndex)
    assert len(back) == len(e.idx) and back.n_slots == e.idx.n_slots
    assert np.array_equal(back.slots(e.ids), e.idx.slots(e.ids))
    a_i, a_s = e.idx.search(e.s.Qd, 10)
    b_i, b_s = back.search(e.s.Qd, 10)
    assert torch.equal(a_i, b_i) and torch.equal(a_s, b_s)
    bm = synth.allowlist_bitmap(synth.allowlists(e.s.Q.shape[0], T, "broad", seed=46), T)
    allow = torch.from_numpy(bm.view(np.int64)).cuda()
    a_i, a_s = e.idx.search(e.s.Qd, 10, allow=allow)
    b_i, b_s = back.search(e.s.Qd, 10, allow=allow)
    assert torch.equal(a_i, b_i) and torch.equal(a_s, b_s)
