"""GPU parity of TQ+ calibration (section II-B) against the oracle.

* The fit (per-coordinate mean and spread of the rotated, normalised first
  batch) matches oracle.tqplus_fit within float32 storage of float64 sums.
* Given the library's installed (mu, kappa), rotation and tables, codes
  equal oracle.encode_tqplus bit for bit and scales agree to one float32
  ulp.
* Searches (unfiltered, tenant-filtered, large k, post-filter; b = 2, 3, 4,
  8) return lists the oracle's calibrated scores validate, as in the plain
  parity tests.
* The identity calibration reproduces the uncalibrated index exactly; the
  calibration persists through save/load; misuse is refused; and on rows in
  a cone (a shared offset) calibration raises recall against exact search."""
import numpy as np
import pytest

import oracle
import synth
from tests.conftest import gpu_available
from tests.parity import assert_codes_equal, assert_scales_close, check_topk, oracle_tables

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402

D = 1536


class Env:
    pass


def _build(d, bits, n, nq, n_fit, n_tenants=1, seed=42):
    e = Env()
    e.d, e.bits = d, bits
    e.X = synth.shifted_mixture(n, d)
    e.Q = synth.isotropic_queries(e.X, nq, seed=47)
    e.cb = tq.Codebook(d, bits)
    e.rot = tq.Rotation(d, seed)
    e.R32 = e.rot.matrix()
    e.ocb = oracle_tables(e.cb)
    e.Xd = torch.from_numpy(e.X).cuda()
    e.Qd = torch.from_numpy(e.Q).cuda()
    e.idx = tq.Index(e.cb, e.rot, n_tenants=n_tenants)
    e.n_fit = n_fit
    print("calibrate d=%d bits=%d m=%d" % (d, bits, n_fit), flush=True)
    e.idx.calibrate(e.Xd[:n_fit].contiguous())
    e.mu, e.kappa = e.idx.calibration()
    e.tenants = None
    if n_tenants > 1:
        e.tenants = synth.zipf_tenants(n, n_tenants, seed=44)
        e.idx.add(e.Xd, torch.from_numpy(e.tenants.view(np.int16)).cuda())
    else:
        e.idx.add(e.Xd)
    torch.cuda.synchronize()
    e.codes, e.norms, e.scales = oracle.encode_tqplus(e.X, e.R32, e.ocb, e.mu, e.kappa)
    e.qrot = oracle.rotate_queries(e.R32, e.Q)
    e.qn = np.linalg.norm(e.Q.astype(np.float64), axis=1)
    return e


@pytest.fixture(scope="module")
def env():
    return _build(D, 4, 6000, 32, 2000, n_tenants=20)


def _check_codes(e):
    codes, scales, _ = e.idx.export()
    assert_codes_equal(codes.cpu().numpy(), e.codes, e.bits)
    assert_scales_close(scales.cpu().numpy(), e.scales)


def test_fit_matches_oracle(env):
    mu_o, kappa_o = oracle.tqplus_fit(env.X[:env.n_fit], env.R32)
    assert np.max(np.abs(env.mu - mu_o)) < 1e-7
    assert np.max(np.abs(env.kappa / kappa_o - 1.0)) < 1e-5


def test_fit_over_several_chunks():
    # more rows than one rotation chunk of the fit (16384), d = 256
    d = 256
    X = synth.shifted_mixture(20000, d)
    rot = tq.Rotation(d, 9)
    R32 = rot.matrix()
    idx = tq.Index(tq.Codebook(d, 4), rot)
    print("calibrate d=256 m=20000", flush=True)
    idx.calibrate(torch.from_numpy(X).cuda())
    mu, kappa = idx.calibration()
    mu_o, kappa_o = oracle.tqplus_fit(X, R32)
    assert np.max(np.abs(mu - mu_o)) < 1e-7
    assert np.max(np.abs(kappa / kappa_o - 1.0)) < 1e-5


def test_codes_bit_exact(env):
    print("tq+ codes d=1536 b=4", flush=True)
    _check_codes(env)


def test_search_matches_oracle(env):
    print("tq+ search k=10", flush=True)
    ids, sc = env.idx.search(env.Qd, 10)
    calib = (env.mu, env.kappa)
    ref_i, ref_s = oracle.search(env.codes, env.scales, env.ocb.cents, env.R32, env.Q, 10, calib=calib)
    differ = check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents,
                        env.qrot, env.qn, 10, ref_i, ref_s, calib=calib)
    assert differ <= 2


def test_filtered_search_matches_oracle(env):
    print("tq+ filtered search k=10", flush=True)
    T = 20
    allowed = synth.allowlists(env.Q.shape[0], T, "selective", seed=45)
    bm = synth.allowlist_bitmap(allowed, T)
    ids, sc = env.idx.search(env.Qd, 10, allow=torch.from_numpy(bm.view(np.int64)).cuda())
    calib = (env.mu, env.kappa)
    ref_i, ref_s = oracle.search(env.codes, env.scales, env.ocb.cents, env.R32, env.Q, 10,
                                 tenants=env.tenants, allow=bm, calib=calib)
    masks = [oracle.allowed_mask(env.tenants, bm[b]) for b in range(bm.shape[0])]
    differ = check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents,
                        env.qrot, env.qn, 10, ref_i, ref_s, allowed=masks, calib=calib)
    assert differ <= 2


def test_large_k_matches_oracle(env):
    print("tq+ search k=300", flush=True)
    k = 300
    Q = env.Q[:6].copy()
    ids, sc = env.idx.search(torch.from_numpy(Q).cuda(), k)
    calib = (env.mu, env.kappa)
    ref_i, ref_s = oracle.search(env.codes, env.scales, env.ocb.cents, env.R32, Q, k, calib=calib)
    check_topk(ids.cpu().numpy(), sc.cpu().numpy(), env.codes, env.scales, env.ocb.cents,
               env.qrot[:6], env.qn[:6], k, ref_i, ref_s, calib=calib)


def test_postfilter_matches_oracle(env):
    print("tq+ post-filter k=10 overfetch=5", flush=True)
    T = 20
    bm = synth.allowlist_bitmap(synth.allowlists(env.Q.shape[0], T, "broad", seed=46), T)
    ids, sc = env.idx.search_postfilter(env.Qd, 10, 5, torch.from_numpy(bm.view(np.int64)).cuda())
    calib = (env.mu, env.kappa)
    ref_i, ref_s = oracle.postfilter_search(env.codes, env.scales, env.ocb.cents, env.R32, env.Q, 10,
                                            5, env.tenants, bm, calib=calib)
    ids = ids.cpu().numpy()
    sc = sc.cpu().numpy().astype(np.float64)
    for b in range(ids.shape[0]):
        nv = int((ids[b] >= 0).sum())
        assert np.all(ids[b][nv:] == -1)
        v = ids[b][:nv]
        assert np.all(oracle.allowed_mask(env.tenants, bm[b])[v]), "disallowed vector returned"
        ref = oracle.scores_for_ids(env.codes, env.scales, env.ocb.cents, env.qrot[b], v, calib=calib)
        tol = np.maximum(1e-4 * np.abs(ref), 1e-6 * env.qn[b])
        assert np.all(np.abs(sc[b][:nv] - ref) <= tol)
    # the oracle's lists, except where scores tie at the over-fetch cut
    assert np.mean(np.all(ids == ref_i, axis=1)) >= 0.9


@pytest.mark.parametrize("bits", [2, 3, 8])
def test_other_widths(bits):
    print("tq+ d=256 bits=%d" % bits, flush=True)
    e = _build(256, bits, 3000, 16, 1000)
    _check_codes(e)
    k = 10
    ids, sc = e.idx.search(e.Qd, k)
    calib = (e.mu, e.kappa)
    ref_i, ref_s = oracle.search(e.codes, e.scales, e.ocb.cents, e.R32, e.Q, k, calib=calib)
    differ = check_topk(ids.cpu().numpy(), sc.cpu().numpy(), e.codes, e.scales, e.ocb.cents,
                        e.qrot, e.qn, k, ref_i, ref_s, calib=calib)
    assert differ <= 2


def test_identity_calibration_is_plain(env):
    print("tq+ identity calibration", flush=True)
    X = env.Xd[:3000].contiguous()
    plain = tq.Index(env.cb, env.rot)
    plain.add(X)
    ident = tq.Index(env.cb, env.rot)
    ident.set_calibration(np.zeros(D, np.float32), np.ones(D, np.float32))
    ident.add(X)
    for a, b in zip(plain.export(), ident.export()):
        assert torch.equal(a, b)
    for k in (10, 300):
        a_i, a_s = plain.search(env.Qd, k)
        b_i, b_s = ident.search(env.Qd, k)
        assert torch.equal(a_i, b_i) and torch.equal(a_s, b_s)


def test_calibration_persists(env, tmp_path):
    print("tq+ save/load", flush=True)
    path = tmp_path / "calibrated.tq"
    env.idx.save(path)
    back = tq.Index.load(env.cb, env.rot, path)
    mu, kappa = back.calibration()
    assert np.array_equal(mu, env.mu) and np.array_equal(kappa, env.kappa)
    for a, b in zip(env.idx.export(), back.export()):
        assert torch.equal(a, b)
    a_i, a_s = env.idx.search(env.Qd, 10)
    b_i, b_s = back.search(env.Qd, 10)
    assert torch.equal(a_i, b_i) and torch.equal(a_s, b_s)
    # vectors added after loading are coded with the loaded calibration
    back.add(env.Xd[:50].contiguous())
    c, s, _ = back.export()
    n = env.X.shape[0]
    assert torch.equal(c[n:].cpu(), c[:50].cpu()) and torch.equal(s[n:].cpu(), s[:50].cpu())


def test_misuse_is_refused(env):
    with pytest.raises(tq.TQError):
        env.idx.calibrate(env.Xd[:10].contiguous())      # vectors already added
    with pytest.raises(tq.TQError):
        env.idx.search(env.Qd[:2].contiguous(), 10, path="mfma")
    fresh = tq.Index(env.cb, env.rot)
    with pytest.raises(tq.TQError):
        fresh.set_calibration(np.zeros(D, np.float32), -np.ones(D, np.float32))
    Z = env.Xd[:8].clone()
    Z[3] = 0
    with pytest.raises(tq.TQError):
        fresh.calibrate(Z)
    assert fresh.calibration() is None


def test_calibration_raises_recall_on_shifted_rows(env):
    print("tq+ recall against exact", flush=True)
    plain = tq.Index(env.cb, env.rot)
    plain.add(env.Xd)
    ex_i, _ = oracle.exact_search(env.X, env.Q, 10)
    a_i, _ = plain.search(env.Qd, 10)
    b_i, _ = env.idx.search(env.Qd, 10)
    r_plain = oracle.recall_at_k(a_i.cpu().numpy(), ex_i, 10)
    r_cal = oracle.recall_at_k(b_i.cpu().numpy(), ex_i, 10)
    print("recall@10 plain %.3f calibrated %.3f" % (r_plain, r_cal), flush=True)
    assert r_cal > r_plain + 0.05
