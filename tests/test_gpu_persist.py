"""GPU round trip of the index file (persistence, section III-A): an index
with tenant ids saved and loaded again holds the same codes, scales and
tenants, answers unfiltered and filtered searches exactly as before, and
keeps accepting vectors."""
import numpy as np
import pytest

import synth
from tests.conftest import gpu_available

pytestmark = pytest.mark.gpu
if not gpu_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2607_16973_amd as tq  # noqa: E402


@pytest.fixture(scope="module")
def env(small_env):
    return small_env


def test_save_load_round_trip(env, tmp_path):
    print("index file round trip", flush=True)
    n, T = env.X.shape[0], 100
    ten = synth.zipf_tenants(n, T, seed=44)
    idx = tq.Index(env.cb, env.rot, n_tenants=T)
    idx.add(env.Xd, torch.from_numpy(ten.view(np.int16)).cuda())
    path = tmp_path / "index.tq"
    idx.save(path)
    assert path.stat().st_size == 48 + n * (1536 * 4 // 8 + 4 + 2) + 8
    back = tq.Index.load(env.cb, env.rot, path)
    assert len(back) == n and back.n_tenants == T
    for a, b in zip(idx.export(), back.export()):
        assert torch.equal(a, b)
    a_i, a_s = idx.search(env.Qd, 10)
    b_i, b_s = back.search(env.Qd, 10)
    assert torch.equal(a_i, b_i) and torch.equal(a_s, b_s)
    bm = synth.allowlist_bitmap(synth.allowlists(env.Q.shape[0], T, "selective", seed=45), T)
    allow = torch.from_numpy(bm.view(np.int64)).cuda()
    a_i, a_s = idx.search(env.Qd, 10, allow=allow)
    b_i, b_s = back.search(env.Qd, 10, allow=allow)
    assert torch.equal(a_i, b_i) and torch.equal(a_s, b_s)
    # the loaded index keeps growing: ids continue after the loaded ones
    back.add(env.Xd[:100].contiguous())
    assert len(back) == n + 100
    c_i, _ = back.search(env.Qd[:4].contiguous(), 1)
    assert np.all(c_i.cpu().numpy() >= 0)
