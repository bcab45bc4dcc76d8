import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")


class SmallSetup:
    """The small workload (10,000 x 1536 isotropic mixture, 64 noisy queries)
    coded by the oracle, plus a GPU index built from the rows."""


@pytest.fixture(scope="session")
def small_env():
    import numpy as np
    import torch

    import oracle
    import paper_2607_16973_amd as tq
    import synth
    from tests.parity import oracle_tables
    d = 1536
    s = SmallSetup()
    s.X, s.Q = synth.workload("small")
    s.cb = tq.Codebook(d, 4)
    s.rot = tq.Rotation(d, 42)
    # the oracle encodes with the library's rotation and tables (the
    # parameters of the encode definition), so codes agree bit for bit
    s.R32 = s.rot.matrix()
    s.ocb = oracle_tables(s.cb)
    s.codes, s.norms, s.scales = oracle.encode(s.X, s.R32, s.ocb)
    s.qrot = oracle.rotate_queries(s.R32, s.Q)
    s.qn = np.linalg.norm(s.Q.astype(np.float64), axis=1)
    s.Xd = torch.from_numpy(s.X).cuda()
    s.Qd = torch.from_numpy(s.Q).cuda()
    s.idx = tq.Index(s.cb, s.rot, n_tenants=1)
    print("index add n=%d" % s.X.shape[0], flush=True)
    s.idx.add(s.Xd)
    torch.cuda.synchronize()
    return s
