"""The Python binding hands raw device pointers to the library, which cannot
see the size of a tensor: every tensor argument's shape is checked first, so
that a mis-sized tensor raises ValueError before any pointer is passed.  Run
on the CPU with CPU tensors: the shape check comes before the device checks,
which then reject the correctly shaped CPU tensors."""
import pytest

torch = pytest.importorskip("torch")

import paper_2607_16973_amd as tq  # noqa: E402

D = 128


@pytest.fixture(scope="module")
def idx():
    cb, rot = tq.Codebook(D, 4), tq.Rotation(D, 3)
    return tq.Index(cb, rot, n_tenants=100)   # 2 allowlist words


def z(*shape, dtype=torch.float32):
    return torch.zeros(shape, dtype=dtype)


@pytest.mark.parametrize("call", [
    lambda i: i.search(z(4, D + 64), 10),                                  # d
    lambda i: i.search(z(4, D), 10, allow=z(3, 2, dtype=torch.int64)),     # rows
    lambda i: i.search(z(4, D), 10, allow=z(4, 1, dtype=torch.int64)),     # words
    lambda i: i.search(z(4, D), 10, ids=z(4, 9, dtype=torch.int64)),       # ids
    lambda i: i.search(z(4, D), 10, scores=z(5, 10)),                      # scores
    lambda i: i.search(z(4, D), 10, slot_allow=z(4, 3, dtype=torch.int64)),
    lambda i: i.search_postfilter(z(4, D), 10, 2, z(4, 1, dtype=torch.int64)),
    lambda i: i.search_alloc(z(4, D - 1), 10),
    lambda i: i.add(z(8, D + 1)),
    lambda i: i.add(z(8, D), z(7, dtype=torch.int16)),
    lambda i: i.add_codes(z(8, D // 2, dtype=torch.uint8), z(8)[:7]),
    lambda i: i.add_codes(z(8, D, dtype=torch.uint8), z(8)),
    lambda i: i.calibrate(z(8, D // 2)),
], ids=["Q-d", "allow-rows", "allow-words", "ids", "scores", "slot-allow", "postfilter-allow",
        "alloc-Q", "add-X", "add-tenants", "codes-scales", "codes-width", "calibrate"])
def test_mis_sized_tensors_raise(idx, call):
    with pytest.raises(ValueError):
        call(idx)


def test_well_sized_cpu_tensors_pass_the_shape_checks(idx):
    # then the device checks reject them: CPU tensors, or no GPU here
    with pytest.raises((TypeError, tq.TQError)):
        idx.search(z(4, D), 10, allow=z(4, 2, dtype=torch.int64))
    with pytest.raises((TypeError, tq.TQError)):
        idx.add(z(8, D), z(8, dtype=torch.int16))


def test_free_functions_check_shapes():
    cb, rot = tq.Codebook(D, 2), tq.Rotation(D, 3)
    with pytest.raises(ValueError):
        tq.rotate_quantize(cb, rot, z(5, D), codes=z(5, D // 8, dtype=torch.uint8))
    with pytest.raises(ValueError):
        tq.rotate_queries(rot, z(5, D + 1))
    with pytest.raises(ValueError):
        tq.rotate_queries(rot, z(5, D), out=z(4, D))
    idm = tq.IdMapIndex(cb, rot, n_tenants=1)
    with pytest.raises(ValueError):
        idm.add(z(3, D), [1, 2, 3], z(2, dtype=torch.int16))
