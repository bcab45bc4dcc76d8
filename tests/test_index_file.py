"""The index file of tq_index_save / tq_index_load (persistence, section
III-A), checked on the CPU: the layout is parsed independently here (header
fields, FNV-1a hash of the preceding bytes), and every damaged or mismatched
file must be rejected before any device work.  Round trips of indexes with
content run on the GPU (tests/test_gpu_persist.py)."""
import struct

import pytest

import paper_2607_16973_amd as tq

HEADER = struct.Struct("<8sIIiiQqii")


def fnv1a64(data: bytes) -> int:
    h = 1469598103934665603
    for b in data:
        h = ((h ^ b) * 1099511628211) & 0xFFFFFFFFFFFFFFFF
    return h


@pytest.fixture(scope="module")
def parts():
    cb, rot = tq.Codebook(256, 4), tq.Rotation(256, 5)
    return cb, rot


def test_empty_index_file_layout(parts, tmp_path):
    cb, rot = parts
    idx = tq.Index(cb, rot, n_tenants=7)
    path = tmp_path / "empty.tq"
    idx.save(path)
    data = path.read_bytes()
    assert len(data) == HEADER.size + 8
    magic, ver, flags, d, bits, seed, n, T, _ = HEADER.unpack(data[:HEADER.size])
    assert (magic, ver, flags, d, bits, seed, n, T) == (b"TQINDEX1", 1, 0, 256, 4, 5, 0, 7)
    assert struct.unpack("<Q", data[-8:])[0] == fnv1a64(data[:-8])
    back = tq.Index.load(cb, rot, path)
    assert len(back) == 0 and back.n_tenants == 7 and back.words == 1


def _expect(status, cb, rot, path, what):
    with pytest.raises(tq.TQError, match=status) as e:
        tq.Index.load(cb, rot, path)
    assert what in str(e.value)


def test_damaged_and_mismatched_files_rejected(parts, tmp_path):
    cb, rot = parts
    good = tmp_path / "good.tq"
    tq.Index(cb, rot, n_tenants=3).save(good)
    data = good.read_bytes()
    bad = tmp_path / "bad.tq"
    flipped = bytearray(data)
    flipped[20] ^= 1                                   # inside the header (d)
    bad.write_bytes(bytes(flipped))
    _expect("TQ_EINVAL", cb, rot, bad, "")
    bad.write_bytes(data[:-3])
    _expect("TQ_EINVAL", cb, rot, bad, "truncated")
    bad.write_bytes(data + b"\0")
    _expect("TQ_EINVAL", cb, rot, bad, "trailing")
    bad.write_bytes(b"NOTINDEX" + data[8:])
    _expect("TQ_EINVAL", cb, rot, bad, "not an index file")
    body = bytearray(data[:-8])
    body[8:12] = struct.pack("<I", 2)                  # another format version
    bad.write_bytes(bytes(body) + struct.pack("<Q", fnv1a64(bytes(body))))
    _expect("TQ_EUNSUPPORTED", cb, rot, bad, "version")
    body = bytearray(data[:-8])
    body[HEADER.size - 8:HEADER.size - 4] = struct.pack("<i", 0)     # n_tenants = 0
    bad.write_bytes(bytes(body) + struct.pack("<Q", fnv1a64(bytes(body))))
    _expect("TQ_EINVAL", cb, rot, bad, "out of range")
    # the codebook and rotation must match the file
    _expect("TQ_EINVAL", tq.Codebook(256, 2), rot, good, "codebook")
    _expect("TQ_EINVAL", cb, tq.Rotation(256, 6), good, "rotation")
    with pytest.raises(tq.TQError, match="TQ_EINVAL"):
        tq.Index.load(cb, rot, tmp_path / "missing.tq")


def test_empty_idmap_index_file(parts, tmp_path):
    cb, rot = parts
    path = tmp_path / "idmap.tq"
    tq.IdMapIndex(cb, rot, n_tenants=2).save(path)
    data = path.read_bytes()
    assert HEADER.unpack(data[:HEADER.size])[2] == 1        # flags: id-map sections
    assert struct.unpack("<Q", data[-8:])[0] == fnv1a64(data[:-8])
    back = tq.Index.load(cb, rot, path)
    assert isinstance(back, tq.IdMapIndex) and len(back) == 0
    body = bytearray(data[:-8])
    body[12:16] = struct.pack("<I", 5)                      # an undefined section flag
    bad = tmp_path / "bad.tq"
    bad.write_bytes(bytes(body) + struct.pack("<Q", fnv1a64(bytes(body))))
    _expect("TQ_EUNSUPPORTED", cb, rot, bad, "sections")


def _with_calibration(data: bytes, mu, kappa) -> bytes:
    """An empty index file with the TQ+ calibration section (flag 2) added."""
    body = bytearray(data[:-8])
    flags = struct.unpack("<I", body[12:16])[0]
    body[12:16] = struct.pack("<I", flags | 2)
    body += struct.pack("<%df" % len(mu), *mu) + struct.pack("<%df" % len(kappa), *kappa)
    return bytes(body) + struct.pack("<Q", fnv1a64(bytes(body)))


def test_calibration_section_checked_before_device_work(parts, tmp_path):
    """A calibration section (mu [d], kappa [d] float32 after the other
    sections) must be whole and hold finite values with kappa >= 0; the
    values are checked before the index touches a device."""
    cb, rot = parts
    good = tmp_path / "plain.tq"
    tq.Index(cb, rot, n_tenants=2).save(good)
    data = good.read_bytes()
    bad = tmp_path / "bad.tq"
    full = _with_calibration(data, [0.0] * 256, [1.0] * 256)
    bad.write_bytes(full[:-8 - 4 * 256] + full[-8:])          # kappa missing
    _expect("TQ_EINVAL", cb, rot, bad, "")
    bad.write_bytes(_with_calibration(data, [0.0] * 256, [1.0] * 255 + [-1.0]))
    _expect("TQ_EINVAL", cb, rot, bad, "kappa")
    bad.write_bytes(_with_calibration(data, [float("nan")] + [0.0] * 255, [1.0] * 256))
    _expect("TQ_EINVAL", cb, rot, bad, "finite")
