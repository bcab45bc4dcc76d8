"""TurboQuant search hot path on AMD Instinct MI355X (gfx950).

Python face of libtq.so (see include/tq.h).  torch provides device memory and
the current stream; every step of the method runs in the HIP library.

    cb = Codebook(1536, 4)                     # analytic Lloyd-Max tables
    rot = Rotation(1536, seed=42)              # Haar rotation, float32
    idx = Index(cb, rot, n_tenants=1)
    idx.add(X)                                 # X: cuda float32 [n, d]
    ids, scores = idx.search(Q, k=10)          # Q: cuda float32 [nq, d]
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from ._lib import FLAG_PREROTATED, FLAG_SLOT_ALLOW, PATHS, TQError, check, lib

__all__ = ["Codebook", "Rotation", "Index", "IdMapIndex", "TQError", "rotate_quantize",
           "rotate_queries", "version", "last_search_fallbacks"]


def version() -> str:
    return lib.tq_version().decode()


def last_search_fallbacks() -> int:
    """Queries of this thread's last search that the matrix-core path re-ran
    on the single-query scan (their top-k certificate failed)."""
    return int(lib.tq_last_search_fallbacks())


def _torch():
    import torch
    return torch


def _stream(device=None):
    torch = _torch()
    raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    if raw is not None:
        # the handle alone, without building a torch Stream object (about
        # 2 us of host time per search call)
        if device is None:
            index = torch.cuda.current_device()
        else:
            index = device.index if device.index is not None else torch.cuda.current_device()
        return ctypes.c_void_p(raw(index))
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _shape(t, shape, name):
    """Raises ValueError unless tensor t has this shape.  The library takes
    raw device pointers and cannot check the size of what they point to."""
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))


def _dev_ptr(t, dtype, name, ndim=None):
    torch = _torch()
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) torch tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must have dtype %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if ndim is not None and t.dim() != ndim:
        raise ValueError("%s must have %d dimensions" % (name, ndim))
    return ctypes.c_void_p(t.data_ptr())


class Codebook:
    """Lloyd-Max boundaries/centroids for (d, bits) -- host tables (float64)."""

    def __init__(self, d: int, bits: int = 4):
        h = ctypes.c_void_p()
        check(lib.tq_build_codebook(d, bits, ctypes.byref(h)))
        self._h = h
        self.d, self.bits = d, bits
        L = 1 << bits
        self.bounds = np.empty(L - 1, dtype=np.float64)
        self.cents = np.empty(L, dtype=np.float64)
        check(lib.tq_codebook_tables(h, self.bounds.ctypes.data_as(ctypes.c_void_p),
                                     self.cents.ctypes.data_as(ctypes.c_void_p)))
        m = ctypes.c_double()
        check(lib.tq_codebook_mse(h, ctypes.byref(m)))
        self.mse = m.value

    # the free function is bound when the class is defined: module globals may
    # already be gone when an object is collected at interpreter exit
    def __del__(self, _free=lib.tq_codebook_free):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            _free(h)
            self._h = None


class Rotation:
    """Seeded Haar orthogonal rotation, float32 row-major."""

    def __init__(self, d: int, seed: int = 42):
        h = ctypes.c_void_p()
        check(lib.tq_rotation_create(d, ctypes.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), ctypes.byref(h)))
        self._h = h
        self.d, self.seed = d, seed

    def matrix(self) -> np.ndarray:
        R = np.empty((self.d, self.d), dtype=np.float32)
        check(lib.tq_rotation_matrix(self._h, R.ctypes.data_as(ctypes.c_void_p)))
        return R

    # the free function is bound when the class is defined: module globals may
    # already be gone when an object is collected at interpreter exit
    def __del__(self, _free=lib.tq_rotation_free):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            _free(h)
            self._h = None


def rotate_quantize(cb: Codebook, rot: Rotation, X, codes=None, scales=None):
    """Encode rows of X (cuda float32 [n, d]) -> (canonical codes uint8
    [n, d*bits/8], scales float32 [n]).  Synchronises the current stream."""
    torch = _torch()
    n = X.shape[0]
    _shape(X, (n, cb.d), "X")
    _shape(codes, (n, cb.d * cb.bits // 8), "codes")
    _shape(scales, (n,), "scales")
    if codes is None:
        codes = torch.empty((n, cb.d * cb.bits // 8), dtype=torch.uint8, device=X.device)
    if scales is None:
        scales = torch.empty((n,), dtype=torch.float32, device=X.device)
    check(lib.tq_rotate_quantize(cb._h, rot._h, _dev_ptr(X, torch.float32, "X", 2), n,
                                 _dev_ptr(codes, torch.uint8, "codes"),
                                 _dev_ptr(scales, torch.float32, "scales"), _stream(X.device)))
    return codes, scales


def rotate_queries(rot: Rotation, Q, out=None):
    """q' = R q for every row of Q (cuda float32 [nq, d])."""
    torch = _torch()
    _shape(Q, (Q.shape[0], rot.d), "Q")
    _shape(out, tuple(Q.shape), "out")
    if out is None:
        out = torch.empty_like(Q)
    check(lib.tq_rotate_queries(rot._h, _dev_ptr(Q, torch.float32, "Q", 2), Q.shape[0],
                                _dev_ptr(out, torch.float32, "out"), _stream(Q.device)))
    return out


class Index:
    """Flat TurboQuant index (positional ids) on the current GPU."""

    def __init__(self, cb: Codebook, rot: Rotation, n_tenants: int = 1):
        h = ctypes.c_void_p()
        check(lib.tq_index_create(cb._h, rot._h, n_tenants, ctypes.byref(h)))
        self._adopt(h)

    def _adopt(self, h) -> None:
        self._h = h
        d, bits, t = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        check(lib.tq_index_info(h, ctypes.byref(d), ctypes.byref(bits), ctypes.byref(t), None, None))
        self.d, self.bits, self.n_tenants = d.value, bits.value, t.value
        self.words = (self.n_tenants + 63) // 64
        self._ws = None

    @property
    def n_slots(self) -> int:
        """Vectors ever added (deleted ones of an id-map index included)."""
        n = ctypes.c_int64()
        check(lib.tq_index_info(self._h, None, None, None, ctypes.byref(n), None))
        return n.value

    def slots(self, ids) -> np.ndarray:
        """Slot of each id (-1 if absent); on a positional index an id is its slot."""
        ids = np.ascontiguousarray(ids, dtype=np.uint64)
        out = np.empty(ids.shape[0], dtype=np.int64)
        check(lib.tq_index_slots(self._h, ids.ctypes.data_as(ctypes.c_void_p), ids.shape[0],
                                 out.ctypes.data_as(ctypes.c_void_p)))
        return out

    def slot_allowlist(self, id_lists, device="cuda"):
        """Slot-level allowlists for search(slot_allow=...): one list of ids
        per query -> cuda int64 [nq, ceil(n_slots/64)] (tq_slot_allowlist)."""
        torch = _torch()
        nq = len(id_lists)
        offs = np.zeros(nq + 1, dtype=np.int64)
        offs[1:] = np.cumsum([len(x) for x in id_lists])
        flat = np.ascontiguousarray(np.concatenate([np.asarray(x, dtype=np.uint64) for x in id_lists])
                                    if nq else np.zeros(0, np.uint64))
        out = torch.zeros((nq, (self.n_slots + 63) // 64), dtype=torch.int64, device=device)
        check(lib.tq_slot_allowlist(self._h, flat.ctypes.data_as(ctypes.c_void_p),
                                    offs.ctypes.data_as(ctypes.c_void_p), nq,
                                    ctypes.c_void_p(out.data_ptr()), _stream(out.device)))
        return out

    def save(self, path) -> None:
        """Writes the index to a file (tq_index_save)."""
        check(lib.tq_index_save(self._h, os.fsencode(path)))

    @classmethod
    def load(cls, cb: Codebook, rot: Rotation, path) -> "Index":
        """Reads an index written by save(); cb and rot must match its d,
        bits and rotation seed (tq_index_load)."""
        h = ctypes.c_void_p()
        check(lib.tq_index_load(os.fsencode(path), cb._h, rot._h, ctypes.byref(h)))
        idm = ctypes.c_int32()
        check(lib.tq_index_info(h, None, None, None, None, ctypes.byref(idm)))
        obj = (IdMapIndex if idm.value else Index).__new__(IdMapIndex if idm.value else Index)
        obj._adopt(h)
        return obj

    def __len__(self) -> int:
        n = ctypes.c_int64()
        check(lib.tq_index_size(self._h, ctypes.byref(n)))
        return n.value

    def reserve(self, capacity: int) -> None:
        check(lib.tq_index_reserve(self._h, capacity))

    def calibrate(self, X) -> None:
        """TQ+ calibration (section II-B) fitted to the rows of X (cuda
        float32 [m, d]) before the first vector is added (tq_index_calibrate)."""
        torch = _torch()
        _shape(X, (X.shape[0], self.d), "X")
        check(lib.tq_index_calibrate(self._h, _dev_ptr(X, torch.float32, "X", 2), X.shape[0],
                                     _stream(X.device)))

    def set_calibration(self, mu, kappa) -> None:
        """Installs a given TQ+ calibration (host float32 [d] each)."""
        mu = np.ascontiguousarray(mu, dtype=np.float32)
        kappa = np.ascontiguousarray(kappa, dtype=np.float32)
        if mu.shape != (self.d,) or kappa.shape != (self.d,):
            raise ValueError("mu and kappa must have shape (d,)")
        check(lib.tq_index_set_calibration(self._h, mu.ctypes.data_as(ctypes.c_void_p),
                                           kappa.ctypes.data_as(ctypes.c_void_p)))

    def calibration(self):
        """The installed TQ+ (mu, kappa) as float32 arrays, or None."""
        mu = np.empty(self.d, dtype=np.float32)
        kappa = np.empty(self.d, dtype=np.float32)
        has = ctypes.c_int32()
        check(lib.tq_index_calibration(self._h, mu.ctypes.data_as(ctypes.c_void_p),
                                       kappa.ctypes.data_as(ctypes.c_void_p), ctypes.byref(has)))
        return (mu, kappa) if has.value else None

    def _check_rows(self, n, X=None, codes=None, scales=None, tenants=None):
        _shape(X, (n, self.d), "X")
        _shape(codes, (n, self.d * self.bits // 8), "codes")
        _shape(scales, (n,), "scales")
        _shape(tenants, (n,), "tenants")

    def add(self, X, tenants=None) -> None:
        torch = _torch()
        self._check_rows(X.shape[0], X=X, tenants=tenants)
        check(lib.tq_index_add(self._h, _dev_ptr(X, torch.float32, "X", 2),
                               _dev_ptr(tenants, torch.int16, "tenants") if tenants is not None else None,
                               X.shape[0], _stream(X.device)))

    def add_codes(self, codes, scales, tenants=None) -> None:
        torch = _torch()
        self._check_rows(codes.shape[0], codes=codes, scales=scales, tenants=tenants)
        check(lib.tq_index_add_codes(self._h, _dev_ptr(codes, torch.uint8, "codes", 2),
                                     _dev_ptr(scales, torch.float32, "scales", 1),
                                     _dev_ptr(tenants, torch.int16, "tenants") if tenants is not None else None,
                                     codes.shape[0], _stream(codes.device)))

    def export(self, device="cuda"):
        """Every slot's (codes, scales, tenants), canonical layout; deleted
        slots of an id-map index included."""
        torch = _torch()
        n = self.n_slots
        codes = torch.empty((n, self.d * self.bits // 8), dtype=torch.uint8, device=device)
        scales = torch.empty((n,), dtype=torch.float32, device=device)
        tenants = torch.empty((n,), dtype=torch.int16, device=device)
        check(lib.tq_index_export(self._h, ctypes.c_void_p(codes.data_ptr()),
                                  ctypes.c_void_p(scales.data_ptr()),
                                  ctypes.c_void_p(tenants.data_ptr()), _stream(codes.device)))
        return codes, scales, tenants

    def workspace_bytes(self, nq: int, k: int, path: str = "auto") -> int:
        b = ctypes.c_size_t()
        check(lib.tq_search_workspace_size(self._h, nq, k, PATHS[path], ctypes.byref(b)))
        return b.value

    def search(self, Q, k: int, allow=None, path: str = "auto", ids=None, scores=None,
               workspace=None, prerotated: bool = False, slot_allow=None):
        """Top-k per query row of Q (cuda float32 [nq, d]).  allow: cuda int64
        tensor [nq, words] (bit patterns of the uint64 allowlist words) or None.
        slot_allow: slot-level allowlists from slot_allowlist() instead.
        prerotated: Q already holds R q (see rotate_queries).
        Returns (ids int64 [nq, k], scores float32 [nq, k]); an id-map index
        returns its external ids (uint64 bit patterns)."""
        torch = _torch()
        nq = Q.shape[0]
        _shape(Q, (nq, self.d), "Q")
        _shape(ids, (nq, k), "ids")
        _shape(scores, (nq, k), "scores")
        flags = FLAG_PREROTATED if prerotated else 0
        if slot_allow is not None:
            if allow is not None:
                raise ValueError("give allow or slot_allow, not both")
            _shape(slot_allow, (nq, (self.n_slots + 63) // 64), "slot_allow")
            allow, flags = slot_allow, flags | FLAG_SLOT_ALLOW
        else:
            _shape(allow, (nq, self.words), "allow")
        if ids is None:
            ids = torch.empty((nq, k), dtype=torch.int64, device=Q.device)
        if scores is None:
            scores = torch.empty((nq, k), dtype=torch.float32, device=Q.device)
        if workspace is None:
            # a workspace the caller passes is checked by the library itself
            need = self.workspace_bytes(nq, k, path)
            if self._ws is None or self._ws.numel() < need:
                self._ws = torch.empty((need,), dtype=torch.uint8, device=Q.device)
            workspace = self._ws
        check(lib.tq_search_ex(self._h, _dev_ptr(Q, torch.float32, "Q", 2), nq, k,
                               _dev_ptr(allow, torch.int64, "allow") if allow is not None else None,
                               PATHS[path] | flags,
                               ctypes.c_void_p(workspace.data_ptr()),
                               workspace.numel() * workspace.element_size(),
                               _dev_ptr(ids, torch.int64, "ids"),
                               _dev_ptr(scores, torch.float32, "scores"), _stream(Q.device)))
        return ids, scores

    def search_postfilter(self, Q, k: int, overfetch: int, allow):
        """Over-fetch post-filter baseline (tq_search_postfilter): the
        unfiltered top k * overfetch, then the first k allowed by `allow`
        (cuda int64 [nq, words])."""
        torch = _torch()
        nq = Q.shape[0]
        _shape(Q, (nq, self.d), "Q")
        _shape(allow, (nq, self.words), "allow")
        ids = torch.empty((nq, k), dtype=torch.int64, device=Q.device)
        scores = torch.empty((nq, k), dtype=torch.float32, device=Q.device)
        check(lib.tq_search_postfilter(self._h, _dev_ptr(Q, torch.float32, "Q", 2), nq, k, overfetch,
                                       _dev_ptr(allow, torch.int64, "allow"),
                                       _dev_ptr(ids, torch.int64, "ids"),
                                       _dev_ptr(scores, torch.float32, "scores"), _stream(Q.device)))
        return ids, scores

    def search_alloc(self, Q, k: int, allow=None):
        """tq_search: the library allocates its own stream-ordered workspace."""
        torch = _torch()
        nq = Q.shape[0]
        _shape(Q, (nq, self.d), "Q")
        _shape(allow, (nq, self.words), "allow")
        ids = torch.empty((nq, k), dtype=torch.int64, device=Q.device)
        scores = torch.empty((nq, k), dtype=torch.float32, device=Q.device)
        check(lib.tq_search(self._h, _dev_ptr(Q, torch.float32, "Q", 2), nq, k,
                            _dev_ptr(allow, torch.int64, "allow") if allow is not None else None,
                            _dev_ptr(ids, torch.int64, "ids"),
                            _dev_ptr(scores, torch.float32, "scores"), _stream(Q.device)))
        return ids, scores

    def search_noalloc(self, Q, k: int, allow=None, ids=None, scores=None):
        """tq_search_noalloc: tq_search with the library's own device scratch
        array as workspace (no device allocation inside the call).  ids and
        scores may be given to write into existing tensors."""
        torch = _torch()
        nq = Q.shape[0]
        _shape(Q, (nq, self.d), "Q")
        _shape(allow, (nq, self.words), "allow")
        _shape(ids, (nq, k), "ids")
        _shape(scores, (nq, k), "scores")
        if ids is None:
            ids = torch.empty((nq, k), dtype=torch.int64, device=Q.device)
        if scores is None:
            scores = torch.empty((nq, k), dtype=torch.float32, device=Q.device)
        check(lib.tq_search_noalloc(self._h, _dev_ptr(Q, torch.float32, "Q", 2), nq, k,
                                    _dev_ptr(allow, torch.int64, "allow") if allow is not None else None,
                                    _dev_ptr(ids, torch.int64, "ids"),
                                    _dev_ptr(scores, torch.float32, "scores"), _stream(Q.device)))
        return ids, scores

    # the free function is bound when the class is defined: module globals may
    # already be gone when an object is collected at interpreter exit
    def __del__(self, _free=lib.tq_index_free):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            _free(h)
            self._h = None


class IdMapIndex(Index):
    """IdMapIndex (tq_idmap_create): vectors carry uint64 ids, deletions are
    O(1), and searches return the ids."""

    def __init__(self, cb: Codebook, rot: Rotation, n_tenants: int = 1):
        h = ctypes.c_void_p()
        check(lib.tq_idmap_create(cb._h, rot._h, n_tenants, ctypes.byref(h)))
        self._adopt(h)

    def add(self, X, ids, tenants=None) -> None:
        torch = _torch()
        ids = np.ascontiguousarray(ids, dtype=np.uint64)
        if ids.shape != (X.shape[0],):
            raise ValueError("ids must have shape (n,)")
        self._check_rows(X.shape[0], X=X, tenants=tenants)
        check(lib.tq_index_add_ids(self._h, _dev_ptr(X, torch.float32, "X", 2),
                                   ids.ctypes.data_as(ctypes.c_void_p),
                                   _dev_ptr(tenants, torch.int16, "tenants") if tenants is not None else None,
                                   X.shape[0], _stream(X.device)))

    def add_codes(self, codes, scales, ids, tenants=None) -> None:
        torch = _torch()
        ids = np.ascontiguousarray(ids, dtype=np.uint64)
        if ids.shape != (codes.shape[0],):
            raise ValueError("ids must have shape (n,)")
        self._check_rows(codes.shape[0], codes=codes, scales=scales, tenants=tenants)
        check(lib.tq_index_add_codes_ids(self._h, _dev_ptr(codes, torch.uint8, "codes", 2),
                                         _dev_ptr(scales, torch.float32, "scales", 1),
                                         ids.ctypes.data_as(ctypes.c_void_p),
                                         _dev_ptr(tenants, torch.int16, "tenants") if tenants is not None else None,
                                         codes.shape[0], _stream(codes.device)))

    def remove(self, ids) -> int:
        """Deletes the vectors with these ids; returns how many were present."""
        ids = np.ascontiguousarray(ids, dtype=np.uint64)
        r = ctypes.c_int64()
        check(lib.tq_index_remove_ids(self._h, ids.ctypes.data_as(ctypes.c_void_p), ids.shape[0],
                                      ctypes.byref(r)))
        return r.value
