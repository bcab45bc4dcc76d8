"""ctypes binding of libtq.so (argument marshalling only).

Every operation runs in the HIP library; this module converts torch tensors
to device pointers, passes the current HIP stream and turns status codes into
exceptions.  If libtq.so has not been built the import fails loudly: there is
no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# TQ_LIBRARY names another build of the same sources (the host-sanitizer
# build of sanitize.py); by default the in-tree libtq.so
LIB_PATH = os.environ.get("TQ_LIBRARY") or os.path.join(HERE, "libtq.so")

TQ_OK, TQ_EINVAL, TQ_ENOMEM, TQ_EDEVICE, TQ_EUNSUPPORTED = 0, -1, -2, -3, -4
PATHS = {"auto": 0, "lut": 1, "mfma": 2}
FLAG_PREROTATED = 0x100
FLAG_SLOT_ALLOW = 0x200
_STATUS = {TQ_EINVAL: "TQ_EINVAL", TQ_ENOMEM: "TQ_ENOMEM", TQ_EDEVICE: "TQ_EDEVICE",
           TQ_EUNSUPPORTED: "TQ_EUNSUPPORTED"}


class TQError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (_STATUS.get(status, str(status)), message))
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libtq.so is not built (run `python paper_2607_16973_amd/build.py`); "
                          "there is no fallback implementation")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U64, SZ = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                            ctypes.c_uint64, ctypes.c_size_t)
    PP = ctypes.POINTER(ctypes.c_void_p)
    sig = {
        "tq_last_error": ([], ctypes.c_char_p),
        "tq_version": ([], ctypes.c_char_p),
        "tq_build_codebook": ([I32, I32, PP], ctypes.c_int),
        "tq_codebook_tables": ([P, P, P], ctypes.c_int),
        "tq_codebook_mse": ([P, P], ctypes.c_int),
        "tq_codebook_free": ([P], None),
        "tq_rotation_create": ([I32, U64, PP], ctypes.c_int),
        "tq_rotation_matrix": ([P, P], ctypes.c_int),
        "tq_rotation_free": ([P], None),
        "tq_rotate_quantize": ([P, P, P, I64, P, P, P], ctypes.c_int),
        "tq_rotate_queries": ([P, P, I64, P, P], ctypes.c_int),
        "tq_index_create": ([P, P, I32, PP], ctypes.c_int),
        "tq_index_reserve": ([P, I64], ctypes.c_int),
        "tq_index_add": ([P, P, P, I64, P], ctypes.c_int),
        "tq_index_add_codes": ([P, P, P, P, I64, P], ctypes.c_int),
        "tq_index_size": ([P, P], ctypes.c_int),
        "tq_index_export": ([P, P, P, P, P], ctypes.c_int),
        "tq_index_info": ([P, P, P, P, P, P], ctypes.c_int),
        "tq_index_calibrate": ([P, P, I64, P], ctypes.c_int),
        "tq_index_set_calibration": ([P, P, P], ctypes.c_int),
        "tq_index_calibration": ([P, P, P, P], ctypes.c_int),
        "tq_idmap_create": ([P, P, I32, P], ctypes.c_int),
        "tq_index_add_ids": ([P, P, P, P, I64, P], ctypes.c_int),
        "tq_index_add_codes_ids": ([P, P, P, P, P, I64, P], ctypes.c_int),
        "tq_index_remove_ids": ([P, P, I64, P], ctypes.c_int),
        "tq_index_slots": ([P, P, I64, P], ctypes.c_int),
        "tq_slot_allowlist": ([P, P, P, I64, P, P], ctypes.c_int),
        "tq_index_save": ([P, ctypes.c_char_p], ctypes.c_int),
        "tq_index_load": ([ctypes.c_char_p, P, P, P], ctypes.c_int),
        "tq_index_free": ([P], None),
        "tq_search": ([P, P, I64, I32, P, P, P, P], ctypes.c_int),
        "tq_search_postfilter": ([P, P, I64, I32, I32, P, P, P, P], ctypes.c_int),
        "tq_search_workspace_size": ([P, I64, I32, I32, P], ctypes.c_int),
        "tq_search_ex": ([P, P, I64, I32, P, I32, P, SZ, P, P, P], ctypes.c_int),
        "tq_search_noalloc": ([P, P, I64, I32, P, P, P, P], ctypes.c_int),
        "tq_last_search_fallbacks": ([], ctypes.c_int32),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


lib = _load()
EXPORTED = ("tq_last_error", "tq_version", "tq_build_codebook", "tq_codebook_tables",
            "tq_codebook_mse", "tq_codebook_free", "tq_rotation_create", "tq_rotation_matrix",
            "tq_rotation_free", "tq_rotate_quantize", "tq_rotate_queries", "tq_index_create",
            "tq_index_reserve", "tq_index_add", "tq_index_add_codes", "tq_index_size",
            "tq_index_export", "tq_index_info", "tq_index_save", "tq_index_load",
            "tq_idmap_create", "tq_index_add_ids", "tq_index_add_codes_ids", "tq_index_remove_ids",
            "tq_index_slots", "tq_slot_allowlist", "tq_index_calibrate",
            "tq_index_set_calibration", "tq_index_calibration",
            "tq_index_free", "tq_search", "tq_search_postfilter", "tq_search_workspace_size",
            "tq_search_ex", "tq_search_noalloc", "tq_last_search_fallbacks")


def check(status: int) -> None:
    if status != TQ_OK:
        msg = lib.tq_last_error()
        raise TQError(status, msg.decode() if msg else "")
