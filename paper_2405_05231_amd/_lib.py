"""ctypes loader for libdg.so (the HIP library).  Fails loudly when the library
has not been built: there is no fallback implementation."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# DG_LIB_PATH: another build of the same library (the host-sanitizer tests
# load one); by default the in-tree build.
LIB_PATH = os.environ.get("DG_LIB_PATH") or os.path.join(_HERE, "libdg.so")

DG_OK, DG_EINVAL, DG_ECAPACITY, DG_EHIP, DG_EWORKSPACE = 0, -1, -2, -3, -4
DG_SAMPLE_LAYERED = 1
DG_SAMPLE_DIRECT = 2
DG_SAMPLE_EXIT_CLEAR = 4
DG_SAMPLE_ENTRY_CLEAR = 8
DG_PACK_CLEAR_MEMBERSHIP = 1
DG_PACK_ROWS_STREAM = 2
DG_PACK_LOC_PENDING = 4
DG_LOC_PENDING = 0x7fffffff
DG_MAX_BATCHES = 64
STATUS_NAMES = {0: "DG_OK", -1: "DG_EINVAL", -2: "DG_ECAPACITY", -3: "DG_EHIP",
                -4: "DG_EWORKSPACE"}

I64 = ctypes.c_int64
I32 = ctypes.c_int32
U64 = ctypes.c_uint64
U32 = ctypes.c_uint32
VP = ctypes.c_void_p
SZ = ctypes.c_size_t
I32P = ctypes.POINTER(ctypes.c_int32)
I64P = ctypes.POINTER(ctypes.c_int64)


class Csr(ctypes.Structure):
    _fields_ = [("num_nodes", I64), ("num_edges", I64), ("offsets", VP), ("indices", VP)]


class Sizes(ctypes.Structure):
    _fields_ = [("max_batch_nodes", I64), ("max_batch_edges", I64), ("total_nodes", I64),
                ("total_edges", I64), ("packed_rows", I64), ("unique_nodes", I64),
                ("unique_packed", I64), ("exact", I32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class Timing(ctypes.Structure):
    _fields_ = [("sample_ms", ctypes.c_float), ("dedup_ms", ctypes.c_float),
                ("relabel_ms", ctypes.c_float), ("mark_ms", ctypes.c_float),
                ("order_ms", ctypes.c_float), ("loc_ms", ctypes.c_float),
                ("gather_ms", ctypes.c_float), ("total_ms", ctypes.c_float)]

    def as_dict(self):
        return {k: float(getattr(self, k)) for k, _ in self._fields_}


# every entry point of include/dg.h with its ctypes signature
SIGNATURES = {
    "dg_version": (ctypes.c_char_p, []),
    "dg_last_error": (ctypes.c_char_p, []),
    "dg_sample_bounds": (ctypes.c_int, [I64, I64, I32, I32P, I32, ctypes.c_uint32, I64P, I64P]),
    "dg_sample_workspace_bytes": (SZ, [I64, I32, I64, I64, U32]),
    "dg_member_lines_bytes": (SZ, [I64]),
    "dg_sample_group": (ctypes.c_int, [ctypes.POINTER(Csr), VP, I32, I32, I64, I32P, I32, U64,
                                       ctypes.c_uint32, I64, VP, I64P, I64, VP, VP, I64P, VP,
                                       VP, VP, VP, VP, SZ, VP,
                                       ctypes.POINTER(Sizes), ctypes.POINTER(Timing)]),
    "dg_pack_workspace_bytes": (SZ, [I64, I32, I64]),
    "dg_pack_group": (ctypes.c_int, [VP, I64, I64, VP, I32, VP, I64, I64P, I64, VP, VP, VP, I64P,
                                     VP, VP, I64, VP, VP, VP, I64, VP, U32, VP, SZ, VP, VP,
                                     ctypes.POINTER(Sizes), ctypes.POINTER(Timing)]),
    "dg_sample_pack_workspace_bytes": (SZ, [I64, I32, I64]),
    "dg_sample_pack_group": (ctypes.c_int, [ctypes.POINTER(Csr), VP, I32, I32, I64, I32P, I32,
                                            U64, ctypes.c_uint32, I64, VP, I64P, I64, VP, VP,
                                            I64P, VP, VP, VP, VP, I64, I64, VP, VP, VP, I64P,
                                            VP, I64, U32, VP, SZ, VP, SZ, VP, VP,
                                            ctypes.POINTER(Sizes), ctypes.POINTER(Timing)]),
    "dg_pack_noalloc_scratch_bytes": (SZ, []),
    "dg_pack_group_noalloc": (ctypes.c_int, [VP, I64, I64, VP, I32, VP, I64, I64P, I64, VP, VP,
                                             VP, I64P, VP, VP, I64, VP, VP, VP, I64, VP, U32,
                                             VP, ctypes.POINTER(Sizes)]),
    "dg_assemble_batch": (ctypes.c_int, [VP, I64, VP, I64, VP, I64, I64, VP, VP, VP]),
    "dg_assemble_batches": (ctypes.c_int, [VP, I64, VP, I64P, VP, I64, I64P, I32, I64,
                                           ctypes.POINTER(VP), I32, VP, VP]),
    "dg_cache_workspace_bytes": (SZ, [I64]),
    "dg_cache_by_frequency": (ctypes.c_int, [VP, I64, I32, I64, VP, VP, I64P, VP, SZ, VP]),
    "dg_gather_rows": (ctypes.c_int, [VP, I64, I64, VP, I64, VP, VP, VP]),
    "dg_minhash_workspace_bytes": (SZ, [I64]),
    "dg_minhash_order": (ctypes.c_int, [VP, I64, I32, VP, I64, VP, I32, VP, VP, VP, SZ, VP]),
}

_lib = None


class DGError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"libdg.so not found at {LIB_PATH}: build it first "
                "(python paper_2405_05231_amd/build.py, or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def check(status: int):
    if status != DG_OK:
        raise DGError(status, load().dg_last_error().decode())
