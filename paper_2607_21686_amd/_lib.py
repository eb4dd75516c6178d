"""ctypes binding of libpcs (include/pcs.h): argument marshalling only.

Every step of the fingerprint / classify / checkpoint / restore path runs in
the library's HIP kernels; this module turns torch tensors into device
pointers and the current torch stream into the context's hipStream_t.  If
libpcs.so is missing or fails to load, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os
import warnings

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpcs.so")

OK = 0
E_INVAL, E_NOMEM, E_HANDLE, E_SHAPE, E_HIP, E_CORRUPT, E_PROBE = -1, -2, -3, -4, -5, -6, -7
CHUNK_BYTES = 4096
FLAT, RING = 0, 1
RECOMPUTABLE, MUST_SNAPSHOT = 0, 1
CKPT_HASH = 1
TIMING_OFF, TIMING_EVENTS, TIMING_DISPATCH = 0, 1, 2

_ERRNAMES = {E_INVAL: "PCS_E_INVAL", E_NOMEM: "PCS_E_NOMEM", E_HANDLE: "PCS_E_HANDLE",
             E_SHAPE: "PCS_E_SHAPE", E_HIP: "PCS_E_HIP", E_CORRUPT: "PCS_E_CORRUPT", E_PROBE: "PCS_E_PROBE"}

# Every symbol include/pcs.h declares.
EXPORTS = ("pcs_ctx_create", "pcs_ctx_destroy", "pcs_last_error", "pcs_chunk_counts", "pcs_fingerprint",
           "pcs_fingerprint_noalloc",
           "pcs_classify", "pcs_checkpoint", "pcs_checkpoint_batch", "pcs_restore", "pcs_restore_batch",
           "pcs_restore_verify", "pcs_fork", "pcs_delete", "pcs_snapshot_info", "pcs_snapshot_payload",
           "pcs_snapshot_view", "pcs_snapshot_hashes",
           "pcs_export", "pcs_import", "pcs_keep_count", "pcs_bank_shrink", "pcs_distance", "pcs_discover", "pcs_arena_stats", "pcs_set_timing", "pcs_kernel_time")


class PcsBuf(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_uint64), ("nbytes", ctypes.c_uint64), ("kind", ctypes.c_uint32),
                ("flags", ctypes.c_uint32), ("row_bytes", ctypes.c_uint64), ("capacity", ctypes.c_uint64),
                ("head", ctypes.c_uint64), ("window", ctypes.c_uint64), ("outer", ctypes.c_uint64),
                ("outer_stride", ctypes.c_uint64)]


class PcsSnapInfo(ctypes.Structure):
    _fields_ = [("state_bytes", ctypes.c_uint64), ("stored_bytes", ctypes.c_uint64),
                ("total_chunks", ctypes.c_uint64), ("dirty_chunks", ctypes.c_uint64),
                ("nbufs", ctypes.c_uint32), ("incremental", ctypes.c_uint32),
                ("has_hashes", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]


class PcsBankPart(ctypes.Structure):
    _fields_ = [("src", ctypes.c_uint64), ("dst", ctypes.c_uint64), ("entry_bytes", ctypes.c_uint64)]


DISCOVER_MAX = 64


class PcsDiscovery(ctypes.Structure):
    _fields_ = [("pcs", ctypes.c_uint8 * DISCOVER_MAX), ("necessary", ctypes.c_uint8 * DISCOVER_MAX),
                ("d_without", ctypes.c_double * DISCOVER_MAX), ("added", ctypes.c_uint32 * DISCOVER_MAX),
                ("d_necessary", ctypes.c_double), ("d_final", ctypes.c_double), ("d_control", ctypes.c_double),
                ("n_added", ctypes.c_uint32), ("probes", ctypes.c_uint32), ("control_ok", ctypes.c_int32),
                ("converged", ctypes.c_int32)]


# int (*)(void *user, pcs_snap snap, const uint8_t *h_mask, uint32_t k, double *d_out)
PROBE_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_uint64, ctypes.POINTER(ctypes.c_uint8),
                            ctypes.c_uint32, ctypes.POINTER(ctypes.c_double))


class PcsError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s: %s" % (_ERRNAMES.get(code, code), msg))
        self.code = code


def load():
    """Loads libpcs.so and declares every entry point's signature.  Warns when
    the library is older than one of its sources (a stale build)."""
    if not os.path.exists(LIB_PATH):
        raise ImportError("libpcs.so is not built (run __graft_entry__.build())")
    from . import build
    if build.stale():
        warnings.warn("libpcs.so is older than its sources; rebuild with __graft_entry__.build()", RuntimeWarning,
                      stacklevel=2)
    lib = ctypes.CDLL(LIB_PATH)
    P, U64, U32, I = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int
    PU64 = ctypes.POINTER(ctypes.c_uint64)
    PB = ctypes.POINTER(PcsBuf)
    sig = {
        "pcs_ctx_create": ([P, U64, P, ctypes.POINTER(P)], I),
        "pcs_ctx_destroy": ([P], I),
        "pcs_last_error": ([P], ctypes.c_char_p),
        "pcs_chunk_counts": ([PB, U32, PU64, PU64], I),
        "pcs_fingerprint": ([P, PB, U32, P, P, P], I),
        "pcs_fingerprint_noalloc": ([P, PB, U32, P, P, P], I),
        "pcs_classify": ([P, P, U32, PU64, U32, P, P], I),
        "pcs_checkpoint": ([P, PB, U32, U64, U32, P, P, P, PU64], I),
        "pcs_checkpoint_batch": ([P, PB, ctypes.POINTER(U32), U32, U32, P, P, P, PU64], I),
        "pcs_restore": ([P, U64, PB, U32], I),
        "pcs_restore_batch": ([P, PU64, U32, PB, ctypes.POINTER(U32)], I),
        "pcs_restore_verify": ([P, U64, PB, U32, P, P], I),
        "pcs_snapshot_view": ([P, U64, PU64, PU64], I),
        "pcs_fork": ([P, U64, PU64], I),
        "pcs_delete": ([P, U64], I),
        "pcs_snapshot_info": ([P, U64, ctypes.POINTER(PcsSnapInfo)], I),
        "pcs_snapshot_payload": ([P, U64, P, U64], I),
        "pcs_snapshot_hashes": ([P, U64, P, U64], I),
        "pcs_export": ([P, U64, P, U64, PU64], I),
        "pcs_import": ([P, P, U64, PU64], I),
        "pcs_keep_count": ([U64, U64, U64, PU64], I),
        "pcs_distance": ([P, PB, U32, P, PU64, ctypes.POINTER(ctypes.c_double)], I),
        "pcs_bank_shrink": ([P, ctypes.POINTER(PcsBankPart), U32, U64, P, U64, P], I),
        "pcs_discover": ([P, PB, U32, ctypes.c_double, ctypes.c_int32, PROBE_FN, P, ctypes.POINTER(PcsDiscovery)], I),
        "pcs_arena_stats": ([P, PU64, PU64, PU64, PU64], I),
        "pcs_set_timing": ([P, I], I),
        "pcs_kernel_time": ([P, ctypes.c_char_p, PU64, ctypes.POINTER(ctypes.c_double)], I),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = load()
    return _lib
