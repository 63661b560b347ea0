"""ctypes declarations of the C ABI in include/tl.h and the library loader.

The shared library is built in-tree (``paper_2408_05235_amd/lib/libtl.so``).
Loading never falls back to anything else: if the library is missing it is
built once; if it cannot be built or loaded an ImportError is raised.
"""
from __future__ import annotations

import ctypes
import os

from . import build as _build

P = ctypes.c_void_p
i32, i64, u32, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_float

TL_OK, TL_EINVAL, TL_ENOMEM, TL_EDEVICE, TL_EUNSUPPORTED = 0, 1, 2, 3, 4
FLAG_BAD_REQUEST, FLAG_LOST, FLAG_OVERCOMMIT, FLAG_OVERFLOW, FLAG_UNSORTED = 1, 2, 4, 8, 16
FLAG_BAD_CANDIDATE = 32
STATUS_OK, STATUS_INFEASIBLE, STATUS_LOST, STATUS_INVALID = 0, 1, 2, 3
ADMIT_OK, ADMIT_LOST, ADMIT_QUEUE_CAPACITY, ADMIT_QUEUE_TBT, ADMIT_QUEUE_E2E, ADMIT_INVALID = 0, 1, 2, 3, 4, 5
MAX_HORIZON, MAX_BLOCK_TOKENS, MAX_FREQS, MAX_FEATURES, MAX_DEPTH = 8192, 65536, 4096, 4, 14

EXPORTED = ("tl_abi_version", "tl_last_error", "tl_forest_create", "tl_forest_destroy",
            "tl_project", "tl_forest_predict", "tl_forest_predict_grid", "tl_select_freq", "tl_admit",
            "tl_select_freq_binary", "tl_adjust_lengths", "tl_lattice_create", "tl_lattice_destroy",
            "tl_lattice_bytes", "tl_lattice_predict_grid", "tl_forest_predict_grid_noalloc")


class ProjectArgs(ctypes.Structure):
    _fields_ = [
        ("struct_size", u32), ("horizon", i32), ("n_scenarios", i64), ("n_requests", i64),
        ("block_tokens", i32), ("n_freqs", i32), ("n_features", i32), ("reserved", i32),
        ("req_offset", P), ("prompt_len", P), ("generated", P), ("remaining", P),
        ("arrival_iter", P), ("deadline_ns", P), ("lost", P), ("kv_capacity", P),
        ("batch_cap", P), ("batch", P), ("kv", P), ("deadline_at", P), ("n_iters", P),
        ("flags", P), ("freqs_mhz", P), ("engine_size", P), ("rows", P),
    ]


class AdmitArgs(ctypes.Structure):
    _fields_ = [
        ("struct_size", u32), ("reserved", u32), ("proj", ProjectArgs), ("forest", P),
        ("max_freq_mhz", f32), ("engine_size", P), ("tbt_slo_ns", P), ("cand_prompt", P),
        ("cand_len", P), ("cand_deadline_ns", P), ("ips", P), ("decision", P), ("lattice", P),
    ]


class TLError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"tl status {status}: {message}")
        self.status = status


_lib = None


def lib():
    """The loaded libtl.so (built first if it does not exist yet)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB_PATH):
        _build.build_library()
    try:
        L = ctypes.CDLL(_build.LIB_PATH)
    except OSError as e:
        raise ImportError(f"cannot load {_build.LIB_PATH}: {e}") from e
    L.tl_abi_version.argtypes = []
    L.tl_abi_version.restype = i32
    L.tl_last_error.argtypes = []
    L.tl_last_error.restype = ctypes.c_char_p
    L.tl_forest_create.argtypes = [i32, i32, i32, f32, P, P, P, ctypes.POINTER(P)]
    L.tl_forest_create.restype = ctypes.c_int
    L.tl_forest_destroy.argtypes = [P]
    L.tl_forest_destroy.restype = None
    L.tl_project.argtypes = [ctypes.POINTER(ProjectArgs), P]
    L.tl_project.restype = ctypes.c_int
    L.tl_forest_predict.argtypes = [P, P, i64, P, P]
    L.tl_forest_predict.restype = ctypes.c_int
    L.tl_forest_predict_grid.argtypes = [P, i64, i32, i32, P, P, P, P, P, P]
    L.tl_forest_predict_grid.restype = ctypes.c_int
    L.tl_forest_predict_grid_noalloc.argtypes = [P, i64, i32, i32, P, P, P, P, P, P]
    L.tl_forest_predict_grid_noalloc.restype = ctypes.c_int
    L.tl_select_freq.argtypes = [P, i64, i32, i32, P, P, P, P, P, P, P]
    L.tl_select_freq.restype = ctypes.c_int
    L.tl_select_freq_binary.argtypes = [P, i64, i32, i32] + [P] * 14
    L.tl_select_freq_binary.restype = ctypes.c_int
    L.tl_lattice_create.argtypes = [P, i32, P, i32, P, i32, i32, P, ctypes.POINTER(P)]
    L.tl_lattice_create.restype = ctypes.c_int
    L.tl_lattice_destroy.argtypes = [P]
    L.tl_lattice_destroy.restype = None
    L.tl_lattice_bytes.argtypes = [P]
    L.tl_lattice_bytes.restype = ctypes.c_uint64
    L.tl_lattice_predict_grid.argtypes = [P, i64, i32, P, P, P, P, P]
    L.tl_lattice_predict_grid.restype = ctypes.c_int
    L.tl_adjust_lengths.argtypes = [i64, i64] + [P] * 8
    L.tl_adjust_lengths.restype = ctypes.c_int
    L.tl_admit.argtypes = [ctypes.POINTER(AdmitArgs), P]
    L.tl_admit.restype = ctypes.c_int
    _lib = L
    return L


def check(status):
    if status != TL_OK:
        msg = lib().tl_last_error()
        raise TLError(status, msg.decode() if msg else "")
    return status
