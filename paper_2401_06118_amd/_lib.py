"""ctypes binding of ``libaqlm_mi355x.so`` (C ABI in ``include/aqlm.h``).

Argument marshalling only: shapes and dtypes are read from torch tensors,
device pointers and the current HIP stream are passed through, and every
step of the computation runs in the library's kernels.  There is no CPU
fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libaqlm_mi355x.so")

AQLM_OK = 0
STATUS_NAMES = {0: "AQLM_OK", 1: "AQLM_ERR_NULL", 2: "AQLM_ERR_SHAPE", 3: "AQLM_ERR_UNSUPPORTED",
                4: "AQLM_ERR_ALIGN", 5: "AQLM_ERR_HIP", 6: "AQLM_ERR_WORKSPACE", 7: "AQLM_ERR_SCRATCH",
                8: "AQLM_ERR_TIMEOUT"}
PATH_AUTO, PATH_GATHER, PATH_TABLE = 0, 1, 2
EXPORTS = ("aqlm_dequantize", "aqlm_gemv", "aqlm_gemv_grouped", "aqlm_gemv_grouped_path", "aqlm_gemm_small_batch",
           "aqlm_gemm_workspace_bytes", "aqlm_gemm", "aqlm_gemm_noalloc", "aqlm_backward", "aqlm_beam_search",
           "aqlm_packed_row_words", "aqlm_gemv_step_plan_bytes", "aqlm_gemv_step_plan", "aqlm_gemv_step",
           "aqlm_gemv_step_status", "aqlm_sort_codes_size", "aqlm_sort_codes", "aqlm_gemv_sorted_workspace_bytes",
           "aqlm_gemv_sorted", "aqlm_gemv_sorted_grouped", "aqlm_status_string", "aqlm_tiled_codes_bytes",
           "aqlm_tile_codes", "aqlm_gemv_grouped_tiled", "aqlm_gemm_small_batch_tiled")
MAX_GROUPED = 8
PACKED = 0x100  # OR-ed into B: bit-packed codes
STEP_SYNC_BYTES = 256


class GemvProblem(ctypes.Structure):
    """Mirror of ``aqlm_gemv_problem`` in include/aqlm.h."""
    _fields_ = [("codes", ctypes.c_void_p), ("codebooks", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("x", ctypes.c_void_p), ("y", ctypes.c_void_p), ("d_out", ctypes.c_int64),
                ("d_in", ctypes.c_int64)]

class SortedProblem(ctypes.Structure):
    """Mirror of ``aqlm_sorted_problem`` in include/aqlm.h."""
    _fields_ = [("entries", ctypes.c_void_p), ("entry_words", ctypes.c_int64), ("index", ctypes.c_void_p),
                ("index_host", ctypes.c_void_p), ("codebooks", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("x", ctypes.c_void_p),
                ("y", ctypes.c_void_p), ("d_out", ctypes.c_int64), ("d_in", ctypes.c_int64)]


_lock = threading.Lock()
_lib = None


class AqlmError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {STATUS_NAMES.get(status, status)} ({status_string(status)})")


def load():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2401_06118_amd.build` "
                "(hipcc, gfx950). There is no CPU fallback.")
        lib = ctypes.CDLL(LIB_PATH)
        p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.aqlm_dequantize.argtypes = [p, p, p, i64, i64, i32, i32, i32, p, p]
        lib.aqlm_dequantize.restype = ctypes.c_int
        lib.aqlm_gemv.argtypes = [p, p, p, i64, i64, i32, i32, i32, p, p, p]
        lib.aqlm_gemv.restype = ctypes.c_int
        lib.aqlm_gemv_grouped.argtypes = [ctypes.POINTER(GemvProblem), i32, i32, i32, i32, p]
        lib.aqlm_gemv_grouped.restype = ctypes.c_int
        lib.aqlm_gemv_grouped_path.argtypes = [ctypes.POINTER(GemvProblem), i32, i32, i32, i32, i32, p]
        lib.aqlm_gemv_grouped_path.restype = ctypes.c_int
        lib.aqlm_tiled_codes_bytes.argtypes = [i64, i64, i32, i32, i32]
        lib.aqlm_tiled_codes_bytes.restype = i64
        lib.aqlm_tile_codes.argtypes = [p, i64, i64, i32, i32, i32, p, i64, p]
        lib.aqlm_tile_codes.restype = ctypes.c_int
        lib.aqlm_gemv_grouped_tiled.argtypes = [ctypes.POINTER(GemvProblem), i32, i32, i32, i32, p]
        lib.aqlm_gemv_grouped_tiled.restype = ctypes.c_int
        lib.aqlm_gemm_small_batch_tiled.argtypes = [p, p, p, i64, i64, i32, i32, i32, i64, p, p, p]
        lib.aqlm_gemm_small_batch_tiled.restype = ctypes.c_int
        lib.aqlm_gemm_small_batch.argtypes = [p, p, p, i64, i64, i32, i32, i32, i64, p, p, p]
        lib.aqlm_gemm_small_batch.restype = ctypes.c_int
        lib.aqlm_gemm_workspace_bytes.argtypes = [i64, i64, i32, i32, i32, i64]
        lib.aqlm_gemm_workspace_bytes.restype = ctypes.c_size_t
        lib.aqlm_gemm.argtypes = [p, p, p, i64, i64, i32, i32, i32, i64, p, p, p, ctypes.c_size_t, p]
        lib.aqlm_gemm.restype = ctypes.c_int
        lib.aqlm_gemm_noalloc.argtypes = [p, p, p, i64, i64, i32, i32, i32, i64, p, p, p]
        lib.aqlm_gemm_noalloc.restype = ctypes.c_int
        lib.aqlm_backward.argtypes = [p, p, p, i64, i64, i32, i32, i32, i64, p, p, p, p, p]
        lib.aqlm_backward.restype = ctypes.c_int
        lib.aqlm_beam_search.argtypes = [p, p, p, p, p, i64, i64, i32, i32, i32, i32, i32, p, p]
        lib.aqlm_beam_search.restype = ctypes.c_int
        lib.aqlm_packed_row_words.argtypes = [i64, i32, i32, i32]
        lib.aqlm_packed_row_words.restype = ctypes.c_int64
        lib.aqlm_gemv_step_plan_bytes.argtypes = [i32]
        lib.aqlm_gemv_step_plan_bytes.restype = ctypes.c_int64
        lib.aqlm_gemv_step_plan.argtypes = [ctypes.POINTER(GemvProblem), ctypes.POINTER(ctypes.c_int32), i32, i32,
                                            i32, i32, p, i64]
        lib.aqlm_gemv_step_plan.restype = ctypes.c_int
        lib.aqlm_gemv_step.argtypes = [p, p, p, ctypes.c_uint32, p]
        lib.aqlm_gemv_step.restype = ctypes.c_int
        lib.aqlm_gemv_step_status.argtypes = [p, p]
        lib.aqlm_gemv_step_status.restype = ctypes.c_int
        lib.aqlm_sort_codes_size.argtypes = [p, i64, i64, i32, i32, i32, ctypes.POINTER(ctypes.c_int64),
                                             ctypes.POINTER(ctypes.c_int64)]
        lib.aqlm_sort_codes_size.restype = ctypes.c_int
        lib.aqlm_sort_codes.argtypes = [p, i64, i64, i32, i32, i32, p, i64, p, i64]
        lib.aqlm_sort_codes.restype = ctypes.c_int
        lib.aqlm_gemv_sorted_workspace_bytes.argtypes = [i64, i32, i32]
        lib.aqlm_gemv_sorted_workspace_bytes.restype = ctypes.c_size_t
        lib.aqlm_gemv_sorted.argtypes = [p, i64, p, p, p, p, i64, i64, i32, i32, i32, p, p, p, ctypes.c_size_t, p]
        lib.aqlm_gemv_sorted.restype = ctypes.c_int
        lib.aqlm_gemv_sorted_grouped.argtypes = [ctypes.POINTER(SortedProblem), i32, i32, i32, i32, p,
                                                 ctypes.c_size_t, p]
        lib.aqlm_gemv_sorted_grouped.restype = ctypes.c_int
        lib.aqlm_status_string.argtypes = [ctypes.c_int]
        lib.aqlm_status_string.restype = ctypes.c_char_p
        _lib = lib
        return lib


def status_string(status: int) -> str:
    try:
        return load().aqlm_status_string(int(status)).decode()
    except RuntimeError:
        return STATUS_NAMES.get(status, "unknown")
