"""ctypes view of the C ABI declared in include/puzzlekv.h (argument marshalling only)."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpuzzlekv.so")

PKV_OK, PKV_E_ARG, PKV_E_SHAPE, PKV_E_RANK, PKV_E_STATE, PKV_E_WORKSPACE, PKV_E_UNSUPPORTED, PKV_E_HIP = range(8)
STATUS_NAMES = ["PKV_OK", "PKV_E_ARG", "PKV_E_SHAPE", "PKV_E_RANK", "PKV_E_STATE", "PKV_E_WORKSPACE",
                "PKV_E_UNSUPPORTED", "PKV_E_HIP"]
PKV_F32, PKV_BF16, PKV_INT4 = 0, 1, 2
PKV_EMPTY, PKV_DENSE, PKV_FACTOR, PKV_GLOBAL = 0, 1, 2, 3
PKV_OP_ATTENTION, PKV_OP_COMPRESS, PKV_OP_PREFILL, PKV_OP_IMPORT = 0, 1, 2, 3
PKV_OP_GLOBAL_PREFILL, PKV_OP_GLOBAL_ATTENTION = 4, 5
PKV_DEV_NOT_DENSE, PKV_DEV_BAD_PAGE, PKV_DEV_RING_OVERRUN, PKV_DEV_NO_CONVERGE, PKV_DEV_BAD_RANK = (
    0x1, 0x2, 0x4, 0x8, 0x10)
PKV_DEV_NOT_ELIGIBLE = 0x20

# Every symbol include/puzzlekv.h declares.
EXPORTS = [
    "pkv_cache_check", "pkv_dense_slots_per_head", "pkv_dense_slot_bytes", "pkv_factor_slot_bytes",
    "pkv_dense_pool_bytes", "pkv_factor_pool_bytes", "pkv_page_table_bytes", "pkv_factor_page_bytes",
    "pkv_workspace_bytes", "pkv_plan_pages", "pkv_eligible_pages", "pkv_cache_reset", "pkv_prefill",
    "pkv_append_kv", "pkv_compress_pages", "pkv_mixed_decode_attention", "pkv_mixed_decode_attention_noalloc",
    "pkv_import_pages",
    "pkv_export_block_elems", "pkv_export_pages", "pkv_int4_blob_bytes", "pkv_export_int4_pages",
    "pkv_device_status", "pkv_compress_sweeps", "pkv_cache_bytes", "pkv_last_error", "pkv_version",
    "pkv_global_basis_bytes", "pkv_global_coef_bytes", "pkv_global_rank", "pkv_global_prefill",
    "pkv_global_attention", "pkv_global_export", "pkv_bandwidth_probe",
]


class PkvFootprint(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int64) for name in ("raw_bytes", "dense_bytes", "factor_bytes",
                                                    "factor_slot_bytes", "dense_pages", "factor_pages")]


class PkvPage(ctypes.Structure):
    _fields_ = [("slot", ctypes.c_int32), ("kind", ctypes.c_uint8), ("rank_k", ctypes.c_uint8),
                ("rank_v", ctypes.c_uint8), ("rows", ctypes.c_uint8)]


class PkvCache(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("batch", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
        ("max_pages", ctypes.c_int32), ("max_rank", ctypes.c_int32), ("sink_tokens", ctypes.c_int32),
        ("window_tokens", ctypes.c_int32), ("dense_dtype", ctypes.c_int32),
        ("factor_dtype", ctypes.c_int32), ("dense_pool", ctypes.c_void_p),
        ("factor_pool", ctypes.c_void_p), ("page_table", ctypes.c_void_p),
        ("adaptive_rank_error", ctypes.c_float), ("key_rope_base", ctypes.c_float),
    ]


class PkvGlobal(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32), ("max_tokens", ctypes.c_int32), ("basis", ctypes.c_void_p),
                ("coef", ctypes.c_void_p)]


_lib = None


def load():
    """Loads libpuzzlekv.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libpuzzlekv.so is not built (%s); run __graft_entry__.build() or "
                          "python paper_2608_23843_amd/build.py" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, u32, sz, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_size_t, ctypes.c_void_p
    cp = ctypes.POINTER(PkvCache)
    gp = ctypes.POINTER(PkvGlobal)
    sig = {
        "pkv_cache_check": ([cp], i32),
        "pkv_dense_slots_per_head": ([cp], i64),
        "pkv_dense_slot_bytes": ([cp], sz),
        "pkv_factor_slot_bytes": ([cp], sz),
        "pkv_dense_pool_bytes": ([cp], sz),
        "pkv_factor_pool_bytes": ([cp], sz),
        "pkv_page_table_bytes": ([cp], sz),
        "pkv_factor_page_bytes": ([cp, i32, i32], sz),
        "pkv_workspace_bytes": ([cp, i32, i64], sz),
        "pkv_plan_pages": ([i64, i32, i32, i32, vp, i64, vp], i32),
        "pkv_eligible_pages": ([i64, i64, i32, i32, i32, vp, i64, vp], i32),
        "pkv_cache_reset": ([cp, i32, vp], i32),
        "pkv_prefill": ([cp, i32, vp, vp, i64, vp, vp, vp, i32, i32, vp, sz, vp], i32),
        "pkv_append_kv": ([cp, i32, vp, vp, vp, vp], i32),
        "pkv_compress_pages": ([cp, i32, i32, vp, vp, vp, vp, vp, vp, sz, vp], i32),
        "pkv_mixed_decode_attention": ([cp, i32, vp, vp, vp, vp, vp, sz, vp], i32),
        "pkv_mixed_decode_attention_noalloc": ([cp, i32, vp, vp, vp, vp, vp], i32),
        "pkv_import_pages": ([cp, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp], i32),
        "pkv_export_block_elems": ([cp], i64),
        "pkv_export_pages": ([cp, i32, i32, vp, vp, vp, vp, vp, sz, vp], i32),
        "pkv_int4_blob_bytes": ([cp, i32, i32], i64),
        "pkv_export_int4_pages": ([cp, i32, i32, vp, vp, vp, vp, vp], i32),
        "pkv_device_status": ([vp, ctypes.POINTER(u32)], i32),
        "pkv_compress_sweeps": ([vp, ctypes.POINTER(ctypes.c_uint64)], i32),
        "pkv_cache_bytes": ([cp, i32, vp, ctypes.POINTER(PkvFootprint), vp], i32),
        "pkv_global_basis_bytes": ([cp, gp], sz),
        "pkv_global_coef_bytes": ([cp, gp], sz),
        "pkv_global_rank": ([i64, i32, i32, i32, i32, ctypes.c_double], i32),
        "pkv_global_prefill": ([cp, gp, i32, vp, vp, i64, vp, vp, sz, vp], i32),
        "pkv_global_attention": ([cp, gp, i32, vp, vp, vp, vp, vp, sz, vp], i32),
        "pkv_global_export": ([cp, gp, i32, i32, i32, i64, vp, vp, vp, vp, vp], i32),
        "pkv_bandwidth_probe": ([vp, vp, i64, i32, i32, i32, i32, ctypes.POINTER(ctypes.c_double), vp], i32),
        "pkv_last_error": ([], ctypes.c_char_p),
        "pkv_version": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


class PuzzleKVError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        self.status = status
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__("%s: %s (%s)" % (where, name, message))


def check(status: int, where: str):
    if status != PKV_OK:
        raise PuzzleKVError(status, where, load().pkv_last_error().decode())
