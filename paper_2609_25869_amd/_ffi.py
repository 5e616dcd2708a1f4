"""ctypes declarations of libbsa.so (the C-ABI in include/bsa.h).

Argument marshalling only: every step of the request path runs in the
library's HIP kernels.  Importing this module fails loudly when the library
has not been built.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbsa.so")

c_i32, c_i64, c_sz, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p

BSA_OK, BSA_ERR_INVALID, BSA_ERR_UNSUPPORTED, BSA_ERR_HIP, BSA_ERR_OOM, BSA_ERR_LUT = range(6)
DTYPE_BF16, DTYPE_F16, DTYPE_F32 = 0, 1, 2
(EXPORT_ROW_PTR, EXPORT_COL_IDX, EXPORT_BH_NNZ, EXPORT_TILE_PTR, EXPORT_TILE_KV, EXPORT_TILE_MEMBER, EXPORT_TASKS,
 EXPORT_DISPATCH) = range(8)
MAX_SEGMENTS = 16


class Shapes(ctypes.Structure):
    _fields_ = [("batch", c_i32), ("heads", c_i32), ("seq_q", c_i32), ("seq_kv", c_i32),
                ("head_dim", c_i32), ("dtype", c_i32),
                ("q_stride", c_i64 * 3), ("k_stride", c_i64 * 3), ("v_stride", c_i64 * 3),
                ("o_stride", c_i64 * 3)]


class Mask(ctypes.Structure):
    _fields_ = [("data", c_vp), ("head_offset", ctypes.POINTER(c_i64)), ("stride_b", c_i64)]


class PlanOpts(ctypes.Structure):
    _fields_ = [("force_plan", c_i32), ("select_mode", c_i32), ("lut", c_vp), ("keep_row_order", c_i32)]


class SegmentInfo(ctypes.Structure):
    _fields_ = [("bq", c_i32), ("bkv", c_i32), ("n_heads", c_i32), ("plan_id", c_i32), ("tq", c_i32),
                ("tkv", c_i32), ("split", c_i32), ("mapping", c_i32), ("regime_hit", c_i32),
                ("reserved", c_i32), ("nnz", c_i64), ("blocks", c_i64), ("run_blocks", c_i64),
                ("max_row_nnz", c_i64), ("n_rows", c_i64), ("n_tiles", c_i64), ("n_tasks", c_i64),
                ("workspace_bytes", c_i64)]


class CatalogEntry(ctypes.Structure):
    _fields_ = [("id", c_i32), ("tq", c_i32), ("tkv", c_i32), ("split", c_i32), ("stages", c_i32),
                ("waves", c_i32), ("xcd_group", c_i32)]


class RegimeQuery(ctypes.Structure):
    _fields_ = [("bq", c_i32), ("bkv", c_i32), ("dtype", c_i32), ("head_dim", c_i32),
                ("batch_heads", c_i64), ("seq_q", c_i64), ("seq_kv", c_i64),
                ("nnz", c_i64), ("blocks", c_i64), ("run_blocks", c_i64), ("max_row_nnz", c_i64)]


# (name, restype, argtypes) of every exported entry point
SIGNATURES = [
    ("bsa_version", c_i32, [ctypes.POINTER(c_i32), ctypes.POINTER(c_i32)]),
    ("bsa_status_string", ctypes.c_char_p, [c_i32]),
    ("bsa_last_error", ctypes.c_char_p, []),
    ("bsa_lut_load", c_i32, [ctypes.c_char_p, ctypes.POINTER(c_vp)]),
    ("bsa_lut_destroy", c_i32, [c_vp]),
    ("bsa_lut_rank", c_i32, [c_vp, ctypes.POINTER(RegimeQuery), ctypes.POINTER(c_i32), c_i32,
                             ctypes.POINTER(c_i32), ctypes.POINTER(c_i32)]),
    ("bsa_select_plan", c_i32, [c_vp, ctypes.POINTER(RegimeQuery), ctypes.POINTER(Shapes),
                                ctypes.POINTER(c_i32)]),
    ("bsa_catalog_size", c_i32, []),
    ("bsa_catalog_get", c_i32, [c_i32, ctypes.POINTER(CatalogEntry)]),
    ("bsa_plan_eligible", c_i32, [c_i32, c_i32, c_i32, ctypes.POINTER(Shapes), ctypes.POINTER(c_i32)]),
    ("bsa_base_plan", c_i32, [c_i32, c_i32, ctypes.POINTER(c_i32)]),
    ("bsa_plan", c_i32, [ctypes.POINTER(Mask), ctypes.POINTER(c_i32), ctypes.POINTER(c_i32), c_i32,
                         ctypes.POINTER(Shapes), ctypes.POINTER(PlanOpts), c_vp, ctypes.POINTER(c_vp)]),
    ("bsa_forward", c_i32, [c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]),
    ("bsa_plan_num_segments", c_i32, [c_vp, ctypes.POINTER(c_i32)]),
    ("bsa_plan_info", c_i32, [c_vp, c_i32, ctypes.POINTER(SegmentInfo)]),
    ("bsa_plan_segment_heads", c_i32, [c_vp, c_i32, ctypes.POINTER(c_i32), c_i32, ctypes.POINTER(c_i32)]),
    ("bsa_plan_export", c_i32, [c_vp, c_i32, c_i32, c_vp, c_sz, ctypes.POINTER(c_sz)]),
    ("bsa_plan_destroy", c_i32, [c_vp]),
    ("bsa_sparsify_topk", c_i32, [c_vp, c_vp, ctypes.POINTER(Shapes), c_i32, c_i32, c_i32, c_i32, c_vp, c_vp]),
    ("bsa_sparsify_topk_noalloc", c_i32, [c_vp, c_vp, ctypes.POINTER(Shapes), c_i32, c_i32, c_i32, c_i32, c_vp,
                                          c_vp]),
]


def load() -> ctypes.CDLL:
    # PyTorch ships its own HIP runtime.  Import it first so that libbsa.so
    # binds to that runtime instead of loading a second one into the process
    # (device pointers and streams must come from one runtime).
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise ImportError("libbsa.so is not built at %s; run `python paper_2609_25869_amd/build.py`" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


class BsaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s (status %d)" % (message, status))
        self.status = status
