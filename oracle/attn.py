"""ctypes front end of the fp64 masked-attention oracle (``attn_fp64.c``).

TEST INFRASTRUCTURE ONLY (see the package docstring).  The arithmetic lives
in ``attn_fp64.c``, which implements Eq. 1 of Section 2.1 row by row in IEEE
double; this module only marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_LIB = None
_LOCK = threading.Lock()


def build(force: bool = False) -> str:
    """Compile attn_fp64.c with gcc -O2 -fopenmp (IEEE double, no fast-math)."""
    src = os.path.join(_HERE, "attn_fp64.c")
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fno-fast-math", "-shared", "-fPIC",
                               src, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _lib():
    global _LIB
    with _LOCK:
        if _LIB is None:
            if not os.path.exists(_LIB_PATH):
                build()
            lib = ctypes.CDLL(_LIB_PATH)
            P = ctypes.c_void_p
            lib.oracle_masked_attention.restype = ctypes.c_int
            lib.oracle_masked_attention.argtypes = [
                ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                P, P, P, P, P, P, P, P, ctypes.c_int64, P, P, P, ctypes.c_int64, P, P]
            lib.oracle_num_threads.restype = ctypes.c_int
            _LIB = lib
    return _LIB


def num_threads() -> int:
    """OpenMP threads the oracle runs with."""
    return int(_lib().oracle_num_threads())


def _strides(x: np.ndarray) -> np.ndarray:
    # [B, N, H, d] element strides, reordered (batch, head, token)
    s = [st // x.itemsize for st in x.strides]
    if s[3] != 1:
        raise ValueError("head dim must be contiguous")
    return np.array([s[0], s[2], s[1]], dtype=np.int64)


def masked_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, mask,
                     rows: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """fp64 masked attention (Eq. 1).

    q: [B, Nq, H, d], k/v: [B, Nkv, H, d] bfloat16 bit arrays (uint16).
    mask: a ``workloads.BlockMask``.
    rows: optional int array [n, 3] of (b, h, i) query rows to evaluate.
    Returns (O, LSE): O is [B, Nq, H, d] (or [n, d] for `rows`) float64 and
    LSE is [B, H, Nq] (or [n]) natural-log log-sum-exp, -inf for empty rows.
    """
    for x in (q, k, v):
        if x.dtype != np.uint16 or x.ndim != 4:
            raise TypeError("q, k, v must be [B, N, H, d] uint16 (bfloat16 bits)")
    B, Nq, H, d = q.shape
    Nkv = k.shape[1]
    if k.shape != (B, Nkv, H, d) or v.shape != k.shape:
        raise ValueError("shape mismatch")
    data = np.ascontiguousarray(mask.data, dtype=np.uint8)
    hoff = np.ascontiguousarray(mask.head_offset, dtype=np.int64)
    bq = np.ascontiguousarray(mask.bq, dtype=np.int32)
    bkv = np.ascontiguousarray(mask.bkv, dtype=np.int32)
    qs, ks, vs = _strides(q), _strides(k), _strides(v)
    if rows is not None:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1, 3)
        n = rows_arr.shape[0]
        rows_ptr = rows_arr.ctypes.data
    else:
        rows_arr = None
        n = B * H * Nq
        rows_ptr = None
    out = np.empty((n, d), dtype=np.float64)
    lse = np.empty(n, dtype=np.float64)
    rc = _lib().oracle_masked_attention(
        B, H, Nq, Nkv, d, q.ctypes.data, qs.ctypes.data, k.ctypes.data, ks.ctypes.data,
        v.ctypes.data, vs.ctypes.data, data.ctypes.data, hoff.ctypes.data, int(mask.stride_b),
        bq.ctypes.data, bkv.ctypes.data, rows_ptr, n if rows is not None else 0,
        out.ctypes.data, lse.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    if rows is not None:
        return out, lse
    # rows were produced in (b, h, i) order
    O = out.reshape(B, H, Nq, d).transpose(0, 2, 1, 3).copy()
    return O, lse.reshape(B, H, Nq)
