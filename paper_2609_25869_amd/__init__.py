"""Dynamic block-sparse attention for AMD Instinct MI355X (gfx950).

Python binding of libbsa.so (include/bsa.h).  Torch supplies device memory
and streams; every step of planning and execution runs in the library's HIP
kernels.  Importing the package raises ImportError if the library has not
been built (``python paper_2609_25869_amd/build.py``, a standalone script:
the package itself cannot be imported before the library exists).

    plan = bsa.plan(mask_dev, head_offset, stride_b, B_Q, B_KV, q, k, v, o)
    bsa.forward(plan, q, k, v, o, lse)          # warm repeats reuse the plan
"""
from __future__ import annotations

import ctypes
from typing import Dict, List, Optional, Sequence, Tuple, Union

import numpy as np

from . import _ffi
from ._ffi import (BsaError, CatalogEntry, Mask, PlanOpts, RegimeQuery, SegmentInfo, Shapes,  # noqa: F401
                   DTYPE_BF16, EXPORT_BH_NNZ, EXPORT_COL_IDX, EXPORT_DISPATCH, EXPORT_ROW_PTR, EXPORT_TASKS,
                   EXPORT_TILE_KV, EXPORT_TILE_MEMBER, EXPORT_TILE_PTR)

_lib = _ffi.load()

MAPPINGS = ("direct", "coarsened", "refined", "mixed")


def library_path() -> str:
    return _ffi.LIB_PATH


def _check(status: int):
    if status != _ffi.BSA_OK:
        msg = _lib.bsa_last_error().decode(errors="replace")
        raise BsaError(status, msg or _lib.bsa_status_string(status).decode())


def version() -> Tuple[int, int]:
    a, b = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.bsa_version(ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


# ----------------------------------------------------------------------------
# Shapes, catalog, plan table (host only)

def make_shapes(batch: int, heads: int, seq_q: int, seq_kv: int, head_dim: int = 128,
                q_stride=None, k_stride=None, v_stride=None, o_stride=None, dtype: int = DTYPE_BF16) -> Shapes:
    """Shapes of [B, N, H, d] tensors; strides (batch, head, token) default to contiguous."""
    s = Shapes()
    s.batch, s.heads, s.seq_q, s.seq_kv, s.head_dim, s.dtype = batch, heads, seq_q, seq_kv, head_dim, dtype
    dq = (seq_q * heads * head_dim, head_dim, heads * head_dim)
    dk = (seq_kv * heads * head_dim, head_dim, heads * head_dim)
    for name, st, dflt in (("q_stride", q_stride, dq), ("k_stride", k_stride, dk),
                           ("v_stride", v_stride, dk), ("o_stride", o_stride, dq)):
        arr = getattr(s, name)
        for i, x in enumerate(st if st is not None else dflt):
            arr[i] = int(x)
    return s


def shapes_of(q, k, v, o) -> Shapes:
    """Shapes of torch tensors laid out [B, N, H, d] (any strides, d contiguous)."""
    import torch
    for t in (q, k, v, o):
        if t.dtype != torch.bfloat16:
            raise TypeError("q, k, v and o must be bfloat16")
        if t.dim() != 4 or t.stride(3) != 1:
            raise ValueError("tensors must be [B, N, H, d] with d contiguous")
    B, Nq, H, d = q.shape
    Nkv = k.shape[1]
    if tuple(k.shape) != (B, Nkv, H, d) or tuple(v.shape) != (B, Nkv, H, d) or tuple(o.shape) != (B, Nq, H, d):
        raise ValueError("inconsistent q/k/v/o shapes")
    st = lambda t: (t.stride(0), t.stride(2), t.stride(1))
    return make_shapes(B, H, Nq, Nkv, d, st(q), st(k), st(v), st(o))


def catalog() -> List[Dict[str, int]]:
    out = []
    e = CatalogEntry()
    for i in range(_lib.bsa_catalog_size()):
        _check(_lib.bsa_catalog_get(i, ctypes.byref(e)))
        out.append(dict(id=e.id, tq=e.tq, tkv=e.tkv, split=e.split, stages=e.stages, waves=e.waves,
                        xcd_group=e.xcd_group))
    return out


def plan_eligible(plan_id: int, bq: int, bkv: int, shapes: Shapes) -> bool:
    r = ctypes.c_int32()
    _check(_lib.bsa_plan_eligible(plan_id, bq, bkv, ctypes.byref(shapes), ctypes.byref(r)))
    return bool(r.value)


def base_plan(bq: int, bkv: int) -> int:
    r = ctypes.c_int32()
    _check(_lib.bsa_base_plan(bq, bkv, ctypes.byref(r)))
    return r.value


class Lut:
    """A loaded plan-table artifact."""

    def __init__(self, path: str):
        h = ctypes.c_void_p()
        _check(_lib.bsa_lut_load(path.encode(), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if self.handle:
            _lib.bsa_lut_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def regime_query(bq: int, bkv: int, batch_heads: int, seq_q: int, seq_kv: int, nnz: int, blocks: int,
                 run_blocks: int, head_dim: int = 128, dtype: int = DTYPE_BF16, max_row_nnz: int = 0) -> RegimeQuery:
    z = RegimeQuery()
    z.bq, z.bkv, z.dtype, z.head_dim = bq, bkv, dtype, head_dim
    z.batch_heads, z.seq_q, z.seq_kv, z.nnz, z.blocks, z.run_blocks = batch_heads, seq_q, seq_kv, nnz, blocks, run_blocks
    z.max_row_nnz = max_row_nnz
    return z


def lut_rank(z: RegimeQuery, lut: Optional[Lut] = None) -> Tuple[List[int], bool]:
    cap = 64
    buf = (ctypes.c_int32 * cap)()
    n, hit = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.bsa_lut_rank(lut.handle if lut else None, ctypes.byref(z), buf, cap, ctypes.byref(n),
                             ctypes.byref(hit)))
    return [buf[i] for i in range(min(n.value, cap))], bool(hit.value)


def select_plan(z: RegimeQuery, shapes: Shapes, lut: Optional[Lut] = None) -> Optional[int]:
    r = ctypes.c_int32()
    st = _lib.bsa_select_plan(lut.handle if lut else None, ctypes.byref(z), ctypes.byref(shapes), ctypes.byref(r))
    if st == _ffi.BSA_ERR_UNSUPPORTED:
        return None
    _check(st)
    return r.value


# ----------------------------------------------------------------------------
# Plans (GPU)

def _stream_handle(stream) -> ctypes.c_void_p:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


class Plan:
    """An executable plan; owns its device metadata until destroy()."""

    def __init__(self, handle: ctypes.c_void_p, shapes: Shapes):
        self.handle = handle
        self.shapes = shapes

    def destroy(self):
        if self.handle:
            _lib.bsa_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def num_segments(self) -> int:
        n = ctypes.c_int32()
        _check(_lib.bsa_plan_num_segments(self.handle, ctypes.byref(n)))
        return n.value

    def info(self, segment: int = 0) -> Dict:
        i = SegmentInfo()
        _check(_lib.bsa_plan_info(self.handle, segment, ctypes.byref(i)))
        d = {f: getattr(i, f) for f, _ in SegmentInfo._fields_ if f != "reserved"}
        d["mapping_name"] = MAPPINGS[i.mapping]
        d["heads"] = self.segment_heads(segment)
        return d

    def segment_heads(self, segment: int) -> List[int]:
        buf = (ctypes.c_int32 * self.shapes.heads)()
        n = ctypes.c_int32()
        _check(_lib.bsa_plan_segment_heads(self.handle, segment, buf, self.shapes.heads, ctypes.byref(n)))
        return [buf[i] for i in range(n.value)]

    def export(self, what: int, segment: int = 0) -> np.ndarray:
        dtype = {EXPORT_ROW_PTR: np.int64, EXPORT_COL_IDX: np.int32, EXPORT_BH_NNZ: np.int64,
                 EXPORT_TILE_PTR: np.int64, EXPORT_TILE_KV: np.int32, EXPORT_TILE_MEMBER: np.uint64,
                 EXPORT_TASKS: np.int64, EXPORT_DISPATCH: np.int64}[what]
        need = ctypes.c_size_t()
        _check(_lib.bsa_plan_export(self.handle, segment, what, None, 0, ctypes.byref(need)))
        out = np.empty(need.value // np.dtype(dtype).itemsize, dtype=dtype)
        if need.value:
            _check(_lib.bsa_plan_export(self.handle, segment, what, out.ctypes.data, need.value, ctypes.byref(need)))
        if what == EXPORT_TASKS:
            out = out.reshape(-1, 6)
        return out

    def forward(self, q, k, v, o, lse=None, stream=None):
        return forward(self, q, k, v, o, lse, stream)


def plan(mask, bq: Union[int, Sequence[int]], bkv: Union[int, Sequence[int]], shapes: Shapes,
         head_offset: Optional[Sequence[int]] = None, stride_b: int = 0, force_plan: int = -1,
         select_mode: int = 0, lut: Optional[Lut] = None, stream=None, keep_row_order: bool = False) -> Plan:
    """Plan a request (bsa_plan).  `mask` is a CUDA uint8/bool tensor holding the
    logical block masks; see include/bsa.h for its layout.  keep_row_order
    dispatches the tasks in row order instead of with equal KV tile lists
    side by side (same output)."""
    import torch
    if not (isinstance(mask, torch.Tensor) and mask.is_cuda and mask.dtype in (torch.uint8, torch.bool)):
        raise TypeError("mask must be a CUDA uint8 or bool tensor")
    bqs = [int(bq)] if np.isscalar(bq) else [int(x) for x in bq]
    bkvs = [int(bkv)] if np.isscalar(bkv) else [int(x) for x in bkv]
    if len(bqs) != len(bkvs):
        raise ValueError("B_Q and B_KV lists differ in length")
    m = Mask()
    m.data = ctypes.c_void_p(mask.data_ptr())
    offs = None
    if head_offset is not None:
        offs = (ctypes.c_int64 * len(head_offset))(*[int(x) for x in head_offset])
        m.head_offset = ctypes.cast(offs, ctypes.POINTER(ctypes.c_int64))
    m.stride_b = int(stride_b)
    opts = PlanOpts()
    opts.force_plan, opts.select_mode = int(force_plan), int(select_mode)
    opts.lut = lut.handle if lut else None
    opts.keep_row_order = 1 if keep_row_order else 0
    gq = (ctypes.c_int32 * len(bqs))(*bqs)
    gk = (ctypes.c_int32 * len(bkvs))(*bkvs)
    h = ctypes.c_void_p()
    _check(_lib.bsa_plan(ctypes.byref(m), gq, gk, len(bqs), ctypes.byref(shapes), ctypes.byref(opts),
                         _stream_handle(stream), ctypes.byref(h)))
    return Plan(h, shapes)


def forward(p: Plan, q, k, v, o, lse=None, stream=None):
    """Run a plan on CUDA bf16 tensors (bsa_forward); returns o."""
    for t in (q, k, v, o):
        if not t.is_cuda:
            raise TypeError("q, k, v and o must be CUDA tensors")
    _check(_lib.bsa_forward(p.handle, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                            ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(o.data_ptr()),
                            ctypes.c_void_p(lse.data_ptr()) if lse is not None else None,
                            _stream_handle(stream)))
    return o


def sparsify_topk(q, k, bq: int, bkv: int, topk: int, diagonal: bool = True, mask=None, stream=None,
                  noalloc: bool = False):
    """Mean-pooled top-k block mask of bf16 [B, N, H, 128] tensors q and k
    (bsa_sparsify_topk): uint8 [B, H, ceil(Nq / bq), ceil(Nkv / bkv)] on the
    device, written into `mask` when given.  Pass it to plan() with
    head_offset = [h * nqb * nkb] and stride_b = H * nqb * nkb.  With
    noalloc=True the library's allocation-free entry point
    (bsa_sparsify_topk_noalloc) runs instead; pass `mask` to allocate
    nothing at all."""
    import torch
    for t in (q, k):
        if not t.is_cuda or t.dtype != torch.bfloat16 or t.dim() != 4 or t.stride(3) != 1:
            raise TypeError("q and k must be CUDA bfloat16 [B, N, H, d] tensors with d contiguous")
    B, Nq, H, d = q.shape
    Nkv = k.shape[1]
    if tuple(k.shape) != (B, Nkv, H, d):
        raise ValueError("inconsistent q/k shapes")
    nqb, nkb = -(-Nq // int(bq)), -(-Nkv // int(bkv))
    if mask is None:
        mask = torch.empty((B, H, nqb, nkb), dtype=torch.uint8, device=q.device)
    elif (tuple(mask.shape) != (B, H, nqb, nkb) or mask.dtype != torch.uint8 or not mask.is_cuda
          or not mask.is_contiguous()):
        raise ValueError("mask must be a contiguous CUDA uint8 tensor of shape %s" % ((B, H, nqb, nkb),))
    st = lambda t: (t.stride(0), t.stride(2), t.stride(1))
    shapes = make_shapes(B, H, Nq, Nkv, d, st(q), st(k), st(k), st(q))
    fn = _lib.bsa_sparsify_topk_noalloc if noalloc else _lib.bsa_sparsify_topk
    _check(fn(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()), ctypes.byref(shapes), int(bq), int(bkv),
              int(topk), 1 if diagonal else 0, ctypes.c_void_p(mask.data_ptr()), _stream_handle(stream)))
    return mask
