"""Failure paths of bsa_plan on the device (needs an MI355X): an allocation
that fails part-way through planning returns BSA_ERR_OOM with *out == NULL
and gives back every allocation the request had already made."""
import ctypes
import os

import numpy as np
import pytest

from tests.gpu_util import log, mask_to_dev
from workloads import BlockMask

pytestmark = pytest.mark.gpu

import paper_2609_25869_amd as bsa  # noqa: E402  (fails loudly if libbsa.so is missing)
from paper_2609_25869_amd import _ffi  # noqa: E402


def _free_bytes():
    import torch
    free, _total = torch.cuda.mem_get_info()
    return free


def test_failed_allocation_returns_oom_and_leaks_nothing():
    import torch
    # 8 heads x 1024 x 1024 blocks at 30%: the block-CSR columns alone take
    # about 10 MB, so a leaked request would show in the device's free memory
    B, H, N = 1, 8, 65536
    rng = np.random.default_rng(5)
    heads = [[(rng.random((N // 64, N // 64)) < 0.3).astype(np.uint8) for _ in range(H)]]
    mask = BlockMask.from_heads(heads, [64] * H, [64] * H, N, N)
    md = mask_to_dev(mask)
    q = torch.zeros((B, N, H, 128), dtype=torch.bfloat16, device="cuda")
    shapes = bsa.shapes_of(q, q, q, q)
    m = _ffi.Mask()
    m.data = md.data_ptr()
    offs = (ctypes.c_int64 * H)(*[int(x) for x in mask.head_offset])
    m.head_offset = offs
    m.stride_b = 0
    bq, bkv = (ctypes.c_int32 * 1)(64), (ctypes.c_int32 * 1)(64)
    lib = bsa._lib

    def plan_once():
        out = ctypes.c_void_p(12345)   # must be overwritten with NULL on failure
        st = lib.bsa_plan(ctypes.byref(m), bq, bkv, 1, ctypes.byref(shapes), None, None, ctypes.byref(out))
        return st, out.value

    st, handle = plan_once()
    assert st == _ffi.BSA_OK and handle
    lib.bsa_plan_destroy(ctypes.c_void_p(handle))
    torch.cuda.synchronize()
    try:
        for n in (1, 2, 3):
            os.environ["BSA_FAULT_ALLOC"] = str(n)
            st, handle = plan_once()
            torch.cuda.synchronize()
            assert st == _ffi.BSA_ERR_OOM, (n, st)
            assert handle is None, "failed plan must leave *out NULL"
            assert b"BSA_FAULT_ALLOC" in lib.bsa_last_error()
            free0 = _free_bytes()
            for _ in range(40):
                assert plan_once()[0] == _ffi.BSA_ERR_OOM
            torch.cuda.synchronize()
            drop = free0 - _free_bytes()
            log("fault at allocation %d: free device memory changed by %d bytes over 40 failed requests" % (n, drop))
            assert drop < (64 << 20), "failed requests kept device memory"
    finally:
        del os.environ["BSA_FAULT_ALLOC"]
    st, handle = plan_once()
    assert st == _ffi.BSA_OK and handle
    lib.bsa_plan_destroy(ctypes.c_void_p(handle))
    torch.cuda.synchronize()
