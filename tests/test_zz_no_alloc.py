"""The allocation-free sparsifier entry point (bsa_sparsify_topk_noalloc)
against the allocating one (bsa_sparsify_topk), through the C-ABI.

The mask is integer output, so the two must agree bit for bit.  Two calls in
a row, the second on a smaller input, check that the shared scratch carries
nothing from one call into the next; a head too large for the scratch is
rejected on the host before any device work.
"""
import ctypes

import numpy as np
import pytest

from tests.gpu_util import log

pytestmark = pytest.mark.gpu

import paper_2609_25869_amd as bsa  # noqa: E402  (fails loudly if libbsa.so is missing)
from paper_2609_25869_amd import _ffi  # noqa: E402

SCRATCH_BYTES = 64 << 20


def _qk(seed, B, H, nq, nkv):
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    q = torch.randn((B, nq, H, 128), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    k = torch.randn((B, nkv, H, 128), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    return q, k


def _both(q, k, bq, bkv, topk, diagonal):
    import torch
    B, nq, H, _ = q.shape
    nkv = k.shape[1]
    nqb, nkb = -(-nq // bq), -(-nkv // bkv)
    # the outputs start as different garbage, so an unwritten byte shows
    ref = torch.full((B, H, nqb, nkb), 7, dtype=torch.uint8, device="cuda")
    out = torch.full((B, H, nqb, nkb), 9, dtype=torch.uint8, device="cuda")
    bsa.sparsify_topk(q, k, bq, bkv, topk, diagonal=diagonal, mask=ref)
    bsa.sparsify_topk(q, k, bq, bkv, topk, diagonal=diagonal, mask=out, noalloc=True)
    torch.cuda.synchronize()
    return ref.cpu().numpy(), out.cpu().numpy()


def test_two_calls_in_a_row_match_the_allocating_entry_point():
    # first call: one head's means and scores take 37.7 MiB, so the scratch
    # holds one head per pass and the three heads need three passes
    cases = [("N131072_H3_g64", 11, 1, 3, 131072, 131072, 64, 64, 245, True),
             ("N3000_H2_b2_ragged", 12, 2, 2, 3000, 2500, 64, 32, 9, False)]
    for name, seed, B, H, nq, nkv, bq, bkv, topk, diag in cases:
        log("no-alloc sparsifier case %s" % name)
        q, k = _qk(seed, B, H, nq, nkv)
        ref, out = _both(q, k, bq, bkv, topk, diag)
        assert set(np.unique(ref)) <= {0, 1}
        assert np.array_equal(out, ref), "%s: %d mask entries differ" % (name, int((out != ref).sum()))
        log("  %d x %d blocks per head, %d active, identical" % (ref.shape[2], ref.shape[3], int(ref.sum())))
        del q, k


def test_head_beyond_the_scratch_is_rejected_before_device_work():
    import torch
    q, k = _qk(13, 1, 1, 64, 64)
    mask = torch.full((4,), 5, dtype=torch.uint8, device="cuda")
    # claim 3000 x 3000 blocks of 64 tokens per head: 72 MB of scores
    n = 3000 * 64
    st = (n * 128, 128, 128)
    shapes = bsa.make_shapes(1, 1, n, n, 128, st, st, st, st)
    lib = bsa._lib
    status = lib.bsa_sparsify_topk_noalloc(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                                           ctypes.byref(shapes), 64, 64, 8, 1, ctypes.c_void_p(mask.data_ptr()), None)
    assert status == _ffi.BSA_ERR_INVALID
    assert b"scratch" in lib.bsa_last_error()
    torch.cuda.synchronize()
    assert mask.cpu().tolist() == [5, 5, 5, 5]
    # the largest head that fits is accepted by the same check: 2048 x 2048
    # blocks need 37.7 MiB (exercised by the first test)
    assert (2048 + 2048) * 1024 + 2048 * 2048 * 8 <= SCRATCH_BYTES < (3000 + 3000) * 1024 + 3000 * 3000 * 8
