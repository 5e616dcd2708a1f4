"""GPU parity of the top-k sparsifier (bsa_sparsify_topk) against the oracle.

The mask is an integer result decided by floating point; both sides compute
the scores in IEEE double with the same steps, so the masks must be equal
bit for bit, ties (equal scores) included.
"""
import numpy as np
import pytest

from oracle import attn as oattn
from oracle import sparsify as osp
from tests.gpu_util import bf16_to_f64, compare, log, to_dev_bf16
from workloads import CONFIGS, BlockMask, bf16_bits_from_f32, make_qkv

pytestmark = pytest.mark.gpu

import paper_2609_25869_amd as bsa  # noqa: E402  (fails loudly if libbsa.so is missing)


def _inputs(seed, B, H, nq, nkv, d=128):
    rng = np.random.default_rng(seed)
    q = bf16_bits_from_f32(rng.standard_normal((B, nq, H, d)).astype(np.float32))
    k = bf16_bits_from_f32(rng.standard_normal((B, nkv, H, d)).astype(np.float32))
    return q, k


def _gpu_mask(q, k, bq, bkv, topk, diagonal=True):
    import torch
    m = bsa.sparsify_topk(to_dev_bf16(q), to_dev_bf16(k), bq, bkv, topk, diagonal=diagonal)
    torch.cuda.synchronize()
    return m.cpu().numpy()


# (name, B, H, Nq, Nkv, bq, bkv, topk, diagonal)
CASES = [
    ("g64_ragged", 1, 2, 1000, 1000, 64, 64, 5, True),
    ("diff_len_b2", 2, 3, 512, 768, 32, 64, 3, True),
    ("q_longer", 1, 2, 700, 300, 16, 32, 4, False),
    ("g128", 1, 1, 2048, 2048, 128, 128, 2, True),
    ("asym_128x32", 1, 2, 640, 640, 128, 32, 6, True),
    ("asym_32x128", 1, 2, 640, 640, 32, 128, 2, True),
    ("diag_only", 1, 2, 256, 256, 64, 64, 0, True),
    ("all_blocks", 1, 2, 256, 256, 64, 64, 100, True),
    ("many_cols", 1, 1, 300, 64 * 700 + 5, 64, 64, 37, True),
    # the largest supported score row: 6144 KV blocks (the host rejects 6145)
    ("max_kv_blocks", 1, 1, 128, 16 * 6144, 16, 16, 50, True),
]


@pytest.mark.parametrize("name", [c[0] for c in CASES])
def test_mask_matches_oracle_bitwise(name):
    _, B, H, nq, nkv, bq, bkv, topk, diag = [c for c in CASES if c[0] == name][0]
    log("sparsify case %s" % name)
    q, k = _inputs(sum(map(ord, name)), B, H, nq, nkv)
    want, _ = osp.sparsify_topk(q, k, bq, bkv, topk, diagonal=diag)
    got = _gpu_mask(q, k, bq, bkv, topk, diag)
    assert got.shape == want.shape
    assert np.array_equal(got, want), "%s: %d of %d mask entries differ" % (name, int((got != want).sum()), got.size)


def test_equal_scores_go_to_the_lower_kv_block():
    """Duplicated key blocks give exactly equal scores; the lower block wins."""
    q, k = _inputs(71, 1, 2, 512, 512)
    bkv = 32
    for src, dst in ((0, 3), (0, 9), (4, 5), (4, 12)):
        k[:, dst * bkv:(dst + 1) * bkv] = k[:, src * bkv:(src + 1) * bkv]
    for topk in (1, 2, 3, 5, 8):
        want, scores = osp.sparsify_topk(q, k, 32, bkv, topk, diagonal=False)
        assert np.any(scores[0, 0, :, 0] == scores[0, 0, :, 3])
        got = _gpu_mask(q, k, 32, bkv, topk, diagonal=False)
        assert np.array_equal(got, want), topk


def test_strided_views_match_contiguous_inputs():
    import torch
    q, k = _inputs(72, 2, 3, 640, 640)
    qd, kd = to_dev_bf16(q), to_dev_bf16(k)
    # [B, H, N, d] storage viewed as [B, N, H, d]
    qs = qd.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
    ks = kd.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
    a = bsa.sparsify_topk(qd, kd, 64, 64, 4)
    b = bsa.sparsify_topk(qs, ks, 64, 64, 4)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_sparsify_plan_forward_on_device_matches_oracle():
    """The whole request on the device: sparsifier mask -> bsa_plan -> bsa_forward."""
    import torch
    B, H, N, bq, bkv, topk = 1, 2, 1000, 64, 64, 3
    rng = np.random.default_rng(73)
    q, k = _inputs(73, B, H, N, N)
    v = bf16_bits_from_f32(rng.standard_normal((B, N, H, 128)).astype(np.float32))
    qd, kd, vd = to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v)
    md = bsa.sparsify_topk(qd, kd, bq, bkv, topk)
    nqb, nkb = md.shape[2], md.shape[3]
    od = torch.empty_like(qd)
    p = bsa.plan(md, bq, bkv, bsa.shapes_of(qd, kd, vd, od), head_offset=[h * nqb * nkb for h in range(H)],
                 stride_b=H * nqb * nkb)
    bsa.forward(p, qd, kd, vd, od)
    torch.cuda.synchronize()
    p.destroy()
    want_mask, _ = osp.sparsify_topk(q, k, bq, bkv, topk)
    mask = BlockMask.from_heads([[want_mask[0, h] for h in range(H)]], [bq] * H, [bkv] * H, N, N)
    O_ref, _ = oattn.masked_attention(q, k, v, mask)
    compare(bf16_to_f64(od), O_ref, "sparsify -> plan -> forward")


def test_full_size_topk_workload_sampled_heads():
    """The 24-head, 115200-token, (64, 64) top-12% workload: the device mask
    of sampled heads equals the oracle's bit for bit."""
    import torch
    cfg = CONFIGS["c3_topk"]
    q, k, _ = make_qkv(cfg)
    nkb = -(-cfg.N // 64)
    topk = int(np.floor(cfg.params["frac"] * nkb + 0.5))
    log("full-size top-k: N %d, %d KV blocks, k = %d" % (cfg.N, nkb, topk))
    md = bsa.sparsify_topk(to_dev_bf16(q), to_dev_bf16(k), 64, 64, topk)
    torch.cuda.synchronize()
    got = md.cpu().numpy()
    for h in (0, 11, cfg.H - 1):
        want, _ = osp.sparsify_topk(q[:, :, h:h + 1], k[:, :, h:h + 1], 64, 64, topk)
        assert np.array_equal(got[:, h], want[:, 0]), "head %d differs in %d entries" % (h, int((got[:, h] != want[:, 0]).sum()))
    dens = got.mean()
    log("full-size top-k density %.4f" % dens)
    assert 0.119 <= dens <= 0.121
