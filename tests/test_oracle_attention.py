"""Pins for the fp64 attention oracle (CPU only).

Each test ties the oracle to something other than itself: an independent
brute-force evaluation of Eq. 1, PyTorch's dense scaled-dot-product
attention, SciPy's logsumexp, closed forms for one- and two-key rows, and
invariants (block permutation, constant V, convexity).
"""
import numpy as np
import pytest
import torch
from scipy.special import expit, logsumexp

from oracle import attn as oattn
from oracle import brute
from workloads import BlockMask, bf16_bits_from_f32, random_case

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def f64(bits):
    return brute.bf16_to_f64(bits)


def _close(a, b, tol=1e-12):
    a, b = np.asarray(a), np.asarray(b)
    fin = np.isfinite(b)
    assert np.array_equal(np.isfinite(a), fin)
    assert np.array_equal(a[~fin], b[~fin])
    if fin.any():
        assert np.max(np.abs(a[fin] - b[fin])) <= tol


@pytest.mark.parametrize("geom,nq,nkv,d", [
    ([(16, 16)], 64, 64, 4),
    ([(32, 16)], 100, 77, 8),
    ([(16, 32)], 77, 100, 128),
    ([(64, 64), (32, 128)], 200, 300, 16),
    ([(8, 24)], 50, 49, 4),
])
def test_matches_brute_force(geom, nq, nkv, d):
    q, k, v, mask = random_case(11, 2, len(geom), nq, nkv, d, geom, 0.35, empty_rows=1)
    O, L = oattn.masked_attention(q, k, v, mask)
    Ob, Lb = brute.masked_attention(q, k, v, mask)
    _close(O, Ob, 1e-12)
    _close(L, Lb, 1e-12)


def test_dense_mask_equals_sdpa():
    rng = np.random.default_rng(3)
    B, N, H, d = 1, 192, 2, 128
    q, k, v = (bf16_bits_from_f32(rng.standard_normal((B, N, H, d), dtype=np.float32)) for _ in range(3))
    ones = [[np.ones((3, 3), bool) for _ in range(H)] for _ in range(B)]
    mask = BlockMask.from_heads(ones, [64] * H, [64] * H, N, N)
    O, L = oattn.masked_attention(q, k, v, mask)
    tq, tk, tv = (torch.from_numpy(f64(x)).permute(0, 2, 1, 3) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv).permute(0, 2, 1, 3).numpy()
    assert np.max(np.abs(O - ref)) < 1e-12
    scores = torch.einsum("bhid,bhjd->bhij", tq, tk) / np.sqrt(d)
    assert np.max(np.abs(L - torch.logsumexp(scores, dim=-1).numpy())) < 1e-12


def test_block_diagonal_is_chunked_dense():
    rng = np.random.default_rng(4)
    B, N, H, d, blk = 2, 256, 1, 32, 64
    q, k, v = (bf16_bits_from_f32(rng.standard_normal((B, N, H, d), dtype=np.float32)) for _ in range(3))
    heads = [[np.eye(N // blk, dtype=bool)] for _ in range(B)]
    mask = BlockMask.from_heads(heads, [blk], [blk], N, N)
    O, _ = oattn.masked_attention(q, k, v, mask)
    for b in range(B):
        for c in range(N // blk):
            sl = slice(c * blk, (c + 1) * blk)
            tq, tk, tv = (torch.from_numpy(f64(x[b, sl, 0, :]))[None] for x in (q, k, v))
            ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)[0].numpy()
            assert np.max(np.abs(O[b, sl, 0, :] - ref)) < 1e-12


def test_empty_rows_are_zero_with_neg_inf_lse():
    q, k, v, mask = random_case(5, 1, 1, 96, 96, 8, [(32, 32)], 0.6, empty_rows=2)
    O, L = oattn.masked_attention(q, k, v, mask)
    m = mask.head(0, 0)
    empty = ~m.any(axis=1)
    assert empty.sum() >= 2
    for qb in np.nonzero(empty)[0]:
        rows = slice(qb * 32, (qb + 1) * 32)
        assert np.all(O[0, rows, 0, :] == 0.0)
        assert np.all(np.isneginf(L[0, 0, rows]))


def test_single_key_rows_copy_v():
    """Token-level permutation mask: each query sees exactly one key."""
    rng = np.random.default_rng(6)
    N, d = 40, 16
    q, k, v = (bf16_bits_from_f32(rng.standard_normal((1, N, 1, d), dtype=np.float32)) for _ in range(3))
    perm = rng.permutation(N)
    m = np.zeros((N, N), bool)
    m[np.arange(N), perm] = True
    mask = BlockMask.from_heads([[m]], [1], [1], N, N)
    O, L = oattn.masked_attention(q, k, v, mask)
    V, Q, K = f64(v[0, :, 0, :]), f64(q[0, :, 0, :]), f64(k[0, :, 0, :])
    assert np.array_equal(O[0, :, 0, :], V[perm])
    z = np.einsum("id,id->i", Q, K[perm]) / np.sqrt(d)
    assert np.max(np.abs(L[0, 0] - z)) < 1e-12


@pytest.mark.parametrize("bq,bkv", [(1, 1), (4, 2), (2, 4)])
def test_two_key_closed_form(bq, bkv):
    """Rows whose allowed set is two keys: O = sigmoid(z1 - z2) v1 + sigmoid(z2 - z1) v2.

    With bq != bkv the mask axes cannot be swapped without breaking this.
    """
    rng = np.random.default_rng(7 + bq)
    nq, nkv, d = 24, 48, 8
    q, k, v = (bf16_bits_from_f32(rng.standard_normal((1, n, 1, d), dtype=np.float32))
               for n in (nq, nkv, nkv))
    nqb, nkb = nq // bq, nkv // bkv
    m = np.zeros((nqb, nkb), bool)
    chosen = {}
    for qb in range(nqb):
        if bkv == 1:
            cols = rng.choice(nkb, 2, replace=False)
            m[qb, cols] = True
            chosen[qb] = sorted(cols)
        else:                                      # one active block of width 2 or 4
            c = int(rng.integers(nkb))
            m[qb, c] = True
            chosen[qb] = [c]
    mask = BlockMask.from_heads([[m]], [bq], [bkv], nq, nkv)
    O, L = oattn.masked_attention(q, k, v, mask)
    Q, K, V = f64(q[0, :, 0, :]), f64(k[0, :, 0, :]), f64(v[0, :, 0, :])
    for i in range(nq):
        cols = chosen[i // bq]
        keys = [j for c in cols for j in range(c * bkv, (c + 1) * bkv)]
        z = K[keys] @ Q[i] / np.sqrt(d)
        if len(keys) == 2:
            ref = expit(z[0] - z[1]) * V[keys[0]] + expit(z[1] - z[0]) * V[keys[1]]
            assert np.max(np.abs(O[0, i, 0] - ref)) < 1e-12
        assert abs(L[0, 0, i] - logsumexp(z)) < 1e-12
        w = np.exp(z - logsumexp(z))
        assert np.max(np.abs(O[0, i, 0] - w @ V[keys])) < 1e-12


def test_constant_v_gives_constant_output():
    q, k, v, mask = random_case(8, 1, 2, 70, 90, 8, [(16, 16), (32, 16)], 0.4, empty_rows=1)
    col = np.linspace(-2, 2, 8, dtype=np.float32)
    v[:] = bf16_bits_from_f32(np.broadcast_to(col, v.shape).copy())
    O, L = oattn.masked_attention(q, k, v, mask)
    live = np.isfinite(L)                      # [B, H, Nq]
    colb = f64(bf16_bits_from_f32(col))
    for h in range(2):
        rows = O[0, live[0, h], h, :]
        assert np.max(np.abs(rows - colb)) < 1e-12


def test_kv_block_permutation_invariance():
    """Permuting whole KV blocks together with the mask columns leaves O unchanged."""
    rng = np.random.default_rng(9)
    q, k, v, mask = random_case(9, 1, 1, 128, 160, 16, [(32, 32)], 0.5)
    perm = rng.permutation(5)
    tok = np.concatenate([np.arange(p * 32, (p + 1) * 32) for p in perm])
    m2 = mask.head(0, 0)[:, perm]
    mask2 = BlockMask.from_heads([[m2]], [32], [32], 128, 160)
    O1, L1 = oattn.masked_attention(q, k, v, mask)
    O2, L2 = oattn.masked_attention(q, np.ascontiguousarray(k[:, tok]), np.ascontiguousarray(v[:, tok]), mask2)
    _close(O1, O2, 1e-12)
    _close(L1, L2, 1e-12)


def test_convex_combination_of_allowed_values():
    q, k, v, mask = random_case(10, 1, 1, 64, 64, 8, [(16, 16)], 0.3, empty_rows=1)
    O, L = oattn.masked_attention(q, k, v, mask)
    V = f64(v[0, :, 0, :])
    E = brute.token_mask(mask.head(0, 0), 16, 16, 64, 64)
    for i in range(64):
        if not E[i].any():
            continue
        lo, hi = V[E[i]].min(axis=0), V[E[i]].max(axis=0)
        assert np.all(O[0, i, 0] >= lo - 1e-12) and np.all(O[0, i, 0] <= hi + 1e-12)


def test_row_subset_matches_full():
    q, k, v, mask = random_case(12, 2, 2, 80, 80, 8, [(16, 16), (16, 32)], 0.4)
    O, L = oattn.masked_attention(q, k, v, mask)
    rng = np.random.default_rng(1)
    rows = np.stack([rng.integers(0, 2, 30), rng.integers(0, 2, 30), rng.integers(0, 80, 30)], axis=1)
    Os, Ls = oattn.masked_attention(q, k, v, mask, rows=rows)
    for r, (b, h, i) in enumerate(rows):
        assert np.array_equal(Os[r], O[b, i, h])
        assert Ls[r] == L[b, h, i] or (np.isneginf(Ls[r]) and np.isneginf(L[b, h, i]))
