"""Pins of the top-k sparsifier oracle (oracle/sparsify.py) against exact
arithmetic, brute force and constructed answers.  CPU only."""
from __future__ import annotations

from fractions import Fraction

import numpy as np
import pytest

from oracle import sparsify as osp


def bits_of(x: np.ndarray) -> np.ndarray:
    """bf16 bits of values that bf16 holds exactly."""
    f = np.asarray(x, dtype=np.float32)
    b = (f.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(osp.bf16_to_f64(b), f.astype(np.float64)), "value not exact in bf16"
    return b


def exact_scores(x_q, x_k, bq, bkv):
    """Block-mean scores in exact rational arithmetic."""
    def means(x, blk):
        n = x.shape[0]
        return [[sum(Fraction(int(v)) for v in x[i:min(n, i + blk), c]) / (min(n, i + blk) - i)
                 for c in range(x.shape[1])] for i in range(0, n, blk)]
    mq, mk = means(x_q, bq), means(x_k, bkv)
    return [[sum(a * b for a, b in zip(qr, kr)) for kr in mk] for qr in mq]


def brute_topk(scores, k):
    """Active iff fewer than k columns beat it (larger score, or equal score and lower column)."""
    n = len(scores)
    return [sum(1 for j in range(n) if scores[j] > scores[i] or (scores[j] == scores[i] and j < i)) < k
            for i in range(n)]


@pytest.mark.parametrize("nq,nkv,bq,bkv,d", [(40, 36, 8, 4, 16), (37, 50, 16, 8, 128), (64, 64, 16, 16, 32)])
def test_scores_are_exact_on_integer_inputs(nq, nkv, bq, bkv, d):
    """Small integers: block sums, means (power-of-two or exact counts) and
    the dot products are all exact in double, so the oracle must reproduce
    the rational scores bit for bit, ragged last blocks included."""
    rng = np.random.default_rng(nq * 7 + bkv)
    xq = rng.integers(-3, 4, size=(nq, d)).astype(np.float32)
    xk = rng.integers(-3, 4, size=(nkv, d)).astype(np.float32)
    got = osp.block_scores(osp.block_means(bits_of(xq), bq), osp.block_means(bits_of(xk), bkv))
    want = exact_scores(xq, xk, bq, bkv)
    pow2 = lambda n: n & (n - 1) == 0
    for i, row in enumerate(want):
        nqi = min(nq, (i + 1) * bq) - i * bq
        for j, w in enumerate(row):
            nkj = min(nkv, (j + 1) * bkv) - j * bkv
            if pow2(nqi) and pow2(nkj):     # dyadic means: every step is exact
                assert got[i, j] == float(w), (i, j, got[i, j], w)
            else:                           # a ragged count such as 5 rounds the mean once
                assert abs(got[i, j] - float(w)) <= 1e-12 * max(1.0, abs(float(w))), (i, j)


def test_ragged_block_mean_divides_by_its_own_row_count():
    x = np.zeros((10, 4), dtype=np.float32)
    x[8:] = 6.0                                   # last block (rows 8, 9) of block size 4
    m = osp.block_means(bits_of(x), 4)
    assert m.shape == (3, 4) and np.all(m[2] == 6.0) and np.all(m[:2] == 0.0)


def test_topk_matches_brute_force_ranking_with_ties():
    rng = np.random.default_rng(3)
    for trial in range(20):
        nkb = int(rng.integers(1, 40))
        # few distinct values, so many ties
        s = rng.integers(-3, 3, size=(5, nkb)).astype(np.float64)
        for k in (0, 1, 2, nkb // 2, nkb - 1, nkb, nkb + 3):
            got = osp.topk_rows(s, k)
            for r in range(5):
                assert list(got[r]) == brute_topk(list(s[r]), k), (trial, k, r)


def test_equal_scores_prefer_the_lower_kv_block():
    s = np.array([[1.0, 5.0, 5.0, 5.0, 2.0]])
    assert list(osp.topk_rows(s, 2)[0]) == [False, True, True, False, False]


@pytest.mark.parametrize("nq,nkv,bq,bkv", [(64, 64, 16, 16), (100, 70, 16, 32), (70, 100, 32, 8), (1000, 1000, 64, 64),
                                            (96, 96, 128, 32)])
def test_diagonal_blocks_by_token_enumeration(nq, nkv, bq, bkv):
    nqb, nkb = -(-nq // bq), -(-nkv // bkv)
    want = np.zeros((nqb, nkb), dtype=bool)
    for i in range(min(nq, nkv)):
        want[i // bq, i // bkv] = True
    assert np.array_equal(osp.diagonal_blocks(nq, nkv, bq, bkv), want)


def test_known_answer_scaled_key_blocks():
    """K block kb = alpha[kb] * u and every query row = u: the scores are
    alpha[kb] * |u|^2, so the selected blocks are the k largest alphas."""
    d, bkv, bq, nkb = 32, 8, 8, 12
    u = np.linspace(-1, 1, d).astype(np.float32)
    u = osp.bf16_to_f64(bits_of(np.round(u * 8) / 8)).astype(np.float32)
    alpha = np.array([3, -1, 7, 2, 0.5, 6, -4, 1, 5, 0.25, 4, -2], dtype=np.float32)
    k_rows = np.concatenate([np.tile(a * u, (bkv, 1)) for a in alpha])
    q_rows = np.tile(u, (2 * bq, 1))
    mask, scores = osp.sparsify_topk(bits_of(q_rows)[None, :, None, :], bits_of(k_rows)[None, :, None, :],
                                     bq, bkv, 4, diagonal=False)
    top = set(np.argsort(-alpha)[:4].tolist())
    for r in range(2):
        assert set(np.nonzero(mask[0, 0, r])[0].tolist()) == top


def test_degenerate_k_values():
    rng = np.random.default_rng(9)
    q = bits_of(np.round(rng.standard_normal((1, 128, 2, 16)) * 16).astype(np.float32) / 16)
    k = bits_of(np.round(rng.standard_normal((1, 96, 2, 16)) * 16).astype(np.float32) / 16)
    full, _ = osp.sparsify_topk(q, k, 16, 16, 1000, diagonal=False)
    assert full.all()
    diag_only, _ = osp.sparsify_topk(q, k, 16, 16, 0, diagonal=True)
    assert np.array_equal(diag_only[0, 0].astype(bool), osp.diagonal_blocks(128, 96, 16, 16))
    m, _ = osp.sparsify_topk(q, k, 16, 16, 3, diagonal=False)
    assert np.all(m.sum(axis=-1) == 3)
