"""Oracle for the top-k block sparsifier that supplies the logical mask.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 2.1: the sparsifier selects the active logical block pairs and hands
the mask M and its geometry B = (B_Q, B_KV) to the runtime.  The dynamic
masks used here follow the mean-pooled top-k rule: for every (b, h) and
query block qb, the scores of all KV blocks kb are

    s(qb, kb) = sum over c = 0 .. d-1 of  qbar(qb)[c] * kbar(kb)[c]

where qbar(qb) is the mean of the bf16 query rows of block qb and kbar(kb)
the mean of the key rows of block kb (a ragged last block averages the rows
it has).  The k KV blocks with the largest score are active, ties going to
the lower kb; optionally every block the token diagonal i == j passes
through is added.

Precision is fixed so that the selection, an integer decided by floating
point, is the same wherever it is computed: block sums of bf16 values in
IEEE double (exact for these magnitudes), the mean as one double division,
and the score accumulated over c in increasing order with a separate
rounding after every multiply and every add (no fused multiply-add).
"""
from __future__ import annotations

from typing import Tuple

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def block_means(x_bits: np.ndarray, block: int) -> np.ndarray:
    """[n, d] bf16 bits -> [ceil(n / block), d] float64 block means (rows summed in order)."""
    x = bf16_to_f64(x_bits)
    n, d = x.shape
    nb = -(-n // block)
    out = np.empty((nb, d))
    for i in range(nb):
        rows = x[i * block:min(n, (i + 1) * block)]
        s = np.zeros(d)
        for r in rows:           # explicit row order
            s = s + r
        out[i] = s / float(rows.shape[0])
    return out


def block_scores(qbar: np.ndarray, kbar: np.ndarray) -> np.ndarray:
    """[nqb, d] x [nkb, d] -> [nqb, nkb]: the sum over c in increasing order,
    one rounding per multiply and per add."""
    nqb, d = qbar.shape
    s = np.zeros((nqb, kbar.shape[0]))
    for c in range(d):
        s = s + qbar[:, c, None] * kbar[None, :, c]
    return s


def topk_rows(scores: np.ndarray, k: int) -> np.ndarray:
    """Boolean [nqb, nkb]: per row the k largest scores, ties to the lower column."""
    nqb, nkb = scores.shape
    out = np.zeros((nqb, nkb), dtype=bool)
    if k <= 0:
        return out
    cols = np.arange(nkb)
    for r in range(nqb):
        order = np.lexsort((cols, -scores[r]))   # by score descending, then column ascending
        out[r, order[:min(k, nkb)]] = True
    return out


def diagonal_blocks(nq: int, nkv: int, bq: int, bkv: int) -> np.ndarray:
    """Boolean [nqb, nkb]: blocks whose token rectangle meets the diagonal i == j."""
    nqb, nkb = -(-nq // bq), -(-nkv // bkv)
    out = np.zeros((nqb, nkb), dtype=bool)
    i = np.arange(min(nq, nkv))
    out[i // bq, i // bkv] = True
    return out


def sparsify_topk(q_bits: np.ndarray, k_bits: np.ndarray, bq: int, bkv: int, k: int,
                  diagonal: bool = True) -> Tuple[np.ndarray, np.ndarray]:
    """q_bits [B, Nq, H, d], k_bits [B, Nkv, H, d] bf16 bits ->
    (mask uint8 [B, H, nqb, nkb], scores float64 [B, H, nqb, nkb])."""
    B, Nq, H, d = q_bits.shape
    Nkv = k_bits.shape[1]
    nqb, nkb = -(-Nq // bq), -(-Nkv // bkv)
    mask = np.zeros((B, H, nqb, nkb), dtype=np.uint8)
    scores = np.zeros((B, H, nqb, nkb))
    diag = diagonal_blocks(Nq, Nkv, bq, bkv) if diagonal else np.zeros((nqb, nkb), dtype=bool)
    for b in range(B):
        for h in range(H):
            s = block_scores(block_means(q_bits[b, :, h, :], bq), block_means(k_bits[b, :, h, :], bkv))
            scores[b, h] = s
            mask[b, h] = (topk_rows(s, k) | diag).astype(np.uint8)
    return mask, scores
