"""Brute-force masked attention with an explicit bias matrix (Eq. 1).

TEST INFRASTRUCTURE ONLY.  For tiny inputs: builds the full N_q x N_kv score
matrix Q K^T / sqrt(d), adds the bias B_M (0 on the effective interaction set
E(M), -inf elsewhere; Section 2.1) and applies a row softmax, all in float64
numpy.  Written independently of ``attn_fp64.c`` so the two can check each
other.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def token_mask(block_mask_2d: np.ndarray, bq: int, bkv: int, nq: int, nkv: int) -> np.ndarray:
    """E(M) as a boolean [nq, nkv] matrix: expand each logical block to its tokens."""
    expanded = np.repeat(np.repeat(np.asarray(block_mask_2d) != 0, bq, axis=0), bkv, axis=1)
    return expanded[:nq, :nkv]


def masked_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, mask):
    """Returns (O [B, Nq, H, d], LSE [B, H, Nq]) in float64."""
    B, Nq, H, d = q.shape
    Nkv = k.shape[1]
    O = np.zeros((B, Nq, H, d))
    LSE = np.full((B, H, Nq), -np.inf)
    for b in range(B):
        for h in range(H):
            Q = bf16_to_f64(q[b, :, h, :])
            K = bf16_to_f64(k[b, :, h, :])
            V = bf16_to_f64(v[b, :, h, :])
            E = token_mask(mask.head(b, h), int(mask.bq[h]), int(mask.bkv[h]), Nq, Nkv)
            bias = np.where(E, 0.0, -np.inf)
            Z = Q @ K.T / np.sqrt(d) + bias
            live = E.any(axis=1)
            m = np.where(live, Z.max(axis=1, initial=-np.inf), 0.0)
            W = np.exp(Z - m[:, None])          # exp(-inf) = 0 off E(M)
            L = W.sum(axis=1)
            with np.errstate(invalid="ignore", divide="ignore"):
                Ob = (W @ V) / L[:, None]
                lse = m + np.log(L)
            Ob[~live] = 0.0
            lse[~live] = -np.inf
            O[b, :, h, :] = Ob
            LSE[b, h, :] = lse
    return O, LSE
