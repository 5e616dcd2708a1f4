"""Enumeration oracle for the planning steps (integers only).

TEST INFRASTRUCTURE ONLY.  Written from the paper's definitions:

* Block-CSR of the shared mask state mu(M): per query-block row, the offsets
  and the ascending active KV block columns (Section 4.2, refine example;
  Section 5.2, regime lookup).
* Mask statistics (Section 5.1): active-block density = active / all logical
  blocks; active-block-run coverage = fraction of active blocks that lie in a
  run (maximal sequence of consecutive active KV blocks in one query-block
  row, Section 4.3) of length >= 2, and 0 for an empty mask.  Exported as
  integer numerators and denominators.
* Physical mapping (Section 4.2): a physical tile (pq, pk) covers the token
  rectangle [pq*T_Q, (pq+1)*T_Q) x [pk*T_KV, (pk+1)*T_KV); its member logical
  blocks are the ones intersecting that rectangle; it is active iff some
  member is active.  Coarsened tiles (several members) carry membership
  metadata: bit a*g_KV + c is set iff member (a, c) is active, with a and c
  counted from the first member row and column.  Direct tiles equal logical
  blocks; refined tiles split a logical block.
* Task organisation (Section 4.3): the active tiles of one physical query
  row are cut into S contiguous chunks [floor(s*n/S), floor((s+1)*n/S));
  empty chunks are dropped.  A physical row with no active tile still gets
  one empty task, which writes the row's zero output.

Rows are ordered (batch, head, row) everywhere.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Sequence, Tuple

import numpy as np


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


# ----------------------------------------------------------------------------
# Block-CSR and statistics of the logical mask
# ----------------------------------------------------------------------------

@dataclass
class BlockCSR:
    row_ptr: np.ndarray   # int64 [R + 1]
    col_idx: np.ndarray   # int32 [nnz]
    row_bh: np.ndarray    # int32 [R], b * H + h of each row


def block_csr(mask) -> BlockCSR:
    """Logical block-CSR over rows (b, h, qb)."""
    counts, cols, bh = [], [], []
    for b in range(mask.B):
        for h in range(mask.H):
            m = mask.head(b, h) != 0
            r, c = np.nonzero(m)          # row-major: rows ascending, columns ascending
            counts.append(m.sum(axis=1).astype(np.int64))
            cols.append(c.astype(np.int32))
            bh.append(np.full(m.shape[0], b * mask.H + h, dtype=np.int32))
    counts = np.concatenate(counts) if counts else np.zeros(0, np.int64)
    row_ptr = np.zeros(counts.size + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    return BlockCSR(row_ptr, np.concatenate(cols) if cols else np.zeros(0, np.int32),
                    np.concatenate(bh) if bh else np.zeros(0, np.int32))


def runs(cols: Sequence[int]) -> List[Tuple[int, int]]:
    """Maximal runs [first, last] of consecutive active columns of one row."""
    out: List[Tuple[int, int]] = []
    for c in sorted(cols):
        if out and c == out[-1][1] + 1:
            out[-1] = (out[-1][0], c)
        else:
            out.append((c, c))
    return out


def _row_run_members(m: np.ndarray) -> np.ndarray:
    """Per row, the number of active blocks whose run has length >= 2."""
    a = m != 0
    left = np.zeros_like(a)
    right = np.zeros_like(a)
    left[:, 1:] = a[:, :-1]
    right[:, :-1] = a[:, 1:]
    return (a & (left | right)).sum(axis=1)


@dataclass
class SegmentStats:
    heads: Tuple[int, ...]
    bq: int
    bkv: int
    nnz: int
    blocks: int          # density denominator
    run_blocks: int      # active blocks in runs of length >= 2
    max_row_nnz: int

    @property
    def density(self) -> float:
        return self.nnz / self.blocks if self.blocks else 0.0

    @property
    def run_coverage(self) -> float:
        return self.run_blocks / self.nnz if self.nnz else 0.0


def segments(mask) -> List[Tuple[Tuple[int, int], Tuple[int, ...]]]:
    """Heads grouped by logical geometry, in order of first appearance."""
    seen: Dict[Tuple[int, int], List[int]] = {}
    for h in range(mask.H):
        seen.setdefault((int(mask.bq[h]), int(mask.bkv[h])), []).append(h)
    return [(g, tuple(hs)) for g, hs in seen.items()]


def mask_stats(mask) -> Tuple[List[SegmentStats], np.ndarray]:
    """Per-segment statistics and per-(b, h) active-block counts."""
    per_bh = np.zeros(mask.B * mask.H, dtype=np.int64)
    out = []
    for (bq, bkv), heads in segments(mask):
        nnz = blocks = run_blocks = max_row = 0
        for b in range(mask.B):
            for h in heads:
                m = mask.head(b, h) != 0
                row_nnz = m.sum(axis=1)
                nnz += int(row_nnz.sum())
                blocks += m.size
                run_blocks += int(_row_run_members(m).sum())
                if m.shape[0]:
                    max_row = max(max_row, int(row_nnz.max()))
                per_bh[b * mask.H + h] = int(row_nnz.sum())
        out.append(SegmentStats(heads, bq, bkv, nnz, blocks, run_blocks, max_row))
    return out, per_bh


# ----------------------------------------------------------------------------
# Physical mapping
# ----------------------------------------------------------------------------

def mapping_kind(bq: int, bkv: int, tq: int, tkv: int) -> str:
    if tq == bq and tkv == bkv:
        return "direct"
    if tq >= bq and tkv >= bkv:
        return "coarsened"
    if tq <= bq and tkv <= bkv:
        return "refined"
    return "mixed"


def ratios(bq: int, bkv: int, tq: int, tkv: int) -> Tuple[int, int, int, int]:
    """(g_Q, g_KV, r_Q, r_KV): members per tile along each axis and tiles per block."""
    for t, bb in ((tq, bq), (tkv, bkv)):
        if not (t % bb == 0 or bb % t == 0):
            raise ValueError("tile %d and block %d do not nest" % (t, bb))
    gq = tq // bq if tq >= bq else 1
    gkv = tkv // bkv if tkv >= bkv else 1
    rq = bq // tq if tq < bq else 1
    rkv = bkv // tkv if tkv < bkv else 1
    return gq, gkv, rq, rkv


def has_membership(bq: int, bkv: int, tq: int, tkv: int) -> bool:
    gq, gkv, _, _ = ratios(bq, bkv, tq, tkv)
    return gq * gkv > 1


@dataclass
class PhysicalTiles:
    row_ptr: np.ndarray   # int64 [Rp + 1]
    kv_tile: np.ndarray   # int32 [ntiles], physical KV tile index pk
    member: np.ndarray    # uint64 [ntiles] (coarsened plans) or empty
    row_bh: np.ndarray    # int32 [Rp]
    row_pq: np.ndarray    # int32 [Rp]


def _head_tiles(m: np.ndarray, bq: int, bkv: int, tq: int, tkv: int, nq: int, nkv: int):
    """Vectorised tile activity and membership for one head: [nPQ, nPK] each."""
    gq, gkv, rq, rkv = ratios(bq, bkv, tq, tkv)
    nqb, nkb = m.shape
    npq, npk = cdiv(nq, tq), cdiv(nkv, tkv)
    a = m != 0
    if tq >= bq:
        pad = np.zeros((npq * gq, nkb), dtype=bool)
        pad[:nqb] = a
        t = pad.reshape(npq, gq, nkb)
    else:
        t = a[np.arange(npq) // rq][:, None, :]
    if tkv >= bkv:
        pad = np.zeros((npq, t.shape[1], npk * gkv), dtype=bool)
        pad[:, :, :nkb] = t
        t = pad.reshape(npq, t.shape[1], npk, gkv)
    else:
        t = t[:, :, np.arange(npk) // rkv][:, :, :, None]
    active = t.any(axis=(1, 3))
    bits = np.zeros((npq, npk), dtype=np.uint64)
    for ai in range(t.shape[1]):
        for ci in range(t.shape[3]):
            bits |= t[:, ai, :, ci].astype(np.uint64) << np.uint64(ai * gkv + ci)
    return active, bits


def physical_tiles(mask, heads: Sequence[int], tq: int, tkv: int) -> PhysicalTiles:
    """Physical tile CSR of one geometry segment, rows ordered (b, h, pq)."""
    counts, kv, mem, rbh, rpq = [], [], [], [], []
    for b in range(mask.B):
        for h in heads:
            bq, bkv = int(mask.bq[h]), int(mask.bkv[h])
            active, bits = _head_tiles(mask.head(b, h), bq, bkv, tq, tkv, mask.nq, mask.nkv)
            r, c = np.nonzero(active)
            counts.append(active.sum(axis=1).astype(np.int64))
            kv.append(c.astype(np.int32))
            mem.append(bits[r, c])
            rbh.append(np.full(active.shape[0], b * mask.H + h, dtype=np.int32))
            rpq.append(np.arange(active.shape[0], dtype=np.int32))
    counts = np.concatenate(counts)
    row_ptr = np.zeros(counts.size + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    h0 = heads[0]
    coarse = has_membership(int(mask.bq[h0]), int(mask.bkv[h0]), tq, tkv)
    return PhysicalTiles(row_ptr, np.concatenate(kv),
                         np.concatenate(mem).astype(np.uint64) if coarse else np.zeros(0, np.uint64),
                         np.concatenate(rbh), np.concatenate(rpq))


def physical_tiles_by_rectangles(mask, heads: Sequence[int], tq: int, tkv: int) -> PhysicalTiles:
    """Pure-loop version for tiny masks, straight from the token-rectangle rule."""
    counts, kv, mem, rbh, rpq = [], [], [], [], []
    h0 = heads[0]
    coarse = has_membership(int(mask.bq[h0]), int(mask.bkv[h0]), tq, tkv)
    for b in range(mask.B):
        for h in heads:
            bq, bkv = int(mask.bq[h]), int(mask.bkv[h])
            m = mask.head(b, h)
            nqb, nkb = m.shape
            for pq in range(cdiv(mask.nq, tq)):
                q0, q1 = pq * tq, min((pq + 1) * tq, mask.nq)
                qbs = [qb for qb in range(nqb) if qb * bq < q1 and min((qb + 1) * bq, mask.nq) > q0]
                n_row = 0
                for pk in range(cdiv(mask.nkv, tkv)):
                    k0, k1 = pk * tkv, min((pk + 1) * tkv, mask.nkv)
                    kbs = [kb for kb in range(nkb) if kb * bkv < k1 and min((kb + 1) * bkv, mask.nkv) > k0]
                    bits = 0
                    any_active = False
                    for a, qb in enumerate(qbs):
                        for c, kb in enumerate(kbs):
                            if m[qb, kb]:
                                any_active = True
                                # member offsets inside the tile's member grid
                                ga = qb - (q0 // bq) if tq >= bq else 0
                                gc = kb - (k0 // bkv) if tkv >= bkv else 0
                                gkv = tkv // bkv if tkv >= bkv else 1
                                bits |= 1 << (ga * gkv + gc)
                    if any_active:
                        kv.append(pk)
                        mem.append(bits)
                        n_row += 1
                counts.append(n_row)
                rbh.append(b * mask.H + h)
                rpq.append(pq)
    row_ptr = np.zeros(len(counts) + 1, dtype=np.int64)
    np.cumsum(np.array(counts, dtype=np.int64), out=row_ptr[1:])
    return PhysicalTiles(row_ptr, np.array(kv, dtype=np.int32),
                         np.array(mem, dtype=np.uint64) if coarse else np.zeros(0, np.uint64),
                         np.array(rbh, dtype=np.int32), np.array(rpq, dtype=np.int32))


# ----------------------------------------------------------------------------
# Task organisation
# ----------------------------------------------------------------------------

TASK_FIELDS = ("bh", "pq", "tile_begin", "tile_end", "split", "nsplit")


def split_tasks(tiles: PhysicalTiles, S: int) -> np.ndarray:
    """Canonical task list [ntasks, 6] int64 in (b, h, pq, split) order."""
    out = []
    for r in range(tiles.row_ptr.size - 1):
        lo, hi = int(tiles.row_ptr[r]), int(tiles.row_ptr[r + 1])
        n = hi - lo
        bh, pq = int(tiles.row_bh[r]), int(tiles.row_pq[r])
        if n == 0:
            out.append((bh, pq, lo, lo, 0, 1))
            continue
        chunks = [(lo + (s * n) // S, lo + ((s + 1) * n) // S) for s in range(S)]
        chunks = [c for c in chunks if c[1] > c[0]]
        for s, (a, z) in enumerate(chunks):
            out.append((bh, pq, a, z, s, len(chunks)))
    return np.array(out, dtype=np.int64).reshape(-1, 6)


def coverage_counts(mask, heads: Sequence[int], tq: int, tkv: int, tasks: np.ndarray,
                    tiles: PhysicalTiles) -> Dict[Tuple[int, int], np.ndarray]:
    """Per (b, h): how many times tasks cover each token pair (tiny masks only).

    A tile contributes the token pairs of its active members (or the whole
    tile when it has no membership metadata), clipped to the sequence.
    """
    out: Dict[Tuple[int, int], np.ndarray] = {}
    for b in range(mask.B):
        for h in heads:
            out[(b, h)] = np.zeros((mask.nq, mask.nkv), dtype=np.int64)
    h0 = heads[0]
    coarse = has_membership(int(mask.bq[h0]), int(mask.bkv[h0]), tq, tkv)
    for (bh, pq, lo, hi, _s, _ns) in tasks:
        b, h = divmod(int(bh), mask.H)
        bq, bkv = int(mask.bq[h]), int(mask.bkv[h])
        gkv = tkv // bkv if tkv >= bkv else 1
        cov = out[(b, h)]
        q0, q1 = int(pq) * tq, min((int(pq) + 1) * tq, mask.nq)
        for t in range(int(lo), int(hi)):
            pk = int(tiles.kv_tile[t])
            k0, k1 = pk * tkv, min((pk + 1) * tkv, mask.nkv)
            if not coarse:
                cov[q0:q1, k0:k1] += 1
                continue
            bits = int(tiles.member[t])
            for i in range(q0, q1):
                a = (i - q0) // bq if tq >= bq else 0
                for j in range(k0, k1):
                    c = (j - k0) // bkv if tkv >= bkv else 0
                    if (bits >> (a * gkv + c)) & 1:
                        cov[i, j] += 1
    return out
