"""Pins for the planning enumerator (CPU only).

The vectorised enumerator is checked against the paper's worked examples,
against a pure-loop evaluation of the token-rectangle rule, and against the
coverage invariant: expanded to token pairs, the tasks of every plan cover
E(M) exactly once.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import brute, plans
from workloads import BlockMask, random_case

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_examples.json")))


def _mask_from_rows(rows, nkb, bq=64, bkv=64):
    m = np.zeros((len(rows), nkb), bool)
    for r, cols in enumerate(rows):
        m[r, cols] = True
    return BlockMask.from_heads([[m]], [bq], [bkv], len(rows) * bq, nkb * bkv)


def test_runs_worked_example():
    ex = GOLDEN["runs_example"]
    assert plans.runs(ex["cols"]) == [tuple(r) for r in ex["runs"]]
    mask = _mask_from_rows([ex["cols"]], 12)
    (seg,), _ = plans.mask_stats(mask)
    assert (seg.run_blocks, seg.nnz) == tuple(ex["run_coverage_derived"])


def test_empty_mask_statistics():
    mask = _mask_from_rows([[], []], 8)
    (seg,), per_bh = plans.mask_stats(mask)
    assert seg.nnz == 0 and seg.run_blocks == 0 and seg.run_coverage == GOLDEN["density_definition"]["empty_mask_run_coverage"]
    assert seg.density == 0.0 and seg.blocks == 16 and per_bh.tolist() == [0]


def test_refine_worked_example():
    ex = GOLDEN["refine_example"]
    rng = np.random.default_rng(0)
    m = rng.random((4, 6)) < 0.5
    B_, T_ = ex["block"], ex["tile"]
    mask = BlockMask.from_heads([[m]], [B_[0]], [B_[1]], 4 * B_[0], 6 * B_[1])
    csr = plans.block_csr(mask)
    tiles = plans.physical_tiles(mask, [0], T_[0], T_[1])
    g = ex["kv_expansion_factor"]
    assert tiles.row_ptr.size - 1 == 4 * ex["q_tiles_per_block_row"]
    for pq in range(tiles.row_ptr.size - 1):
        qb = pq // ex["q_tiles_per_block_row"]
        cols = csr.col_idx[csr.row_ptr[qb]:csr.row_ptr[qb + 1]]
        expect = [x for c in cols for x in (g * c, g * c + 1)]
        assert tiles.kv_tile[tiles.row_ptr[pq]:tiles.row_ptr[pq + 1]].tolist() == expect
    assert tiles.member.size == 0          # refined tiles carry no membership


def test_direct_plan_is_the_block_csr():
    q, k, v, mask = random_case(1, 2, 2, 300, 260, 4, [(64, 32), (64, 32)], 0.3)
    csr = plans.block_csr(mask)
    tiles = plans.physical_tiles(mask, [0, 1], 64, 32)
    assert np.array_equal(tiles.row_ptr, csr.row_ptr)
    assert np.array_equal(tiles.kv_tile, csr.col_idx)
    assert tiles.member.size == 0


def test_block_csr_matches_loops():
    q, k, v, mask = random_case(2, 2, 3, 200, 170, 4, [(32, 16), (16, 32), (64, 64)], 0.3, empty_rows=1)
    csr = plans.block_csr(mask)
    ptr, cols = [0], []
    for b in range(2):
        for h in range(3):
            m = mask.head(b, h)
            for r in range(m.shape[0]):
                row = [c for c in range(m.shape[1]) if m[r, c]]
                cols += row
                ptr.append(ptr[-1] + len(row))
    assert csr.row_ptr.tolist() == ptr and csr.col_idx.tolist() == cols


def test_statistics_match_loops():
    q, k, v, mask = random_case(3, 2, 2, 256, 256, 4, [(32, 32), (16, 64)], 0.4)
    segs, per_bh = plans.mask_stats(mask)
    for seg in segs:
        nnz = blocks = rb = mx = 0
        for b in range(2):
            for h in seg.heads:
                m = mask.head(b, h)
                blocks += m.size
                for r in range(m.shape[0]):
                    cols = [c for c in range(m.shape[1]) if m[r, c]]
                    nnz += len(cols)
                    mx = max(mx, len(cols))
                    rb += sum(hi - lo + 1 for lo, hi in plans.runs(cols) if hi > lo)
        assert (seg.nnz, seg.blocks, seg.run_blocks, seg.max_row_nnz) == (nnz, blocks, rb, mx)
    assert per_bh.sum() == sum(s.nnz for s in segs)


GEOMS = [(16, 16), (32, 16), (16, 32), (64, 64), (128, 32), (32, 128)]
TILES = [(32, 32), (64, 64), (64, 32), (128, 64), (128, 128), (256, 64), (64, 128), (32, 64)]


def _nests(b, t):
    return t % b == 0 or b % t == 0


@pytest.mark.parametrize("geom", GEOMS)
def test_vectorised_tiles_match_rectangle_rule(geom):
    for seed, (nq, nkv) in enumerate([(256, 256), (200, 330), (97, 161)]):
        q, k, v, mask = random_case(20 + seed, 1, 1, nq, nkv, 4, [geom], 0.25)
        for tq, tkv in TILES:
            if not (_nests(geom[0], tq) and _nests(geom[1], tkv)):
                continue
            a = plans.physical_tiles(mask, [0], tq, tkv)
            b = plans.physical_tiles_by_rectangles(mask, [0], tq, tkv)
            for f in ("row_ptr", "kv_tile", "member", "row_bh", "row_pq"):
                assert np.array_equal(getattr(a, f), getattr(b, f)), (geom, tq, tkv, f)


@pytest.mark.parametrize("geom", GEOMS)
def test_every_plan_covers_interactions_exactly_once(geom):
    q, k, v, mask = random_case(40, 2, 1, 190, 230, 4, [geom], 0.3, empty_rows=1)
    E = {(b, 0): brute.token_mask(mask.head(b, 0), geom[0], geom[1], 190, 230).astype(np.int64)
         for b in range(2)}
    for (tq, tkv), S in itertools.product(TILES, (1, 2, 3, 8)):
        if not (_nests(geom[0], tq) and _nests(geom[1], tkv)):
            continue
        tiles = plans.physical_tiles(mask, [0], tq, tkv)
        tasks = plans.split_tasks(tiles, S)
        cov = plans.coverage_counts(mask, [0], tq, tkv, tasks, tiles)
        for key in E:
            assert np.array_equal(cov[key], E[key]), (geom, tq, tkv, S)


def test_split_chunks_partition_rows():
    q, k, v, mask = random_case(41, 1, 2, 512, 512, 4, [(32, 32), (32, 32)], 0.2, empty_rows=2)
    tiles = plans.physical_tiles(mask, [0, 1], 64, 64)
    for S in (1, 2, 4, 7):
        tasks = plans.split_tasks(tiles, S)
        for r in range(tiles.row_ptr.size - 1):
            lo, hi = tiles.row_ptr[r], tiles.row_ptr[r + 1]
            mine = tasks[(tasks[:, 0] == tiles.row_bh[r]) & (tasks[:, 1] == tiles.row_pq[r])]
            n = hi - lo
            assert len(mine) == (1 if n == 0 else min(S, n))
            assert mine[0, 2] == lo and mine[-1, 3] == hi
            assert np.all(mine[1:, 2] == mine[:-1, 3])
            assert mine[:, 4].tolist() == list(range(len(mine)))
            assert np.all(mine[:, 5] == len(mine))
            if n:
                sizes = mine[:, 3] - mine[:, 2]
                assert sizes.max() - sizes.min() <= 1


def test_intensity_accounting_table4():
    """Q-resident accounting: per tile 4*d*T_Q*T_KV flop over 4*d*T_KV K/V bytes -> T_Q flop/byte
    (Section 2.3; Table 3 lists intensity = B_Q for Direct tiles)."""
    table4 = {(128, 128): 128.0, (128, 64): 128.0, (64, 64): 64.0, (64, 32): 64.0,
              (32, 32): 32.0, (32, 16): 32.0, (16, 16): 16.0}
    d = 128
    for (bq, bkv), inten in table4.items():
        flop = 4 * d * bq * bkv
        kv_bytes = 4 * d * bkv       # bf16 K and V rows: 2 tensors x 2 bytes
        assert flop / kv_bytes == inten
