"""Parity at the full workload sizes (needs an MI355X).

Each workload runs through the C-ABI exactly as the benchmark runs it (the
library's own plan selection, default launch configuration).  The fp64
oracle evaluates a seeded sample of query rows one by one; at full size the
integer planning state (block-CSR, statistics, physical tiles, membership,
tasks) is compared with the oracle's enumeration in full, bit for bit, and
every output element must be finite.
"""
import gc

import numpy as np
import pytest

from oracle import attn as oattn
from oracle import plans
from tests.gpu_util import compare, compare_lse, expected_dispatch, log, run_plan
from workloads import CONFIGS, make_mask, make_qkv

pytestmark = pytest.mark.gpu

import paper_2609_25869_amd as bsa  # noqa: E402  (fails loudly if libbsa.so is missing)

FULL = ["c2_window15", "c2_window", "c3_topk", "c4_asym", "c5_mixed"]


def sample_rows(B, H, N, tq_of_head, seed):
    """Per (b, h): the first and last query token, and one seeded random token
    inside every physical query tile of the plan that runs the head (tiles of
    tq_of_head[h] rows), so every task of a split-free plan is checked."""
    rng = np.random.default_rng(seed)
    rows = []
    for b in range(B):
        for h in range(H):
            tq = int(tq_of_head[h])
            lo = np.arange(0, N, tq, dtype=np.int64)
            hi = np.minimum(lo + tq, N)
            toks = lo + (rng.random(len(lo)) * (hi - lo)).astype(np.int64)
            toks = np.concatenate([[0, N - 1], toks])
            rows.append(np.stack([np.full(len(toks), b), np.full(len(toks), h), toks], axis=1))
    return np.concatenate(rows).astype(np.int64)


@pytest.mark.parametrize("name", FULL)
def test_full_size_parity(name):
    import torch
    cfg = CONFIGS[name]
    log("full-size case %s: B%d H%d N%d" % (name, cfg.B, cfg.H, cfg.N))
    q, k, v = make_qkv(cfg)
    mask = make_mask(cfg, q, k)
    p, od, lsed, _ = run_plan(bsa, mask, q, k, v)
    log("  planned and ran: %s" % [(i["plan_id"], i["mapping_name"]) for i in
                                   (p.info(s) for s in range(p.num_segments()))])

    # every output element is finite (checked on the device, at full size)
    assert bool(torch.isfinite(od).all().item()), "non-finite output"
    assert bool((torch.isfinite(lsed) | (lsed == -float("inf"))).all().item())

    # one row of every physical query tile against the oracle
    tq_of_head = np.zeros(cfg.H, dtype=np.int64)
    for si in range(p.num_segments()):
        info = p.info(si)
        tq_of_head[list(info["heads"])] = info["tq"]
    rows = sample_rows(cfg.B, cfg.H, cfg.N, tq_of_head, seed=len(name))
    O_ref, L_ref = oattn.masked_attention(q, k, v, mask, rows=rows)
    rb, rh, ri = (torch.from_numpy(rows[:, c]).cuda() for c in range(3))
    O_gpu = od[rb, ri, rh].float().cpu().numpy().astype(np.float64)
    L_gpu = lsed[rb, rh, ri].cpu().numpy().astype(np.float64)
    err = compare(O_gpu, O_ref, name)
    compare_lse(L_gpu, L_ref, name)
    log("  %d rows (one per physical query tile, plus each head's first and last): max_abs %.2e mean_abs %.2e"
        % (len(rows), err["max_abs"], err["mean_abs"]))

    # integer planning state, in full
    csr = plans.block_csr(mask)
    segs, per_bh = plans.mask_stats(mask)
    assert np.array_equal(p.export(bsa.EXPORT_ROW_PTR), csr.row_ptr)
    assert np.array_equal(p.export(bsa.EXPORT_COL_IDX), csr.col_idx)
    assert np.array_equal(p.export(bsa.EXPORT_BH_NNZ), per_bh)
    assert p.num_segments() == len(segs)
    for si, seg in enumerate(segs):
        info = p.info(si)
        assert tuple(info["heads"]) == seg.heads
        assert (info["nnz"], info["blocks"], info["run_blocks"], info["max_row_nnz"]) == \
            (seg.nnz, seg.blocks, seg.run_blocks, seg.max_row_nnz)
        tiles = plans.physical_tiles(mask, seg.heads, info["tq"], info["tkv"])
        assert np.array_equal(p.export(bsa.EXPORT_TILE_PTR, si), tiles.row_ptr)
        assert np.array_equal(p.export(bsa.EXPORT_TILE_KV, si), tiles.kv_tile)
        assert np.array_equal(p.export(bsa.EXPORT_TILE_MEMBER, si), tiles.member)
        tasks = plans.split_tasks(tiles, info["split"])
        assert np.array_equal(p.export(bsa.EXPORT_TASKS, si), tasks)
        want = np.arange(len(tasks))
        if len(tasks) > 512:
            want = expected_dispatch(tasks, tiles.kv_tile, tiles.member if len(tiles.member) else None)
        assert np.array_equal(p.export(bsa.EXPORT_DISPATCH, si), want)
    log("  planning state and dispatch order match the enumeration (%d segments)" % len(segs))
    p.destroy()
    del od, lsed
    gc.collect()
    torch.cuda.empty_cache()


def test_tiny_workload_in_full_under_every_eligible_plan():
    """The 2048-token workload (two heads, (64,64) blocks, 32% density): every
    output element and LSE of every eligible catalog plan against the oracle."""
    import torch
    cfg = CONFIGS["c1_tiny"]
    q, k, v = make_qkv(cfg)
    mask = make_mask(cfg, q, k)
    O_ref, L_ref = oattn.masked_attention(q, k, v, mask)
    shapes = bsa.make_shapes(cfg.B, cfg.H, cfg.N, cfg.N)
    plans_run = [e["id"] for e in bsa.catalog() if bsa.plan_eligible(e["id"], 64, 64, shapes)]
    assert len(plans_run) >= 24
    for pid in plans_run:
        p, od, lsed, _ = run_plan(bsa, mask, q, k, v, force_plan=pid)
        err = compare(od.float().cpu().numpy().astype(np.float64), O_ref, "c1_tiny plan %d" % pid)
        compare_lse(lsed.cpu().numpy().astype(np.float64), L_ref, "c1_tiny plan %d" % pid)
        log("c1_tiny plan %d: max_abs %.2e mean_abs %.2e" % (pid, err["max_abs"], err["mean_abs"]))
        p.destroy()
        del od, lsed
    torch.cuda.empty_cache()
