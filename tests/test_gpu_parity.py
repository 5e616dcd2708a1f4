"""GPU parity of the HIP path against the fp64 oracle (needs an MI355X).

Every case runs through the C-ABI (bsa_plan + bsa_forward) and is compared
element by element with the oracle on the same seeded inputs.  Plan exports
(block-CSR, statistics, physical tiles, membership, tasks) must equal the
oracle's enumeration bit for bit.
"""
import numpy as np
import pytest

from oracle import attn as oattn
from oracle import brute, plans
from tests.gpu_util import bf16_to_f64, compare, compare_lse, expected_dispatch, log, run_plan, to_dev_bf16
from workloads import BlockMask, bf16_bits_from_f32, random_case

pytestmark = pytest.mark.gpu

import paper_2609_25869_amd as bsa  # noqa: E402  (fails loudly if libbsa.so is missing)

# (name, B, H, Nq, Nkv, geometry per head, density, empty q-block rows per head)
CASES = [
    ("g64_ragged", 2, 2, 1000, 1000, [(64, 64)] * 2, 0.3, 1),
    ("g128_ragged", 1, 2, 700, 700, [(128, 128)] * 2, 0.35, 1),
    ("g16", 1, 2, 333, 333, [(16, 16)] * 2, 0.2, 2),
    ("g32x16", 1, 1, 512, 480, [(32, 16)], 0.25, 1),
    ("asym_heads", 1, 4, 777, 777, [(128, 32), (32, 128), (128, 32), (32, 128)], 0.3, 1),
    ("qkv_diff_len", 1, 2, 300, 517, [(64, 32)] * 2, 0.4, 0),
    # sparse small blocks: tiles of 64-256 query rows span 2-8 query blocks,
    # so waves often have no active member in a tile (and skip it)
    ("g32_sparse", 1, 2, 1100, 1100, [(32, 32)] * 2, 0.08, 1),
    # word-aligned mask rows (nKB % 4 == 0) whose last block has fewer
    # refined tiles than the others (980 = 15 * 64 + 20, 950 = 7 * 128 + 54)
    ("g64_tail", 1, 2, 980, 980, [(64, 64)] * 2, 0.3, 1),
    ("g128_tail", 1, 2, 950, 950, [(128, 128)] * 2, 0.35, 1),
]


def _case(name):
    spec = [c for c in CASES if c[0] == name][0]
    _, B, H, nq, nkv, geom, dens, empty = spec
    seed = sum(map(ord, name))
    return random_case(seed, B, H, nq, nkv, 128, geom, dens, diag=False, empty_rows=empty)


def _eligible_plans(mask):
    shapes = bsa.make_shapes(mask.B, mask.H, mask.nq, mask.nkv)
    out = []
    for e in bsa.catalog():
        if all(bsa.plan_eligible(e["id"], int(mask.bq[h]), int(mask.bkv[h]), shapes) for h in range(mask.H)):
            out.append(e["id"])
    return out


_ORACLE_CACHE = {}


def _oracle(name, q, k, v, mask):
    if name not in _ORACLE_CACHE:
        _ORACLE_CACHE[name] = oattn.masked_attention(q, k, v, mask)
    return _ORACLE_CACHE[name]


@pytest.mark.parametrize("name", [c[0] for c in CASES])
def test_every_eligible_plan_matches_oracle(name):
    q, k, v, mask = _case(name)
    O_ref, L_ref = _oracle(name, q, k, v, mask)
    ids = _eligible_plans(mask)
    assert ids, "no eligible plan"
    for pid in ids:
        log("case %s plan %d" % (name, pid))
        p, od, lsed, _ = run_plan(bsa, mask, q, k, v, force_plan=pid)
        err = compare(bf16_to_f64(od), O_ref, "%s plan %d" % (name, pid))
        compare_lse(lsed.cpu().numpy().astype(np.float64), L_ref, "%s plan %d" % (name, pid))
        p.destroy()
        log("  ok max_abs %.2e mean_abs %.2e" % (err["max_abs"], err["mean_abs"]))


@pytest.mark.parametrize("name", [c[0] for c in CASES])
def test_plan_exports_match_enumeration(name):
    q, k, v, mask = _case(name)
    csr = plans.block_csr(mask)
    segs, per_bh = plans.mask_stats(mask)
    for pid in _eligible_plans(mask):
        log("case %s plan %d exports" % (name, pid))
        p, od, lsed, _ = run_plan(bsa, mask, q, k, v, force_plan=pid, lse=False)
        assert np.array_equal(p.export(bsa.EXPORT_ROW_PTR), csr.row_ptr)
        assert np.array_equal(p.export(bsa.EXPORT_COL_IDX), csr.col_idx)
        assert np.array_equal(p.export(bsa.EXPORT_BH_NNZ), per_bh)
        assert p.num_segments() == len(segs)
        entry = bsa.catalog()[pid]
        for si, seg in enumerate(segs):
            info = p.info(si)
            assert tuple(info["heads"]) == seg.heads
            assert (info["nnz"], info["blocks"], info["run_blocks"], info["max_row_nnz"]) == \
                (seg.nnz, seg.blocks, seg.run_blocks, seg.max_row_nnz)
            tiles = plans.physical_tiles(mask, seg.heads, entry["tq"], entry["tkv"])
            assert np.array_equal(p.export(bsa.EXPORT_TILE_PTR, si), tiles.row_ptr)
            assert np.array_equal(p.export(bsa.EXPORT_TILE_KV, si), tiles.kv_tile)
            assert np.array_equal(p.export(bsa.EXPORT_TILE_MEMBER, si), tiles.member)
            tasks = plans.split_tasks(tiles, entry["split"])
            assert np.array_equal(p.export(bsa.EXPORT_TASKS, si), tasks)
            assert info["n_tiles"] == tiles.kv_tile.size and info["n_tasks"] == tasks.shape[0]
        p.destroy()


def test_inactive_blocks_contribute_nothing():
    """Huge (finite) K/V values in blocks a query-block row does not use leave that row bitwise unchanged."""
    q, k, v, mask = random_case(501, 1, 2, 640, 640, 128, [(64, 64)] * 2, 0.3)
    for pid in _eligible_plans(mask):
        p, od, _, _ = run_plan(bsa, mask, q, k, v, force_plan=pid, lse=False)
        base = od.clone()
        k2, v2 = k.copy(), v.copy()
        rows = {}
        for h in range(2):
            m = mask.head(0, h)
            S = [2, 5, 7]                     # perturbed KV blocks
            rows[h] = [r for r in range(m.shape[0]) if not m[r, S].any()]
            for kb in S:
                sl = slice(kb * 64, (kb + 1) * 64)
                k2[0, sl, h, :] = bf16_bits_from_f32(np.full((64, 128), 1000.0, np.float32))
                v2[0, sl, h, :] = bf16_bits_from_f32(np.full((64, 128), -3000.0, np.float32))
        assert sum(len(r) for r in rows.values()) > 0
        p2, od2, _, _ = run_plan(bsa, mask, q, k2, v2, force_plan=pid, lse=False)
        for h in range(2):
            for r in rows[h]:
                assert (base[0, r * 64:(r + 1) * 64, h] == od2[0, r * 64:(r + 1) * 64, h]).all().item(), (pid, h, r)
        p.destroy()
        p2.destroy()


def test_kv_block_permutation_invariance():
    rng = np.random.default_rng(502)
    q, k, v, mask = random_case(502, 1, 1, 512, 768, 128, [(64, 64)], 0.35)
    perm = rng.permutation(12)
    tok = np.concatenate([np.arange(pb * 64, (pb + 1) * 64) for pb in perm])
    mask2 = BlockMask.from_heads([[mask.head(0, 0)[:, perm]]], [64], [64], 512, 768)
    k2, v2 = np.ascontiguousarray(k[:, tok]), np.ascontiguousarray(v[:, tok])
    O_ref, _ = oattn.masked_attention(q, k, v, mask)
    for pid in _eligible_plans(mask):
        p1, o1, _, _ = run_plan(bsa, mask, q, k, v, force_plan=pid, lse=False)
        p2, o2, _, _ = run_plan(bsa, mask2, q, k2, v2, force_plan=pid, lse=False)
        a, b = bf16_to_f64(o1), bf16_to_f64(o2)
        assert np.max(np.abs(a - b)) <= 1e-2, pid     # bf16 output: a few ulps at most
        assert np.mean(np.abs(a - b)) <= 1e-3, pid
        compare(b, O_ref, "permuted plan %d" % pid)
        p1.destroy()
        p2.destroy()


def _scale_rows(q_bits, factors):
    """Q rows multiplied by per-row factors (exactly representable scalings of bf16 values)."""
    from workloads import f32_from_bf16_bits
    q = f32_from_bf16_bits(q_bits) * factors
    return bf16_bits_from_f32(q.astype(np.float32))


@pytest.mark.parametrize("name", ["g64_ragged", "asym_heads", "g16", "g32_sparse"])
@pytest.mark.parametrize("mode", ["all_large", "mixed", "extreme"])
def test_large_scores_use_the_running_maximum(name, mode):
    """Scores beyond the fixed-reference bound (scale |q| max|k| > 32 in log2
    units) take the running-maximum path; wavefronts of one task may take
    different paths.  Every eligible plan must still match the oracle."""
    q, k, v, mask = _case(name)
    B, Nq, H, d = q.shape
    rng = np.random.default_rng(5)
    if mode == "all_large":
        f = np.full((B, Nq, H, 1), 6.0, dtype=np.float32)       # bounds ~100: running maximum
    elif mode == "mixed":
        # alternate 32-row groups (one wavefront each): bounded and running-maximum paths in one task
        grp = (np.arange(Nq) // 32) % 2 == 0
        f = np.where(grp[None, :, None, None], 8.0, 1.0).astype(np.float32) * np.ones((B, 1, H, 1), np.float32)
    else:
        f = np.full((B, Nq, H, 1), 64.0, dtype=np.float32)      # scores in the hundreds
    q = _scale_rows(q, f)
    O_ref, L_ref = oattn.masked_attention(q, k, v, mask)
    for pid in _eligible_plans(mask):
        log("case %s mode %s plan %d" % (name, mode, pid))
        p, od, lsed, _ = run_plan(bsa, mask, q, k, v, force_plan=pid)
        compare(bf16_to_f64(od), O_ref, "%s %s plan %d" % (name, mode, pid))
        compare_lse(lsed.cpu().numpy().astype(np.float64), L_ref, "%s %s plan %d" % (name, mode, pid))
        p.destroy()


def test_rows_are_convex_combinations_of_allowed_values():
    q, k, v, mask = random_case(503, 1, 2, 384, 384, 128, [(32, 32)] * 2, 0.2, empty_rows=1)
    p, od, _, _ = run_plan(bsa, mask, q, k, v)
    O = bf16_to_f64(od)
    V = brute.bf16_to_f64(v)
    for h in range(2):
        E = brute.token_mask(mask.head(0, h), 32, 32, 384, 384)
        for i in range(384):
            if not E[i].any():
                assert np.all(O[0, i, h] == 0.0)
                continue
            lo, hi = V[0, E[i], h].min(axis=0), V[0, E[i], h].max(axis=0)
            slack = 2.0 ** -7 * np.maximum(np.abs(lo), np.abs(hi)) + 1e-6   # bf16 output rounding
            assert np.all(O[0, i, h] >= lo - slack) and np.all(O[0, i, h] <= hi + slack), (h, i)


def test_split_k_partitions_agree():
    q, k, v, mask = random_case(504, 1, 2, 1024, 1024, 128, [(64, 64)] * 2, 0.5)
    cat = bsa.catalog()
    for tq, tkv in [(64, 64), (128, 32), (256, 64)]:
        outs = []
        for e in cat:
            if (e["tq"], e["tkv"]) == (tq, tkv):
                p, od, _, _ = run_plan(bsa, mask, q, k, v, force_plan=e["id"], lse=False)
                outs.append(bf16_to_f64(od))
                p.destroy()
        for o in outs[1:]:
            assert np.max(np.abs(o - outs[0])) <= 1e-2 and np.mean(np.abs(o - outs[0])) <= 1e-3


def test_run_to_run_bitwise_determinism():
    q, k, v, mask = random_case(505, 1, 2, 900, 900, 128, [(64, 64)] * 2, 0.4)
    for pid in (4, 13, 22):
        p, o1, l1, (qd, kd, vd, _) = run_plan(bsa, mask, q, k, v, force_plan=pid)
        o2 = o1.clone().zero_()
        l2 = l1.clone().zero_()
        bsa.forward(p, qd, kd, vd, o2, l2)
        import torch
        torch.cuda.synchronize()
        assert torch.equal(o1, o2) and torch.equal(l1, l2), pid
        p.destroy()


def test_empty_mask_gives_zero_and_neg_inf():
    q, k, v, mask = random_case(506, 1, 2, 500, 500, 128, [(64, 64)] * 2, 0.0)
    assert mask.data.sum() == 0
    for pid in (4, 13):
        p, od, lsed, _ = run_plan(bsa, mask, q, k, v, force_plan=pid)
        assert (od.float() == 0).all().item()
        assert np.all(np.isneginf(lsed.cpu().numpy()))
        p.destroy()


def test_broadcast_mask_over_batch_and_strided_tensors():
    import torch
    q, k, v, mask = random_case(507, 1, 2, 640, 640, 128, [(64, 64)] * 2, 0.3)
    B = 2
    rng = np.random.default_rng(507)
    q2 = bf16_bits_from_f32(rng.standard_normal((B, 640, 2, 128), dtype=np.float32))
    k2 = bf16_bits_from_f32(rng.standard_normal((B, 640, 2, 128), dtype=np.float32))
    v2 = bf16_bits_from_f32(rng.standard_normal((B, 640, 2, 128), dtype=np.float32))
    # broadcast: batch stride 0 over a one-batch mask
    mask_b = BlockMask(mask.data, mask.head_offset, 0, mask.bq, mask.bkv, B, 2, 640, 640)
    O_ref, L_ref = oattn.masked_attention(q2, k2, v2, mask_b)
    # strided Q/O: every token row padded to 384 elements (head_dim 128 is a view)
    big_q = torch.zeros((B, 640, 2, 384), dtype=torch.bfloat16, device="cuda")
    big_q[..., :128] = to_dev_bf16(q2)
    qd = big_q[..., :128]
    kd, vd = to_dev_bf16(k2), to_dev_bf16(v2)
    big_o = torch.zeros((B, 640, 2, 256), dtype=torch.bfloat16, device="cuda")
    od = big_o[..., 128:]
    md = torch.from_numpy(mask.data).cuda()
    shapes = bsa.shapes_of(qd, kd, vd, od)
    p = bsa.plan(md, 64, 64, shapes, head_offset=list(mask.head_offset), stride_b=0)
    lse = torch.empty((B, 2, 640), dtype=torch.float32, device="cuda")
    bsa.forward(p, qd, kd, vd, od, lse)
    torch.cuda.synchronize()
    compare(bf16_to_f64(od), O_ref, "broadcast/strided")
    compare_lse(lse.cpu().numpy().astype(np.float64), L_ref, "broadcast/strided")
    assert (big_o[..., :128] == 0).all().item()      # nothing written outside O
    p.destroy()


def test_plan_is_reusable_for_new_inputs():
    import torch
    q, k, v, mask = random_case(508, 1, 2, 512, 512, 128, [(64, 64)] * 2, 0.3)
    p, od, _, _ = run_plan(bsa, mask, q, k, v, lse=False)
    rng = np.random.default_rng(9)
    for trial in range(2):
        q2, k2, v2 = (bf16_bits_from_f32(rng.standard_normal(q.shape, dtype=np.float32)) for _ in range(3))
        O_ref, _ = oattn.masked_attention(q2, k2, v2, mask)
        o2 = torch.empty_like(od)
        bsa.forward(p, to_dev_bf16(q2), to_dev_bf16(k2), to_dev_bf16(v2), o2)
        torch.cuda.synchronize()
        compare(bf16_to_f64(o2), O_ref, "reuse %d" % trial)
    p.destroy()


def test_kv_rows_beyond_2_gib():
    """One head's K/V rows reach past 2^31 bytes from the head's first token
    (12 heads x 128 bf16 = 3 KB per token, 720,896 tokens): the kernel's
    per-head 32-bit offsets must stay unsigned.  Every query block attends
    to the same blocks on both sides of the 2 GiB mark plus one of its own;
    the oracle evaluates the compact problem made of exactly those blocks
    (Eq. 1 depends only on the active token pairs)."""
    import torch
    B, H, Nq, d, blk = 1, 12, 256, 128, 64
    nkb = 11264
    Nkv = nkb * blk
    nqb = Nq // blk
    g = torch.Generator(device="cuda")
    g.manual_seed(2024)
    qd = torch.randn((B, Nq, H, d), generator=g, device="cuda").to(torch.bfloat16)
    kd = torch.randn((B, Nkv, H, d), generator=g, device="cuda").to(torch.bfloat16)
    vd = torch.randn((B, Nkv, H, d), generator=g, device="cuda").to(torch.bfloat16)
    boundary = (1 << 31) // (H * d * 2) // blk          # first block past 2 GiB from token 0
    common = [0, 5000, boundary - 1, boundary, boundary + 77, nkb - 1]
    heads = []
    for h in range(H):
        m = np.zeros((nqb, nkb), dtype=np.uint8)
        for qb in range(nqb):
            m[qb, common] = 1
            m[qb, boundary + 100 + 7 * qb + h] = 1
        heads.append(m)
    mask = BlockMask.from_heads([heads], [blk] * H, [blk] * H, Nq, Nkv)
    md = torch.from_numpy(np.ascontiguousarray(mask.data)).cuda()
    shapes = bsa.shapes_of(qd, kd, vd, qd)
    assert all(bsa.plan_eligible(pid, blk, blk, shapes) for pid in (0, 4, 12, 16))

    # the compact problem: the union of the active blocks, in order
    union = sorted(set(common) | {boundary + 100 + 7 * qb + h for qb in range(nqb) for h in range(H)})
    idx = torch.tensor([b * blk + t for b in union for t in range(blk)], device="cuda")
    to_bits = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    q_bits = to_bits(qd)
    k_bits, v_bits = to_bits(kd[:, idx]), to_bits(vd[:, idx])
    pos = {b: i for i, b in enumerate(union)}
    compact = []
    for h in range(H):
        mc = np.zeros((nqb, len(union)), dtype=np.uint8)
        for qb in range(nqb):
            for kb in np.nonzero(heads[h][qb])[0]:
                mc[qb, pos[int(kb)]] = 1
        compact.append(mc)
    cmask = BlockMask.from_heads([compact], [blk] * H, [blk] * H, Nq, len(union) * blk)
    O_ref, L_ref = oattn.masked_attention(q_bits, k_bits, v_bits, cmask)

    for pid in (-1, 4, 0, 12, 16):
        od = torch.empty_like(qd)
        lsed = torch.empty((B, H, Nq), dtype=torch.float32, device="cuda")
        p = bsa.plan(md, blk, blk, shapes, head_offset=list(mask.head_offset), stride_b=mask.stride_b,
                     force_plan=pid)
        bsa.forward(p, qd, kd, vd, od, lsed)
        torch.cuda.synchronize()
        log("  K/V past 2 GiB, plan %d" % p.info(0)["plan_id"])
        compare(bf16_to_f64(od), O_ref, "kv>2GiB plan %d" % pid)
        compare_lse(lsed.cpu().numpy().astype(np.float64), L_ref, "kv>2GiB plan %d" % pid)
        p.destroy()
    del qd, kd, vd
    torch.cuda.empty_cache()


def test_dispatch_order_does_not_change_the_output():
    """Tasks dispatched with equal KV lists side by side (the default above 512
    tasks) and in row order give the same bits, every row is written (outputs
    start as NaN), and both match the oracle.  A 3-D window over an (8, 4, 4)
    grid of 64-token blocks whose middle half-width covers the whole grid, so
    the four query blocks of a (t, w) pair have equal KV lists and sit a grid
    stride apart in row order; 10 heads."""
    import torch
    from workloads.gen import window_mask
    grid, half, bs, H = (8, 4, 4), (1, 3, 1), 64, 10
    blocks = window_mask(grid, half).astype(np.uint8)
    N = blocks.shape[0] * bs
    rng = np.random.default_rng(91)
    q, k, v = (bf16_bits_from_f32(rng.standard_normal((1, N, H, 128), dtype=np.float32)) for _ in range(3))
    mask = BlockMask.from_heads([[blocks] * H], [bs] * H, [bs] * H, N, N)
    O_ref, L_ref = oattn.masked_attention(q, k, v, mask)
    ids = _eligible_plans(mask)
    split_ids = [e["id"] for e in bsa.catalog() if e["id"] in ids and e["split"] > 1]
    assert split_ids
    ordered = 0
    for pid in [-1] + ids:
        log("dispatch order, plan %d" % pid)
        p1, o1, l1, _ = run_plan(bsa, mask, q, k, v, force_plan=pid)
        p2, o2, l2, _ = run_plan(bsa, mask, q, k, v, force_plan=pid, keep_row_order=True)
        n_tasks = p1.info()["n_tasks"]
        ordered += n_tasks > 512
        tasks = p1.export(bsa.EXPORT_TASKS)
        want = np.arange(len(tasks))
        if n_tasks > 512:
            member = p1.export(bsa.EXPORT_TILE_MEMBER)
            want = expected_dispatch(tasks, p1.export(bsa.EXPORT_TILE_KV), member if len(member) else None)
        assert np.array_equal(p1.export(bsa.EXPORT_DISPATCH), want), "plan %d: dispatch order" % pid
        assert np.array_equal(p2.export(bsa.EXPORT_DISPATCH), np.arange(len(tasks)))
        assert torch.equal(o1, o2) and torch.equal(l1, l2), "plan %d: the dispatch order changed the output" % pid
        compare(bf16_to_f64(o1), O_ref, "dispatch order plan %d" % pid)
        compare_lse(l1.cpu().numpy().astype(np.float64), L_ref, "dispatch order plan %d" % pid)
        p1.destroy()
        p2.destroy()
    assert ordered >= len(ids) // 2, "too few plans with more than 512 tasks"
