"""Host-side checks of the C-ABI library (no GPU needed).

The library must load on a machine without a GPU, export exactly the entry
points include/bsa.h declares, and its host logic (catalog, eligibility,
base plans, plan-table artifact, Algorithm 2 selection) must agree with the
plain restatement of Section 5 in oracle/regime.py.
"""
from __future__ import annotations

import ctypes
import itertools
import json
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bsa.h")

bsa = pytest.importorskip("paper_2609_25869_amd")
from paper_2609_25869_amd import _ffi  # noqa: E402
from oracle import regime  # noqa: E402


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^BSA_API\s+[\w\s\*]*?\b(bsa_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_request_entry_points():
    names = header_functions()
    for required in ("bsa_plan", "bsa_forward", "bsa_plan_destroy", "bsa_lut_load", "bsa_plan_export",
                     "bsa_plan_info", "bsa_status_string", "bsa_last_error", "bsa_sparsify_topk"):
        assert required in names
    assert len(names) == 20


def test_library_exports_exactly_the_header():
    lib = ctypes.CDLL(_ffi.LIB_PATH)
    for name in header_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", _ffi.LIB_PATH], stdout=subprocess.PIPE, text=True,
                         check=True).stdout
    exported = sorted(line.split()[-1] for line in out.splitlines() if line.split()[1] == "T")
    assert exported == header_functions()


def test_binding_covers_every_entry_point():
    assert sorted(n for n, _, _ in _ffi.SIGNATURES) == header_functions()


def test_version_and_status_strings():
    assert bsa.version() == (1, 1)
    lib = bsa._lib
    for s in range(6):
        assert lib.bsa_status_string(s)
    assert b"unknown" in lib.bsa_status_string(99).lower()


def test_catalog_layout():
    """Every catalog entry names the kernel that runs it: wavefronts and ring
    depth as launched (one wave per 32 query rows and 64 KB rings, except
    T = (256, 32), four waves of 64 rows with an eight-slot ring); ids 24-29
    repeat the split-free tiles with the all-XCD traversal order; ids 30-32
    are the other ring depth of (64, 32), (128, 32) and (256, 64) (XCD pairs),
    ids 33-34 the first two of those with the all-XCD order."""
    cat = bsa.catalog()
    assert len(cat) == 35
    tqs, tkvs, splits = (64, 128, 256), (32, 64), (1, 2, 4, 8)

    def launched(tq, tkv):
        return (8, 4) if (tq, tkv) == (256, 32) else ((4 if tkv == 32 else 2), tq // 32)

    for e in cat[:24]:
        i = e["id"]
        assert (e["tq"], e["tkv"], e["split"]) == (tqs[i // 8], tkvs[(i // 4) % 2], splits[i % 4])
        assert (e["stages"], e["waves"]) == launched(e["tq"], e["tkv"])
        assert e["xcd_group"] == 2
    for j, e in enumerate(cat[24:30]):
        assert (e["id"], e["tq"], e["tkv"], e["split"], e["xcd_group"]) == (24 + j, tqs[j // 2], tkvs[j % 2], 1, 8)
        assert (e["stages"], e["waves"]) == launched(e["tq"], e["tkv"])
    # the (256, 32) plans run four 64-row waves through an eight-slot ring
    assert [(e["stages"], e["waves"]) for e in cat[16:20]] == [(8, 4)] * 4
    assert [(e["id"], e["tq"], e["tkv"], e["split"], e["stages"], e["waves"], e["xcd_group"]) for e in cat[30:]] == [
        (30, 64, 32, 1, 2, 2, 2), (31, 128, 32, 1, 2, 4, 2), (32, 256, 64, 1, 4, 8, 2),
        (33, 64, 32, 1, 2, 2, 8), (34, 128, 32, 1, 2, 4, 8)]
    st = bsa._lib.bsa_catalog_get(35, ctypes.byref(_ffi.CatalogEntry()))
    assert st == _ffi.BSA_ERR_INVALID


def test_base_plans():
    # Direct plan at T = B when the catalog has that tile; otherwise the nearest tile.
    assert bsa.base_plan(64, 64) == 4
    assert bsa.base_plan(128, 32) == 8
    assert bsa.base_plan(256, 64) == 20
    assert bsa.base_plan(128, 128) == 12
    assert bsa.base_plan(16, 16) == 0
    for bq, bkv in itertools.product((16, 32, 64, 128, 256, 512), repeat=2):
        p = bsa.base_plan(bq, bkv)
        assert bsa.catalog()[p]["split"] == 1


def test_eligibility_rules():
    s = bsa.make_shapes(1, 2, 1000, 1000)
    assert all(bsa.plan_eligible(p, 64, 64, s) for p in range(24))
    # head dim other than 128: nothing is eligible, so selection reports no eligible plan
    s64 = bsa.make_shapes(1, 2, 1000, 1000, head_dim=64)
    assert not any(bsa.plan_eligible(p, 64, 64, s64) for p in range(24))
    z = bsa.regime_query(64, 64, 2, 1000, 1000, nnz=10, blocks=256, run_blocks=0, head_dim=64)
    assert bsa.select_plan(z, s64) is None
    # bf16 only
    sf = bsa.make_shapes(1, 2, 1000, 1000, dtype=_ffi.DTYPE_F16)
    assert not bsa.plan_eligible(12, 64, 64, sf)
    # coarsening needs power-of-two ratios and at most 64 member blocks per tile
    assert not bsa.plan_eligible(12, 48, 48, s)
    assert bsa.plan_eligible(20, 16, 16, s)       # (256,64) over (16,16): 16*4 = 64 members, the limit
    assert not bsa.plan_eligible(20, 16, 8, s)    # 16*8 = 128 members
    assert bsa.plan_eligible(20, 32, 16, s) and bsa.plan_eligible(4, 16, 16, s)
    # strides must keep 16-byte rows
    bad = bsa.make_shapes(1, 2, 1000, 1000)
    bad.q_stride[2] = 129
    assert not bsa.plan_eligible(4, 64, 64, bad)


SCHEMA = [("seq_q", [4096, 32768]), ("batch_heads", [8]), ("density", [500, 2000]), ("run_coverage", [5000])]
ARCH_OK = "gfx950"


def artifact(table, schema=SCHEMA, **over):
    doc = {
        "format": "bsa-plan-table", "version": 1, "arch": ARCH_OK,
        "catalog": [[e["id"], e["tq"], e["tkv"], e["split"], e["stages"], e["waves"], e["xcd_group"]]
                    for e in bsa.catalog()],
        "schema": [[n, list(e)] for n, e in schema],
        "regimes": [{"key": list(k), "bucket": list(b), "ranking": list(r)}
                    for k, bt in table.items() for b, r in bt.items()],
    }
    doc.update(over)
    return doc


def write(tmp_path, doc, name="t.json"):
    p = tmp_path / name
    p.write_text(doc if isinstance(doc, str) else json.dumps(doc))
    return str(p)


def synthetic_table(seed=0):
    """An oracle-compiled table from a synthetic latency table."""
    rng = np.random.default_rng(seed)
    keys = [(64, 64, 0, 128), (128, 128, 0, 128), (128, 32, 0, 128)]
    cases, lat = [], {}
    for cid in range(120):
        key = keys[cid % 3]
        feats = {"seq_q": int(rng.choice([2048, 8192, 65536])), "batch_heads": int(rng.choice([2, 24])),
                 "density": (int(rng.integers(0, 1000)), 1000), "run_coverage": (int(rng.integers(0, 50)), 50)}
        cases.append({"id": cid, "key": key, "features": feats})
        for p in range(24):
            if rng.random() < 0.9:
                lat[(cid, p)] = float(rng.choice([1.0, 1.5, 2.0, 3.0]))   # ties on purpose
    base = lambda key: bsa.base_plan(key[0], key[1])
    return regime.compile_table(cases, lat, SCHEMA, base), base


def features_of(z):
    return {"seq_q": z.seq_q, "seq_kv": z.seq_kv, "batch_heads": z.batch_heads,
            "density": (z.nnz, z.blocks), "run_coverage": (z.run_blocks, z.nnz)}


def test_sparsifier_rejects_bad_requests_before_any_launch():
    """Argument errors surface before any device work (null pointers, block
    sizes, dtype, head dim, KV blocks per row)."""
    s = bsa.make_shapes(1, 2, 1024, 1024)
    fake = ctypes.c_void_p(16)      # never dereferenced: every case fails validation first
    call = lambda q, k, sh, bq, bkv, m: bsa._lib.bsa_sparsify_topk(q, k, ctypes.byref(sh), bq, bkv, 4, 1, m, None)
    assert call(None, fake, s, 64, 64, fake) == _ffi.BSA_ERR_INVALID
    assert call(fake, fake, s, 64, 64, None) == _ffi.BSA_ERR_INVALID
    assert call(fake, fake, s, 0, 64, fake) == _ffi.BSA_ERR_INVALID
    assert call(fake, fake, bsa.make_shapes(1, 2, 1024, 1024, head_dim=64), 64, 64, fake) == _ffi.BSA_ERR_UNSUPPORTED
    assert call(fake, fake, bsa.make_shapes(1, 2, 1024, 1024, dtype=_ffi.DTYPE_F16), 64, 64, fake) == \
        _ffi.BSA_ERR_UNSUPPORTED
    assert call(fake, fake, bsa.make_shapes(1, 2, 64, 6145 * 16), 16, 16, fake) == _ffi.BSA_ERR_UNSUPPORTED
    assert b"KV blocks per row" in bsa._lib.bsa_last_error()


def test_kv_rows_of_one_head_must_fit_32_bit_offsets():
    """K and V rows of a head are addressed with 32-bit byte offsets, up to
    a tile past the sequence end: larger requests have no eligible plan."""
    # [B, N, H, 128] bf16: a token row of all heads is H * 256 bytes
    ok = bsa.make_shapes(1, 24, 1024, 131072)              # 131136 * 6144 B = 0.75 GiB
    assert all(bsa.plan_eligible(p, 64, 64, ok) for p in range(24))
    big = bsa.make_shapes(1, 64, 1024, 300000)              # 300064 * 16384 B > 4 GiB
    assert not any(bsa.plan_eligible(p, 64, 64, big) for p in range(24))
    # the limit is on the token stride of K and V, not on the head count
    edge_rows = (0xFFFFFFFF - 256) // (2 * 24 * 128) - 64
    assert bsa.plan_eligible(4, 64, 64, bsa.make_shapes(1, 24, 64, edge_rows))
    assert not bsa.plan_eligible(4, 64, 64, bsa.make_shapes(1, 24, 64, edge_rows + 1))


def test_lut_rank_and_select_match_the_reference(tmp_path):
    table, base = synthetic_table()
    assert table
    lut = bsa.Lut(write(tmp_path, artifact(table)))
    rng = np.random.default_rng(1)
    hits = 0
    for t in range(400):
        bq, bkv = [(64, 64), (128, 128), (128, 32), (32, 32)][t % 4]
        blocks = int(rng.integers(1, 5000))
        nnz = int(rng.integers(0, blocks + 1))
        z = bsa.regime_query(bq, bkv, int(rng.choice([2, 24])), int(rng.choice([2048, 8192, 65536])), 4096,
                             nnz=nnz, blocks=blocks, run_blocks=int(rng.integers(0, nnz + 1)))
        key = (bq, bkv, 0, 128)
        bucket = regime.bucket_of(features_of(z), SCHEMA)
        ranking, hit = bsa.lut_rank(z, lut)
        ref = table.get(key, {}).get(bucket)
        assert hit == (ref is not None)
        assert ranking == (ref if ref is not None else [base(key)])
        hits += hit
        shapes = bsa.make_shapes(1, z.batch_heads, z.seq_q, z.seq_kv)
        elig = lambda p: bsa.plan_eligible(p, bq, bkv, shapes)
        assert bsa.select_plan(z, shapes, lut) == regime.select(table, key, bucket, base, elig)
    assert hits > 50
    lut.close()


def test_density_bucket_edges_are_exact_integers(tmp_path):
    table = {(64, 64, 0, 128): {(0, 0, 1, 0): [8], (0, 0, 2, 0): [16]}}
    lut = bsa.Lut(write(tmp_path, artifact(table)))
    # edge 500 (5.00%): 5 of 100 blocks is exactly on the edge and belongs to the upper bucket
    for nnz, blocks, want in [(5, 100, [8]), (4999999, 100000000, [4]), (200, 1000, [16]), (199, 1000, [8])]:
        z = bsa.regime_query(64, 64, 2, 1000, 1000, nnz=nnz, blocks=blocks, run_blocks=0)
        assert bsa.lut_rank(z, lut)[0] == want, (nnz, blocks)


@pytest.mark.parametrize("mutate,needle", [
    (lambda d: d.update(format="other"), "artifact"),
    (lambda d: d.update(version=3), "version"),
    (lambda d: d.update(arch="gfx942"), "gfx950"),
    (lambda d: d["catalog"].pop(), "catalog"),
    (lambda d: d["catalog"][3].__setitem__(2, 999), "catalog"),
    (lambda d: d["regimes"][0].__setitem__("ranking", [77]), "unknown plan"),
    (lambda d: d["regimes"][0].__setitem__("ranking", []), "regime"),
    (lambda d: d["schema"][0].__setitem__(1, [5, 5]), "increase"),
    (lambda d: d["schema"].append(["entropy", [1]]), "unknown feature"),
])
def test_lut_rejects_bad_artifacts(tmp_path, mutate, needle):
    table = {(64, 64, 0, 128): {(0, 0, 0, 0): [4]}}
    doc = artifact(table)
    mutate(doc)
    with pytest.raises(_ffi.BsaError) as e:
        bsa.Lut(write(tmp_path, doc))
    assert e.value.status == _ffi.BSA_ERR_LUT
    assert needle in str(e.value).lower()


def test_lut_rejects_malformed_json_and_missing_file(tmp_path):
    with pytest.raises(_ffi.BsaError) as e:
        bsa.Lut(write(tmp_path, '{"format": "bsa-plan-table", '))
    assert e.value.status == _ffi.BSA_ERR_LUT
    with pytest.raises(_ffi.BsaError) as e:
        bsa.Lut(str(tmp_path / "missing.json"))
    assert e.value.status == _ffi.BSA_ERR_LUT


def test_null_arguments_are_rejected():
    lib = bsa._lib
    assert lib.bsa_lut_load(None, None) == _ffi.BSA_ERR_INVALID
    assert lib.bsa_plan(None, None, None, 1, None, None, None, None) == _ffi.BSA_ERR_INVALID
    assert lib.bsa_forward(None, None, None, None, None, None, None) == _ffi.BSA_ERR_INVALID
    assert lib.bsa_plan_destroy(None) == _ffi.BSA_OK
    assert lib.bsa_last_error()


def test_query_rows_feature_is_counted_from_its_definition(tmp_path):
    """The derived feature query_rows = batch x heads x ceil(seq_q / B_Q) (the
    number of logical query-block rows) is computed by the library from the
    regime query, so a grid over it buckets like the oracle's restatement."""
    schema = [("query_rows", [1024, 4096]), ("density", [500, 2000])]
    rng = np.random.default_rng(3)
    table = {}
    for key in [(64, 64, 0, 128), (128, 32, 0, 128), (16, 16, 0, 128)]:
        for b0 in range(3):
            for b1 in range(3):
                table.setdefault(key, {})[(b0, b1)] = [int(x) for x in rng.choice(24, 3, replace=False)]
    doc = artifact(table, schema)
    lut = bsa.Lut(write(tmp_path, doc))
    for t in range(300):
        bq, bkv = [(64, 64), (128, 32), (16, 16)][t % 3]
        seq_q = int(rng.choice([1, 1000, 1024, 4095, 4096, 65536, 131071]))
        bh = int(rng.choice([1, 2, 8, 24, 48]))
        # half the probes sit exactly on an edge of the row count
        if t % 2:
            bh = 1
            seq_q = bq * int(rng.choice([1023, 1024, 4095, 4096]))
        blocks = int(rng.integers(1, 5000))
        nnz = int(rng.integers(0, blocks + 1))
        z = bsa.regime_query(bq, bkv, bh, seq_q, seq_q, nnz=nnz, blocks=blocks, run_blocks=0)
        feats = {"query_rows": bh * -(-seq_q // bq), "density": (nnz, blocks)}
        want = table[(bq, bkv, 0, 128)][regime.bucket_of(feats, schema)]
        assert bsa.lut_rank(z, lut) == (want, 1), (bq, seq_q, bh)
    lut.close()


def test_row_imbalance_feature_is_counted_from_its_definition(tmp_path):
    """row_imbalance = max_row_nnz * query_rows / nnz, compared with its
    edges exactly as integers like the other ratios (0 when nnz is 0)."""
    schema = [("row_imbalance", [15000, 30000])]
    table = {(64, 64, 0, 128): {(0,): [0], (1,): [8], (2,): [16]}}
    lut = bsa.Lut(write(tmp_path, artifact(table, schema)))
    rng = np.random.default_rng(4)
    cases = [(0, 0, 7, 0), (1, 100, 150, 1), (1, 100, 151, 1), (2, 1000, 3000, 64)]
    for _ in range(200):
        cases.append((int(rng.integers(1, 5)), int(rng.integers(0, 5000)), int(rng.integers(0, 3000)),
                      int(rng.integers(64, 20000))))
    for bh, nnz, max_row, seq_q in cases:
        rows = bh * -(-seq_q // 64)
        z = bsa.regime_query(64, 64, bh, seq_q, seq_q, nnz=nnz, blocks=max(1, nnz) * 4, run_blocks=0,
                             max_row_nnz=max_row)
        feats = {"row_imbalance": (max_row * rows, nnz)}
        want = table[(64, 64, 0, 128)][regime.bucket_of(feats, schema)]
        assert bsa.lut_rank(z, lut) == (want, 1), (bh, nnz, max_row, seq_q)
    # exactly on an edge: one row of 3 blocks against a mean of 1 (3.0 = 30000 / 1e4)
    z = bsa.regime_query(64, 64, 1, 64 * 4, 64 * 4, nnz=4, blocks=16, run_blocks=0, max_row_nnz=3)
    assert bsa.lut_rank(z, lut) == ([16], 1)
    lut.close()
