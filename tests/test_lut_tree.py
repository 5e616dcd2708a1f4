"""Decision-tree regimes (Section 5.1) and the version-2 plan table: the
learned regions, their rankings and the library's lookup (CPU only)."""
from __future__ import annotations

import json
import math

import numpy as np
import pytest

bsa = pytest.importorskip("paper_2609_25869_amd")
from oracle import regime  # noqa: E402
from paper_2609_25869_amd.lut import compile as lutc  # noqa: E402
from paper_2609_25869_amd.lut import tree  # noqa: E402


def base(key):
    return bsa.base_plan(key[0], key[1])


def oracle_features(f, bq=64):
    """Regime features from their definitions (query_rows = batch x heads x
    ceil(seq_q / B_Q), row_imbalance = max_row_nnz * query_rows / nnz)."""
    rows = f["batch_heads"] * math.ceil(f["seq_q"] / bq)
    return {"seq_q": f["seq_q"], "batch_heads": f["batch_heads"], "density": (f["nnz"], f["blocks"]),
            "run_coverage": (f["run_blocks"], f["nnz"]), "query_rows": rows,
            "row_imbalance": (f["max_row_nnz"] * rows, f["nnz"])}


def structured_records(seed, n=240, key=(64, 64, 0, 128)):
    """Plan 12 wins below 20% density, plan 4 above; plan 8 is always a bit
    slower than the winner; five sources (families)."""
    rng = np.random.default_rng(seed)
    recs = []
    for i in range(n):
        blocks = 10000
        nnz = int(rng.integers(100, 6000))
        dens = nnz / blocks
        lat = {"12": 1.0 if dens < 0.2 else 1.6, "4": 1.5 if dens < 0.2 else 1.0,
               "8": 1.1, "0": 2.0 + rng.random()}
        lat = {p: t * (1 + 0.01 * rng.random()) for p, t in lat.items()}
        feats = {"seq_q": int(rng.choice([8192, 65536])), "seq_kv": 8192, "batch_heads": int(rng.choice([4, 24])),
                 "nnz": nnz, "blocks": blocks, "run_blocks": int(rng.integers(0, nnz + 1)),
                 "max_row_nnz": int(rng.integers(0, nnz + 1))}
        recs.append(lutc.with_query_rows({"id": "t%d" % i, "key": list(key), "family": "f%d" % (i % 5),
                                          "rho": 0.1, "features": feats, "latency_ms": lat}))
    return recs


def test_tree_splits_where_the_best_plan_changes():
    recs = structured_records(0)
    regions = tree.compile_regions(recs, base)
    ent = regions[(64, 64, 0, 128)]
    assert ent["depth"] >= 1
    leaves = ent["regimes"]
    assert len(leaves) >= 2
    for region, ranking, n in leaves:
        assert n >= tree.MIN_LEAF
        members = [r for r in recs if tree.in_region(r["features"], region)]
        assert len(members) == n
        # the leaf ranking is Algorithm 1 over the leaf's cases, base plan appended
        cases = [{"id": r["id"], "key": tuple(r["key"]), "features": oracle_features(r["features"])} for r in members]
        lat = {(r["id"], int(p)): t for r in members for p, t in r["latency_ms"].items()}
        one = [("seq_q", [])]
        want = regime.compile_table(cases, lat, one, base)[(64, 64, 0, 128)][(0,)]
        assert ranking == want
    # the density split separates the two winners
    first = {ranking[0] for _, ranking, _ in leaves}
    assert first == {12, 4}


def test_regions_partition_every_case_and_random_query():
    recs = structured_records(1)
    regions = tree.compile_regions(recs, base)
    leaves = regions[(64, 64, 0, 128)]["regimes"]
    rng = np.random.default_rng(2)
    probes = [r["features"] for r in recs]
    for _ in range(300):
        blocks = int(rng.integers(1, 20000))
        nnz = int(rng.integers(0, blocks + 1))
        f = {"seq_q": int(rng.integers(1, 200000)), "batch_heads": int(rng.integers(1, 64)),
             "nnz": nnz, "blocks": blocks, "run_blocks": int(rng.integers(0, nnz + 1)),
             "max_row_nnz": int(rng.integers(0, nnz + 1))}
        probes.append(lutc.with_query_rows({"key": [64, 64, 0, 128], "features": f})["features"])
    for f in probes:
        inside = [region for region, _, _ in leaves if tree.in_region(f, region)]
        assert len(inside) == 1
        assert regime.region_contains(oracle_features(f), inside[0], tree.FEATURES)


def test_too_few_cases_give_one_regime_per_key():
    recs = structured_records(3, n=50)
    ent = tree.compile_regions(recs, base)[(64, 64, 0, 128)]
    assert len(ent["regimes"]) == 1 and ent["regimes"][0][2] == 50


def write_v2(tmp_path, regions):
    doc = lutc.artifact_v2(regions, bsa.catalog(), {})
    p = tmp_path / "v2.json"
    p.write_text(json.dumps(doc))
    return str(p), doc


def test_library_lookup_matches_the_regions(tmp_path):
    recs = structured_records(4) + structured_records(5, key=(128, 128, 0, 128))
    regions = tree.compile_regions(recs, base)
    path, doc = write_v2(tmp_path, regions)
    lut = bsa.Lut(path)
    rng = np.random.default_rng(6)
    edges = sorted({b for r in doc["regimes"] for iv in r["region"] for b in iv if b is not None})
    for t in range(400):
        bq, bkv = [(64, 64), (128, 128), (32, 32)][t % 3]
        blocks = 10000 if t % 2 else int(rng.integers(1, 20000))
        # half the probes sit exactly on a learned density edge
        nnz = edges[t % len(edges)] if (t % 4 == 1 and edges and edges[t % len(edges)] <= 10000) \
            else int(rng.integers(0, blocks + 1))
        z = bsa.regime_query(bq, bkv, int(rng.choice([4, 24])), int(rng.choice([8192, 65536])), 8192,
                             nnz=nnz, blocks=blocks, run_blocks=int(rng.integers(0, nnz + 1)),
                             max_row_nnz=int(rng.integers(0, nnz + 1)))
        feats = {"seq_q": z.seq_q, "batch_heads": z.batch_heads, "nnz": nnz, "blocks": blocks,
                 "run_blocks": z.run_blocks, "max_row_nnz": z.max_row_nnz}
        key = (bq, bkv, 0, 128)
        # Algorithm 2's lookup over the key's regions, by the oracle's leaf test
        leaves = [(region, ranking) for region, ranking, _ in regions.get(key, {}).get("regimes", [])]
        want, hit = regime.lookup_regions(leaves, oracle_features(feats, bq), tree.FEATURES, base(key))
        assert sum(regime.region_contains(oracle_features(feats, bq), r, tree.FEATURES) for r, _ in leaves) <= 1
        got, ghit = bsa.lut_rank(z, lut)
        assert (got, ghit) == (want, hit), (t, key, feats)
        assert tree.select(regions, key, feats, base(key)) == (want, hit)
    lut.close()


@pytest.mark.parametrize("mutate,needle", [
    (lambda d: d["regimes"][0].__setitem__("region", d["regimes"][0]["region"][:-1]), "regime"),
    (lambda d: d["regimes"][0]["region"].__setitem__(2, [500, 500]), "interval"),
    (lambda d: d.__setitem__("features", ["seq_q", "batch_heads", "density", "colour"]), "feature"),
    (lambda d: d["regimes"][0].__setitem__("ranking", [99]), "plan"),
])
def test_v2_artifact_validation(tmp_path, mutate, needle):
    regions = tree.compile_regions(structured_records(7), base)
    _, doc = write_v2(tmp_path, regions)
    mutate(doc)
    p = tmp_path / "bad.json"
    p.write_text(json.dumps(doc))
    with pytest.raises(bsa.BsaError) as e:
        bsa.Lut(str(p))
    assert needle in str(e.value)
