"""The offline plan table: compilation rules, the shipped artifact, its use by the library (CPU only)."""
from __future__ import annotations

import json
import math
import os

import numpy as np
import pytest

bsa = pytest.importorskip("paper_2609_25869_amd")
from oracle import regime  # noqa: E402
from paper_2609_25869_amd.lut import compile as lutc  # noqa: E402

LUT_DIR = os.path.dirname(lutc.__file__)
ARTIFACT = os.path.join(LUT_DIR, "gfx950_v1.json")
PROFILE = lutc.PROFILES
EVAL = lutc.EVALS


def base(key):
    return bsa.base_plan(key[0], key[1])


def synthetic_records(seed, n=200):
    rng = np.random.default_rng(seed)
    keys = [[64, 64, 0, 128], [128, 128, 0, 128], [16, 16, 0, 128]]
    recs = []
    for i in range(n):
        blocks = int(rng.integers(100, 100000))
        nnz = int(rng.integers(0, blocks + 1))
        feats = {"seq_q": int(rng.choice([4096, 65536, 131072])), "seq_kv": 4096,
                 "batch_heads": int(rng.choice([2, 48])), "nnz": nnz, "blocks": blocks,
                 "run_blocks": int(rng.integers(0, nnz + 1)), "max_row_nnz": int(rng.integers(0, 4 * nnz // 3 + 2))}
        lat = {str(p): float(rng.choice([0.5, 1.0, 1.25, 2.0])) for p in range(24) if rng.random() < 0.85}
        recs.append(lutc.with_query_rows({"id": "s%d" % i, "key": keys[i % 3], "features": feats, "latency_ms": lat}))
    return recs


def oracle_features(f, key):
    """The regime features of Eq. 3 from their definitions: query_rows is
    batch x heads x ceil(seq_q / B_Q) logical query-block rows, and
    row_imbalance is max_row_nnz * query_rows / nnz."""
    rows = f["batch_heads"] * math.ceil(f["seq_q"] / key[0])
    return {"seq_q": f["seq_q"], "seq_kv": f["seq_kv"], "batch_heads": f["batch_heads"], "query_rows": rows,
            "density": (f["nnz"], f["blocks"]), "run_coverage": (f["run_blocks"], f["nnz"]),
            "row_imbalance": (f["max_row_nnz"] * rows, f["nnz"])}


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_compile_matches_the_algorithm_restatement(seed):
    recs = synthetic_records(seed)
    got = lutc.compile_table(recs, lutc.SCHEMA, base)
    cases = [{"id": r["id"], "key": tuple(r["key"]), "features": oracle_features(r["features"], r["key"])} for r in recs]
    lat = {(r["id"], int(p)): t for r in recs for p, t in r["latency_ms"].items()}
    want = regime.compile_table(cases, lat, lutc.SCHEMA, base)
    assert got == want


def test_bucket_matches_the_algorithm_restatement():
    for r in synthetic_records(5, 300):
        assert lutc.bucket(r["features"], lutc.SCHEMA) == regime.bucket_of(oracle_features(r["features"], r["key"]), lutc.SCHEMA)


def test_shipped_artifact_is_the_compiled_profile():
    doc = json.load(open(ARTIFACT))
    table = lutc.compile_table(lutc.load_records(PROFILE), lutc.SCHEMA, base)
    want = lutc.artifact(table, lutc.SCHEMA, bsa.catalog(), {})
    assert doc["regimes"] == want["regimes"]
    assert doc["schema"] == want["schema"] and doc["catalog"] == want["catalog"]
    assert doc["arch"] == "gfx950" and doc["format"] == "bsa-plan-table" and doc["version"] == 1


def test_profile_covers_every_geometry_and_validated_every_plan():
    recs = lutc.load_records(PROFILE)
    keys = {tuple(r["key"][:2]) for r in recs}
    assert {(128, 128), (128, 64), (64, 64), (64, 32), (32, 32), (32, 16), (16, 16), (128, 32), (32, 128)} <= keys
    for r in recs:
        eligible = [e["id"] for e in bsa.catalog() if bsa.plan_eligible(e["id"], r["key"][0], r["key"][1],
                                                                        bsa.make_shapes(1, 1, 1024, 1024))]
        assert sorted(int(p) for p in r["latency_ms"]) == eligible, r["id"]
        assert not r.get("invalid")


def test_library_uses_the_shipped_table_by_default():
    """With no table given, the library's lookup equals the artifact's rankings."""
    table = lutc.compile_table(lutc.load_records(PROFILE), lutc.SCHEMA, base)
    for r in lutc.load_records(EVAL)[::7]:
        f = r["features"]
        z = bsa.regime_query(r["key"][0], r["key"][1], f["batch_heads"], f["seq_q"], f["seq_kv"], f["nnz"],
                             f["blocks"], f["run_blocks"],
                             max_row_nnz=f["max_row_nnz"])
        ranking, hit = bsa.lut_rank(z)
        want = table.get(tuple(r["key"]), {}).get(lutc.bucket(f, lutc.SCHEMA))
        assert hit == (want is not None)
        assert ranking == (want if want is not None else [base(r["key"])])
        shapes = bsa.make_shapes(1, f["batch_heads"], f["seq_q"], f["seq_kv"])
        assert bsa.select_plan(z, shapes) == ranking[0]


def test_held_out_selection_regret():
    """Selected-plan regret on the held-out splits (measured latencies, 1 = optimal):
    within a few percent overall, and within 3% for kernels of 1 ms or more
    (the fastest measured plan includes both ring depths of every tile that
    has two)."""
    table = lutc.compile_table(lutc.load_records(PROFILE), lutc.SCHEMA, base)
    held = lutc.load_records(EVAL)
    rep = lutc.regret_report(table, lutc.SCHEMA, base, held)["all"]
    assert rep["cases"] >= 700
    assert rep["gm"] < 1.04
    long = [r for r in held if min(r["latency_ms"].values()) >= 1.0]
    rep_long = lutc.regret_report(table, lutc.SCHEMA, base, long)["all"]
    assert rep_long["cases"] >= 150 and rep_long["gm"] < 1.03


def test_kernel_ablations_on_constructed_records():
    """A0 = base plan, A1 = fastest, A2 = the pick; O-variants keep the base tile."""
    cat = bsa.catalog()
    key = [64, 64, 0, 128]
    b = base(tuple(key))                         # Direct (64,64), split 1
    same_tile = [e["id"] for e in cat if (e["tq"], e["tkv"]) == (64, 64) and e["id"] != b]
    other = [e["id"] for e in cat if (e["tq"], e["tkv"]) != (64, 64)][0]
    recs = [{"key": key, "features": {}, "latency_ms": {str(b): 2.0, str(same_tile[0]): 1.6, str(other): 1.0}}]
    out = lutc.kernel_ablations(lambda r: [same_tile[0]], base, cat, recs)
    assert math.isclose(out["kernel_speedup_over_A0"]["A1_exhaustive"], 2.0)
    assert math.isclose(out["kernel_speedup_over_A0"]["A2_table"], 2.0 / 1.6)
    o = out["organization_at_base_tile"]
    assert math.isclose(o["O1_speedup_over_O0"], 2.0 / 1.6) and math.isclose(o["O1_regret_vs_O2"], 1.0)
    assert o["O1_vs_O0_wins_ties_losses"] == [1, 0, 0]


def test_mapping_names_follow_section_4_2():
    assert lutc.mapping_name(64, 64, 64, 64) == "Direct"
    assert lutc.mapping_name(16, 16, 64, 32) == "Coarsened"
    assert lutc.mapping_name(128, 128, 128, 64) == "Refined"
    assert lutc.mapping_name(32, 128, 64, 32) == "mixed"


def test_request_ablation_summary():
    from paper_2609_25869_amd.lut import ablation
    recs = [{"plans": {"A0": 4, "A1": 8, "A2": 8},
             "request_ms": {"A0": [2.0, 2.0, 2.0, 2.0], "A1": [40.0, 1.5, 1.5, 1.5], "A2": [1.6, 1.0, 1.0, 1.0]},
             "kernel_ms": {"A0": 1.8, "A1": 1.2, "A2": 1.2}}]
    s = ablation.summarize(recs)
    assert math.isclose(s["cold"]["A1/A2"], 40.0 / 1.6) and math.isclose(s["warm"]["A0/A2"], 2.0)
    assert math.isclose(s["amortized"]["A0/A1"], 2.0 / ((40 + 4.5) / 4))
    assert math.isclose(s["kernel"]["A0/A2"], 1.5) and s["same_plan_as_A1"] == 1.0


def test_dispatch_summary_on_constructed_records():
    from paper_2609_25869_amd.lut import ablation
    recs = [{"key": [64, 64], "plan_ms": [0.30, 0.10, 0.12, 0.11], "select_us": {"mean": 1.0, "p95": 1.2}},
            {"key": [128, 128], "plan_ms": [0.50, 0.20, 0.20, 0.20], "select_us": {"mean": 2.0, "p95": 2.5}},
            {"key": [64, 64], "request_ms": {}}]  # a record without dispatch timings is left out
    d = ablation.dispatch_summary(recs)
    assert d["cases"] == 2
    assert math.isclose(d["plan_first_ms"]["mean"], 0.40) and d["plan_first_ms"]["n"] == 2
    assert d["plan_repeat_ms"]["n"] == 6 and math.isclose(d["plan_repeat_ms"]["mean"], (0.33 + 0.6) / 6)
    assert math.isclose(d["select_mean_us"]["mean"], 1.5)
    one = ablation.dispatch_summary(recs, (64, 64))
    assert one["cases"] == 1 and math.isclose(one["plan_first_ms"]["p95"], 0.30)
    assert ablation.dispatch_summary(recs, (32, 32))["plan_first_ms"] is None
