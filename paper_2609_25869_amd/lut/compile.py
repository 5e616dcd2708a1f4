"""Plan-table compilation (Section 5.1, Algorithm 1, regimes-and-rankings part).

Input: the JSON lines written by ``profile.py`` (one per profiling case: the
request key, the regime features and the validated median latency of every
plan).  Output: the ``bsa-plan-table`` artifact that ``bsa_lut_load`` reads.

Rules:
* cases are grouped by request key (B_Q, B_KV, dtype, head dim);
* within a key, each case falls in the bucket given by the feature schema:
  for every feature, the number of bucket edges <= its value; density
  (active / all logical blocks) and run coverage (active blocks in runs of
  length >= 2 / active blocks) are compared exactly as integers,
  num * 10000 >= edge * den;
* in every bucket the plans with a valid latency on *every* case of the
  bucket are ranked by increasing geometric-mean latency over the bucket,
  exact ties by plan id, and the key's base plan is appended.

    python -m paper_2609_25869_amd.lut.compile --profile P.jsonl [--eval E.jsonl] --out gfx950_v1.json
"""
from __future__ import annotations

import argparse
import json
import math
import os
from typing import Dict, List, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))

# Feature schema of the gfx950 table: predefined bucket edges.  query_rows
# is batch x heads x ceil(seq_q / B_Q), the number of logical query-block
# rows of the request (u_A of Eq. 3 folded into one count: how many
# query-tile tasks there are to spread over 256 CUs, which decides whether
# Split-K and small tiles pay); ratios in units of 1e-4.  Chosen among
# candidate grids by source-grouped 4-fold cross-validation on the training
# records (gfx950_report.md lists the candidates with their held-out
# regret).
SCHEMA: List[Tuple[str, List[int]]] = [
    ("query_rows", [1024, 4096, 32768]),
    ("density", [700, 2000]),
    ("run_coverage", [9000]),
]
# A candidate that adds row_imbalance = max_row_nnz * query_rows / nnz, the
# longest row against the mean row (near 1 for top-k and window masks, well
# above 1 when heads differ in density).
IMBALANCE_SCHEMA: List[Tuple[str, List[int]]] = [
    ("query_rows", [1024, 4096]),
    ("density", [700, 2000]),
    ("run_coverage", [9000]),
    ("row_imbalance", [30000]),
]
# The grid of the previous table, kept for the report's comparison.
SEQ_HEADS_SCHEMA: List[Tuple[str, List[int]]] = [
    ("seq_q", [6144, 24576, 98304]),
    ("batch_heads", [3, 12]),
    ("density", [700, 2000]),
    ("run_coverage", [5000]),
]

# Profiling records the shipped table is built from, and held-out records.
PROFILES = [os.path.join(HERE, "gfx950_profile.jsonl"), os.path.join(HERE, "gfx950_wide.jsonl"),
            os.path.join(HERE, "gfx950_mixture.jsonl"), os.path.join(HERE, "gfx950_large.jsonl")]
EVALS = [os.path.join(HERE, "gfx950_eval.jsonl"), os.path.join(HERE, "gfx950_wide_eval.jsonl"),
         os.path.join(HERE, "gfx950_mixture_eval.jsonl"), os.path.join(HERE, "gfx950_large_eval.jsonl"),
         os.path.join(HERE, "gfx950_grid2.jsonl")]


def with_query_rows(rec: Dict) -> Dict:
    """Add the derived features: query_rows = batch_heads * ceil(seq_q / B_Q)
    and, when max_row_nnz is recorded, the numerator of row_imbalance =
    max_row_nnz * query_rows / nnz."""
    f = rec.get("features")
    if f and "query_rows" not in f and "key" in rec:
        f["query_rows"] = int(f["batch_heads"]) * (-(-int(f["seq_q"]) // int(rec["key"][0])))
    if f and "max_row_nnz" in f and "imbalance_num" not in f:
        f["imbalance_num"] = int(f["max_row_nnz"]) * int(f["query_rows"])
    return rec


def load_records(path) -> List[Dict]:
    """Records of one JSON-lines file, or of several (a list of paths)."""
    if not isinstance(path, str):
        return [r for p in path for r in load_records(p)]
    with open(path) as f:
        return [with_query_rows(json.loads(line)) for line in f if line.strip()]


def feature_value(feats: Dict, name: str):
    if name == "density":
        return feats["nnz"], feats["blocks"]
    if name == "run_coverage":
        return feats["run_blocks"], feats["nnz"]
    if name == "row_imbalance":
        return feats["imbalance_num"], feats["nnz"]
    return feats[name]


def bucket(feats: Dict, schema: Sequence[Tuple[str, Sequence[int]]]) -> Tuple[int, ...]:
    out = []
    for name, edges in schema:
        v = feature_value(feats, name)
        if isinstance(v, tuple):
            num, den = v
            if den <= 0:
                num, den = 0, 1
            out.append(sum(1 for e in edges if num * 10000 >= e * den))
        else:
            out.append(sum(1 for e in edges if v >= e))
    return tuple(out)


def source_of(rec: Dict) -> Tuple:
    """Mask source of a profiling case: generator family and density (the
    stand-in for the model a mask came from).  A mixture request composes
    its heads from several families and densities, so each one is a source
    of its own (the stand-in for one model's mix of heads)."""
    if rec.get("family") == "mixture":
        return ("mixture", rec.get("id"))
    return (rec.get("family"), rec.get("rho"))


def cv_regret(records: Sequence[Dict], schema, base_plan, folds: int = 4) -> float:
    """Geometric-mean selector regret of a grid schema under source-grouped
    cross-validation on the training records: each fold's table is built
    without the fold's sources and scored on them."""
    sources = sorted({source_of(r) for r in records}, key=repr)
    fold_of = {s: i % folds for i, s in enumerate(sources)}
    total, n = 0.0, 0
    for f in range(folds):
        train = [r for r in records if fold_of[source_of(r)] != f]
        test = [r for r in records if fold_of[source_of(r)] == f]
        if not train or not test:
            continue
        a = regret_report(compile_table(train, schema, base_plan), schema, base_plan, test)["all"]
        total += math.log(a["gm"]) * a["cases"]
        n += a["cases"]
    return math.exp(total / n) if n else float("nan")


# Candidate grids the shipped schema was chosen from (lowest cross-validated
# regret on the training records).
CANDIDATE_SCHEMAS: List[List[Tuple[str, List[int]]]] = [
    SCHEMA,
    IMBALANCE_SCHEMA,
    [("query_rows", [1024, 4096]), ("density", [700, 2000]), ("run_coverage", [9000]), ("row_imbalance", [25000])],
    [("query_rows", [512, 2048, 8192]), ("density", [700, 2000]), ("run_coverage", [9000]),
     ("row_imbalance", [30000])],
    [("query_rows", [1024, 4096]), ("density", [700, 2000]), ("run_coverage", [5000, 9000])],
    [("query_rows", [1024, 4096]), ("density", [700, 2000]), ("run_coverage", [9000])],
    [("query_rows", [1024, 4096]), ("density", [700, 2000]), ("run_coverage", [5000])],
    [("query_rows", [1024, 4096, 16384]), ("density", [700, 2000]), ("run_coverage", [9000])],
    [("query_rows", [1024, 4096]), ("density", [700, 2000]), ("run_coverage", [8000])],
    [("query_rows", [1024, 4096]), ("density", [700, 2000]), ("run_coverage", [9000]), ("row_imbalance", [20000])],
    [("query_rows", [512, 2048, 8192]), ("density", [700, 2000]), ("run_coverage", [8000])],
    [("query_rows", [512, 2048, 8192]), ("density", [700, 2000]), ("run_coverage", [5000])],
    [("query_rows", [256, 1024, 4096, 16384]), ("density", [700, 2000]), ("run_coverage", [5000])],
    [("query_rows", [1024, 4096]), ("density", [500, 1500, 3000]), ("run_coverage", [8000])],
    [("query_rows", [1024, 4096]), ("seq_q", [24576]), ("density", [700, 2000]), ("run_coverage", [5000])],
    SEQ_HEADS_SCHEMA,
    [("seq_q", [32768, 98304]), ("batch_heads", [12]), ("density", [700, 2000]), ("run_coverage", [5000])],
]


def compile_table(records: Sequence[Dict], schema, base_plan) -> Dict[Tuple[int, ...], Dict[Tuple[int, ...], List[int]]]:
    """{key: {bucket: ranking}} from profiling records."""
    groups: Dict[Tuple[int, ...], Dict[Tuple[int, ...], List[Dict]]] = {}
    for r in records:
        key = tuple(r["key"])
        groups.setdefault(key, {}).setdefault(bucket(r["features"], schema), []).append(r)
    table = {}
    for key, buckets in groups.items():
        base = base_plan(key)
        for b, cases in buckets.items():
            common = None
            for c in cases:
                valid = {int(p) for p in c["latency_ms"]}
                common = valid if common is None else common & valid
            if not common:
                continue

            def geo_mean(p):
                return math.exp(sum(math.log(c["latency_ms"][str(p)]) for c in cases) / len(cases))

            ranking = sorted(common, key=lambda p: (geo_mean(p), p))
            table.setdefault(key, {})[b] = ranking + [base]
    return table


def artifact(table, schema, catalog, provenance: Dict) -> Dict:
    regimes = []
    for key in sorted(table):
        for b in sorted(table[key]):
            regimes.append({"key": list(key), "bucket": list(b), "ranking": table[key][b]})
    return {
        "format": "bsa-plan-table",
        "version": 1,
        "arch": "gfx950",
        "catalog": [[e["id"], e["tq"], e["tkv"], e["split"], e["stages"], e["waves"], e["xcd_group"]]
                    for e in catalog],
        "schema": [[n, list(e)] for n, e in schema],
        "regimes": regimes,
        "provenance": provenance,
    }


def select(table, schema, base_plan, key, feats) -> int:
    """First plan of the ranking (every catalog plan is eligible for the corpus requests)."""
    ranking = table.get(tuple(key), {}).get(bucket(feats, schema))
    return ranking[0] if ranking else base_plan(tuple(key))


def regret_report(table, schema, base_plan, records) -> Dict:
    """Selected / fastest measured latency per case (1 is optimal)."""
    regrets, misses, per_key = [], 0, {}
    for r in records:
        lat = {int(p): t for p, t in r["latency_ms"].items()}
        if not lat:
            continue
        sel = select(table, schema, base_plan, r["key"], r["features"])
        if tuple(r["key"]) not in table or bucket(r["features"], schema) not in table[tuple(r["key"])]:
            misses += 1
        best = min(lat.values())
        g = lat.get(sel, float("nan")) / best
        regrets.append(g)
        per_key.setdefault("%d:%d" % tuple(r["key"][:2]), []).append(g)
    regrets = [g for g in regrets if g == g]

    def summary(xs):
        xs = sorted(xs)
        if not xs:
            return {}
        pct = lambda q: xs[min(len(xs) - 1, int(math.ceil(q * len(xs))) - 1)]
        return {"cases": len(xs), "gm": math.exp(sum(math.log(x) for x in xs) / len(xs)), "p95": pct(0.95),
                "p99": pct(0.99), "max": xs[-1], "within_3pct": sum(1 for x in xs if x <= 1.03) / len(xs)}

    return {"all": summary(regrets), "lookup_misses": misses,
            "per_key": {k: summary(v) for k, v in sorted(per_key.items())}}


def artifact_v2(regions, catalog, provenance: Dict) -> Dict:
    """Version-2 artifact: per key, the decision-tree leaves as disjoint regions."""
    from . import tree
    regimes = []
    for key in sorted(regions):
        for region, ranking, n in regions[key]["regimes"]:
            regimes.append({"key": list(key), "region": [[lo, hi] for lo, hi in region], "ranking": ranking,
                            "cases": n})
    return {
        "format": "bsa-plan-table",
        "version": 2,
        "arch": "gfx950",
        "catalog": [[e["id"], e["tq"], e["tkv"], e["split"], e["stages"], e["waves"], e["xcd_group"]]
                    for e in catalog],
        "features": list(tree.FEATURES),
        "regimes": regimes,
        "partition": {"%d:%d" % key[:2]: {"kind": regions[key]["kind"], "depth": regions[key]["depth"],
                                          "cv_regret": regions[key]["cv_regret"]} for key in sorted(regions)},
        "provenance": provenance,
    }


def regret_report_v2(regions, base_plan, records) -> Dict:
    """Selected / fastest measured latency per case for a region table."""
    from . import tree
    regrets, misses, per_key = [], 0, {}
    for r in records:
        lat = {int(p): t for p, t in r["latency_ms"].items()}
        if not lat:
            continue
        base = base_plan(tuple(r["key"]))
        rk, hit = tree.select(regions, r["key"], r["features"], base)
        misses += not hit
        sel = next((p for p in rk if p in lat), None)
        g = lat[sel] / min(lat.values()) if sel is not None else float("nan")
        regrets.append(g)
        per_key.setdefault("%d:%d" % tuple(r["key"][:2]), []).append(g)
    return _regret_summary(regrets, misses, per_key)


def _regret_summary(regrets, misses, per_key):
    regrets = [g for g in regrets if g == g]

    def summary(xs):
        xs = sorted(g for g in xs if g == g)
        if not xs:
            return {}
        pct = lambda q: xs[min(len(xs) - 1, int(math.ceil(q * len(xs))) - 1)]
        return {"cases": len(xs), "gm": math.exp(sum(math.log(x) for x in xs) / len(xs)), "p95": pct(0.95),
                "p99": pct(0.99), "max": xs[-1], "within_3pct": sum(1 for x in xs if x <= 1.03) / len(xs)}

    return {"all": summary(regrets), "lookup_misses": misses,
            "per_key": {k: summary(v) for k, v in sorted(per_key.items())}}


def kernel_ablations(pick, base_plan, catalog, records) -> Dict:
    """Kernel-time ablations from profiling records (organization: Section 7.3, Table 5; selection: Section 7.4).

    A0 / A1 / A2: the key's base plan, the fastest measured eligible plan
    (what an exhaustive search finds), and the table's pick (`pick(record)`
    -> ranking).  The paper's A0 is Direct (physical tile = logical block);
    the catalog has that tile only for some keys, so the A0 ratios are also
    given separately over the keys whose base plan is Direct and over the
    others (whose base plan is the nearest tile).  O0 / O1 / O2 hold the
    physical tile at the base plan's tile and vary only the task
    organization (Split-K factor, traversal order and ring depth): the base organization,
    the table's first-ranked plan with that tile, and the fastest measured
    one.  Paired-case geometric means; wins / ties / losses against O0 use a
    3% tie band.
    """
    tile = {e["id"]: (e["tq"], e["tkv"]) for e in catalog}
    gm = lambda xs: math.exp(sum(math.log(x) for x in xs) / len(xs)) if xs else float("nan")
    a0a2, a0a1, a2a1, o_sp, o_reg, o1_reg, wtl = [], [], [], [], [], [], [0, 0, 0]
    by_base = {True: ([], []), False: ([], [])}   # direct base? -> (A0/A1, A0/A2)
    keys_by_base = {True: set(), False: set()}
    for r in records:
        lat = {int(p): t for p, t in r["latency_ms"].items()}
        base = base_plan(tuple(r["key"]))
        if not lat or base not in lat:
            continue
        rk = pick(r)
        sel = next((p for p in rk if p in lat), base)
        best = min(lat.values())
        a0a1.append(lat[base] / best)
        a0a2.append(lat[base] / lat[sel])
        a2a1.append(lat[sel] / best)
        direct = tile[base] == tuple(r["key"][:2])
        by_base[direct][0].append(lat[base] / best)
        by_base[direct][1].append(lat[base] / lat[sel])
        keys_by_base[direct].add("%d:%d" % tuple(r["key"][:2]))
        same = {p: t for p, t in lat.items() if tile[p] == tile[base]}
        o1 = next((p for p in rk if p in same), base)
        o2 = min(same.values())
        o_sp.append(lat[base] / lat[o1])
        o_reg.append(lat[base] / o2)
        o1_reg.append(lat[o1] / o2)
        ratio = lat[base] / lat[o1]
        wtl[0 if ratio > 1.03 else 2 if ratio < 1 / 1.03 else 1] += 1
    return {"cases": len(a0a1),
            "kernel_speedup_over_A0": {"A1_exhaustive": gm(a0a1), "A2_table": gm(a0a2)},
            "by_base_kind": {("direct" if d else "nearest_tile"): {
                "keys": sorted(keys_by_base[d]), "cases": len(by_base[d][0]),
                "A1_exhaustive": gm(by_base[d][0]), "A2_table": gm(by_base[d][1])} for d in (True, False)},
            "A2_regret_vs_A1": gm(a2a1),
            "organization_at_base_tile": {"O1_speedup_over_O0": gm(o_sp), "O2_speedup_over_O0": gm(o_reg),
                                          "O1_regret_vs_O2": gm(o1_reg), "O0_regret_vs_O2": gm(o_reg),
                                          "O1_vs_O0_wins_ties_losses": wtl}}


def mapping_name(bq: int, bkv: int, tq: int, tkv: int) -> str:
    """Section 4.2 mapping of logical blocks onto a physical tile."""
    if tq == bq and tkv == bkv:
        return "Direct"
    if tq >= bq and tkv >= bkv:
        return "Coarsened"
    if tq <= bq and tkv <= bkv:
        return "Refined"
    return "mixed"


def mapping_census(catalog, records) -> Dict[str, Dict[str, float]]:
    """Per key, the share of cases whose fastest measured plan uses each mapping."""
    tile = {e["id"]: (e["tq"], e["tkv"]) for e in catalog}
    out: Dict[str, Dict[str, int]] = {}
    for r in records:
        lat = {int(p): t for p, t in r["latency_ms"].items()}
        if not lat:
            continue
        bq, bkv = r["key"][:2]
        best = min(lat, key=lat.get)
        kind = mapping_name(bq, bkv, *tile[best])
        c = out.setdefault("%d:%d" % (bq, bkv), {})
        c[kind] = c.get(kind, 0) + 1
    return {k: {m: n / sum(v.values()) for m, n in sorted(v.items())} for k, v in sorted(out.items())}


def write_report(path: str, table, base, catalog, prof_recs, eval_recs, candidates=None) -> None:
    """Markdown summary of the shipped table: regret, census, ablations."""
    pick = lambda r: table.get(tuple(r["key"]), {}).get(bucket(r["features"], SCHEMA), [base(tuple(r["key"]))])
    lines = ["# gfx950 plan table: selection quality on MI355X", "",
             "Generated by `python -m paper_2609_25869_amd.lut.compile --report` from the committed profiling "
             "records: the table is built from %s; %s hold held-out cases of the same generators with "
             "other seeds.  Latencies are kernel times: the median of 3 timed batches after 1 warm-up launch, "
             % (", ".join("`%s`" % os.path.basename(x) for x in PROFILES),
                ", ".join("`%s`" % os.path.basename(x) for x in EVALS)) +
             "where a launch shorter than 1 ms is timed in batches of back-to-back launches of about 1 ms "
             "(HIP events around each batch).",
             "", "## Selector regret (selected / fastest measured latency per case)", "",
             "| cases | GM | P95 | P99 | max | within 3% |", "|---|---:|---:|---:|---:|---:|"]
    for name, recs in (("profile (in-sample)", prof_recs), ("eval (held-out)", eval_recs)):
        a = regret_report(table, SCHEMA, base, recs)["all"]
        lines.append("| %s: %d | %.4f | %.4f | %.4f | %.4f | %.1f%% |" % (
            name, a["cases"], a["gm"], a["p95"], a["p99"], a["max"], 100 * a["within_3pct"]))
    hold = list(eval_recs)
    lines += ["", "Held-out regret by the kernel time of the fastest plan (short kernels carry most of the regret: "
              "there a plan's launch geometry matters most and the regimes are coarsest):", "",
              "| fastest kernel | cases | GM | P95 | within 3% |", "|---|---:|---:|---:|---:|"]
    for lo, hi in ((0, 0.05), (0.05, 0.2), (0.2, 1.0), (1.0, float("inf"))):
        sub = [r for r in hold if r["latency_ms"] and lo <= min(r["latency_ms"].values()) < hi]
        if sub:
            a = regret_report(table, SCHEMA, base, sub)["all"]
            lines.append("| %s ms | %d | %.4f | %.4f | %.1f%% |" % (
                "%g-%g" % (lo, hi) if hi != float("inf") else ">= %g" % lo, a["cases"], a["gm"], a["p95"],
                100 * a["within_3pct"]))
    if candidates:
        lines += ["", "## Regime partitions (Section 5.1: predefined intervals or decision-tree thresholds)", "",
                  "The shipped grid is the candidate with the lowest source-grouped 4-fold cross-validated regret "
                  "on the training records (CV GM); the held-out columns are reported, not used for the choice.",
                  "", "| partition (built from the profiling records) | CV GM | held-out GM | P95 | P99 | within 3% |",
                  "|---|---:|---:|---:|---:|---:|"]
        for name, cv, a in candidates:
            lines.append("| %s | %s | %.4f | %.4f | %.4f | %.1f%% |" % (
                name, "%.4f" % cv if cv is not None else "-", a["gm"], a["p95"], a["p99"], 100 * a["within_3pct"]))
    lines += ["", "Held-out regret per request key (B_Q:B_KV):", "",
              "| key | cases | GM | P95 | max |", "|---|---:|---:|---:|---:|"]
    for k, a in regret_report(table, SCHEMA, base, eval_recs)["per_key"].items():
        lines.append("| %s | %d | %.4f | %.4f | %.4f |" % (k, a["cases"], a["gm"], a["p95"], a["max"]))
    lines += ["", "## Mapping census: share of held-out cases whose fastest plan uses each mapping (Section 4.2)", "",
              "| key | Direct | Coarsened | Refined | mixed |", "|---|---:|---:|---:|---:|"]
    for k, c in mapping_census(catalog, eval_recs).items():
        lines.append("| %s | %s |" % (k, " | ".join("%.0f%%" % (100 * c.get(m, 0))
                                                   for m in ("Direct", "Coarsened", "Refined", "mixed"))))
    ab = kernel_ablations(pick, base, catalog, eval_recs)
    o = ab["organization_at_base_tile"]
    bk = ab["by_base_kind"]
    lines += ["", "## Kernel-time ablations on the held-out cases (paired-case geometric means)", "",
              "A0 is the key's base plan. It is Direct (T = B) for the keys %s; for %s the catalog has no T = B "
              "kernel and the base plan is the nearest tile, so those keys are listed separately." % (
                  ", ".join(bk["direct"]["keys"]), ", ".join(bk["nearest_tile"]["keys"])), "",
              "| variant | all keys: speedup over A0 | Direct-base keys (%d cases) | nearest-tile keys (%d cases) |"
              % (bk["direct"]["cases"], bk["nearest_tile"]["cases"]), "|---|---:|---:|---:|",
              "| A1: fastest measured eligible plan (exhaustive search) | %.3f | %.3f | %.3f |" % (
                  ab["kernel_speedup_over_A0"]["A1_exhaustive"], bk["direct"]["A1_exhaustive"],
                  bk["nearest_tile"]["A1_exhaustive"]),
              "| A2: plan-table selection | %.3f | %.3f | %.3f |" % (
                  ab["kernel_speedup_over_A0"]["A2_table"], bk["direct"]["A2_table"], bk["nearest_tile"]["A2_table"]),
              "", "A2 / A1 kernel time: %.4f." % ab["A2_regret_vs_A1"], "",
              "Task organization at the base tile (Split-K factor, traversal order and ring depth vary, the tile "
              "does not):",
              "",
              "| variant | speedup over O0 | regret vs O2 |", "|---|---:|---:|",
              "| O0: base organization (no split) | 1.000 | %.4f |" % o["O0_regret_vs_O2"],
              "| O1: table's first plan with that tile | %.3f | %.4f |" % (o["O1_speedup_over_O0"], o["O1_regret_vs_O2"]),
              "| O2: fastest measured organization | %.3f | 1.0000 |" % o["O2_speedup_over_O0"],
              "", "O1 against O0 with a 3%% tie band: %d wins, %d ties, %d losses." % tuple(o["O1_vs_O0_wins_ties_losses"]),
              ""]
    abl = os.path.join(HERE, "gfx950_ablation.jsonl")
    if os.path.exists(abl):
        from . import ablation
        recs = load_records(abl)
        sm = ablation.summarize(recs)
        lines += ["## Complete requests: A0 Direct, A1 exhaustive online search, A2 plan table", "",
                  "`gfx950_ablation.jsonl`, written by `python -m paper_2609_25869_amd.lut.ablation --split eval "
                  "--every 4` (every fourth held-out case of the grid split, %d cases; "
                  "pass 1 is the cold unique request, passes 2-4 warm exact repeats, amortized = mean of the four). "
                  "Paired-case geometric means of latency ratios:" % sm["cases"], "",
                  "| population | T_A0 / T_A1 | T_A1 / T_A2 | T_A0 / T_A2 |", "|---|---:|---:|---:|"]
        for pop in ("cold", "warm", "amortized"):
            lines.append("| %s | %.3f | %.2f | %.3f |" % (pop, sm[pop]["A0/A1"], sm[pop]["A1/A2"], sm[pop]["A0/A2"]))
        lines += ["", "Kernel time of the plan each variant executes: A0 / A1 %.3f, A0 / A2 %.3f, A2 / A1 %.4f; "
                  "A2 picks A1's plan in %.0f%% of the cases." % (sm["kernel"]["A0/A1"], sm["kernel"]["A0/A2"],
                                                                  sm["kernel"]["A2/A1"], 100 * sm["same_plan_as_A1"]),
                  ""]
        rows = [("all keys", ablation.dispatch_summary(recs)),
                ("64:64", ablation.dispatch_summary(recs, (64, 64)))]
        if rows[0][1]["cases"]:
            lines += ["## Dispatch overhead per request (the measurement of Table 6)", "",
                      "`bsa_plan` is the whole request-path preprocessing: the mask state on the device, the one "
                      "statistics copy and synchronisation, lookup and eligibility on the host, and the metadata "
                      "launches of the selected plan (wall time, stream synchronised). The lookup and "
                      "eligibility step alone is `bsa_select_plan` on the same statistics, called through the "
                      "Python binding.", "",
                      "| cases | n | `bsa_plan` first request mean / P95 (us) | `bsa_plan` repeats mean / P95 (us) "
                      "| lookup + eligibility mean / P95 (us) |", "|---|---:|---:|---:|---:|"]
            for name, d in rows:
                if not d["cases"]:
                    continue
                pf, pr, se = d["plan_first_ms"], d["plan_repeat_ms"], d["select_mean_us"]
                lines.append("| %s | %d | %.1f / %.1f | %.1f / %.1f | %.2f / %.2f |" % (
                    name, d["cases"], 1e3 * pf["mean"], 1e3 * pf["p95"], 1e3 * pr["mean"], 1e3 * pr["p95"],
                    se["mean"], se["p95"]))
            lines.append("")
    with open(path, "w") as f:
        f.write("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--profile", nargs="+", default=PROFILES)
    ap.add_argument("--eval", nargs="+", default=EVALS)
    ap.add_argument("--out", default=None)
    ap.add_argument("--report", action="store_true", help="also write gfx950_report.md beside the table")
    ap.add_argument("--tree", action="store_true",
                    help="learn the regimes with per-key decision trees (version-2 artifact)")
    args = ap.parse_args()
    import paper_2609_25869_amd as bsa

    base = lambda key: bsa.base_plan(key[0], key[1])
    recs = load_records(args.profile)
    if args.tree:
        from . import tree
        regions = tree.compile_regions(recs, base, grid_schema=SCHEMA)
        prov = {"profiled_on": "MI355X (gfx950)", "profile_cases": len(recs),
                "regimes": "per key, the lower source-grouped 4-fold cross-validated regret of a regret decision "
                           "tree (>= %d cases per leaf, depth from %s) and of the predefined intervals %s"
                           % (tree.MIN_LEAF, list(tree.DEPTHS), SCHEMA),
                "latency": "median of 3 timed batches after 1 warm-up launch; launches under 1 ms timed as back-to-back batches of about 1 ms (HIP events)"}
        if all(os.path.exists(e) for e in args.eval):
            ev = load_records(args.eval)
            prov["eval_cases"] = len(ev)
            prov["eval_regret"] = regret_report_v2(regions, base, ev)["all"]
        prov["profile_regret"] = regret_report_v2(regions, base, recs)["all"]
        doc = artifact_v2(regions, bsa.catalog(), prov)
        with open(args.out or os.path.join(HERE, "gfx950_v2.json"), "w") as f:
            json.dump(doc, f, indent=1)
            f.write("\n")
        print(json.dumps(prov, indent=1))
        print(json.dumps(doc["partition"], indent=1))
        if all(os.path.exists(e) for e in args.eval):
            print(json.dumps(regret_report_v2(regions, base, load_records(args.eval)), indent=1))
        return
    args.out = args.out or os.path.join(HERE, "gfx950_v1.json")
    table = compile_table(recs, SCHEMA, base)
    prov = {"profiled_on": "MI355X (gfx950)", "profile_cases": len(recs),
            "corpus": "seeded synthetic masks (frame windows, Bernoulli + diagonal, pooled q.k top-k, per-head "
                      "mixtures) on the nine paper geometries + (128,32)/(32,128): the grid split (N in {16K, 64K, "
                      "115K}, 4 or 24 batch x heads, 6 sources), the wide split (N from 2K to 115K, 1 to 24 batch "
                      "x heads, 12 sources, 96 random draws per key), the mixture split (N from 16K to 131K, 8 to "
                      "48 batch x heads, 12 draws per key), the large split (N from 64K to 131K, 8 to 48 batch "
                      "x heads, 12 sources and mixtures, 12 draws per key)",
            "latency": "median of 3 timed batches after 1 warm-up launch; launches under 1 ms timed as back-to-back batches of about 1 ms (HIP events)"}
    if all(os.path.exists(e) for e in args.eval):
        ev = load_records(args.eval)
        prov["eval_cases"] = len(ev)
        prov["eval_regret"] = regret_report(table, SCHEMA, base, ev)["all"]
    prov["profile_regret"] = regret_report(table, SCHEMA, base, recs)["all"]
    doc = artifact(table, SCHEMA, bsa.catalog(), prov)
    with open(args.out, "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    print(json.dumps(prov, indent=1))
    if all(os.path.exists(e) for e in args.eval):
        print(json.dumps(regret_report(table, SCHEMA, base, load_records(args.eval)), indent=1))
        if args.report:
            from . import tree
            ev = load_records(args.eval)
            cands = []
            for sch in CANDIDATE_SCHEMAS:
                cands.append(("predefined intervals %s%s" % (sch, " (shipped)" if sch is SCHEMA else ""),
                              cv_regret(recs, sch, base),
                              regret_report(compile_table(recs, sch, base), sch, base, ev)["all"]))
            cands += [("decision trees per key (>= %d cases per leaf, depth by grouped CV)" % tree.MIN_LEAF, None,
                       regret_report_v2(tree.compile_regions(recs, base), base, ev)["all"]),
                      ("per key, tree or shipped intervals by grouped CV", None,
                       regret_report_v2(tree.compile_regions(recs, base, grid_schema=SCHEMA), base, ev)["all"])]
            write_report(os.path.join(HERE, "gfx950_report.md"), table, base, bsa.catalog(), recs, ev, cands)


if __name__ == "__main__":
    main()
