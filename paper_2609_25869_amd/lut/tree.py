"""Decision-tree regimes for the plan table (Section 5.1, Algorithm 1).

The second stage of the two-stage hierarchy partitions the profiling cases of
one request key by thresholds learned with a decision tree; the tree's
leaves are the performance regimes.  Each leaf is a box, one half-open
interval [lo, hi) per feature (None = unbounded), so the artifact stores a
key's regimes as disjoint regions and the runtime finds the one that
contains a request.

Learning (per request key):
* a node's plan is the first plan of the Algorithm 1 ranking over its cases
  (plans valid on every case, by geometric-mean latency, ties by id); its
  cost is the summed log regret of that plan, log(latency / best latency of
  the case);
* a node splits on the feature threshold that lowers the summed cost of its
  two children the most, when both children keep at least `min_leaf`
  cases (32, as in the paper) and some plan is valid on all of each child's
  cases; otherwise, or at the depth limit, it is a leaf;
* the depth limit is chosen by cross-validation over folds in which the
  cases of one source (mask family and density, the stand-in for the model
  a mask came from) stay together; ties go to the shallower tree.

Thresholds: integer features split at the midpoint of two neighbouring
values; ratio features (density = active / all blocks, run coverage =
active blocks in runs of length >= 2 / active blocks) at an edge in units of
1e-4 between the two ratios, compared exactly as integers,
num * 10000 >= edge * den, as at lookup.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

FEATURES = ["seq_q", "batch_heads", "density", "run_coverage", "query_rows", "row_imbalance"]
RATIOS = {"density": ("nnz", "blocks"), "run_coverage": ("run_blocks", "nnz"), "row_imbalance": ("imbalance_num", "nnz")}
MIN_LEAF = 32
DEPTHS = (0, 1, 2, 3, 4)

Region = List[Tuple[Optional[int], Optional[int]]]


def _ratio(feats: Dict, name: str) -> Tuple[int, int]:
    num, den = feats[RATIOS[name][0]], feats[RATIOS[name][1]]
    return (0, 1) if den <= 0 else (int(num), int(den))


def _ge(feats: Dict, name: str, edge: int) -> bool:
    """feature >= edge (ratio edges in units of 1e-4, compared as integers)."""
    if name in RATIOS:
        num, den = _ratio(feats, name)
        return num * 10000 >= edge * den
    return int(feats[name]) >= edge


def in_region(feats: Dict, region: Region) -> bool:
    for name, (lo, hi) in zip(FEATURES, region):
        if lo is not None and not _ge(feats, name, lo):
            return False
        if hi is not None and _ge(feats, name, hi):
            return False
    return True


def _lat(case: Dict) -> Dict[int, float]:
    return {int(p): t for p, t in case["latency_ms"].items()}


def ranking(cases: Sequence[Dict]) -> List[int]:
    """Algorithm 1 over a set of cases: plans valid on all of them, by
    increasing geometric-mean latency, exact ties by plan id."""
    common = None
    for c in cases:
        valid = set(_lat(c))
        common = valid if common is None else common & valid
    if not common:
        return []
    gm = {p: sum(math.log(_lat(c)[p]) for c in cases) / len(cases) for p in common}
    return sorted(common, key=lambda p: (gm[p], p))


def _value(feats: Dict, name: str) -> float:
    if name in RATIOS:
        num, den = _ratio(feats, name)
        return num / den
    return float(feats[name])


def _edge_between(a: Dict, b: Dict, name: str) -> Optional[int]:
    """A threshold e with value(a) < e <= value(b), compared as at lookup."""
    if name in RATIOS:
        (na, da), (nb, db) = _ratio(a, name), _ratio(b, name)
        mid = int(math.floor((na / da + nb / db) / 2 * 10000 + 0.5))
        for e in (mid, int(math.ceil(na * 10000 / da)), int(math.floor(nb * 10000 / db))):
            if na * 10000 < e * da and nb * 10000 >= e * db:
                return e
        return None
    va, vb = int(a[name]), int(b[name])
    return (va + vb + 1) // 2 if va < vb else None


def _plan_costs(cases: Sequence[Dict]):
    """Per-case log latency of every plan (0 where invalid), validity, log of the case's best latency."""
    plans = sorted({int(p) for c in cases for p in c["latency_ms"]})
    L = np.zeros((len(cases), len(plans)))
    V = np.zeros((len(cases), len(plans)), dtype=np.int64)
    best = np.zeros(len(cases))
    for i, c in enumerate(cases):
        lat = _lat(c)
        for j, p in enumerate(plans):
            if p in lat:
                L[i, j] = math.log(lat[p])
                V[i, j] = 1
        best[i] = math.log(min(lat.values()))
    return plans, L, V, best


def _side_cost(sumL, cntV, n, sum_best):
    """Regret of the Algorithm 1 winner of a side: plans valid on all n cases,
    the smallest summed log latency (first plan id on ties)."""
    ok = cntV == n
    if not ok.any():
        return math.inf
    return float(np.min(np.where(ok, sumL, np.inf)) - sum_best)


def _grow(cases: List[Dict], region: Region, depth: int, min_leaf: int, out: List[Tuple[Region, List[Dict]]]):
    best = None
    n = len(cases)
    if depth > 0 and n >= 2 * min_leaf:
        plans, L, V, lb = _plan_costs(cases)
        here = _side_cost(L.sum(0), V.sum(0), n, lb.sum())
        for fi, name in enumerate(FEATURES):
            vals = np.array([_value(c["features"], name) for c in cases])
            order = np.argsort(vals, kind="stable")
            cl, cv, cb = np.cumsum(L[order], 0), np.cumsum(V[order], 0), np.cumsum(lb[order])
            for i in range(min_leaf - 1, n - min_leaf):
                a, b = cases[order[i]], cases[order[i + 1]]
                if not vals[order[i]] < vals[order[i + 1]]:
                    continue
                cost = _side_cost(cl[i], cv[i], i + 1, cb[i]) + \
                    _side_cost(cl[-1] - cl[i], cv[-1] - cv[i], n - i - 1, cb[-1] - cb[i])
                if not (cost < here - 1e-9 and (best is None or cost < best[0] - 1e-12)):
                    continue
                e = _edge_between(a["features"], b["features"], name)
                if e is None:
                    continue
                hi_side = [c for c in cases if _ge(c["features"], name, e)]
                lo_side = [c for c in cases if not _ge(c["features"], name, e)]
                if len(hi_side) >= min_leaf and len(lo_side) >= min_leaf:
                    best = (cost, fi, e, lo_side, hi_side)
    if best is None:
        out.append((region, cases))
        return
    _, fi, e, lo_side, hi_side = best
    lo, hi = region[fi]
    r_lo, r_hi = list(region), list(region)
    r_lo[fi] = (lo, e)
    r_hi[fi] = (e, hi)
    _grow(lo_side, r_lo, depth - 1, min_leaf, out)
    _grow(hi_side, r_hi, depth - 1, min_leaf, out)


def grow(cases: Sequence[Dict], depth: int, min_leaf: int = MIN_LEAF) -> List[Tuple[Region, List[Dict]]]:
    """Leaves (region, cases) of the regret tree of one key's cases."""
    out: List[Tuple[Region, List[Dict]]] = []
    _grow(list(cases), [(None, None)] * len(FEATURES), depth, min_leaf, out)
    return out


def source_of(case: Dict) -> Tuple:
    """Generator family and density; each mixture request is its own source."""
    if case.get("family") == "mixture":
        return ("mixture", case.get("id"))
    return (case.get("family"), case.get("rho"))


def _select(leaves, case: Dict, base: int) -> int:
    for region, members in leaves:
        if in_region(case["features"], region):
            rk = ranking(members)
            lat = _lat(case)
            for p in rk + [base]:
                if p in lat:
                    return p
            return base
    return base


def _fold_of(cases: Sequence[Dict], folds: int) -> Dict:
    sources = sorted({source_of(c) for c in cases}, key=repr)
    return {s: i % folds for i, s in enumerate(sources)}


def _cv_regret(cases: Sequence[Dict], base: int, build: Callable, folds: int = 4) -> float:
    """Held-out mean log regret of the regimes `build(train_cases)` returns
    (a list of (region, member cases)); sources stay in one fold."""
    fold_of = _fold_of(cases, folds)
    total, n = 0.0, 0
    for f in range(folds):
        train = [c for c in cases if fold_of[source_of(c)] != f]
        test = [c for c in cases if fold_of[source_of(c)] == f]
        if not train or not test:
            continue
        leaves = build(train)
        for c in test:
            lat = _lat(c)
            p = _select(leaves, c, base)
            if lat and p in lat:
                total += math.log(lat[p] / min(lat.values()))
                n += 1
    return total / n if n else math.inf


def grid_regions(cases: Sequence[Dict], schema) -> List[Tuple[Region, List[Dict]]]:
    """Predefined intervals: the occupied cells of a bucket grid (Section 5.1),
    as regions.  `schema` lists (feature, edges); features not in it are
    unbounded."""
    cells: Dict[Tuple, List[Dict]] = {}
    edges_of = dict(schema)
    for c in cases:
        idx = []
        for name in FEATURES:
            edges = edges_of.get(name, [])
            idx.append(sum(1 for e in edges if _ge(c["features"], name, e)))
        cells.setdefault(tuple(idx), []).append(c)
    out = []
    for idx, members in sorted(cells.items()):
        region = []
        for name, i in zip(FEATURES, idx):
            edges = list(edges_of.get(name, []))
            region.append((edges[i - 1] if i > 0 else None, edges[i] if i < len(edges) else None))
        out.append((region, members))
    return out


def cv_depth(cases: Sequence[Dict], base: int, depths=DEPTHS, folds: int = 4, min_leaf: int = MIN_LEAF) -> int:
    """Depth with the lowest held-out mean log regret; ties go to the shallower tree."""
    best_d, best_r = depths[0], math.inf
    for d in depths:
        r = _cv_regret(cases, base, lambda tr: grow(tr, d, min_leaf), folds)
        if r < best_r - 1e-12:
            best_d, best_r = d, r
    return best_d


def compile_regions(records: Sequence[Dict], base_plan: Callable[[Tuple], int], min_leaf: int = MIN_LEAF,
                    depths=DEPTHS, grid_schema=None) -> Dict[Tuple, Dict]:
    """{key: {"depth": d or None, "kind": "tree" | "grid", "cv_regret": r,
    "regimes": [(region, ranking incl. base, n_cases)]}}.

    Per key, the learned tree (depth by cross-validation) is compared, by the
    same cross-validation, with the predefined intervals of `grid_schema`
    when one is given, and the lower held-out regret wins (ties: the tree).
    """
    by_key: Dict[Tuple, List[Dict]] = {}
    for r in records:
        if r["latency_ms"]:
            by_key.setdefault(tuple(r["key"]), []).append(r)
    out = {}
    for key, cases in sorted(by_key.items()):
        base = base_plan(key)
        d = cv_depth(cases, base, depths, min_leaf=min_leaf)
        r_tree = _cv_regret(cases, base, lambda tr: grow(tr, d, min_leaf))
        kind, leaves = "tree", grow(cases, d, min_leaf)
        r_best = r_tree
        if grid_schema is not None:
            r_grid = _cv_regret(cases, base, lambda tr: grid_regions(tr, grid_schema))
            if r_grid < r_tree - 1e-12:
                kind, leaves, r_best = "grid", grid_regions(cases, grid_schema), r_grid
        regimes = []
        for region, members in leaves:
            rk = ranking(members)
            if rk:
                regimes.append((region, rk + [base], len(members)))
        out[key] = {"depth": d if kind == "tree" else None, "kind": kind, "cv_regret": math.exp(r_best),
                    "regimes": regimes}
    return out


def select(table: Dict[Tuple, Dict], key, feats: Dict, base: int) -> Tuple[List[int], bool]:
    """Ranking of the region that contains the request (hit), else [base]."""
    ent = table.get(tuple(key))
    if ent:
        for region, rk, _ in ent["regimes"]:
            if in_region(feats, region):
                return rk, True
    return [base], False
