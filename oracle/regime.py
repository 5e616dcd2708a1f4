"""Reference for profile-guided regime selection (Algorithms 1 and 2).

TEST INFRASTRUCTURE ONLY.  Plain Python restatement of the rules of
Section 5:

Table compilation (Algorithm 1): cases are grouped by request key; each group
is partitioned into buckets by the feature schema; in every nonempty bucket
the plans with a valid latency on *every* case of the bucket are sorted by
increasing geometric-mean latency over the bucket, exact ties broken by plan
identifier, and the key's base plan is appended.

Online selection (Algorithm 2): the regime signature (key, bucketed request
dimensions, mask statistics) is looked up; a hit yields its ranking, a miss
yields the base plan alone; the first eligible plan in rank order is
returned, or None (no eligible plan).

Bucket boundaries are half-open: a value v falls in bucket i when exactly i
edges are <= v.  Ratio features (density, run coverage) are compared exactly
as integers: num * 10000 >= edge * den, with edges in units of 1e-4.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, Iterable, List, Optional, Sequence, Tuple

Key = Tuple
Bucket = Tuple[int, ...]


def bucket_index(value, edges: Sequence[int]) -> int:
    """Number of edges <= value; `value` is an int or a (num, den) ratio."""
    if isinstance(value, tuple):
        num, den = value
        if den == 0:
            num, den = 0, 1
        return sum(1 for e in edges if num * 10000 >= e * den)
    return sum(1 for e in edges if value >= e)


def bucket_of(features: Dict[str, object], schema: Sequence[Tuple[str, Sequence[int]]]) -> Bucket:
    return tuple(bucket_index(features[name], edges) for name, edges in schema)


def compile_table(cases: Iterable[Dict], latency: Dict[Tuple[str, int], float],
                  schema: Sequence[Tuple[str, Sequence[int]]],
                  base_plan: Callable[[Key], int]) -> Dict[Key, Dict[Bucket, List[int]]]:
    """Algorithm 1, regimes-and-rankings half.

    cases: dicts with 'id', 'key' (hashable) and 'features'.
    latency: (case id, plan id) -> median latency, present only for runs that
    passed numerical validation.
    """
    by_key: Dict[Key, List[Dict]] = {}
    for c in cases:
        by_key.setdefault(c["key"], []).append(c)
    table: Dict[Key, Dict[Bucket, List[int]]] = {}
    for key, group in by_key.items():
        p_base = base_plan(key)
        buckets: Dict[Bucket, List[Dict]] = {}
        for c in group:
            buckets.setdefault(bucket_of(c["features"], schema), []).append(c)
        for b, members in buckets.items():
            plans = None
            for c in members:
                valid = {p for (cid, p) in latency if cid == c["id"]}
                plans = valid if plans is None else plans & valid
            if not plans:
                continue
            def geo(p):
                return math.exp(sum(math.log(latency[(c["id"], p)]) for c in members) / len(members))
            ranked = sorted(plans, key=lambda p: (geo(p), p))
            table.setdefault(key, {})[b] = ranked + [p_base]
    return table


def select(table: Dict[Key, Dict[Bucket, List[int]]], key: Key, bucket: Bucket,
           base_plan: Callable[[Key], int], eligible: Callable[[int], bool]) -> Optional[int]:
    """Algorithm 2 after the mask state is built: lookup, ranked fallback."""
    ranking = table.get(key, {}).get(bucket)
    candidates = list(ranking) if ranking is not None else [base_plan(key)]
    for p in candidates:
        if eligible(p):
            return p
    return None


def region_contains(features: Dict[str, object], region: Sequence[Tuple[Optional[int], Optional[int]]],
                    names: Sequence[str]) -> bool:
    """Regimes given as leaves of a decision tree (Section 5.1): one
    half-open interval [lo, hi) per feature, None for an unbounded side.
    Ratio features compare exactly as integers, num * 10000 >= edge * den."""
    for name, (lo, hi) in zip(names, region):
        v = features[name]
        if isinstance(v, tuple):
            num, den = v
            if den == 0:
                num, den = 0, 1
            at_least = lambda e: num * 10000 >= e * den
        else:
            at_least = lambda e: v >= e
        if lo is not None and not at_least(lo):
            return False
        if hi is not None and at_least(hi):
            return False
    return True
