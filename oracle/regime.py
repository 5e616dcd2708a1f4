"""Reference for profile-guided regime selection (Algorithms 1 and 2).

TEST INFRASTRUCTURE ONLY.  Plain Python restatement of the rules of
Section 5:

* A regime's ranking (Section 5.1): among the plans measured valid on every
  profiling case of the regime, increasing geometric-mean latency over those
  cases, equal means ordered by plan identifier; the request key's base plan
  closes the list.  A regime with no plan valid on all its cases gets no
  entry.
* Regimes (Section 5.1) are the nonempty cells of a key's feature partition:
  either predefined intervals (buckets) or the leaves of a decision tree
  (regions, one half-open interval per feature).
* Online selection (Algorithm 2, Section 5.2): the request's regime is looked
  up; a hit gives its ranking, a miss gives the base plan alone; the answer
  is the first plan of that list that is eligible for the request, or None
  (no eligible plan).

Bucket boundaries are half-open: a value v falls in bucket i when exactly i
edges are <= v.  Ratio features (density, run coverage) are compared exactly
as integers: num * 10000 >= edge * den, with edges in units of 1e-4, and a
ratio with a zero denominator counts as zero.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, Iterable, List, Optional, Sequence, Tuple

Key = Tuple
Bucket = Tuple[int, ...]


def at_least(value, edge: int) -> bool:
    """value >= edge; `value` is an int, or a (num, den) ratio compared with
    an edge in units of 1e-4 as integers (den == 0 reads as 0)."""
    if isinstance(value, tuple):
        num, den = value
        if den == 0:
            num, den = 0, 1
        return num * 10000 >= edge * den
    return value >= edge


def bucket_index(value, edges: Sequence[int]) -> int:
    """Number of edges <= value."""
    return sum(1 for e in edges if at_least(value, e))


def bucket_of(features: Dict[str, object], schema: Sequence[Tuple[str, Sequence[int]]]) -> Bucket:
    return tuple(bucket_index(features[name], edges) for name, edges in schema)


def regime_ranking(members: Sequence[Dict], latency: Dict[Tuple[str, int], float]) -> List[int]:
    """The ranking of one regime (Section 5.1), without the base plan.

    members: the regime's profiling cases; latency: (case id, plan id) ->
    median latency, present only for runs that passed validation."""
    valid_everywhere = set.intersection(*({p for (cid, p) in latency if cid == c["id"]} for c in members))

    def geo_mean(p):
        return math.exp(sum(math.log(latency[(c["id"], p)]) for c in members) / len(members))

    return sorted(valid_everywhere, key=lambda p: (geo_mean(p), p))


def compile_table(cases: Iterable[Dict], latency: Dict[Tuple[str, int], float],
                  schema: Sequence[Tuple[str, Sequence[int]]],
                  base_plan: Callable[[Key], int]) -> Dict[Key, Dict[Bucket, List[int]]]:
    """Plan table over predefined intervals: key -> bucket -> ranking.

    cases: dicts with 'id', 'key' (hashable) and 'features'."""
    regimes: Dict[Tuple[Key, Bucket], List[Dict]] = {}
    for c in cases:
        regimes.setdefault((c["key"], bucket_of(c["features"], schema)), []).append(c)
    table: Dict[Key, Dict[Bucket, List[int]]] = {}
    for (key, bucket), members in regimes.items():
        ranked = regime_ranking(members, latency)
        if ranked:
            table.setdefault(key, {})[bucket] = ranked + [base_plan(key)]
    return table


def first_eligible(candidates: Sequence[int], eligible: Callable[[int], bool]) -> Optional[int]:
    return next((p for p in candidates if eligible(p)), None)


def select(table: Dict[Key, Dict[Bucket, List[int]]], key: Key, bucket: Bucket,
           base_plan: Callable[[Key], int], eligible: Callable[[int], bool]) -> Optional[int]:
    """Algorithm 2 after the mask state is built, for a bucketed table."""
    return first_eligible(table.get(key, {}).get(bucket, [base_plan(key)]), eligible)


def region_contains(features: Dict[str, object], region: Sequence[Tuple[Optional[int], Optional[int]]],
                    names: Sequence[str]) -> bool:
    """Whether a request lies in a decision-tree leaf (Section 5.1): for every
    feature, lo <= value < hi, with None for an unbounded side."""
    return all((lo is None or at_least(features[name], lo)) and (hi is None or not at_least(features[name], hi))
               for name, (lo, hi) in zip(names, region))


def lookup_regions(regimes: Sequence[Tuple[Sequence[Tuple[Optional[int], Optional[int]]], Sequence[int]]],
                   features: Dict[str, object], names: Sequence[str], base: int) -> Tuple[List[int], bool]:
    """Algorithm 2's lookup for a key whose regimes are regions: the ranking
    of the (first) region containing the request and True, or the base plan
    alone and False on a miss."""
    for region, ranking in regimes:
        if region_contains(features, region, names):
            return list(ranking), True
    return [base], False
