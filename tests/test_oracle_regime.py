"""Pins for the regime-selection reference (Algorithms 1 and 2), CPU only.

Expected rankings below were worked out by hand from the rules of
Section 5.1 (valid on every case of the bucket, increasing geometric-mean
latency, exact ties by plan id, base plan appended) and Section 5.2 (hit ->
ranking, miss -> base plan only, first eligible, else no-eligible-plan).
"""
from oracle import regime

SCHEMA = [("seq", [4096, 65536]), ("density", [500, 1500])]   # density edges: 5%, 15%


def _case(cid, key, seq, nnz, blocks):
    return {"id": cid, "key": key, "features": {"seq": seq, "density": (nnz, blocks)}}


def test_bucket_edges_are_half_open_and_exact():
    assert regime.bucket_index(4095, [4096, 65536]) == 0
    assert regime.bucket_index(4096, [4096, 65536]) == 1
    assert regime.bucket_index(10 ** 6, [4096, 65536]) == 2
    # 5% exactly falls in the upper bucket, 4.99% below; 0/0 counts as zero
    assert regime.bucket_index((5, 100), [500]) == 1
    assert regime.bucket_index((499, 10000), [500]) == 0
    assert regime.bucket_index((0, 0), [500]) == 0


def test_table_compilation_rules():
    K = ("gfx950", 64, 64)
    cases = [_case("a", K, 8192, 10, 100), _case("b", K, 8192, 12, 100),    # bucket (1, 1)
             _case("c", K, 2048, 1, 100)]                                  # bucket (0, 0)
    lat = {
        ("a", 1): 2.0, ("b", 1): 8.0,        # geo 4.0
        ("a", 2): 4.0, ("b", 2): 4.0,        # geo 4.0 -> tie with plan 1, id 1 first
        ("a", 3): 1.0, ("b", 3): 9.0,        # geo 3.0 -> best
        ("a", 4): 0.5,                       # missing on case b -> excluded
        ("c", 4): 1.0, ("c", 2): 3.0,
    }
    base = lambda key: 7
    t = regime.compile_table(cases, lat, SCHEMA, base)
    assert t[K][(1, 1)] == [3, 1, 2, 7]
    assert t[K][(0, 0)] == [4, 2, 7]
    assert set(t[K]) == {(1, 1), (0, 0)}


def test_bucket_without_valid_plan_gets_no_ranking():
    K = ("k",)
    cases = [_case("a", K, 100, 1, 10), _case("b", K, 100, 1, 10)]
    lat = {("a", 1): 1.0, ("b", 2): 1.0}
    assert regime.compile_table(cases, lat, SCHEMA, lambda k: 0) == {}


def test_online_selection_rules():
    K = ("gfx950", 64, 64)
    table = {K: {(1, 1): [3, 1, 2, 7]}}
    base = lambda key: 7
    assert regime.select(table, K, (1, 1), base, lambda p: True) == 3
    assert regime.select(table, K, (1, 1), base, lambda p: p != 3) == 1
    assert regime.select(table, K, (1, 1), base, lambda p: p == 7) == 7
    # a miss (unknown bucket or key) considers the base plan only
    assert regime.select(table, K, (0, 2), base, lambda p: p in (3, 7)) == 7
    assert regime.select(table, ("other",), (1, 1), base, lambda p: p == 3) is None
    # nothing eligible -> no-eligible-plan
    assert regime.select(table, K, (1, 1), base, lambda p: False) is None
