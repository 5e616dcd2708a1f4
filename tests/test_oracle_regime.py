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


# ---- decision-tree leaves (Section 5.1): one half-open interval per feature.
# Every expected answer below is worked out by hand from lo <= v < hi, with
# ratios compared as num * 10000 >= edge * den.
NAMES = ["seq_q", "batch_heads", "density", "run_coverage"]


def _f(seq_q=8192, bh=24, dens=(15, 100), run=(49, 100)):
    return {"seq_q": seq_q, "batch_heads": bh, "density": dens, "run_coverage": run}


# seq_q in [8192, 65536), batch_heads unbounded, density >= 15%, run coverage < 50%
LEAF = [(8192, 65536), (None, None), (1500, None), (None, 5000)]


def test_region_integer_feature_edges():
    assert regime.region_contains(_f(seq_q=8192), LEAF, NAMES)           # exactly on lo: inside
    assert regime.region_contains(_f(seq_q=65535), LEAF, NAMES)
    assert not regime.region_contains(_f(seq_q=65536), LEAF, NAMES)      # exactly on hi: outside
    assert not regime.region_contains(_f(seq_q=8191), LEAF, NAMES)       # below lo


def test_region_unbounded_sides():
    assert regime.region_contains(_f(bh=1), LEAF, NAMES)
    assert regime.region_contains(_f(bh=10 ** 9), LEAF, NAMES)
    assert regime.region_contains(_f(dens=(1, 1)), LEAF, NAMES)          # density 100%, no hi
    assert regime.region_contains(_f(run=(0, 7)), LEAF, NAMES)           # run coverage 0, no lo
    everything = [(None, None)] * 4
    assert regime.region_contains(_f(seq_q=1, bh=1, dens=(0, 9), run=(9, 9)), everything, NAMES)


def test_region_ratio_feature_on_a_1e4_edge():
    # 15 / 100 is exactly the 1500 edge: 15 * 10000 == 1500 * 100
    assert regime.region_contains(_f(dens=(15, 100)), LEAF, NAMES)
    assert not regime.region_contains(_f(dens=(1499, 10000)), LEAF, NAMES)
    # run coverage 1/2 is exactly the 5000 edge, which is the (open) hi side
    assert not regime.region_contains(_f(run=(1, 2)), LEAF, NAMES)
    assert regime.region_contains(_f(run=(4999, 10000)), LEAF, NAMES)
    # 3/7 = 0.42857...: 30000 >= 4285 * 7 = 29995 but 30000 < 4286 * 7 = 30002
    inside = [(None, None), (None, None), (4285, 4286), (None, None)]
    assert regime.region_contains(_f(dens=(3, 7)), inside, NAMES)
    assert not regime.region_contains(_f(dens=(3, 7)), [(None, None), (None, None), (4286, None), (None, None)],
                                      NAMES)
    assert not regime.region_contains(_f(dens=(3, 7)), [(None, None), (None, None), (None, 4285), (None, None)],
                                      NAMES)


def test_region_zero_denominator_reads_as_zero():
    # an empty mask: density 0/0 and run coverage 0/0 are both 0
    assert not regime.region_contains(_f(dens=(0, 0)), LEAF, NAMES)      # 0 < 15%
    low = [(None, None), (None, None), (0, 1), (0, 1)]
    assert regime.region_contains(_f(dens=(0, 0), run=(0, 0)), low, NAMES)
    assert not regime.region_contains(_f(dens=(0, 0), run=(0, 0)), [(None, None), (None, None), (1, None),
                                                                       (None, None)], NAMES)


def test_region_needs_every_feature():
    assert not regime.region_contains(_f(seq_q=4096, run=(1, 100)), LEAF, NAMES)
    assert not regime.region_contains(_f(dens=(1, 100)), LEAF, NAMES)
    assert not regime.region_contains(_f(run=(99, 100)), LEAF, NAMES)


def test_region_lookup_hit_and_miss():
    # two leaves of one key with a gap between 8192 and 16384 tokens
    leaves = [([(None, 8192), (None, None), (None, None), (None, None)], [4, 12]),
              ([(16384, None), (None, None), (None, None), (None, None)], [12, 8])]
    assert regime.lookup_regions(leaves, _f(seq_q=100), NAMES, 0) == ([4, 12], True)
    assert regime.lookup_regions(leaves, _f(seq_q=16384), NAMES, 0) == ([12, 8], True)
    assert regime.lookup_regions(leaves, _f(seq_q=8192), NAMES, 0) == ([0], False)     # in no leaf
    assert regime.lookup_regions(leaves, _f(seq_q=16383), NAMES, 0) == ([0], False)
