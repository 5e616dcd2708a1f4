"""The clock factor of plans timed into existing profiling records (host only).

`finalize_added` puts the latencies of plans added to a split's records on
the clock the split was first profiled at: one factor per pass, the
geometric mean of the per-case reference ratios over the cases whose
reference kernels take at least FINALIZE_MIN_MS.  These records are
constructed by hand, with the expected latencies worked out here.
"""
import json
import math

from paper_2609_25869_amd.lut import profile as prof


def _write(path, recs):
    with open(path, "w") as f:
        for r in recs:
            f.write(json.dumps(r) + "\n")


def _read(path):
    return [json.loads(l) for l in open(path) if l.strip()]


def test_factor_is_the_geometric_mean_over_long_references(tmp_path):
    p = str(tmp_path / "recs.jsonl")
    recs = [
        # long references (>= 0.5 ms): ratios 0.9 and 1.0 -> factor sqrt(0.9)
        {"id": "a", "latency_ms": {"0": 2.0, "9": 0.0}, "invalid": [],
         "added": [{"plans": [9], "refs": [0], "scale": 0.9, "raw": {"9": 3.0}, "ref_ms": 2.0}]},
        {"id": "b", "latency_ms": {"0": 1.0, "9": 0.0}, "invalid": [],
         "added": [{"plans": [9], "refs": [0], "scale": 1.0, "raw": {"9": 5.0}, "ref_ms": 1.0}]},
        # a short reference: its ratio (1.5) must not enter the factor
        {"id": "c", "latency_ms": {"0": 0.01, "9": 0.0}, "invalid": [],
         "added": [{"plans": [9], "refs": [0], "scale": 1.5, "raw": {"9": 0.02}, "ref_ms": 0.01}]},
    ]
    _write(p, recs)
    prof.finalize_added(p)
    f = math.sqrt(0.9)
    out = {r["id"]: r for r in _read(p)}
    assert math.isclose(out["a"]["latency_ms"]["9"], 3.0 * f, rel_tol=1e-12)
    assert math.isclose(out["b"]["latency_ms"]["9"], 5.0 * f, rel_tol=1e-12)
    assert math.isclose(out["c"]["latency_ms"]["9"], 0.02 * f, rel_tol=1e-12)
    assert all(math.isclose(r["added"][0]["factor"], f, rel_tol=1e-12) for r in out.values())
    # recorded latencies of other plans are untouched
    assert out["a"]["latency_ms"]["0"] == 2.0 and out["c"]["latency_ms"]["0"] == 0.01
    # a second finalisation changes nothing
    before = _read(p)
    prof.finalize_added(p)
    assert _read(p) == before


def test_later_passes_win_and_legacy_entries_are_reconstructed(tmp_path):
    p = str(tmp_path / "recs.jsonl")
    # pass 0 (written before raw times were kept): stored 4.4 = raw 4.0 * scale 1.1;
    # pass 1 times plan 7 again (raw 3.0) with scale 0.8
    recs = [{"id": "a", "latency_ms": {"1": 1.0, "7": 4.4}, "invalid": [],
             "added": [{"plans": [7], "refs": [1], "scale": 1.1},
                       {"plans": [7], "refs": [1], "scale": 0.8, "raw": {"7": 3.0}, "ref_ms": 1.0}]}]
    _write(p, recs)
    prof.finalize_added(p)
    r = _read(p)[0]
    # each pass has one case with a long reference, so its factor is that case's ratio
    assert math.isclose(r["added"][0]["raw"]["7"], 4.0, rel_tol=1e-12)
    assert math.isclose(r["added"][0]["factor"], 1.1, rel_tol=1e-12)
    assert math.isclose(r["latency_ms"]["7"], 3.0 * 0.8, rel_tol=1e-12)
