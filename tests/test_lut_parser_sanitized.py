"""The plan-table reader (catalog.cpp, host C++) under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only): the shipped artifact, a version-2
artifact, and damaged copies of both (truncations, byte flips, nesting, huge
numbers) must be read or rejected without any sanitizer report."""
import json
import os
import random
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2609_25869_amd", "csrc")
SHIPPED = os.path.join(ROOT, "paper_2609_25869_amd", "lut", "gfx950_v1.json")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    out = str(tmp_path_factory.mktemp("asan") / "lut_parse_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", CSRC, "-I", os.path.join(ROOT, "include"),
           os.path.join(HERE, "sanitize", "lut_parse_driver.cpp"), os.path.join(CSRC, "catalog.cpp"), "-o", out]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    return out


def _damaged(text, rng, n):
    out = []
    for i in range(n):
        kind = i % 5
        if kind == 0:
            out.append(text[:rng.randrange(len(text))])
        elif kind == 1:
            b = bytearray(text.encode())
            for _ in range(8):
                b[rng.randrange(len(b))] = rng.randrange(256)
            out.append(b.decode("latin-1"))
        elif kind == 2:
            out.append("[" * 5000 + "]" * 5000)
        elif kind == 3:
            out.append(text.replace("128", "1" + "9" * 400, 3))
        else:
            out.append(text.replace('"', "", rng.randrange(1, 40)))
    return out


def test_reader_is_clean_under_sanitizers(driver, tmp_path):
    shipped = open(SHIPPED).read()
    # a version-2 artifact with one region per key, written like the compiler writes it
    doc = json.loads(shipped)
    v2 = {"format": doc["format"], "version": 2, "arch": doc["arch"], "catalog": doc["catalog"],
          "features": ["seq_q", "batch_heads", "density", "run_coverage"],
          "regimes": [{"key": [64, 64, 0, 128], "region": [[None, 65536], [None, None], [1500, None], [None, 5000]],
                       "ranking": [12, 4]},
                      {"key": [64, 64, 0, 128], "region": [[65536, None], [None, None], [None, None], [None, None]],
                       "ranking": [27, 12, 4]}],
          "provenance": {}}
    texts = [shipped, json.dumps(v2)] + _damaged(shipped, random.Random(0), 40) + \
        _damaged(json.dumps(v2), random.Random(1), 20) + ["", "{", "null", "{\"format\": 1e999}"]
    paths = []
    for i, t in enumerate(texts):
        p = tmp_path / ("in%03d.json" % i)
        p.write_bytes(t.encode("latin-1", errors="replace") if isinstance(t, str) else t)
        paths.append(str(p))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([driver] + paths, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env,
                       timeout=600)
    assert r.returncode == 0, r.stdout[-4000:]
    assert "Sanitizer" not in r.stdout and "runtime error" not in r.stdout, r.stdout[-4000:]
    lines = r.stdout.splitlines()
    assert "accepted" in lines[0] and "accepted" in lines[1], lines[:2]
    assert sum("rejected" in l for l in lines) >= 40
