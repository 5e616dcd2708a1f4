"""The ctypes structures of the Python binding have the size and field offsets
that a C compiler gives the structures of include/bsa.h."""
import ctypes
import os
import shutil
import subprocess

import pytest

from paper_2609_25869_amd import _ffi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PAIRS = [("bsa_shapes", _ffi.Shapes), ("bsa_mask", _ffi.Mask), ("bsa_plan_opts", _ffi.PlanOpts),
         ("bsa_segment_info", _ffi.SegmentInfo), ("bsa_catalog_entry", _ffi.CatalogEntry),
         ("bsa_regime_query", _ffi.RegimeQuery)]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_ctypes_layout_matches_the_header(tmp_path):
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "bsa.h"', "int main(void) {"]
    for cname, cls in PAIRS:
        lines.append('  printf("%s size %%zu\\n", sizeof(%s));' % (cname, cname))
        for f, _ in cls._fields_:
            lines.append('  printf("%s %s %%zu\\n", offsetof(%s, %s));' % (cname, f, cname, f))
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, stdout=subprocess.PIPE, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for cname, cls in PAIRS:
        assert got[(cname, "size")] == ctypes.sizeof(cls), cname
        for f, _ in cls._fields_:
            assert got[(cname, f)] == getattr(cls, f).offset, (cname, f)
