"""The bounded cache of device work plans, host logic only: compiled with g++ from
the same header the library uses (csrc/plan_cache.h) and driven with fake plans, so
eviction, retirement and pinning are checked without a GPU."""
import os
import shutil
import subprocess

import pytest

from tests.conftest import ROOT

CSRC = os.path.join(ROOT, "paper_2502_06155_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_plan_cache_bounds_and_retirement(tmp_path):
    exe = tmp_path / "plan_cache_check"
    src = os.path.join(ROOT, "tests", "plan_cache_check.cpp")
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-I", CSRC, src, "-o", str(exe)],
                   check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    print(res.stdout)
    assert res.returncode == 0, res.stdout
    assert "plan cache ok" in res.stdout
    assert "many: size 256 retired 0 released 9744" in res.stdout


def test_cache_capacity_matches_the_header():
    with open(os.path.join(ROOT, "include", "tile_attn.h")) as f:
        assert "#define TA_PLAN_CACHE_ENTRIES 256" in f.read()
