"""The forward launch schedule, host logic only: a C++ check compiled against the built
library replays the schedule of several shapes and confirms every kept tile of every
query block is computed exactly once, by a whole-block workgroup or by one of the
parts a ragged last round is cut into, that every query block with rows runs (also one
that keeps no tile), and that MM-DiT plans run each XCD's share longest first."""
import os
import re
import shutil
import subprocess

import pytest

from tests.conftest import ROOT

PKG = os.path.join(ROOT, "paper_2502_06155_amd")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_schedule_covers_every_tile_once(tmp_path):
    lib = os.path.join(PKG, "libtileattn.so")
    if not os.path.exists(lib):
        pytest.skip("library not built")
    exe = tmp_path / "schedule_check"
    cmd = ["g++", "-std=c++17", "-O1", "-I", os.path.join(PKG, "csrc"), "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "schedule_check.cpp"), "-o", str(exe), "-L", PKG, "-ltileattn",
           f"-Wl,-rpath,{PKG}"]
    rocm_lib = "/opt/rocm/lib"
    if os.path.isdir(rocm_lib):
        cmd += ["-L", rocm_lib, "-lamdhip64", f"-Wl,-rpath,{rocm_lib}"]
    subprocess.run(cmd, check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    print(res.stdout)
    assert res.returncode == 0, res.stdout + res.stderr
    got = {m.group(1): tuple(int(m.group(i)) for i in range(2, 8))
           for m in re.finditer(r"^(\S+) units (\d+) whole (\d+) parts (\d+) slots (\d+) table (\d) short (\d+)$",
                                res.stdout, re.M)}
    assert len(got) == 17
    assert "short-last orders 32" in res.stdout
    # a launch whose XCDs run whole rounds only keeps every block whole
    assert got["93f-col"] == (8640, 8640, 0, 0, 0, 0)
    # the GPU parity shapes are cut into parts, so those tests cover the merge
    for name in ("gpu-a", "gpu-b", "gpu-c", "gpu-d", "gpu-e", "gpu-f", "gpu-h"):
        assert got[name][3] > 0, name
    # among them, short last query blocks (16 rows, d = 128)
    assert got["gpu-h"][5] > 0
    # where every segment ends on a short block at d = 64 or 96 (video only), the kernel
    # runs those blocks last in each share and the schedule cuts no parts
    for name in ("gpu-g", "29f-col", "sp-col", "93f-col"):
        assert got[name][2] == 0 and got[name][4] == 0, name
    # plans with split frames keep their pieces whole
    for name in ("sp-sym", "cog-sym"):
        assert got[name][2] == 0, name
    # an MM-DiT plan without split frames runs longest first from a table that leaves
    # out the text query blocks past the text's end (5 of 6 per head at 226 text
    # tokens); with split frames (one global frame) it keeps the natural order for the
    # kernel's persistent loop
    assert got["cog-sym2"][4] == 1 and got["cog-sym2"][1] == got["cog-sym2"][0] - 48 * 5
    assert got["cog-sym"][4] == 0
