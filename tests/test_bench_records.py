"""The committed rocprofv3 summaries keep the per-launch figures bench.py reads from
them (HBM bytes, matrix FLOP seen by the MFMA op counter, the hash of the kernel
sources they were taken on), in a form its parser accepts."""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILES = sorted(f for f in os.listdir(os.path.join(ROOT, "profiles"))
                  if f.startswith("tile_attn_") and f.endswith(".md"))


@pytest.mark.parametrize("name", PROFILES)
def test_profile_records(name):
    text = open(os.path.join(ROOT, "profiles", name)).read()
    rec = {}
    for line in text.splitlines():
        m = re.fullmatch(r"([a-z0-9_]+): (\S+)", line)
        if m:
            rec[m.group(1)] = m.group(2)
    assert re.fullmatch(r"[0-9a-f]{64}", rec["kernel_sha256"])
    read = float(rec["hbm_read_bytes_per_launch"])
    write = float(rec["hbm_write_bytes_per_launch"])
    assert read > 0 and write > 0
    assert float(rec["hbm_bytes_per_launch"]) == pytest.approx(read + write, abs=2)
    assert float(rec["mfma_bf16_flop_per_launch"]) > 0
    # the command lines of the summary run committed files only
    for cmd in re.findall(r"^(?:timeout .*|rocprofv3 .*)$", text, flags=re.M):
        assert "_work" not in cmd and "python3 bench.py" in cmd


def test_bench_parser_reads_the_fwd_record():
    import bench

    # the record is returned when the hash matches the sources, None otherwise
    got = bench.profile_record("fwd", "mfma_bf16_flop_per_launch")
    assert got is None or got > 5.0e12
    got = bench.profile_record("fwd", "mfma_bf16_flop_per_launch", "29f", "col", 1)
    assert got is None or got > 1.7e12


def test_every_summary_is_named_for_its_pass_workload_and_mask():
    import bench
    import workloads

    assert len(PROFILES) >= 5
    for name in PROFILES:
        m = re.fullmatch(r"tile_attn_(fwd|bwd)_(\w+)_(col|sym|dense)_g(\d+)\.md", name)
        assert m, name
        assert m.group(2) in workloads.WORKLOADS, name
        assert bench.profile_md(m.group(1), m.group(2), m.group(3), int(m.group(4))).endswith(name)
