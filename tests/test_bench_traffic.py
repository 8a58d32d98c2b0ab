"""Host-side checks of the benchmark's traffic bookkeeping: the measured HBM
bytes are reported only for the kernel sources they were taken on."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


@pytest.fixture(scope="module")
def bench():
    import bench as b
    return b


def _summary(path, nbytes, sha):
    with open(path, "w") as fh:
        fh.write(f"# traffic\n\n- bytes_per_launch: {nbytes}\n- kernel_sources_sha256: `{sha}`\n")


def test_traffic_read_when_sources_match(bench, tmp_path):
    p = tmp_path / "t.md"
    _summary(p, 123456, bench.bwd_sources_sha256())
    assert bench.read_traffic(str(p)) == 123456


def test_traffic_null_when_sources_differ(bench, tmp_path):
    p = tmp_path / "t.md"
    _summary(p, 123456, "0" * 64)
    assert bench.read_traffic(str(p)) is None


def test_traffic_null_without_summary(bench, tmp_path):
    assert bench.read_traffic(str(tmp_path / "missing.md")) is None


def test_committed_summary_parses(bench):
    # the committed summary names a byte count; it is reported only while
    # its hash matches the sources
    fields = {}
    for line in open(bench.TRAFFIC_SUMMARY):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    assert int(fields["bytes_per_launch"]) > 0
    assert len(fields["kernel_sources_sha256"]) == 64
