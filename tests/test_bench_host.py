"""Host-side logic of bench.py (no GPU): more than one GPU is refused before anything touches a device, and a
recorded counter value (HBM bytes per launch) applies only while the text of the kernel's sources is unchanged."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.fixture
def tree(tmp_path, monkeypatch):
    """A copy of the kernel sources bench.py hashes, under a temporary root."""
    names = sorted({f for fs in bench.KERNEL_SOURCES.values() for f in fs})
    csrc = tmp_path / "paper_2609_12378_amd" / "csrc"
    csrc.mkdir(parents=True)
    for f in names:
        shutil.copy(os.path.join(ROOT, "paper_2609_12378_amd", "csrc", f), csrc / f)
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return tmp_path


def write_rows(tree, rows):
    lines = ["| class | kernel | sources sha | fetch B | write B | total B per launch | algorithmic B | launches |",
             "|---|---|---|---|---|---|---|---|"]
    lines += ["| %s | k | %s | 1 | 2 | %s | - | 1 |" % r for r in rows]
    (tree / "profiles" / "pmc_traffic.md").write_text("\n".join(lines) + "\n")


def test_traffic_applies_only_to_unchanged_sources(tree):
    sha = bench.sources_sha("ntt_row_mac")
    assert sha is not None and len(sha) == 16
    write_rows(tree, [("ntt_row_mac", sha, "2.5e+10"), ("ntt_fwd_col", "0" * 16, "3e+10")])
    assert bench.load_traffic("ntt_row_mac") == 2.5e10
    # a row recorded for other source text does not apply
    assert bench.load_traffic("ntt_fwd_col") is None
    # one byte changed in a source the kernel is built from retires the recorded value
    path = tree / "paper_2609_12378_amd" / "csrc" / bench.KERNEL_SOURCES["ntt_row_mac"][0]
    path.write_bytes(path.read_bytes() + b"\n")
    assert bench.sources_sha("ntt_row_mac") != sha
    assert bench.load_traffic("ntt_row_mac") is None


def test_traffic_absent_or_unknown(tree):
    assert bench.load_traffic("ntt_row_mac") is None  # no counter file
    assert bench.sources_sha("not_a_kernel") is None
    write_rows(tree, [("ntt_row_mac", bench.sources_sha("ntt_row_mac"), "not a number")])
    assert bench.load_traffic("ntt_row_mac") is None
