"""Host checks of bench.py: the multi-GPU refusal and the algorithmic bytes
per position it prices each kernel class with (the figures of the kernel
table in the design notes)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU only" in res.stderr and res.stdout == ""


@pytest.fixture(scope="module")
def bench():
    import bench as B
    return B


@pytest.mark.parametrize("name,op,expected", [
    ("c3", "restore", 4), ("c3", "update", 4), ("c3", "perturb", (6 + 29 * 4) / 30),
    ("c4", "restore", 12), ("c4", "perturb", 12 + 2 / 30), ("c4", "update", 12),
    ("c4u", "restore", 8), ("c4c", "restore", 4),
    ("c5", "perturb", 4), ("c5", "restore", 4), ("c5", "update", 10), ("c5", "stage_master", 6), ("c5", "backup", 4),
    ("c1", "restore", 8), ("c1", "perturb", (12 + 7 * 8) / 8),
    ("c3h", "perturb", 4), ("c3h", "backup_host", 2), ("c3h", "restore_host", 2),
])
def test_bytes_per_position(bench, name, op, expected):
    import synthetic as S
    assert bench.bytes_per_position(S.workload(name), op) == pytest.approx(expected)


def test_extras_default_to_the_other_benchmark_workloads(bench):
    assert bench.parse([]).extras == ["c1", "c2", "c4", "c5"]
    assert bench.parse(["--workload", "c4"]).extras == []
    assert bench.parse(["--no-extras"]).extras == []
    assert bench.parse(["--extras", "c1,c2"]).extras == ["c1", "c2"]


def test_counter_figures_are_keyed_to_the_kernel_sources(bench):
    sha = bench.sources_sha256()
    assert len(sha) == 64
    assert sha == bench.sources_sha256()          # a pure function of the sources
