"""Host logic of bench.py's command line: the benchmark measures one GPU and
refuses a multi-GPU request before it touches a device."""
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


@pytest.mark.parametrize("n", [0, 2, 8])
def test_bench_refuses_other_gpu_counts(n, capsys):
    assert bench.main(["--gpus", str(n)]) == 2
    assert "one GPU" in capsys.readouterr().err


def test_bench_refuses_multi_rank_launch(monkeypatch, capsys):
    monkeypatch.setenv("WORLD_SIZE", "4")
    assert bench.main([]) == 2
    assert "--gpus 1" in capsys.readouterr().err
