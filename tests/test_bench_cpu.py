"""bench.py's host-side contract, on the CPU: one GPU only, no GPU means an
error rather than a number, and the counter traffic is used only for the
kernel sources it was taken on."""

import os
import re

import pytest

import bench


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err


def test_traffic_only_for_the_sources_it_was_taken_on():
    path = os.path.join(bench.ROOT, "profiles", "traffic.txt")
    lines = [l for l in open(path) if l.startswith("kernel=")]
    assert lines, "no counter lines committed"
    f = dict(kv.split("=", 1) for kv in lines[0].split())
    assert re.fullmatch(r"[0-9a-f]{16}", f["sha"])
    got = bench.read_traffic(f["kernel"], f["workload"], f["sha"])
    assert got == float(f["bytes_per_launch"])
    assert bench.read_traffic(f["kernel"], f["workload"], "0" * 16) is None
    assert bench.read_traffic("no_such_kernel", f["workload"], f["sha"]) is None


def test_sources_hash_covers_every_kernel_file():
    sha = bench.kernel_sources_sha()
    assert re.fullmatch(r"[0-9a-f]{16}", sha)
    assert bench.kernel_sources_sha() == sha


def test_no_gpu_is_an_error_not_a_number(capsys):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present: the bench itself runs there")
    assert bench.main(["--cpu-seconds", "0"]) == 1
    captured = capsys.readouterr()
    assert "needs a GPU" in captured.err
    assert captured.out == ""
