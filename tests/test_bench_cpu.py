"""The benchmark's command-line contract and its committed counter data, checked without a GPU."""
import json
import os
import subprocess
import sys

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def run_bench(*args):
    return subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True, timeout=300, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    res = run_bench("--gpus", "2", "--steps", "1", "--warmup", "0")
    assert res.returncode == 2
    assert "one GPU" in res.stderr


def test_help_lists_the_contract_flags():
    res = run_bench("--help")
    assert res.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--no-cpu", "--no-prefill", "--pipeline"):
        assert flag in res.stdout


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-GPU path")
def test_without_a_gpu_the_bench_stops_before_measuring():
    res = run_bench("--steps", "1", "--warmup", "0")
    assert res.returncode == 2
    assert "needs a GPU" in res.stderr


def test_committed_traffic_counters_are_well_formed():
    """Every counted kernel names the sources it was counted on (files in the tree), a digest,
    per-launch FETCH/WRITE medians and the calibration the bench applies."""
    path = os.path.join(ROOT, "profiles", "traffic_counters.json")
    data = json.load(open(path))
    cal = data["calibration"]
    assert 1.9 < cal["fetch_factor"] < 2.1 and 0.9 < cal["write_factor"] < 1.1
    assert "sparse_attn_kernel<4, 8>" in data["kernels"]  # the kernel the headline roofline reports
    for name, e in data["kernels"].items():
        assert e["launches"] >= 1, name
        assert len(e["sources_sha256"]) == 64, name
        for src in e["sources"]:
            assert os.path.exists(os.path.join(ROOT, src)), (name, src)
        want = e["fetch_kib_per_launch"] * 1024 * cal["fetch_factor"] + e["write_kib_per_launch"] * 1024 * cal[
            "write_factor"]
        assert abs(e["traffic_bytes"] - want) <= 1e-6 * want, name
        assert abs(e["ratio"] - e["traffic_bytes"] / e["algorithmic_bytes"]) < 1e-9, name
