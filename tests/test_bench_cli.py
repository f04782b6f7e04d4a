"""bench.py without a GPU: the single-GPU contract (more than one GPU exits with a message),
the per-configuration FLOP counts it reads, the traffic record that is used only while the
kernel source matches the one the counters were taken on, and the CPU baseline's record."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


@pytest.mark.parametrize("argv, env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_exits_with_a_message(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       env=dict(os.environ, **env), timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_flops_per_config_come_from_the_counting_oracle():
    with open(bench.FLOPS_FILE) as f:
        stored = json.load(f)["workloads"]
    for name, w in stored.items():
        # The algorithmic unit is the shared-level count (the oracle's nested loops); the
        # from-scratch count is reported beside it.
        fsh, fpc = bench.flops_per_config(name)
        assert fpc == w["flops_per_config"] and fsh == w["flops_per_config_shared_levels"]
        assert 0 < fsh < fpc
    assert bench.flops_per_config("no such workload") == (None, None)


def test_traffic_is_reported_only_for_the_kernel_it_was_measured_on(monkeypatch):
    with open(bench.TRAFFIC_FILE) as f:
        rec = json.load(f)["gpt2.7b-d16"]
    monkeypatch.setattr(bench, "kernel_hash", lambda: rec["kernel_sha"])
    assert bench.traffic_record("gpt2.7b-d16", 0) == rec["bytes_per_launch"]
    monkeypatch.setattr(bench, "kernel_hash", lambda: "0" * 16)
    assert bench.traffic_record("gpt2.7b-d16", 0) is None
    assert bench.traffic_record("no such workload", 0) is None


def test_cpu_baseline_record():
    from paper_2503_19050_amd import workloads as W
    rec = bench.cpu_baseline(W.workload("gpt1.3b-d8"), 0.5, 2)
    assert rec["kind"] == "oracle" and rec["cores"] == 1 and rec["unit"] == "configs/s"
    assert rec["value"] > 0 and "gpt1.3b-d8" in rec["sample"]
    assert rec["nproc"] >= 1 and isinstance(rec["cpu_model"], str)
    sh = rec["sharded"]
    assert sh["processes"] == 2 and sh["value"] > 0 and sh["unit"] == "configs/s"


def test_counter_record_only_for_the_kernel_it_was_measured_on(monkeypatch, tmp_path):
    rec = {"w": {"kernel_sha": "abc", "executed_fp64_per_config": 50.0, "valu_per_config": 90.0}}
    p = tmp_path / "t.json"
    p.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(p))
    monkeypatch.setattr(bench, "kernel_hash", lambda: "abc")
    assert bench.counter_record("w") == 50.0
    assert bench.counter_record("w", "valu_per_config") == 90.0
    monkeypatch.setattr(bench, "kernel_hash", lambda: "abd")
    assert bench.counter_record("w") is None
    assert bench.counter_record("w", "valu_per_config") is None


def test_committed_counter_records_match_the_kernel_source():
    """profiles/traffic.json holds the headline workload's record, taken on the committed kernel
    source: the bench line's traffic and counter figures are then not null."""
    with open(bench.TRAFFIC_FILE) as f:
        rec = json.load(f)["llama42b-d128-hw64"]
    assert rec["kernel_sha"] == bench.kernel_hash()
    assert bench.traffic_record("llama42b-d128-hw64", 0) == rec["bytes_per_launch"]
    assert rec["fetch_bytes"] + rec["write_bytes"] == rec["bytes_per_launch"]
    # The kernel shares more work than the oracle's loop nest, so it executes fewer FP64
    # operations than the algorithmic unit, but at least a configuration's own: the host streams
    # of its first microbatch, at least two interference rounds on them, its memory, bucket index,
    # delta and objective (above 30 with fma counted as 2).
    flops, _ = bench.flops_per_config("llama42b-d128-hw64")
    assert 30.0 < rec["executed_fp64_per_config"] < flops
    assert rec["executed_fp64_per_config"] < rec["valu_per_config"] < 200.0
