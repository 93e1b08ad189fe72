"""bench.py's host-side contract, checked without a GPU."""

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_ragged_plan_is_seeded_and_in_range():
    sys.path.insert(0, ROOT)
    import bench
    w = bench.WORKLOADS["phi4-ragged"]
    lps, gens = bench.sequence_plan("phi4-ragged", w, 80)
    assert (lps, gens) == bench.sequence_plan("phi4-ragged", w, 80)
    assert len(lps) == len(gens) == w["B"] == 128
    assert all(64 <= x <= 2048 for x in lps)
    assert all(4096 <= x <= 32768 for x in gens)
    assert gens == sorted(gens, reverse=True)
    lps, starts = bench.sequence_plan("qwen3-14b", bench.WORKLOADS["qwen3-14b"], 320)
    assert lps == [1024] * 32 and starts == [32768 - 320] * 32


def test_traffic_is_reported_only_for_the_profiled_run(monkeypatch):
    """The stored counter traffic is the mean over the timed launches of one
    run (the default bench line); a run with other settings, or kernels
    changed since, reports none."""
    sys.path.insert(0, ROOT)
    import bench
    with open(os.path.join(ROOT, "profiles", "attention_traffic_qwen3-14b.json")) as f:
        stored = json.load(f)
    default = bench.run_signature(bench.build_parser().parse_args([]))
    assert stored["run"] == default
    monkeypatch.setattr(bench, "kernel_source_hash", lambda read=None: stored["kernel_source_hash"])
    assert bench.read_traffic(default) == stored["hbm_bytes_per_launch"]
    for key, other in [("steps", 2), ("warmup", 0), ("layout", "holefill"),
                       ("policy", "shared"), ("attn_split", 4096)]:
        assert bench.read_traffic(dict(default, **{key: other})) is None, key
    full = bench.build_parser().parse_args(["--full-run"])
    full.warmup, full.steps = 0, bench.WORKLOADS["qwen3-14b"]["T"]   # as main() sets them
    assert bench.read_traffic(bench.run_signature(full)) is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda read=None: "0" * 16)
    assert bench.read_traffic(default) is None


def test_tiny_cpu_baseline_replays_the_whole_run():
    """--tiny's CPU baseline is the oracle on the whole tiny run: 1024 steps
    from the prompt with all 11 eviction events."""
    sys.path.insert(0, ROOT)
    import bench
    r = bench.tiny_cpu_baseline(128, 256, 1024, 4, 2, 1000 * 1000003, 0)
    assert r["events"] == 11 and r["kind"] == "oracle" and r["unit"] == "us/step"
    assert r["value"] > 0 and r["cores"] >= 1
