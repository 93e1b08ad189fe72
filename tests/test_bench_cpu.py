"""bench.py's host-side contract, checked without a GPU."""

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
