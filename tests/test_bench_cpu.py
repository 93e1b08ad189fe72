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
    run (the bench line the driver runs: --gpus 1 --steps 20 --warmup 5); a
    run with other settings, or kernels changed since, reports none."""
    sys.path.insert(0, ROOT)
    import bench
    with open(os.path.join(ROOT, "profiles", "attention_traffic_qwen3-14b.json")) as f:
        stored = json.load(f)
    default = bench.run_signature(bench.build_parser().parse_args(
        ["--gpus", "1", "--steps", "20", "--warmup", "5"]))
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


def test_traffic_summary_parses_counter_csvs(tmp_path, monkeypatch):
    """The summary takes the last steps x layers attention dispatches of a
    FETCH_SIZE and a WRITE_SIZE run (the timed ones), scales them by the 1 GiB
    copy's counts, and records the run's signature."""
    sys.path.insert(0, ROOT)
    import bench
    cols = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id",
            "Thread_Id", "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size",
            "LDS_Block_Size", "Scratch_Size", "VGPR_Count", "SGPR_Count",
            "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]

    def write(d, counter, rows):
        d.mkdir()
        with open(d / "run_counter_collection.csv", "w") as f:
            f.write(",".join(cols) + "\n")
            for i, (name, v) in enumerate(rows):
                vals = {c: "0" for c in cols}
                vals.update(Dispatch_Id=str(i + 1), Kernel_Name='"%s"' % name,
                            Counter_Name=counter, Counter_Value=str(v))
                f.write(",".join(vals[c] for c in cols) + "\n")

    steps, L = 2, bench.WORKLOADS["qwen3-14b"]["L"]
    attn = "void ra::attn_bf16_kernel<12, 1, false>(ra::AttnLaunch, ra::Paging, int)"
    full = "void ra::evict_kernel<1024, 9, unsigned short, false, 0>(ra::SeqMeta const*)"
    warm = [(attn, 999.0)] * L                       # warm-up launches: not sampled
    write(tmp_path / "f", "FETCH_SIZE", warm + [(attn, 100.0)] * (steps * L) + [(full, 50.0)])
    write(tmp_path / "w", "WRITE_SIZE", warm + [(attn, 2.0)] * (steps * L) + [(full, 40.0)])
    write(tmp_path / "cf", "FETCH_SIZE", [("copy_kernel", 524288.0)] * 3)
    write(tmp_path / "cw", "WRITE_SIZE", [("copy_kernel", 1048576.0)] * 3)
    written = {}
    monkeypatch.setattr(bench.json, "dump", lambda obj, f, **kw: written.update(obj))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda read=None: "0" * 16)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    args = bench.build_parser().parse_args(
        ["--steps", str(steps), "--warmup", "1", "--traffic-summary",
         str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"), str(tmp_path / "cw")])
    bench.traffic_summary(args)
    assert written["launches_sampled"] == steps * L
    assert written["copy_calibration"]["fetch_scale"] == 2.0
    assert written["fetch_bytes_per_launch"] == 100.0 * 1024 * 2.0
    assert written["write_bytes_per_launch"] == 2.0 * 1024
    assert written["evict_full_event"] == {"fetch_bytes": 50.0 * 2048, "write_bytes": 40.0 * 1024}
    assert written["evict_deferred_event"] is None
    assert written["run"]["steps"] == steps and written["run"]["warmup"] == 1


def test_traffic_summary_deferred_event(tmp_path, monkeypatch):
    """An event whose moves ride on the next step's attention: the summary
    samples the plain launches of the timed steps (not the move launches),
    takes the last positions-only eviction (the fast forward's come first)
    as the selection, and reports the move launches' bytes above as many
    plain launches."""
    sys.path.insert(0, ROOT)
    import bench
    cols = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]

    def write(d, counter, rows):
        d.mkdir()
        with open(d / "run_counter_collection.csv", "w") as f:
            f.write(",".join(cols) + "\n")
            for i, (name, v) in enumerate(rows):
                f.write('%d,"%s",%s,%s\n' % (i + 1, name, counter, v))

    steps, L = 2, bench.WORKLOADS["qwen3-14b"]["L"]
    attn = "void ra::attn_bf16_kernel<12, 1, false>(ra::AttnLaunch, ra::Paging, int)"
    mv = "void ra::(anonymous namespace)::attn_bf16_move_kernel<8>(ra::AttnLaunch, int)"
    sel = "void ra::evict_kernel<1024, 9, unsigned short, true, 0>(ra::SeqMeta const*)"
    ff = [(sel, 7.0)] * 3                             # fast forward: not the event
    write(tmp_path / "f", "FETCH_SIZE", ff + [(attn, 999.0)] * L + [(attn, 100.0)] * L +
          [(sel, 5.0)] + [(mv, 150.0)] * L)
    write(tmp_path / "w", "WRITE_SIZE", ff + [(attn, 9.0)] * L + [(attn, 2.0)] * L +
          [(sel, 4.0)] + [(mv, 80.0)] * L)
    write(tmp_path / "cf", "FETCH_SIZE", [("copy_kernel", 524288.0)] * 3)
    write(tmp_path / "cw", "WRITE_SIZE", [("copy_kernel", 1048576.0)] * 3)
    written = {}
    monkeypatch.setattr(bench.json, "dump", lambda obj, f, **kw: written.update(obj))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda read=None: "0" * 16)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    args = bench.build_parser().parse_args(
        ["--steps", str(steps), "--warmup", "1", "--traffic-summary",
         str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"), str(tmp_path / "cw")])
    bench.traffic_summary(args)
    assert written["launches_sampled"] == L
    assert written["fetch_bytes_per_launch"] == 100.0 * 2048
    assert written["evict_full_event"] is None
    d = written["evict_deferred_event"]
    assert d["select_fetch_bytes"] == 5.0 * 2048 and d["select_write_bytes"] == 4.0 * 1024
    assert d["move_attention_launches"] == L
    assert d["moves_fetch_bytes"] == L * 50.0 * 2048
    assert d["moves_write_bytes"] == L * 78.0 * 1024


def test_timeline_summary_reads_kernel_trace(tmp_path, capsys):
    """The timeline takes the last steps x layers attention dispatches of a
    kernel trace and measures each one, the merge that follows it (if any)
    and the gap to the next layer's attention within a step."""
    sys.path.insert(0, ROOT)
    import bench
    L = bench.WORKLOADS["qwen3-4b"]["L"]
    attn = "void ra::(anonymous namespace)::attn_bf16_kernel<8, 1, false>(ra::AttnLaunch)"
    comb = "void ra::(anonymous namespace)::combine_kernel<unsigned short>(ra::AttnLaunch)"
    adv = "ra::(anonymous namespace)::advance_kernel(ra::SeqMeta*, int)"
    rows, t = [], 1000
    for step in range(3):                       # one warm-up step, two timed
        for l in range(L):
            rows.append((attn, t, t + 90000))          # 90 us
            rows.append((comb, t + 90010, t + 94810))  # 10 ns gap, 4.8 us
            t += 94820                                  # 10 ns to the next layer
        rows.append((adv, t, t + 3000))
        t += 5000
    d = tmp_path / "trace"
    d.mkdir()
    with open(d / "run_kernel_trace.csv", "w") as f:
        f.write("Kernel_Name,Start_Timestamp,End_Timestamp\n")
        for n, s, e in rows:
            f.write('"%s",%d,%d\n' % (n, s, e))
    args = bench.build_parser().parse_args(
        ["--workload", "qwen3-4b", "--steps", "2", "--timeline-summary", str(d)])
    bench.timeline_summary(args)
    out = json.loads(capsys.readouterr().out)
    assert out["launches"] == 2 * L
    assert out["attention_us"]["n"] == 2 * L and abs(out["attention_us"]["mean"] - 90.0) < 1e-9
    assert abs(out["merge_us"]["mean"] - 4.8) < 1e-9
    assert abs(out["gap_to_merge_us"]["mean"] - 0.01) < 1e-9
    assert out["gap_to_next_layer_us"]["n"] == 2 * (L - 1)
    assert abs(out["layer_span_us"]["mean"] - 94.82) < 1e-9
    assert out["move_attention_us"] is None
