"""bench.py's command line on the CPU: more than one GPU, and options that do not fit the workload,
are refused with exit status 2 before anything touches a device, and the record-store timing
runs on the host alone."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_record_store_timing_prints_one_json_line():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--records"],
                       capture_output=True, text=True, cwd=ROOT, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1
    line = json.loads(lines[0])
    assert line["unit"] == "tasks/s" and line["value"] > 0
    assert line["config"]["workload"].startswith("records:")


def test_default_workload_is_the_largest_logits_streaming_one():
    """With no flags the bench measures the long single-turn reasoning batch (8 x 16,384 tokens,
    79.7 GB of logits), one GPU, and a step count that finishes in seconds."""
    sys.path.insert(0, ROOT)
    import bench
    args = bench.build_parser().parse_args([])
    assert args.workload == "reasoning" and args.gpus == 1
    assert 1 <= args.steps <= 100 and args.warmup >= 1


def test_band_order_timing_needs_the_fused_workload():
    """--band-ab times the fused projection's tile order; with another workload it is refused
    before anything touches a device."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--band-ab", "4"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "--workload fused" in r.stderr
