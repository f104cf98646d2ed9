"""bench.py's host-only paths on the CPU: the one-JSON-line contract of the
control-plane component, and the refusal of a multi-GPU request."""

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CONTRACT_KEYS = {"metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                 "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                 "roofline", "cpu_baseline"}


def run_bench(*args, timeout=300):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=timeout)


def test_multi_gpu_request_exits_with_a_message():
    r = run_bench("--gpus", "2", timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_control_plane_line_keeps_the_contract():
    r = run_bench("--component", "control_plane")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    line = json.loads(lines[-1])
    assert CONTRACT_KEYS <= set(line)
    assert line["n_gpus"] == 0 and line["higher_is_better"] is False
    assert line["value"] > 0 and line["unit"] == "us"
    assert isinstance(line["config"], dict) and "workload" in line["config"]
    base = line["cpu_baseline"]
    assert base["kind"] == "oracle" and base["cores"] >= 1 and base["value"] > 0
