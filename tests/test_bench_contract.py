"""bench.py's command-line contract, on the CPU: more than one GPU is refused with a message, and
the scheduler leg (host code only) prints one JSON line with every field the contract names."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FIELDS = ["metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
          "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config", "roofline",
          "cpu_baseline"]


def run(*args, timeout=600):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=timeout)


def test_more_than_one_gpu_is_refused():
    r = run("--gpus", "2")
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_scheduler_leg_prints_one_contract_line():
    r = run("--workload", "sched_scale", "--steps", "1", "--cpu-seconds", "2")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    assert all(k in d for k in FIELDS)
    assert d["n_gpus"] == 1 and d["higher_is_better"] is False and d["unit"] == "ms"
    assert d["config"]["workload"] == "sched_scale" and d["roofline"] is None
    assert d["cpu_baseline"]["kind"] == "oracle" and d["cpu_baseline"]["value"] > 0
    per = d["config"]["per_cluster"]
    assert set(per) == {"4", "16", "64", "256"}
    for m, v in per.items():
        assert v["gap_to_minmax_optimum_max"] >= 0.0
        assert v["scale_out_migrations"] == (int(m) // 2) * 4  # half of K = 8 per new GPU
    assert d["value"] == max(per["256"]["decision_ms_max"], per["256"]["scale_out_epoch_ms"])
