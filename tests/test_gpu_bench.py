"""bench.py's contract on the GPU: one JSON line with every field the contract names, the roofline
of the attention launch, the oracle's rate and parity on a row sample, and the context
references, for a dense workload (the 1024-token tiny case) and a chunk workload."""
import json
import os
import subprocess
import sys

import pytest

from test_bench_contract import FIELDS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pytestmark = pytest.mark.gpu


def bench(*args, timeout=240):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                       capture_output=True, text=True, timeout=timeout)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout[-2000:]
    return json.loads(lines[0])


def check_common(d, workload):
    assert all(k in d for k in FIELDS)
    assert d["n_gpus"] == 1 and d["higher_is_better"] is True and d["unit"] == "TFLOP/s"
    assert d["config"]["workload"] == workload and d["dtype"] == "bf16"
    assert d["value"] > 0 and d["ms_per_step"] > 0
    roof = d["roofline"]
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s" and roof["peak"] == 2516.6
    assert roof["achieved"] > 0 and abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-9
    base = d["cpu_baseline"]
    assert base["kind"] == "oracle" and base["value"] > 0 and base["cores"] >= 1
    ps = d["parity_sample"]
    assert ps["rows"] > 0 and ps["max_abs"] <= 2e-2 and ps["mean_abs"] <= 2e-3


def test_dense_bench_line():
    d = bench("--workload", "tiny", "--steps", "3", "--warmup", "1", "--cpu-seconds", "1")
    check_common(d, "tiny")
    c = d["config"]
    assert c["segments"] == [1024] and c["H"] == 2 and c["d"] == 64
    assert c["gemm_bf16_reference"]["tflops"] > 0
    sdpa = c["sdpa_flash_reference"]
    assert "tflops" in sdpa or "unavailable" in sdpa
    assert set(c["input_rounding"]) == {"oracle_on_bf16_inputs", "oracle_on_fp32_inputs"}


def test_chunk_bench_line_without_references():
    d = bench("--workload", "kv_chunk_1s", "--steps", "3", "--warmup", "1", "--cpu-seconds", "1",
              "--no-gemm-reference", "--no-sdpa-reference")
    check_common(d, "kv_chunk_1s")
    c = d["config"]
    assert "gemm_bf16_reference" not in c and "sdpa_flash_reference" not in c
    assert c["query_segments"] == [1560] and c["key_segments"] == [32760]
