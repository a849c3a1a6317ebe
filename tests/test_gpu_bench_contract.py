"""bench.py on a small workload: one JSON line with the fields the benchmark
contract names (metric, value, unit, counts, timing, scaling, dtype, config,
the attention roofline and the oracle's CPU baseline), in a child process."""
from __future__ import annotations

import json
import os
import subprocess
import sys

import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("args", [["--workload", "small_bf16"],
                                  ["--workload", "small_bf16", "--last-row-only", "--tasks", "2"],
                                  ["--mode", "recursive", "--workload", "small_bf16_sp5"]],
                         ids=["one_pass", "tasks_last_row", "recursive"])
def test_bench_prints_the_contract_line(args):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"[bench contract] {' '.join(args)}", flush=True)
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args, "--steps", "3", "--warmup", "1",
                          "--cpu-seconds", "1"], capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert res.returncode == 0, res.stderr[-2000:]
    lines = [l for l in res.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, res.stdout
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["dtype"].startswith("bf16 storage") and isinstance(d["config"], dict) and "workload" in d["config"]
    assert d["config"]["weights"] == "fp16 image"
    dist = d["step_time_distribution"]
    assert dist["steps"] >= 50 and 0 < dist["p10_ms"] <= dist["median_ms"] <= dist["p90_ms"]
    r = d["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in r, key
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000
    assert r["frac"] > 0 and r["frac"] == pytest.approx(r["achieved"] / r["peak"], abs=1e-4)
    assert r["measured_read_peak_gbps"] > 0
    assert r["frac_of_measured_read_peak"] == pytest.approx(r["achieved"] / r["measured_read_peak_gbps"], abs=1e-3)
    # the device's own ceilings: a streaming read below the 8 TB/s nameplate, an
    # fp16 matrix-core rate below 2.5 PFLOP/s, each projection below both
    assert r["measured_read_peak_gbps"] < 8000
    pr = d["projections"]
    assert 0 < pr["measured_mfma_peak_tflops"] < 2500
    for name in ("o_proj", "gate_up", "down"):
        assert 0 < pr[name]["frac_of_peak"] <= pr[name]["frac_of_measured_mfma_peak"] < 1.05
    # the attention stage (split + merge) takes longer than the split kernel alone
    assert r["mean_launch_ms"] >= r["split_kernel_only"]["mean_launch_ms"]
    # a KV cache this small is rotated over copies exceeding 1 GB
    assert d["config"]["kv_copies_rotated"] >= 2
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["value"] > 0 and c["cores"] >= 1 and c["sample"]
