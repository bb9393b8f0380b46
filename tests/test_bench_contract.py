"""The benchmark's output contract: one JSON line with the fields the
measurement depends on (throughput, HBM roofline of the dominant kernel,
the CPU oracle beside it), and a clear refusal of more than one GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


@pytest.mark.gpu
def test_bench_json_line():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # the benchmark runs as a child process of its own
    r = subprocess.run([sys.executable, BENCH, "--config", "mlp", "--steps", "3", "--warmup", "1",
                        "--cpu-seconds", "1", "--no-other-calls", "--no-other-configs"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, lines
    res = json.loads(lines[0])
    import bench

    assert res["metric"] == bench.METRIC
    assert res["unit"] == "elements/s" and res["value"] > 0
    assert res["n_gpus"] == 1 and res["steps"] == 3 and res["warmup"] == 1
    assert res["ms_per_step"] > 0 and res["higher_is_better"] is True
    assert res["graph_ms_per_step"] > 0  # the same step replayed as a captured HIP graph
    assert res["scaling"] == "weak" and res["vs_baseline"] is None
    assert res["dtype"] == "f32" and res["data"] == "synthetic"
    assert res["config"]["workload"] == "mlp"
    # value is the whole step's throughput over the W worker rows
    W, n = res["config"]["W"], res["config"]["n"]
    assert abs(res["value"] - W * n / (res["ms_per_step"] * 1e-3)) <= 1e-6 * res["value"]
    rf = res["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert rf["achieved"] > 0 and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-12
    assert "traffic" in rf and rf["kernel"].startswith("k_")
    cb = res["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["unit"] == "elements/s"
    assert cb["value"] > 0 and cb["cores"] >= 1 and cb["sample"]
    assert cb["cpu_model"] and "physical_cores" in cb and "logical_cpus" in cb
