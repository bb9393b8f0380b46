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


def test_counter_summary_is_tied_to_its_kernel_sources(tmp_path, monkeypatch):
    # the HBM bytes of a counter summary count only while the files it names
    # are unchanged (comments aside)
    import json as _json

    sys.path.insert(0, ROOT)
    import bench

    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    src = ["paper_1911_08907_amd/csrc/aps_sync.hip", "include/aps.h"]
    summary = {"fetch_kib_per_dispatch": 3.0, "write_kib_per_dispatch": 5.0, "fetch_scale": 2.0,
               "write_scale": 1.0, "sources": src, "source_digest": bench.source_digest(src)}
    path = tmp_path / "sync_spec_demo_1-5-2_counters.json"
    path.write_text(_json.dumps(summary))
    got, where = bench.traffic_from_profile("sync_spec", "demo", "1-5-2")
    assert got == (3.0 * 2.0 + 5.0) * 1024 and where.endswith("_counters.json")
    summary["source_digest"] = "0" * 16
    path.write_text(_json.dumps(summary))
    assert bench.traffic_from_profile("sync_spec", "demo", "1-5-2") == (None, "kernel changed since the counters were taken")
    assert bench.traffic_from_profile("sync_spec", "other", "1-5-2") == (None, "no counter summary")
    # the committed summary of the dominant kernel names the files it was taken on
    with open(os.path.join(ROOT, "profiles", "sync_spec_resnet50_w256_1-5-2_counters.json")) as fh:
        committed = _json.load(fh)
    assert "paper_1911_08907_amd/csrc/aps_sync.hip" in committed["sources"]
