"""The benchmark's output contract: one JSON line with the fields the
measurement reports (the metric, the step time, the roofline of the
dominant kernel class, the CPU baseline).  The multi-GPU refusal runs on
the CPU; one full run on the smallest workload needs a GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_default_chunk_rule():
    sys.path.insert(0, ROOT)
    import bench
    import synthetic as sy
    assert bench.default_chunk(sy.WORKLOADS["strassen3_8192x27648x5120_sign512"]) == 16
    assert bench.default_chunk(sy.WORKLOADS["strassen2_2048x4096x4096_sign512"]) == 32


@pytest.mark.gpu
def test_json_line_on_the_smallest_workload():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    print("[bench] strassen1_256_gl64, 1 step", flush=True)
    r = subprocess.run([sys.executable, BENCH, "--workload", "strassen1_256_gl64", "--steps", "2",
                        "--warmup", "1"], capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "pipeline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1 and d["value"] > 0
    assert d["config"]["workload"] == "strassen1_256_gl64"
    ro = d["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in ro, k
    assert 0 < ro["frac"] < 1 and abs(ro["achieved"] / ro["peak"] - ro["frac"]) < 1e-3
    cb = d["cpu_baseline"]
    for k in ("value", "unit", "cores", "kind", "sample"):
        assert k in cb, k
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1
