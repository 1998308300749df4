"""The benchmark script on short batched runs (GPU): the JSON line keeps its
contract, every sequence of the batch is built (a batch-1 prompt handed to a
batch-2 cache would read past its buffers), and the routing cadence of the
workload is followed."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

KEYS = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
        "scaling", "vs_baseline", "dtype", "data", "config", "roofline")


@pytest.mark.gpu
@pytest.mark.parametrize("workload,routing,batch,interval", [("c3s", "async", 2, 1),
                                                              ("c3s", "sync", 2, 1),
                                                              ("c5s", "async", 2, 8)])
def test_bench_line_on_batched_workloads(workload, routing, batch, interval):
    print(f"[bench] {workload} {routing}", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", workload,
                        "--routing", routing, "--instances", "2", "--steps", "16", "--warmup", "4",
                        "--no-cpu"], capture_output=True, text=True, timeout=180, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-3000:]
    d = json.loads(r.stdout.strip().splitlines()[-1])
    for k in KEYS:
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 16 and d["value"] > 0
    assert d["config"]["global_batch"] == batch and d["config"]["routing_interval"] == interval
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and 0 < rf["frac"] < 1 and rf["traffic"] is None
