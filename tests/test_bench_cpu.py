"""Host-side pieces of the benchmark (CPU): the one-GPU contract, the
algorithmic byte count the roofline is stated on, and the workload line."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synthetic as syn  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_algorithmic_bytes_per_window():
    # 8 KV heads x 32 tokens x 128 channels: a bf16 window is K + V at 2 bytes
    # (128 KiB); an int4 window is 4-bit K + V codes (32 KiB) plus fp16 scale and
    # zero per (head, channel) for keys and per (head, token, 32-channel group)
    # for values (8 KiB); an int2 window has half the codes.  Each live window's
    # score is read and written (8 bytes).
    wl = syn.get_workload("c2")
    base = bench.attend_bytes(wl, 0, 0, 0, 0)
    assert base == 2 * 32 * 128 * 2 + 8                      # query + output, open-window score
    assert bench.attend_bytes(wl, 1, 0, 0, 0) - base == 131072 + 8
    assert bench.attend_bytes(wl, 0, 1, 0, 0) - base == 32768 + 8192 + 8
    assert bench.attend_bytes(wl, 0, 0, 1, 0) - base == 16384 + 8192 + 8
    assert bench.attend_bytes(wl, 0, 0, 0, 5) - base == 5 * 2 * 8 * 128 * 2
    # the benchmark shape: 1024 windows, 20% bf16 / 30% int4 -> about 39.4 MB per call
    n_f, n_q = wl.capacity_full, wl.capacity_quant
    mb = bench.attend_bytes(wl, n_f, n_q, 0, 1) / 1e6
    assert 39.0 < mb < 39.8


@pytest.mark.parametrize("name,words", [("c2", ["32768-token", "batch 1", "int4"]),
                                        ("c3", ["batch 8", "int4"]),
                                        ("c5", ["batch 4", "64 query", "int4 / int2"]),
                                        ("c6", ["byte budget", "sink 5", "recent 32"])])
def test_workload_line_names_the_shape(name, words):
    d = bench.workload_desc(syn.get_workload(name))
    for w in words:
        assert w in d, (w, d)


def test_whole_model_workload_line():
    d = bench.workload_desc(syn.get_workload("c3"))
    assert d.startswith("32 layers back to back per step"), d


def test_host_cpu_reports_count():
    model, n = bench.host_cpu()
    assert n == os.cpu_count() and n >= 1
