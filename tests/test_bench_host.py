"""Host-side behaviour of bench.py that needs no GPU: the one-GPU contract
(any other GPU count is refused with a message), the refusal without a
visible GPU, and the committed HBM traffic record (used only while the
kernel sources it was measured on are unchanged, and then within a few
percent of the algorithmic bytes)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


def test_bench_refuses_more_than_one_gpu():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_bench_without_a_gpu_says_so():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is visible")
    r = _run("--steps", "1", "--warmup", "0")
    assert r.returncode == 1
    assert json.loads(r.stdout.strip().splitlines()[-1]) == {"error": "no GPU visible"}


def test_traffic_record_is_current_or_withheld():
    sys.path.insert(0, ROOT)
    import bench
    rec = json.load(open(os.path.join(ROOT, "profiles", "attn_l64_self_hbm_traffic.json")))
    t = bench.recorded_traffic()
    if t is None:
        pytest.skip("kernel sources changed since the counters were taken: the bench reports null")
    assert rec["algorithmic_bytes"] <= t <= 1.05 * rec["algorithmic_bytes"]
