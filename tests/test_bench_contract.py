"""bench.py's command-line contract on the CPU: it refuses more than one GPU with a one-line
JSON message, and reports the absence of a GPU instead of falling back to anything."""

import json
import os
import subprocess
import sys

import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       timeout=300, cwd=ROOT)
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    return r.returncode, lines


def test_more_than_one_gpu_is_refused():
    rc, lines = _run("--gpus", "2", "--steps", "1", "--warmup", "0")
    assert rc == 2 and len(lines) == 1
    msg = json.loads(lines[0])
    assert "error" in msg and "one GPU" in msg["error"]


def test_no_gpu_is_reported_not_emulated():
    if torch.cuda.is_available():
        return
    rc, lines = _run("--steps", "1", "--warmup", "0")
    assert rc == 2 and len(lines) == 1
    assert json.loads(lines[0]) == {"error": "no GPU visible"}


def test_cpu_baseline_repeats_a_small_sample():
    # a workload with fewer rows than the sample asks for repeats them: 16 rows, 40 asked -> 3 passes
    sys.path.insert(0, ROOT)
    import bench
    from paper_2607_02461_amd.workloads import Linear
    lin = Linear("tiny", 16, 256, 128, 4, 4)
    g = torch.Generator()
    g.manual_seed(0)
    layers = [dict(lin=lin, X=torch.randn((16, 256), generator=g).to(torch.bfloat16),
                   W=(torch.randn((128, 256), generator=g) * 0.02).to(torch.bfloat16))]
    out = bench.cpu_baseline(layers, 40, min_seconds=0.0)
    assert out["kind"] == "oracle" and out["unit"] == "TFLOP/s" and out["value"] > 0
    assert "16 token rows" in out["sample"] and "3 passes" in out["sample"]


def test_cpu_baseline_one_thread_leg_runs_in_a_child_process():
    # the single-thread leg re-times the oracle on the first rows in a child process whose thread
    # pools are pinned to one thread
    sys.path.insert(0, ROOT)
    import bench
    from paper_2607_02461_amd.workloads import Linear
    lin = Linear("tiny", 16, 256, 128, 4, 4)
    g = torch.Generator()
    g.manual_seed(1)
    layers = [dict(lin=lin, X=torch.randn((16, 256), generator=g).to(torch.bfloat16),
                   W=(torch.randn((128, 256), generator=g) * 0.02).to(torch.bfloat16))]
    out = bench.cpu_baseline(layers, 16, min_seconds=0.0, one_thread_rows=8)
    one = out["one_thread"]
    assert "error" not in one, one
    assert one["kind"] == "oracle" and one["cores"] == 1 and one["value"] > 0
    assert "8 token rows" in one["sample"] and "one thread" in one["sample"]
    assert out["host_cpu_count"] == os.cpu_count()
