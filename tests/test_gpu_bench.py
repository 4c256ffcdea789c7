"""The measurement path: bench.py's one-layer line in a fresh process.

Runs `bench.py --workload 7b-layer-mixed` for a few steps as a child process and checks the line's
contract: one JSON line with the metric, value and units; the dominant kernel's roofline timed by
events inside the timed steps (not named by the first launches' one-time costs); the HBM traffic,
when given, above the algorithmic bytes (it is null once the GEMM sources differ from those the
committed counter summary was taken on).
"""
import json
import os
import subprocess
import sys

import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


def test_one_layer_line_contract():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "7b-layer-mixed", "--steps", "3",
                        "--warmup", "2", "--no-cpu-baseline"], capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    out = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "roofline", "config"):
        assert k in out, k
    assert out["n_gpus"] == 1 and out["steps"] == 3 and out["value"] > 0
    roof = out["roofline"]
    assert roof["kernel"] == "gemm_gate_up" and roof["bound"] == "mfma"
    assert "inside the timed steps" in roof["timing"], roof["timing"]
    assert 0 < roof["frac"] < 1 and abs(roof["achieved"] / roof["peak"] - roof["frac"]) < 1e-9
    assert roof["traffic"] is None or roof["traffic"] > roof["algorithmic_bytes_per_launch"]
    print(json.dumps({k: out[k] for k in ("value", "ms_per_step")}), roof["frac"], flush=True)
