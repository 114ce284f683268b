"""The benchmark's host-side accounting (CPU only): the algorithmic bytes it divides by, the counter
summary it reads its HBM traffic from, and its refusal of more than one GPU."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth.workloads import WORKLOADS  # noqa: E402


def test_gate_up_bytes_per_launch():
    """The dominant kernel's algorithmic bytes at the 8B shapes, k = 16: the bf16 gate and up weights
    (2 x 12288 x 4096 x 2 B) plus the bf16 operand read (16 x 4096) and the bf16 activation written
    (16 x 12288)."""
    wl = WORKLOADS["8b"]
    kb = bench.kernel_bytes(wl.shape, 1, 16, wl.prefix_lengths())
    assert kb["gate_up"] == 2 * 12288 * 4096 * 2 + 2 * 16 * 4096 + 2 * 16 * 12288 == 201850880


def test_pass_bytes_are_weights_kv_and_small_activations():
    """A pass's algorithmic bytes are every weight once (the workload registry's own count), the K/V of
    the prefix and the block once per layer, and activations that stay under 1% of the total."""
    wl = WORKLOADS["8b"]
    s, k = wl.shape, 16
    plens = wl.prefix_lengths()
    total = bench.pass_bytes(s, 1, k, plens)
    kv = s.n_layers * 2 * 2 * int(np.sum(plens + k)) * s.kv_dim
    rest = total - s.weight_bytes() - kv
    assert 0 < rest < 0.01 * total


def test_measured_traffic_follows_the_kernel_sources(monkeypatch):
    """bench reads the gate/up traffic from the committed counter summary only while the kernel sources
    hash to the value recorded there."""
    path = os.path.join(ROOT, "profiles", "gate_up_8b_hbm_traffic.md")
    recorded = None
    for line in open(path):
        if line.startswith("- kernel sources sha256[:16]:"):
            recorded = line.split(": ", 1)[1].strip().strip("`")
    assert recorded
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: recorded)
    t = bench.measured_traffic("gate_up")
    assert isinstance(t, int) and t > bench.kernel_bytes(WORKLOADS["8b"].shape, 1, 16, [4096])["gate_up"]
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 16)
    assert bench.measured_traffic("gate_up") is None
    assert bench.measured_traffic("no_such_kernel") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
