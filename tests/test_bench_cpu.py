"""bench.py logic that needs no GPU: the one-GPU refusal, the use of committed HBM
counters only for the kernel source they were taken on, and the Newton-Schulz FLOP count
of the Gefen-Muon roofline."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_device_work():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert out.returncode == 2
    assert "one GPU" in out.stdout + out.stderr


def test_counters_are_used_only_for_the_source_they_were_taken_on(monkeypatch):
    with open(os.path.join(ROOT, "profiles", "traffic_llama3_1p5b.json")) as f:
        rec = json.load(f)
    key, ent = next(iter(rec["kernels"].items()))
    kind, vpl, gdt = key.split("/")[:3]
    args = ("llama3_1p5b", kind, int(vpl[3:]), gdt)
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: rec["source_hash"])
    assert bench.read_traffic(*args) == ent["bytes_per_launch"]
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0" * 16)
    assert bench.read_traffic(*args) is None
    assert bench.read_traffic("no_such_workload", kind, int(vpl[3:]), gdt) is None


def test_newton_schulz_flops_of_gpt2_small():
    """Counted from the GPT-2 small architecture (12 layers, d = 768, MLP 3072, vocabulary
    50257, 1024 positions), independently of the workload's tensor list: per matrix and
    iteration 4 m^2 n + 2 m^3 with m the short side; 1-D tensors as 1 x n."""
    d, L, V, P = 768, 12, 50257, 1024
    mats = [(V, d), (P, d)] + L * [(d, 3 * d), (d, d), (d, 4 * d), (4 * d, d)]
    vecs = L * [d, d, 3 * d, d, d, d, 4 * d, d] + [d, d]
    per_iter = sum(4 * min(a, b) ** 2 * max(a, b) + 2 * min(a, b) ** 3 for a, b in mats)
    per_iter += sum(4 * n + 2 for n in vecs)
    assert bench.muon_ns_flops(W.get("gpt2_125m"), 5) == 5 * per_iter
