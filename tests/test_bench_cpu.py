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


def test_all_core_oracle_baseline_equals_one_core():
    """The all-core CPU baseline deals disjoint whole-block ranges to worker processes
    that run the unchanged oracle; their parameters must equal the one-core run's bit
    for bit (time_oracle raises otherwise), and every element is counted once."""
    import numpy as np
    import oracle
    rng = np.random.default_rng(5)
    h = np.zeros(4096, dtype=np.uint64)
    g0 = rng.standard_normal(4096).astype(np.float32)
    oracle.histogram_uniform(g0, 64, 4096, h)
    cb, _, _, _ = oracle.dp_codebook(h, 256)
    jobs = []
    for p, nb in ((64, 300), (100, 7), (1, 50)):
        n = p * nb
        jobs.append((rng.standard_normal(n) * 0.02, rng.standard_normal(n).astype(np.float32),
                     rng.integers(0, 256, n).astype(np.uint8), rng.uniform(0, 1, nb),
                     rng.uniform(0, 1, nb), np.arange(0, n + 1, p, dtype=np.int64)))
    ref = [j[0].copy() for j in jobs]
    for (th0, g, c, s, v, offs), r in zip([tuple(a.copy() for a in j) for j in jobs], ref):
        oracle.step_blocks(r, g, c, s, v, offs, cb, cb, 1e-3, 0.9, 0.999, 1e-8, 0.1, 3)
    hp = {"lr": 1e-3, "b1": 0.9, "b2": 0.999, "eps": 1e-8, "wd": 0.1, "t": 3}
    n, par_dt, one_dt, pieces, procs = bench.time_oracle(jobs, cb, hp, 3)
    assert n == sum(j[0].size for j in jobs)
    assert procs == 3 and pieces >= 3 and par_dt > 0 and one_dt > 0
    for j, r in zip(jobs, ref):
        np.testing.assert_array_equal(j[0], r)
