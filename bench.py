#!/usr/bin/env python
"""Benchmark of the Gefen optimizer step on one MI355X.

Metric: optimizer-step Gparams/s (parameters updated per second) and achieved HBM GB/s
(algorithmic bytes / time) as a fraction of MI355X's 8 TB/s peak, on one GPU.

A step is one ``gefen_step`` over every tensor of the workload (all kernel classes),
with parameters, gradients and optimizer state resident in HBM. The default workload
is the Llama-3 1.5B shape (1,498,482,688 fp32 parameters, bf16 gradients with
Student-t(3) noise and per-row / per-head scales); gradients for two steps are drawn
before timing and alternated, so the timed region contains only optimizer steps.

Per-step times come from HIP events between steps (median / mean / min over the steps
without a refit; with codebook refits, the refit step and the amortised step time
separately). ``ceiling`` holds the practical streaming ceilings on the same GPU: the
library's hand-written pass over the step's own byte mix (``mix_gbps``: parameter read +
write, gradient read, code byte read + write, no arithmetic), and torch's device copy and
two-input add.

Prints one JSON line. ``roofline`` describes the dominant kernel class: algorithmic
bytes per launch over its mean launch time, from HIP events recorded on the step's
stream around every class launch during a second pass of as many plain steps (kept out
of the timed steps, whose whole-step time the extra events would lengthen). ``traffic`` comes from committed rocprofv3 counter summaries when they were
taken on the current kernel source, else null. ``cpu_baseline`` is the float64 oracle
(as it stands) timed on a bounded sample of the same workload, over one process per
available core (at most 16), with the one-core rate beside it.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
METRIC = "optimizer-step Gparams/s and achieved HBM GB/s (% of MI355X peak), 1 GPU"


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for name in ("step.hip", "step_device.h", "gefen_internal.h"):
        with open(os.path.join(ROOT, "paper_2606_13894_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(workload: str, kind: str, vpl: int, gdt: str, code_bits: int = 8):
    """Counter-derived HBM bytes per launch from profiles/, if taken on this source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_hash") != kernel_source_hash():
        return None
    key = f"{kind}/vpl{vpl}/{gdt}" + ("" if code_bits == 8 else f"/cb{code_bits}")
    ent = d.get("kernels", {}).get(key)
    return None if ent is None else ent.get("bytes_per_launch")


def _baseline_jobs(w, params, grads, st, sample_elems: int):
    """A bounded sample of the workload for the oracle: whole blocks from the start of
    every tensor in turn (largest first) until `sample_elems` elements are covered, with
    the state the GPU holds for them. Each job is (theta, grad bits, codes, s, v, block
    offsets relative to the job)."""
    import numpy as np
    import paper_2606_13894_amd as gf
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import grad_bits, unpack_codes

    lay = st.layout()
    periods = st.periods
    codes = unpack_codes(st.read(gf.STATE_CODES).cpu().numpy(), st.k)
    scale = st.read(gf.STATE_SCALE).cpu().numpy().astype(np.float64)
    vm = st.read(gf.STATE_V).cpu().numpy().astype(np.float64)
    explicit = None
    if any(p == 0 for p in periods):
        import workloads as W
        explicit = W.stress_block_offsets(w.numel, w.n_blocks)
    jobs = []
    left = sample_elems
    order = sorted(range(len(params)), key=lambda i: -params[i].numel())
    per_tensor = max(1, sample_elems // max(1, len(order)))
    for i in order:
        if left <= 0:
            break
        want = min(per_tensor, left)
        if periods[i] > 0:
            p = periods[i]
            take = min(params[i].numel(), max(p, (want // p) * p))
            offs = np.arange(0, take + 1, p, dtype=np.int64)
        else:
            # explicit blocks (one tensor spans the whole table): the first whole blocks
            nb = int(np.searchsorted(explicit, want, side="right")) - 1
            nb = max(1, nb)
            offs = np.ascontiguousarray(explicit[:nb + 1], dtype=np.int64)
            take = int(offs[-1])
        nb = offs.size - 1
        th = params[i].detach().reshape(-1)[:take].double().cpu().numpy()
        g = grad_bits(grads[i].reshape(-1)[:take])
        c0 = lay["code_offsets"][i]
        b0 = lay["block_index"][i]
        jobs.append((th, g, codes[c0:c0 + take].copy(), scale[b0:b0 + nb].copy(),
                     vm[b0:b0 + nb].copy(), offs))
        left -= take
    return jobs


def _cpu_worker(job_dir: str, idx: int):
    """--cpu-worker: run the oracle's step over this worker's share of the sample
    (disjoint whole-block ranges written by cpu_baseline), write the results back and
    print the wall-clock interval of the oracle calls. Touches no GPU."""
    import numpy as np
    import oracle
    with open(os.path.join(job_dir, "hp.json")) as f:
        hp = json.load(f)
    cb = np.load(os.path.join(job_dir, "cb.npy"))
    pieces = hp["shares"][idx]
    arrays = []
    for name in pieces:
        base = os.path.join(job_dir, name)
        arrays.append([np.load(f"{base}.{k}.npy") for k in ("th", "g", "c", "s", "v", "o")])
    t0 = time.time()
    for th, g, c, s_, v, o in arrays:
        oracle.step_blocks(th, g, c, s_, v, o, cb, cb, hp["lr"], hp["b1"], hp["b2"], hp["eps"],
                           hp["wd"], hp["t"])
    t1 = time.time()
    for name, (th, g, c, s_, v, o) in zip(pieces, arrays):
        np.save(os.path.join(job_dir, f"{name}.out.npy"), th)
    print(json.dumps({"t0": t0, "t1": t1, "elems": int(sum(a[0].size for a in arrays))}),
          flush=True)


def time_oracle(jobs, cb, hp: dict, ncpu: int):
    """Time the oracle's step over `jobs` (see _baseline_jobs) once on one core and once
    over disjoint whole-block ranges in `ncpu` worker processes, each running the same
    oracle routine. The all-core parameters must equal the one-core ones bit for bit.
    Returns (elements, all-core seconds, one-core seconds, pieces, processes)."""
    import shutil
    import subprocess
    import tempfile
    import numpy as np
    import oracle

    n = sum(j[0].size for j in jobs)
    job_dir = tempfile.mkdtemp(prefix="gefen_cpu_", dir="/dev/shm" if os.path.isdir("/dev/shm")
                               else None)
    try:
        np.save(os.path.join(job_dir, "cb.npy"), cb)
        pieces = []   # (name, job index, first element, end element, size)
        target = max(1, n // (4 * ncpu))
        for ji, (th, g, c, s_, v, offs) in enumerate(jobs):
            b = 0
            nb = offs.size - 1
            while b < nb:
                e = int(np.searchsorted(offs, offs[b] + target, side="right")) - 1
                e = min(nb, max(b + 1, e))
                lo, hi = int(offs[b]), int(offs[e])
                name = f"j{ji}_b{b}"
                base = os.path.join(job_dir, name)
                for k, a in (("th", th[lo:hi]), ("g", g[lo:hi]), ("c", c[lo:hi]),
                             ("s", s_[b:e]), ("v", v[b:e]), ("o", offs[b:e + 1] - lo)):
                    np.save(f"{base}.{k}.npy", np.ascontiguousarray(a))
                pieces.append((name, ji, lo, hi, hi - lo))
                b = e
        shares = [[] for _ in range(ncpu)]
        load = [0] * ncpu
        for name, _, _, _, sz in sorted(pieces, key=lambda q: -q[4]):
            k = load.index(min(load))
            shares[k].append(name)
            load[k] += sz
        with open(os.path.join(job_dir, "hp.json"), "w") as f:
            json.dump(dict(hp, shares=shares), f)
        procs = [subprocess.Popen([sys.executable, os.path.abspath(__file__), "--cpu-worker",
                                   job_dir, str(k)], stdout=subprocess.PIPE, text=True)
                 for k in range(ncpu) if shares[k]]
        outs = [p.communicate()[0] for p in procs]
        if any(p.returncode for p in procs):
            raise RuntimeError("an oracle worker failed")
        spans = [json.loads(o.strip().splitlines()[-1]) for o in outs]
        par_dt = max(x["t1"] for x in spans) - min(x["t0"] for x in spans)
        if sum(x["elems"] for x in spans) != n:
            raise RuntimeError("the workers did not cover the sample")

        t0 = time.perf_counter()
        for th, g, c, s_, v, offs in jobs:
            oracle.step_blocks(th, g, c, s_, v, offs, cb, cb, hp["lr"], hp["b1"], hp["b2"],
                               hp["eps"], hp["wd"], hp["t"])
        one_dt = time.perf_counter() - t0
        for name, ji, lo, hi, _ in pieces:
            got = np.load(os.path.join(job_dir, f"{name}.out.npy"))
            if not np.array_equal(got, jobs[ji][0][lo:hi]):
                raise RuntimeError("the all-core oracle run differs from the one-core run")
    finally:
        shutil.rmtree(job_dir, ignore_errors=True)
    return n, par_dt, one_dt, len(pieces), len(procs)


def cpu_baseline(w, params, grads, st, sample_elems: int, t: int):
    """The oracle's step (float64, as it stands) on a bounded sample of the workload, on
    one core and on every available core (at most 16 processes). The rate is the
    sample's, extrapolated to the workload (the step costs the same per element
    everywhere)."""
    import numpy as np
    import paper_2606_13894_amd as gf

    jobs = _baseline_jobs(w, params, grads, st, sample_elems)
    cb = st.read(gf.STATE_CB_DEC).cpu().numpy().astype(np.float64)
    hp = {"lr": w.lr, "b1": w.betas[0], "b2": w.betas[1], "eps": w.eps, "wd": w.wd, "t": t}
    ncpu = min(16, host_cpu()["cpus_available"] or 1)
    n, par_dt, one_dt, npieces, nproc = time_oracle(jobs, cb, hp, ncpu)
    kind = ("explicit blocks from the start of the block table" if any(
        p == 0 for p in st.periods) else f"whole blocks from the start of the {len(jobs)} "
        "largest tensors")
    return {"value": n / par_dt / 1e9, "unit": "Gparams/s", "cores": nproc, "kind": "oracle",
            "sample": f"oracle step (float64) on {n} of {w.numel} elements ({kind}), "
                      f"{npieces} disjoint block ranges over {nproc} processes; "
                      "rate extrapolated from the sample",
            "seconds": par_dt,
            "single_thread": {"value": n / one_dt / 1e9, "cores": 1, "seconds": one_dt},
            "host": host_cpu()}


def host_cpu():
    """The host's CPU model and the logical CPUs this process may use."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:
        ncpu = os.cpu_count()
    return {"cpu_model": model, "cpus_available": ncpu}


def adamw_comparator(torch, w, params, grads, steps: int, gefen_state_bytes: int,
                     gefen_peak_bytes: int, gefen_ms: float):
    """torch.optim.AdamW (fused) on the same parameters and gradients: step time, state
    bytes (after the first step), peak bytes above parameters and gradients over its
    steps, and algorithmic bytes per element (parameter read + write 8, fp32 gradient
    4, m and v read + write 16). Fused AdamW takes gradients in the parameter dtype, so
    bf16 gradients are widened to fp32 once, outside the timed loop. Gefen's peak is
    its persistent state plus its workspace: the library allocates nothing in a step."""
    ps = [torch.nn.Parameter(p.detach().clone()) for p in params]
    g32 = [[g.float() for g in gs] for gs in grads]
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    opt = torch.optim.AdamW(ps, lr=w.lr, betas=w.betas, eps=w.eps, weight_decay=w.wd,
                            fused=True)
    for p, g in zip(ps, g32[0]):
        p.grad = g
    opt.step()
    torch.cuda.synchronize()
    state_bytes = torch.cuda.memory_allocated() - base
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        for p, g in zip(ps, g32[i % 2]):
            p.grad = g
        opt.step()
    e1.record()
    torch.cuda.synchronize()
    peak_bytes = torch.cuda.max_memory_allocated() - base
    ms = e0.elapsed_time(e1) / steps
    n = w.numel
    bytes_step = 28 * n
    out = {"optimizer": "torch.optim.AdamW(fused=True)", "ms_per_step": round(ms, 4),
           "gparams_per_s": round(n / (ms * 1e-3) / 1e9, 3),
           "hbm_gbps": round(bytes_step / (ms * 1e-3) / 1e9, 1),
           "bytes_per_elem": 28, "state_bytes": state_bytes, "peak_bytes": peak_bytes,
           "gefen_state_bytes": gefen_state_bytes, "gefen_peak_bytes": gefen_peak_bytes,
           "state_ratio": round(state_bytes / gefen_state_bytes, 3),
           "peak_ratio": round(peak_bytes / gefen_peak_bytes, 3),
           "gefen_speedup": round(ms / gefen_ms, 3)}
    del opt, ps, g32
    torch.cuda.empty_cache()
    return out


PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA


def muon_ns_flops(w, steps: int) -> int:
    """Newton-Schulz FLOPs of one Gefen-Muon step: per tensor (m = min side, n = max
    side) and iteration, X X^T (2 m^2 n), A A (2 m^3) and B X (2 m^2 n)."""
    total = 0
    for t in w.tensors:
        r = t.rows
        c = t.numel // r
        m, n = min(r, c), max(r, c)
        total += steps * (4 * m * m * n + 2 * m * m * m)
    return total


def bench_muon(args, torch, w, dev):
    """Gefen-Muon steps (quantized Muon momentum + bf16 Newton-Schulz + update) on the
    workload's tensors as matrices (1-D tensors as 1 x n), against torch.optim.Muon."""
    import workloads as W
    import paper_2606_13894_amd as gf
    fields = W.scale_fields(w)
    params = W.init_params(w, dev)
    grads = [W.make_grads(w, fields, t, dev) for t in (1, 2)]
    rows = [t.rows for t in w.tensors]
    lr, mu, wd, ns_steps = 1e-3, 0.95, 0.1, 5
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    st = gf.GefenState(grads[0], eps_part=w.eps, code_bits=args.code_bits)
    st.muon_init(rows)
    torch.cuda.synchronize()
    init_s = time.perf_counter() - t0
    for i in range(args.warmup):
        st.muon_step(params, grads[i % 2], lr, mu, wd, True, ns_steps)
    torch.cuda.synchronize()
    st.profile_begin(args.steps)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        st.muon_step(params, grads[i % 2], lr, mu, wd, True, ns_steps)
    e1.record()
    torch.cuda.synchronize()
    prof = st.muon_profile_end()
    ms = e0.elapsed_time(e1) / args.steps
    flops = muon_ns_flops(w, ns_steps)
    ortho_ms = prof["ortho_ms"] / max(1, prof["steps"])
    codec_ms = prof["codec_ms"] / max(1, prof["steps"])
    gb = 2 if w.grad_dtype == "bf16" else 4
    codec_bytes = w.numel * (gb + (2 if args.code_bits == 8 else 1) + 2)
    persistent, workspace = st.state_bytes()
    out = {
        "metric": METRIC + " (Gefen-Muon)",
        "value": round(w.numel / (ms * 1e-3) / 1e9, 3),
        "unit": "Gparams/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "optimizer": "gefen_muon", "params": w.numel,
                   "tensors": len(w.tensors), "grad_dtype": w.grad_dtype,
                   "code_bits": args.code_bits, "ns_steps": ns_steps, "nesterov": True},
        "phases_ms": {"codec": round(codec_ms, 4), "orthogonalise_update": round(ortho_ms, 4)},
        "roofline": {"bound": "mfma", "achieved": None, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": None, "traffic": None,
                     "kernel": "Newton-Schulz bf16 matrix-core products (k_ns_gemm), timed "
                               "with the prep and update kernels around them (wall time of "
                               "that phase)",
                     "flops_per_step": flops},
        "codec": {"bytes_per_step": codec_bytes,
                  "gbps": round(codec_bytes / (codec_ms * 1e-3) / 1e9, 1)},
        "memory": {"gefen_muon_persistent_bytes": persistent,
                   "gefen_muon_workspace_bytes": workspace},
        "init_s": round(init_s, 3),
    }
    achieved = flops / (ortho_ms * 1e-3) / 1e12
    out["roofline"]["achieved"] = round(achieved, 1)
    out["roofline"]["frac"] = round(achieved / PEAK_BF16_TFLOPS, 4)
    if args.no_torch_muon:
        out["torch_muon"] = None
        return out
    # torch.optim.Muon on the same matrices
    ps = [torch.nn.Parameter(p.detach().clone().view(r, p.numel() // r))
          for p, r in zip(params, rows)]
    gm = [[g.float().view(r, g.numel() // r) for g, r in zip(gs, rows)] for gs in grads]
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    opt = torch.optim.Muon(ps, lr=lr, momentum=mu, weight_decay=wd, nesterov=True,
                           ns_steps=ns_steps)
    for p, g in zip(ps, gm[0]):
        p.grad = g
    opt.step()
    torch.cuda.synchronize()
    muon_state = torch.cuda.memory_allocated() - base
    m0 = torch.cuda.Event(enable_timing=True)
    m1 = torch.cuda.Event(enable_timing=True)
    reps = min(args.steps, 10)
    m0.record()
    for i in range(reps):
        for p, g in zip(ps, gm[i % 2]):
            p.grad = g
        opt.step()
    m1.record()
    torch.cuda.synchronize()
    muon_ms = m0.elapsed_time(m1) / reps
    out["torch_muon"] = {"ms_per_step": round(muon_ms, 4), "state_bytes": muon_state,
                         "state_ratio": round(muon_state / persistent, 3),
                         "gefen_speedup": round(muon_ms / ms, 3)}
    return out


def copy_ceiling(torch, dev, nbytes: int = 4 << 30, reps: int = 10):
    """Practical streaming ceiling on this GPU: torch's device copy (one read, one write)
    and an add of two tensors (two reads, one write) over `nbytes` per tensor."""
    n = nbytes // 4
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    c = torch.empty_like(a)
    out = {}
    for name, fn, moved in (("copy_gbps", lambda: b.copy_(a), 2 * nbytes),
                            ("add_gbps", lambda: torch.add(a, b, out=c), 3 * nbytes)):
        fn()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        out[name] = round(moved * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    del a, b, c
    torch.cuda.empty_cache()
    out["bytes_per_tensor"] = nbytes
    return out


def mix_ceiling(torch, gf, dev, grad_dtype: str, n: int = 1_500_000_000, reps: int = 10):
    """The step's byte mix (12 or 14 B per element) through the library's streaming
    kernel, with no optimizer arithmetic: the practical ceiling for the step kernels."""
    theta = torch.zeros(n, dtype=torch.float32, device=dev)
    grad = torch.zeros(n, dtype=torch.bfloat16 if grad_dtype == "bf16" else torch.float32,
                       device=dev)
    codes = torch.zeros(n, dtype=torch.uint8, device=dev)
    gf.stream_mix(theta, grad, codes)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        gf.stream_mix(theta, grad, codes)
    e1.record()
    torch.cuda.synchronize()
    per = 8 + (2 if grad_dtype == "bf16" else 4) + 2
    gbps = per * n * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del theta, grad, codes
    torch.cuda.empty_cache()
    return {"mix_gbps": round(gbps, 1), "mix_elements": n, "mix_bytes_per_element": per}


def main():
    if len(sys.argv) == 4 and sys.argv[1] == "--cpu-worker":
        _cpu_worker(sys.argv[2], int(sys.argv[3]))
        return
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None,
                    help="llama3_1p5b for gefen, gpt2_125m for gefen_muon by default")
    ap.add_argument("--code-bits", type=int, default=8, choices=(8, 4),
                    help="momentum code width: 8 (k = 256) or 4 (k = 16, two codes per byte)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--optimizer", default="gefen", choices=("gefen", "gefen_muon"),
                    help="gefen (the default, Alg. 1) or gefen_muon (quantized Muon momentum "
                         "with Newton-Schulz; default workload gpt2_125m)")
    ap.add_argument("--no-adamw", action="store_true",
                    help="skip the torch AdamW comparison (always skipped for explicit blocks)")
    ap.add_argument("--no-torch-muon", action="store_true",
                    help="skip the torch.optim.Muon comparison of --optimizer gefen_muon")
    ap.add_argument("--cpu-sample-elems", type=int, default=100_000_000)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain device-to-device copy of a known byte count "
                         "(scales rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the Gefen step needs no collectives, and a run on "
              "N GPUs would be N independent copies of this one (see the sharding notes). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as W
    import paper_2606_13894_amd as gf

    dev = torch.device("cuda", 0)
    if args.copy_calibration:
        nbytes = 1 << 30
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": nbytes, "launches": 3}), flush=True)
        return
    if args.workload is None:
        args.workload = "gpt2_125m" if args.optimizer == "gefen_muon" else "llama3_1p5b"
    w = W.get(args.workload)
    if args.optimizer == "gefen_muon":
        if w.n_blocks:
            print("gefen_muon needs matrix-shaped tensors", file=sys.stderr)
            sys.exit(2)
        import paper_2606_13894_amd as gf
        try:
            line = bench_muon(args, torch, w, dev)
        except gf.GefenError as e:
            print(f"gefen_muon on {w.name}: {e}", file=sys.stderr)
            sys.exit(2)
        print(json.dumps(line), flush=True)
        return
    fields = W.scale_fields(w)
    offsets = None
    bscales = None
    if w.n_blocks:
        offsets = W.stress_block_offsets(w.numel, w.n_blocks)
        bscales = W.stress_block_scales(w.n_blocks)
    params = W.init_params(w, dev)
    grads = [W.make_grads(w, fields, t, dev, block_scales=bscales, offsets=offsets)
             for t in (1, 2)]
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    st = gf.GefenState(grads[0], block_offsets=offsets, eps_part=w.eps,
                       code_bits=args.code_bits)
    torch.cuda.synchronize()
    init_s = time.perf_counter() - t0

    hp = (w.lr, w.betas, w.eps, w.wd)
    t = 0
    for _ in range(args.warmup):
        t += 1
        st.step(params, grads[(t - 1) % 2], *hp, t,
                fit=bool(w.refit_every and t % w.refit_every == 0))
    torch.cuda.synchronize()

    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    refit_at = []
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    marks[0].record()
    for i in range(args.steps):
        t += 1
        refit = bool(w.refit_every and t % w.refit_every == 0)
        # a refit step refits the codebook on its own gradients (gefen_step_fit: the
        # histogram is taken inside the step kernels, then the DP)
        st.step(params, grads[(t - 1) % 2], *hp, t, fit=refit)
        if refit:
            refit_at.append(i)
        marks[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    # The kernel classes' launch durations come from a second pass of as many plain steps
    # with HIP events around every class launch (events between the launches would add
    # their own gaps to the whole-step time measured above: 4 % on the GPT-2 125M shapes,
    # whose step is two launches).
    st.profile_begin(args.steps)
    for i in range(args.steps):
        st.step(params, grads[(t + i) % 2], *hp, t + 1 + i)
    torch.cuda.synchronize()
    classes = st.profile_end()
    ms_per_step = marks[0].elapsed_time(marks[-1]) / args.steps
    per_step = [marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)]
    plain = [x for i, x in enumerate(per_step) if i not in refit_at]
    step_stats = {"median_ms": round(statistics.median(plain), 4),
                  "mean_ms": round(statistics.fmean(plain), 4), "min_ms": round(min(plain), 4),
                  "amortised_ms": round(ms_per_step, 4)}
    if refit_at:
        step_stats["refit_step_ms"] = round(statistics.fmean(per_step[i] for i in refit_at), 4)
        step_stats["refits_timed"] = len(refit_at)
    ceiling = dict(mix_ceiling(torch, gf, dev, w.grad_dtype), **copy_ceiling(torch, dev))

    n = w.numel
    step_bytes = sum(c["bytes_per_launch"] for c in classes)
    gparams = n / (ms_per_step * 1e-3) / 1e9
    gbps = step_bytes / (ms_per_step * 1e-3) / 1e9
    dom = max(classes, key=lambda c: c["bytes_per_launch"])
    dom_ms = dom["total_ms"] / max(1, dom["launches"])
    achieved = dom["bytes_per_launch"] / (dom_ms * 1e-3) / 1e9
    traffic = read_traffic(w.name, dom["kind"], dom["vpl"], dom["grad_dtype"], args.code_bits)
    persistent, workspace = st.state_bytes()

    line = {
        "metric": METRIC,
        "value": round(gparams, 3),
        "unit": "Gparams/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "params": n, "tensors": len(w.tensors),
                   "grad_dtype": w.grad_dtype, "code_bits": args.code_bits,
                   "refit_every": w.refit_every or None},
        "hbm_gbps": round(gbps, 1),
        "pct_peak_hbm": round(100.0 * gbps / PEAK_HBM_GBPS, 2),
        "step_ms": step_stats,
        "ceiling": dict(ceiling, dominant_kernel_pct_of_mix=round(
            100.0 * achieved / ceiling["mix_gbps"], 1)),
        "bytes_per_step": step_bytes,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": traffic,
                     "kernel": f"{dom['kind']}/vpl{dom['vpl']}/{dom['grad_dtype']}",
                     "bytes_per_launch": dom["bytes_per_launch"],
                     "mean_launch_ms": round(dom_ms, 4)},
        "kernels": [{k: (round(v, 4) if isinstance(v, float) else v) for k, v in c.items()}
                    for c in classes],
        "init_s": round(init_s, 3),
        "wall_s_timed": round(wall, 3),
        "state_bytes": {"persistent": persistent, "workspace": workspace},
        "source_hash": kernel_source_hash(),
    }
    if not args.no_adamw and not w.n_blocks:
        line["adamw"] = adamw_comparator(torch, w, params, grads, min(args.steps, 20),
                                         persistent, persistent + workspace, ms_per_step)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, params, grads[t % 2], st, args.cpu_sample_elems,
                                            t + 1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
