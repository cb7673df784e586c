"""The oracle over a full-size workload, in parallel worker processes.

Test infrastructure. A parent (a GPU test) writes the arrays a check needs into a job
directory -- the state before and after one library step, the gradient bits, block
offsets, hyperparameters -- and a task list. Worker processes
(``python tests/oracle_pool.py <dir> <k>``) take a share of the tasks; they import numpy,
the oracle and the gates only (no torch, no HIP library), and print one JSON line of
results. Blocks are independent in the step, so any run of whole blocks is checked
completely on its own; a partition task runs the oracle's Alg. 2 on one whole tensor.

Task kinds:

* ``{"kind": "step", "tensor": i, "b0": b0, "b1": b1}``: the oracle's step (Alg. 1) on
  blocks [b0, b1) of tensor i, loaded with the library's state before the step, then
  the parity gates against the library's state after it;
* ``{"kind": "partition", "tensor": i}``: the oracle's block inference (Sec. 5.1,
  Alg. 2) on tensor i's gradient; returns the period and every divisor's score.
"""
from __future__ import annotations

import json
import os
import shutil
import subprocess
import sys
import tempfile
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def make_dir(nbytes: int) -> str:
    """A job directory in /dev/shm when it has room for `nbytes`, else in the default
    temporary directory."""
    base = None
    if os.path.isdir("/dev/shm"):
        try:
            if shutil.disk_usage("/dev/shm").free > nbytes + (1 << 30):
                base = "/dev/shm"
        except OSError:
            pass
    return tempfile.mkdtemp(prefix="gefen_oracle_", dir=base)


def save(job_dir: str, name: str, a: np.ndarray):
    np.save(os.path.join(job_dir, name + ".npy"), np.ascontiguousarray(a))


def deal(tasks: list, sizes: list, nproc: int) -> list:
    """Tasks to workers, largest first, each to the least loaded worker."""
    shares = [[] for _ in range(nproc)]
    load = [0] * nproc
    for i in sorted(range(len(tasks)), key=lambda j: -sizes[j]):
        k = load.index(min(load))
        shares[k].append(tasks[i])
        load[k] += sizes[i]
    return [s for s in shares if s]


def run(job_dir: str, meta: dict, tasks: list, sizes: list, nproc: int, timeout: float):
    """Run the tasks over `nproc` workers; returns the results in task order of the
    workers' shares (each result carries its task). Raises if a worker fails."""
    shares = deal(tasks, sizes, nproc)
    with open(os.path.join(job_dir, "meta.json"), "w") as f:
        json.dump(dict(meta, shares=shares), f)
    procs = [subprocess.Popen([sys.executable, os.path.abspath(__file__), job_dir, str(k)],
                              stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
             for k in range(len(shares))]
    results = []
    errors = []
    t0 = time.time()
    t_end = t0 + timeout
    for k, p in enumerate(procs):
        try:
            out, err = p.communicate(timeout=max(1.0, t_end - time.time()))
        except subprocess.TimeoutExpired:
            for q in procs:
                q.kill()
            raise RuntimeError("oracle workers timed out")
        print(f"  oracle worker {k + 1}/{len(procs)} done after {time.time() - t0:.1f} s",
              flush=True)
        if p.returncode != 0:
            errors.append(err[-2000:])
            continue
        results.extend(json.loads(out.strip().splitlines()[-1]))
    if errors:
        raise RuntimeError("oracle worker failed:\n" + "\n".join(errors))
    return results


# ---------------------------------------------------------------------------- worker
def _load(job_dir, name):
    return np.load(os.path.join(job_dir, name + ".npy"), mmap_mode="r")


def _step_task(job_dir, meta, task):
    import gates
    import oracle
    i, b0, b1 = task["tensor"], task["b0"], task["b1"]
    e0, blk0 = meta["elem_off"][i], meta["blk_off"][i]
    offs = np.asarray(_load(job_dir, f"offs_{i}")[b0:b1 + 1], dtype=np.int64)
    lo, hi = int(offs[0]), int(offs[-1])
    rel = offs - lo
    sl = slice(e0 + lo, e0 + hi)
    bl = slice(blk0 + b0, blk0 + b1)
    g = np.array(_load(job_dir, "grad")[sl])
    pre_theta = np.asarray(_load(job_dir, "theta_pre")[sl], dtype=np.float64)
    pre_codes = np.array(_load(job_dir, "codes_pre")[sl])
    pre_s = np.asarray(_load(job_dir, "s_pre")[bl], dtype=np.float64)
    pre_v = np.asarray(_load(job_dir, "v_pre")[bl], dtype=np.float64)
    cb_dec = np.asarray(_load(job_dir, "cb_dec"), dtype=np.float64)
    cb_enc = np.asarray(_load(job_dir, "cb_enc"), dtype=np.float64)
    hp = meta["hp"]
    th, cq, s, v = pre_theta.copy(), pre_codes.copy(), pre_s.copy(), pre_v.copy()
    m = np.zeros_like(th)
    oracle.step_blocks(th, g, cq, s, v, rel, cb_dec, cb_enc, hp["lr"], hp["b1"], hp["b2"],
                       hp["eps"], hp["wd"], hp["t"], m_out=m)
    gd = (g.astype(np.float32) if g.dtype == np.float32 else
          (g.astype(np.uint32) << 16).view(np.float32)).astype(np.float64)
    rep = gates.check_tensor(
        pre_theta, pre_codes, pre_s,
        np.asarray(_load(job_dir, "theta_post")[sl], dtype=np.float64),
        np.array(_load(job_dir, "codes_post")[sl]),
        np.asarray(_load(job_dir, "s_post")[bl], dtype=np.float64),
        np.asarray(_load(job_dir, "v_post")[bl], dtype=np.float64),
        th, cq, s, v, m, gd, rel, cb_dec, cb_enc, hp["lr"], (hp["b1"], hp["b2"]),
        hp["eps"], hp["wd"], hp["t"], f"{meta.get('where', '')} tensor {i} blocks {b0}-{b1}")
    return rep


def _partition_task(job_dir, meta, task):
    import oracle
    i = task["tensor"]
    e0, n = meta["elem_off"][i], meta["numel"][i]
    g = np.array(_load(job_dir, "grad")[e0:e0 + n])
    divs, scores, per = oracle.partition(g, meta["eps_part"])
    return {"period": per, "divisors": divs.tolist(), "scores": scores.tolist()}


def _worker(job_dir: str, k: int):
    sys.path.insert(0, HERE)
    sys.path.insert(0, ROOT)
    with open(os.path.join(job_dir, "meta.json")) as f:
        meta = json.load(f)
    out = []
    for task in meta["shares"][k]:
        try:
            if task["kind"] == "step":
                res = _step_task(job_dir, meta, task)
            elif task["kind"] == "partition":
                res = _partition_task(job_dir, meta, task)
            else:
                raise ValueError(task["kind"])
            out.append({"task": task, "ok": True, "result": res})
        except AssertionError as e:
            out.append({"task": task, "ok": False, "error": str(e)})
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    _worker(sys.argv[1], int(sys.argv[2]))
