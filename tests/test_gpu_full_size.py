"""Every element of the GPT-2 1B and Llama-3 1.5B shapes against the oracle, at full
size, in the launch configuration bench.py times (one whole-model gefen_step).

* Block inference (Sec. 5.1, Alg. 2): the period of every tensor, the embedding and
  output tables included, against the oracle's partition of the same gradient, one
  worker process per tensor.
* Steps (Alg. 1), teacher-forced: t = 1 and 2 (codes filling from zero), and t = 50,
  a steady state reached after 47 unchecked steps. Every output of every block -- codes,
  scales, second moments, parameters -- passes the parity gates (tests/gates.py). The
  oracle runs over disjoint whole-block ranges in worker processes
  (tests/oracle_pool.py), loaded with the library's state before the step.
"""
import gc
import os

import numpy as np
import pytest
import torch

import oracle
import oracle_pool
import workloads as W

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")

PIECE_ELEMS = 8 << 20   # elements per step task (whole blocks; one larger block alone)


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _nproc():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _flat(tensors, np_dtype):
    out = np.empty(sum(t.numel() for t in tensors), dtype=np_dtype)
    e = 0
    for t in tensors:
        n = t.numel()
        if t.dtype == torch.bfloat16:
            out[e:e + n] = t.detach().reshape(-1).view(torch.int16).cpu().numpy().view(np.uint16)
        else:
            out[e:e + n] = t.detach().reshape(-1).cpu().numpy()
        e += n
    return out


class FullRun:
    def __init__(self, name):
        dev = _dev()
        self.w = W.get(name)
        self.dev = dev
        self.fields = W.scale_fields(self.w)
        self.params = W.init_params(self.w, dev)
        self.g1 = W.make_grads(self.w, self.fields, 1, dev)
        self.st = gf.GefenState(self.g1, eps_part=self.w.eps)
        self.periods = self.st.periods
        lay = self.st.layout()
        self.code_off = lay["code_offsets"]
        self.blk_idx = lay["block_index"]
        self.numel = [p.numel() for p in self.params]
        self.elem_off = np.concatenate([[0], np.cumsum(self.numel)]).astype(np.int64).tolist()
        self.t = 0
        self.hp = (self.w.lr, self.w.betas, self.w.eps, self.w.wd)

    def grads(self, t):
        return self.g1 if t == 1 else W.make_grads(self.w, self.fields, t, self.dev)

    def _codes_flat(self):
        from parity import unpack_codes
        codes = unpack_codes(self.st.read(gf.STATE_CODES).cpu().numpy(), self.st.k)
        return np.concatenate([codes[c:c + n] for c, n in zip(self.code_off, self.numel)])

    def _write_state(self, job, tag):
        torch.cuda.synchronize()
        oracle_pool.save(job, f"theta_{tag}", _flat(self.params, np.float32))
        oracle_pool.save(job, f"codes_{tag}", self._codes_flat())
        oracle_pool.save(job, f"s_{tag}", self.st.read(gf.STATE_SCALE).cpu().numpy())
        oracle_pool.save(job, f"v_{tag}", self.st.read(gf.STATE_V).cpu().numpy())

    def advance(self, t_target):
        """Unchecked steps until the next step is t_target."""
        while self.t + 1 < t_target:
            self.t += 1
            self.st.step(self.params, self.grads(self.t), *self.hp, self.t)
        torch.cuda.synchronize()

    def checked_step(self, t):
        self.advance(t)
        assert self.t + 1 == t
        n = self.elem_off[-1]
        job = oracle_pool.make_dir(24 * n)
        try:
            grads = self.grads(t)
            self._write_state(job, "pre")
            oracle_pool.save(job, "grad", _flat(grads, np.uint16 if self.w.grad_dtype == "bf16"
                                                else np.float32))
            oracle_pool.save(job, "cb_dec",
                             self.st.read(gf.STATE_CB_DEC).cpu().numpy().astype(np.float64))
            oracle_pool.save(job, "cb_enc",
                             self.st.read(gf.STATE_CB_ENC).cpu().numpy().astype(np.float64))
            self.st.step(self.params, grads, *self.hp, t)
            self.t = t
            del grads
            self._write_state(job, "post")
            tasks, sizes = [], []
            for i, (n_i, p) in enumerate(zip(self.numel, self.periods)):
                offs = np.arange(0, n_i + 1, p, dtype=np.int64)
                oracle_pool.save(job, f"offs_{i}", offs)
                nb = offs.size - 1
                per = max(1, PIECE_ELEMS // p)
                for b0 in range(0, nb, per):
                    b1 = min(nb, b0 + per)
                    tasks.append({"kind": "step", "tensor": i, "b0": b0, "b1": b1})
                    sizes.append((b1 - b0) * p)
            lr, (b1_, b2_), eps, wd = self.hp
            meta = {"elem_off": self.elem_off, "blk_off": [int(b) for b in self.blk_idx],
                    "hp": {"lr": lr, "b1": b1_, "b2": b2_, "eps": eps, "wd": wd, "t": t},
                    "where": f"{self.w.name} t={t}"}
            res = oracle_pool.run(job, meta, tasks, sizes, _nproc(), timeout=900)
        finally:
            import shutil
            shutil.rmtree(job, ignore_errors=True)
        bad = [r for r in res if not r["ok"]]
        assert not bad, bad[0]["error"]
        assert len(res) == len(tasks)
        rep = {"codes": sum(r["result"]["codes"] for r in res),
               "code_ties": sum(r["result"]["code_ties"] for r in res),
               "max_theta_gate": max(r["result"]["max_theta_gate"] for r in res),
               "max_rel_v": max(r["result"]["max_rel_v"] for r in res)}
        assert rep["codes"] == n, (rep["codes"], n)
        print(f"{self.w.name} t={t}: every element checked: {rep}", flush=True)
        return rep

    def close(self):
        self.st.close()
        self.params = self.g1 = None
        gc.collect()
        torch.cuda.empty_cache()


@pytest.fixture(scope="module", params=["gpt2_1b", "llama3_1p5b"])
def full(request):
    run = FullRun(request.param)
    yield run
    run.close()


@pytest.mark.timeout(900)
def test_every_period(full):
    """Alg. 2 at full size: every tensor's period equals the oracle's on the same
    gradient bits (the embedding and output tables take the partition kernel's sub-chunk
    mode)."""
    n = full.elem_off[-1]
    job = oracle_pool.make_dir(2 * n)
    try:
        oracle_pool.save(job, "grad", _flat(full.g1, np.uint16))
        tasks = [{"kind": "partition", "tensor": i} for i in range(len(full.numel))]
        sizes = [n_i * max(1, oracle.divisors(n_i).size) for n_i in full.numel]
        meta = {"elem_off": full.elem_off, "numel": full.numel, "eps_part": full.w.eps}
        res = oracle_pool.run(job, meta, tasks, sizes, _nproc(), timeout=900)
    finally:
        import shutil
        shutil.rmtree(job, ignore_errors=True)
    assert len(res) == len(tasks)
    for r in res:
        i = r["task"]["tensor"]
        assert r["ok"]
        assert full.periods[i] == r["result"]["period"], (full.w.tensors[i].name,
                                                         full.periods[i], r["result"]["period"])
    big = max(range(len(full.numel)), key=lambda i: full.numel[i])
    print(f"{full.w.name}: {len(res)} periods equal the oracle's; largest tensor "
          f"{full.w.tensors[big].name} ({full.numel[big]} elements) period {full.periods[big]}",
          flush=True)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("t", [1, 2, 50])
def test_every_element_of_a_step(full, t):
    rep = full.checked_step(t)
    assert rep["max_theta_gate"] <= 1.0
