"""GPU parity of the five workloads at full size, in the configuration bench.py times.

* ``gpt2_125m``: every element of two teacher-forced steps, periods of every tensor.
* ``gpt2_1b`` and ``llama3_1p5b`` with 8-bit codes: every element of three steps and
  every period, in tests/test_gpu_full_size.py. Here the Llama-3 shape with 4-bit codes:
  whole-model steps, every output of sampled blocks checked against the oracle (first
  and last two blocks of every tensor plus a seeded random 0.2 %).
* ``stress_4b``: 4e9 elements (int64 indexing) in 1e6 explicit blocks, sampled as
  follows: a seeded random 1 % of blocks, every block under 128 elements, the first and
  last 100 blocks and the 100 largest; two steps, the second refitting the codebook on
  its gradients inside the step (gefen_step_fit: the histogram the step kernels take is
  checked exactly, as is the histogram kernel's, and the DP codebook bit-identical), and
  the step after the refit (decode with the old codebook, encode with the new one). The other reading of its block sizes
  (log-uniform sizes drawn until 4e9 is covered) is checked the same way over two steps.

Blocks are independent in the step, so a sample checks its blocks completely.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _free():
    gc.collect()
    torch.cuda.empty_cache()


class Sampled:
    """Teacher-forced checks on selected blocks of a whole-model state."""

    def __init__(self, st, params, offsets, blocks):
        from parity import Run
        self.st = st
        self.params = params
        self.offsets = offsets          # per tensor: tensor-relative block offsets
        self.blocks = blocks            # per tensor: sorted block indices to check
        lay = st.layout()
        self.code_off = lay["code_offsets"]
        self.blk_idx = lay["block_index"]
        # element ranges of the sample, and their offsets inside the sample
        self.elem_idx, self.sub_offs = [], []
        for i, b in enumerate(blocks):
            offs = offsets[i]
            lens = offs[b + 1] - offs[b]
            self.elem_idx.append(np.concatenate([np.arange(offs[j], offs[j + 1]) for j in b])
                                 if len(b) else np.zeros(0, np.int64))
            self.sub_offs.append(np.concatenate([[0], np.cumsum(lens)]).astype(np.int64))
        self._check = Run.check

    def snapshot(self):
        torch.cuda.synchronize()
        from parity import unpack_codes
        codes = torch.from_numpy(unpack_codes(self.st.read(gf.STATE_CODES).cpu().numpy(),
                                              self.st.k))
        scale = self.st.read(gf.STATE_SCALE)
        v = self.st.read(gf.STATE_V)
        snap = {"theta": [], "codes": [], "s": [], "v": [],
                "cb_dec": self.st.read(gf.STATE_CB_DEC).cpu().numpy().astype(np.float64),
                "cb_enc": self.st.read(gf.STATE_CB_ENC).cpu().numpy().astype(np.float64)}
        for i, p in enumerate(self.params):
            ei = torch.from_numpy(self.elem_idx[i]).to(p.device)
            bi = torch.from_numpy(np.asarray(self.blocks[i], dtype=np.int64)).to(p.device)
            snap["theta"].append(p.reshape(-1)[ei].double().cpu().numpy())
            snap["codes"].append(codes[self.code_off[i] + ei.cpu()].numpy())
            snap["s"].append(scale[self.blk_idx[i] + bi].double().cpu().numpy())
            snap["v"].append(v[self.blk_idx[i] + bi].double().cpu().numpy())
        del codes, scale, v
        return snap

    def grads_sample(self, grads):
        out = []
        for i, g in enumerate(grads):
            ei = torch.from_numpy(self.elem_idx[i]).to(g.device)
            out.append(g.reshape(-1)[ei])
        return out

    def oracle(self, pre, gs, lr, betas, eps, wd, t):
        from parity import grad_bits
        ref = {"theta": [], "codes": [], "s": [], "v": [], "m": []}
        for i in range(len(self.params)):
            th, cq = pre["theta"][i].copy(), pre["codes"][i].copy()
            s, v = pre["s"][i].copy(), pre["v"][i].copy()
            m = np.zeros_like(th)
            if th.size:
                oracle.step_blocks(th, grad_bits(gs[i]), cq, s, v, self.sub_offs[i],
                                   pre["cb_dec"], pre["cb_enc"], lr, betas[0], betas[1], eps, wd,
                                   t, m_out=m)
            for key, val in (("theta", th), ("codes", cq), ("s", s), ("v", v), ("m", m)):
                ref[key].append(val)
        return ref

    def step(self, grads, lr, betas, eps, wd, t, where, fit=False):
        pre = self.snapshot()
        gs = self.grads_sample(grads)
        self.st.step(self.params, grads, lr, betas, eps, wd, t, fit=fit)
        post = self.snapshot()
        ref = self.oracle(pre, gs, lr, betas, eps, wd, t)
        shim = type("S", (), {})()
        shim.params = [None] * len(self.params)
        shim.offsets = self.sub_offs
        return self._check(shim, pre, post, ref, gs, lr, betas, eps, wd, t, where)


def _uniform_offsets(params, periods):
    return [np.arange(0, p.numel() + 1, per, dtype=np.int64) for p, per in zip(params, periods)]


def _sample_uniform(offsets, frac, seed):
    rng = np.random.default_rng(seed)
    out = []
    for offs in offsets:
        nb = offs.size - 1
        pick = set(range(min(2, nb))) | set(range(max(0, nb - 2), nb))
        k = max(2, int(frac * nb))
        pick |= set(rng.choice(nb, size=min(k, nb), replace=False).tolist())
        out.append(np.array(sorted(pick), dtype=np.int64))
    return out


def _check_periods(w, grads, periods, which):
    from parity import grad_bits
    for i in which:
        _, _, per = oracle.partition(grad_bits(grads[i]), w.eps)
        assert periods[i] == per, (w.tensors[i].name, periods[i], per)


def test_gpt2_125m_full_coverage():
    from parity import Run
    dev = _dev()
    w = W.get("gpt2_125m")
    fields = W.scale_fields(w)
    params = W.init_params(w, dev)
    g1 = W.make_grads(w, fields, 1, dev)
    run = Run(params, g1, eps_part=w.eps)
    _check_periods(w, g1, run.periods, range(len(w.tensors)))
    hp = (w.lr, w.betas, w.eps, w.wd)
    for t in (1, 2):
        run.teacher_forced_step(W.make_grads(w, fields, t, dev), *hp, t, where=f"gpt2_125m t={t}")
    del run, params, g1
    _free()


@pytest.mark.parametrize("name,code_bits", [("llama3_1p5b", 4)])
def test_large_shapes_sampled(name, code_bits):
    """Whole-model steps at full size with two codes per byte at the Llama-3 shape (its
    periods are those of the 8-bit case, checked in full elsewhere)."""
    dev = _dev()
    w = W.get(name)
    fields = W.scale_fields(w)
    params = W.init_params(w, dev)
    g1 = W.make_grads(w, fields, 1, dev)
    st = gf.GefenState(g1, eps_part=w.eps, code_bits=code_bits)
    periods = st.periods
    offsets = _uniform_offsets(params, periods)
    smp = Sampled(st, params, offsets, _sample_uniform(offsets, 0.002, seed=w.index))
    hp = (w.lr, w.betas, w.eps, w.wd)
    g = g1
    for t in (1, 2):
        if t > 1:
            g = W.make_grads(w, fields, t, dev)
        rep = smp.step(g, *hp, t, where=f"{name} cb{code_bits} t={t}")
        assert rep["codes"] > 1_000_000
    del st, params, g1, g, smp
    _free()


def _stress_sample(offs, seed):
    sizes = np.diff(offs)
    nb = sizes.size
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(nb, size=nb // 100, replace=False).tolist())
    pick |= set(np.nonzero(sizes < 128)[0].tolist())
    pick |= set(range(100)) | set(range(nb - 100, nb))
    pick |= set(np.argsort(-sizes, kind="stable")[:100].tolist())
    return np.array(sorted(pick), dtype=np.int64)


def test_stress_4b_sampled_with_refit():
    from parity import grad_bits
    dev = _dev()
    w = W.get("stress_4b")
    offs = W.stress_block_offsets(w.numel, w.n_blocks)
    bsc = W.stress_block_scales(w.n_blocks)
    params = W.init_params(w, dev)
    g1 = W.make_grads(w, W.scale_fields(w), 1, dev, block_scales=bsc, offsets=offs)
    st = gf.GefenState(g1, block_offsets=offs, eps_part=w.eps)
    blocks = _stress_sample(offs, seed=5)
    smp = Sampled(st, params, [offs], [blocks])
    hp = (w.lr, w.betas, w.eps, w.wd)
    smp.step(g1, *hp, 1, where="stress t=1")
    del g1
    _free()
    g2 = W.make_grads(w, W.scale_fields(w), 2, dev, block_scales=bsc, offsets=offs)
    # step 2 refits on g2 inside the step (gefen_step_fit): the histogram the step kernels
    # took equals the oracle's exactly, and so does the standalone histogram kernel's; the
    # DP codebook is bit-identical (a sampled histogram is not enough for the DP, so the
    # oracle histogram is built over all blocks in chunks)
    smp.step(g2, *hp, 2, where="stress t=2 (refit inside the step)", fit=True)
    h_fit = st.read(gf.STATE_HIST).cpu().numpy().view(np.uint64)
    h_gpu = st.histogram(g2).cpu().numpy().view(np.uint64)
    h_ref = np.zeros(16 * 256, dtype=np.uint64)
    chunk_blocks = 50_000
    for b0 in range(0, w.n_blocks, chunk_blocks):
        b1 = min(w.n_blocks, b0 + chunk_blocks)
        e0, e1 = int(offs[b0]), int(offs[b1])
        gb = grad_bits(g2[0][e0:e1])
        oracle.histogram_blocks(gb, offs[b0:b1 + 1] - e0, 16 * 256, h_ref)
    np.testing.assert_array_equal(h_fit, h_ref)
    np.testing.assert_array_equal(h_gpu, h_ref)
    cb_ref, _, _, _ = oracle.dp_codebook(h_ref, 256)
    torch.cuda.synchronize()
    enc = st.read(gf.STATE_CB_ENC).cpu().numpy()
    np.testing.assert_array_equal(enc, cb_ref.astype(np.float32))
    rep = smp.step(g2, *hp, 3, where="stress t=3 (after refit)")
    assert rep["codes"] > 10_000_000
    np.testing.assert_array_equal(st.read(gf.STATE_CB_DEC64).cpu().numpy(), cb_ref)
    del st, params, g2, smp
    _free()


def test_stress_sequential_variant_sampled():
    """The other reading of the stress block sizes: log-uniform [64, 65536] drawn until
    4e9 elements are covered (about 4.2e5 blocks, the largest at 65536, a short last
    block). Two teacher-forced steps on the same kind of sample."""
    dev = _dev()
    w = W.get("stress_4b")
    offs = W.stress_block_offsets(w.numel, variant="sequential")
    nb = offs.size - 1
    assert 400_000 < nb < 450_000 and np.diff(offs).max() <= 65536
    bsc = W.stress_block_scales(nb)
    params = W.init_params(w, dev)
    g1 = W.make_grads(w, W.scale_fields(w), 1, dev, block_scales=bsc, offsets=offs)
    st = gf.GefenState(g1, block_offsets=offs, eps_part=w.eps)
    smp = Sampled(st, params, [offs], [_stress_sample(offs, seed=7)])
    hp = (w.lr, w.betas, w.eps, w.wd)
    smp.step(g1, *hp, 1, where="stress sequential t=1")
    del g1
    _free()
    g2 = W.make_grads(w, W.scale_fields(w), 2, dev, block_scales=bsc, offsets=offs)
    rep = smp.step(g2, *hp, 2, where="stress sequential t=2")
    assert rep["codes"] > 10_000_000
    del st, params, g2, smp
    _free()


@pytest.mark.parametrize("code_bits", [8, 4])
def test_gpt2_125m_persistent_state_accounting(code_bits):
    """The library's persistent state on the GPT-2 125M shapes, with the periods it
    infers: exactly codes + 8 bytes per block + two codebook slots, and, at 8 bits, the
    x0.25 of parameter memory that the paper's memory table prints
    (tests/golden/optimizer_state_memory.txt)."""
    from test_memory_accounting import _golden, codebook_bytes
    dev = _dev()
    w = W.get("gpt2_125m")
    g1 = W.make_grads(w, W.scale_fields(w), 1, dev)
    st = gf.GefenState(g1, eps_part=w.eps, code_bits=code_bits)
    lay = st.layout()
    persistent, _ = st.state_bytes()
    codes = sum((t.numel + 31) // 32 * 32 for t in w.tensors) * code_bits // 8
    assert lay["code_bytes"] == codes
    assert persistent == codes + 8 * lay["total_blocks"] + codebook_bytes(1 << code_bits)
    if code_bits == 8:
        assert round(persistent / (4 * w.numel), 2) == _golden()["gpt2_125m_gefen_persistent"][0]
    del st, g1
    _free()


@pytest.mark.parametrize("code_bits", [8, 4])
def test_uniform_tensor_beyond_2p31_elements_sampled(code_bits):
    """One bf16 tensor of 2048 x 1,048,600 elements (2^31 + 49,152) with period 2048, so
    the register kernel and the state tables index past 2^31 elements (the init
    histogram and fit run over all of them too). Two steps; sampled blocks (the first two, the last 100, those around element 2^31,
    and a seeded random 0.01 %) checked completely against the oracle."""
    dev = _dev()
    p, nb = 2048, 1_048_600
    n = p * nb
    assert n > 2 ** 31
    gen = torch.Generator(device=dev)
    gen.manual_seed(71)
    params = [torch.randn(n, device=dev, generator=gen) * 0.02]
    row_scale = torch.exp(torch.empty(nb, device=dev).uniform_(np.log(1e-3), 0, generator=gen))

    def grads(t):
        g = torch.empty(n, device=dev, dtype=torch.bfloat16)
        gen.manual_seed(1000 + t)
        for r0 in range(0, nb, 1 << 17):      # in slices, to bound the float32 temporary
            r1 = min(nb, r0 + (1 << 17))
            x = torch.randn((r1 - r0) * p, device=dev, generator=gen)
            g[r0 * p:r1 * p] = (x.view(r1 - r0, p) * row_scale[r0:r1, None]).reshape(-1).bfloat16()
        return [g]

    g1 = grads(1)
    st = gf.GefenState(g1, period_override=[p], code_bits=code_bits)
    offs = _uniform_offsets(params, [p])
    mid = 2 ** 31 // p
    rng = np.random.default_rng(5)
    pick = set(range(2)) | set(range(nb - 100, nb)) | set(range(mid - 3, mid + 3))
    pick |= set(rng.choice(nb, size=nb // 10000, replace=False).tolist())
    blocks = [np.array(sorted(pick), dtype=np.int64)]
    smp = Sampled(st, params, offs, blocks)
    hp = (1e-3, (0.9, 0.999), 1e-8, 0.1)
    smp.step(g1, *hp, 1, where="2^31+ t=1")
    del g1
    _free()
    smp.step(grads(2), *hp, 2, where="2^31+ t=2")
    st.close()
    del params, smp
    _free()
