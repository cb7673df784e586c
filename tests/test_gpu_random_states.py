"""Seeded random states against the oracle: each seed draws a few tensors of random sizes
and gradient types, with either explicit block tables (block lengths from every kernel
class's range: lane per block, register runs, one workgroup, split over workgroups) or
uniform periods (small, register-held, streamed, split), at 8- or 4-bit codes. Two
teacher-forced steps (Alg. 1), then a step that refits the codebook on its own gradients
(Alg. 3) checked bit for bit against a step and a separate fit on a second state, then a
teacher-forced step that decodes with the old codebook and encodes with the new one.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")

HP = (1e-3, (0.9, 0.999), 1e-8, 0.1)


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _draw(seed):
    rng = np.random.default_rng(7000 + seed)
    code_bits = int(rng.choice([8, 4]))
    explicit = bool(rng.integers(2))
    sizes, offs, pers, dts = [], [], [], []
    for _ in range(int(rng.integers(1, 5))):
        dts.append(torch.float32 if rng.integers(2) else torch.bfloat16)
        if explicit:
            ranges = [(1, 33), (33, 2043), (2043, 65537), (65537, 140000)]
            lens = [int(rng.integers(*ranges[int(rng.choice(4, p=[0.3, 0.45, 0.2, 0.05]))]))
                    for _ in range(int(rng.integers(1, 60)))]
            sizes.append(int(sum(lens)))
            offs.append(lens)
        else:
            p = int(rng.choice([1, 3, 4, 20, 32, 64, 768, 999, 2048, 8192, 8196, 70000]))
            nb = int(rng.integers(1, 200 if p < 8192 else 6))
            sizes.append(p * nb)
            pers.append(p)
    block_offsets = None
    if explicit:
        block_offsets = np.concatenate([[0], np.cumsum(np.concatenate(offs))]).astype(np.int64)
    return code_bits, sizes, dts, block_offsets, (pers if not explicit else None)


def _grad(n, seed, dt, dev):
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    g = torch.randn(n, generator=gen, device=dev)
    u = torch.rand(n, generator=gen, device=dev).clamp_min(1e-4)
    return (g * u).to(dt)   # a normal times a uniform: a spread of magnitudes


@pytest.mark.parametrize("seed", range(40))
def test_random_state(seed):
    from parity import Run
    dev = _dev()
    code_bits, sizes, dts, offs, pers = _draw(seed)
    kw = dict(code_bits=code_bits)
    if offs is not None:
        kw["block_offsets"] = offs
    else:
        kw["period_override"] = pers
    gr = lambda t: [_grad(n, 100 * seed + 10 * i + t, dt, dev)
                    for i, (n, dt) in enumerate(zip(sizes, dts))]
    p0 = [torch.randn(n, device=dev) * 0.02 for n in sizes]
    run = Run([p.clone() for p in p0], gr(1), **kw)
    where = f"seed {seed} ({code_bits}-bit, {'explicit' if offs is not None else 'periods'})"
    for t in (1, 2):
        run.teacher_forced_step(gr(t), HP[0], HP[1], HP[2], HP[3], t, where=f"{where} step {t}")
    # step 3 refits inside the step; a second state does step then fit
    other = gf.GefenState(gr(1), **kw)
    q = [p.clone() for p in p0]
    for t in (1, 2):
        other.step(q, gr(t), *HP, t)
    g3 = gr(3)
    run.state.step(run.params, g3, *HP, 3, fit=True)
    other.step(q, g3, *HP, 3)
    other.fit_codebook(g3)
    torch.cuda.synchronize()
    for a, b in zip(run.params, q):
        assert torch.equal(a, b), where
    for which in (gf.STATE_CODES, gf.STATE_SCALE, gf.STATE_V, gf.STATE_CB_DEC64, gf.STATE_CB_ENC):
        x, y = run.state.read(which), other.read(which)
        if x.dtype == torch.float64:
            x, y = x.view(torch.uint8), y.view(torch.uint8)
        assert torch.equal(x, y), (where, which)
    run.teacher_forced_step(gr(4), HP[0], HP[1], HP[2], HP[3], 4, where=f"{where} step 4")
