"""4-bit momentum codes (k = 16, 256 histogram bins, two codes per byte) against the
oracle, teacher-forced, through the C ABI.

Code j of the state lives in byte j / 2 (low nibble for even j). Blocks of odd length
or at odd offsets share a byte with their neighbour, which another lane or workgroup
updates in the same launch; these cases (odd periods, explicit irregular blocks, block
size 1 and 3, blocks split across workgroups at odd offsets) are the ones that check
the shared-byte updates.
"""
import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _grad(n, seed, dtype, rows=None, dev=None):
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    g = torch.randn(n, generator=gen, device=dev)
    if rows:
        sc = torch.exp(torch.empty(rows, device=dev).uniform_(np.log(1e-3), 0, generator=gen))
        g = (g.view(rows, -1) * sc[:, None]).reshape(-1)
    return g.to(dtype)


HP = (1e-3, (0.9, 0.999), 1e-8, 0.1)


def _steps(run, grads_fn, steps, where, t0=1):
    for t in range(t0, t0 + steps):
        run.teacher_forced_step(grads_fn(t), *HP, t, where=f"{where} step {t}")


PERIODS4 = [(1, 3001), (2, 701), (3, 513), (4, 1000), (5, 301), (12, 257), (33, 41),
            (64, 70), (768, 19), (999, 40), (2048, 9), (5003, 9), (8192, 3), (8196, 2),
            (40000, 2), (65537, 2), (200001, 2)]


@pytest.mark.parametrize("p,nb", PERIODS4)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_four_bit_uniform_periods(p, nb, dtype):
    from parity import Run
    dev = _dev()
    n = p * nb
    theta = torch.randn(n, device=dev) * 0.02
    run = Run([theta], [_grad(n, 1, dtype, rows=nb, dev=dev)], period_override=[p],
              code_bits=4)
    assert run.k == 16 and run.periods == [p]
    _steps(run, lambda t: [_grad(n, 100 + t, dtype, rows=nb, dev=dev)], 3, f"4-bit p={p}")


def test_four_bit_explicit_irregular_blocks():
    """Block boundaries at every parity; small (lane), streamed and split blocks."""
    from parity import Run
    dev = _dev()
    rng = np.random.default_rng(11)
    sizes = np.concatenate([[1, 1, 2, 3, 5, 31, 32, 33, 63, 65, 1001, 9001, 70001, 131075],
                            rng.integers(1, 40, size=400), rng.integers(40, 3000, size=80)])
    rng.shuffle(sizes)
    n1 = int(sizes[:250].sum())
    n = int(sizes.sum())
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    params = [torch.randn(n1, device=dev) * 0.02, torch.randn(n - n1, device=dev) * 0.02]
    gr = lambda t: [_grad(n1, 20 + t, torch.bfloat16, dev=dev),
                    _grad(n - n1, 60 + t, torch.bfloat16, dev=dev)]
    run = Run(params, gr(1), block_offsets=offs, code_bits=4)
    _steps(run, gr, 3, "4-bit explicit")


def test_four_bit_misaligned_tensors():
    from parity import Run
    dev = _dev()
    p, nb = 2048, 5
    n = p * nb
    pbuf = torch.randn(n + 3, device=dev) * 0.02
    theta = pbuf[1:1 + n]
    gbufs = {t: _grad(n + 1, 30 + t, torch.bfloat16, dev=dev) for t in range(1, 4)}
    run = Run([theta], [gbufs[1][1:]], period_override=[p], code_bits=4)
    _steps(run, lambda t: [gbufs[t][1:]], 3, "4-bit misaligned")


def test_four_bit_mixed_tensors():
    from parity import Run
    dev = _dev()
    specs = [(2048, 12, torch.bfloat16), (768, 7, torch.float32), (12, 300, torch.bfloat16),
             (3, 501, torch.float32), (999, 6, torch.bfloat16), (40000, 2, torch.float32),
             (7, 77, torch.bfloat16)]
    params = [torch.randn(p * nb, device=dev) * 0.02 for p, nb, _ in specs]
    gr = lambda t: [_grad(p * nb, 900 + 10 * i + t, dt, dev=dev)
                    for i, (p, nb, dt) in enumerate(specs)]
    run = Run(params, gr(1), period_override=[p for p, _, _ in specs], code_bits=4)
    _steps(run, gr, 3, "4-bit mixed")


def test_four_bit_block_size_one_is_adamw():
    """p = 1: m / s' = +-1 are the forced end entries, so the 4-bit step is AdamW too.
    Free-running against torch.optim.AdamW (fp32); every byte holds two blocks."""
    dev = _dev()
    n = 40_001
    torch.manual_seed(1)
    theta0 = torch.randn(n, device=dev) * 0.02
    p_gef = theta0.clone()
    p_ref = torch.nn.Parameter(theta0.clone())
    opt = torch.optim.AdamW([p_ref], lr=1e-3, betas=(0.9, 0.999), eps=1e-8,
                            weight_decay=0.1, foreach=False)
    g1 = torch.randn(n, device=dev)
    st = gf.GefenState([g1], period_override=[1], code_bits=4)
    for t in range(1, 21):
        g = g1 if t == 1 else torch.randn(n, device=dev)
        st.step([p_gef], [g], 1e-3, (0.9, 0.999), 1e-8, 0.1, t)
        p_ref.grad = g.clone()
        opt.step()
    torch.cuda.synchronize()
    a, b = p_gef.double(), p_ref.detach().double()
    err = (a - b).abs()
    assert (err <= 1e-5 * b.abs() + 1e-5 * 1e-3).all(), float((err / (b.abs() + 1e-3)).max())


def test_four_bit_refit_and_checkpoint():
    """Refit at 4 bits (256-bin histogram, exact 16-entry DP) and a bitwise resume."""
    from parity import Run, grad_bits
    import oracle
    dev = _dev()
    w = W.get("tiny")
    fields = W.scale_fields(w)
    params = W.init_params(w, dev)
    gr = lambda t: W.make_grads(w, fields, t, dev)
    run = Run(params, gr(1), code_bits=4)
    st = run.state
    assert st.layout()["code_bytes"] == sum((p.numel() + 31) // 32 * 16 for p in params)
    _steps(run, gr, 2, "4-bit tiny")
    g3 = gr(3)
    h = st.histogram(g3).cpu().numpy().view(np.uint64)
    assert h.size == 256
    h_ref = np.zeros(256, dtype=np.uint64)
    for p, g, per in zip(params, g3, run.periods):
        oracle.histogram_uniform(grad_bits(g), per, 256, h_ref)
    np.testing.assert_array_equal(h, h_ref)
    st.fit_codebook(g3)
    cb_ref, _, _, _ = oracle.dp_codebook(h_ref, 16)
    np.testing.assert_array_equal(st.read(gf.STATE_CB_ENC).cpu().numpy(),
                                  cb_ref.astype(np.float32))
    _steps(run, gr, 2, "4-bit after refit", t0=3)
    ck = st.export(device=torch.device("cpu"))
    pb = [p.clone() for p in params]
    for t in (5, 6):
        st.step(params, gr(t), *HP, t)
    b = gf.GefenState(gr(1), code_bits=4)
    b.import_(ck.to(dev))
    for t in (5, 6):
        b.step(pb, gr(t), *HP, t)
    for x, y in zip(params, pb):
        assert torch.equal(x, y)
    for which in (gf.STATE_CODES, gf.STATE_SCALE, gf.STATE_V):
        assert torch.equal(st.read(which), b.read(which))
