"""gefen_step_fit: one step (Alg. 1) and the codebook refit (Alg. 3) on the same gradients,
the histogram taken inside the step kernels of explicit and irregular blocks.

Against gefen_step followed by gefen_fit_codebook on a second state from the same start:
every state array, the parameters, both codebooks and the histogram equal bit for bit,
at the refit step and at the two steps after it (the new codebook encodes at the first
and is used for both at the second). The histogram also equals the oracle's on the same
gradient bits (Alg. 3), so the refit is pinned to the paper's definition and not only to
the library's other path. Cases take every kernel class: register runs of short explicit
blocks, one workgroup per block, small blocks one lane each, uniform blocks in
registers and huge blocks split over workgroups, with 8- and 4-bit codes.
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")

HP = (1e-3, (0.9, 0.999), 1e-8, 0.1)


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _grad(n, seed, heavy, dev):
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    g = torch.randn(n, generator=gen, device=dev)
    if heavy:   # a heavier tail than the start's, so that the refit changes the codebook
        u = torch.rand(n, generator=gen, device=dev).clamp_min(1e-6)
        g = g / u.sqrt()
    return g.to(torch.bfloat16)


def _explicit_offsets(seed):
    rng = np.random.default_rng(seed)
    sizes = np.concatenate([[1, 3, 32, 33, 65536, 65537, 9000, 2042, 2043],
                            rng.integers(1, 33, size=150),      # one lane per block
                            rng.integers(33, 600, size=400),    # register runs
                            rng.integers(600, 40000, size=40)])  # one workgroup per block
    rng.shuffle(sizes)
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)


def _case(name):
    """(tensor sizes, block offsets or None, period overrides or None)."""
    if name == "explicit":
        offs = _explicit_offsets(3)
        n = int(offs[-1])
        cut = int(offs[300])
        return [cut, n - cut], offs, None
    # uniform periods: one lane per block (20), registers (768), one workgroup per block
    # (999, odd), split over workgroups (200000)
    pers = [20, 768, 999, 200000]
    counts = [500, 40, 30, 2]
    return [p * c for p, c in zip(pers, counts)], None, pers


def _state(sizes, offs, pers, g, code_bits):
    kw = dict(code_bits=code_bits)
    if offs is not None:
        kw["block_offsets"] = offs
    else:
        kw["period_override"] = pers
    return gf.GefenState(g, **kw)


def _arrays(st, params):
    torch.cuda.synchronize()
    out = {f"param{i}": p.clone() for i, p in enumerate(params)}
    for name, w in (("codes", gf.STATE_CODES), ("scale", gf.STATE_SCALE), ("v", gf.STATE_V),
                    ("cb_dec", gf.STATE_CB_DEC64), ("cb_enc", gf.STATE_CB_ENC)):
        out[name] = st.read(w).clone()
    return out


def _assert_same(a, b, where):
    for key in a:
        assert torch.equal(a[key].view(torch.uint8) if a[key].dtype == torch.float64 else a[key],
                           b[key].view(torch.uint8) if b[key].dtype == torch.float64 else b[key]), \
            (where, key)


@pytest.mark.parametrize("code_bits", [8, 4])
@pytest.mark.parametrize("name", ["explicit", "periods"])
def test_step_fit_equals_step_then_fit(name, code_bits):
    from parity import grad_bits
    dev = _dev()
    sizes, offs, pers = _case(name)
    gr = lambda t: [_grad(n, 1000 * t + i, heavy=(t == 2), dev=dev) for i, n in enumerate(sizes)]
    g1 = gr(1)
    a = _state(sizes, offs, pers, g1, code_bits)
    b = _state(sizes, offs, pers, g1, code_bits)
    p0 = [torch.randn(n, device=dev) * 0.02 for n in sizes]
    pa = [p.clone() for p in p0]
    pb = [p.clone() for p in p0]
    a.step(pa, g1, *HP, 1)
    b.step(pb, g1, *HP, 1)
    g2 = gr(2)
    a.step(pa, g2, *HP, 2)
    a.fit_codebook(g2)
    b.step(pb, g2, *HP, 2, fit=True)
    _assert_same(_arrays(a, pa), _arrays(b, pb), f"{name} refit step")
    ha = a.read(gf.STATE_HIST).cpu().numpy().view(np.uint64)
    hb = b.read(gf.STATE_HIST).cpu().numpy().view(np.uint64)
    np.testing.assert_array_equal(ha, hb)
    # the histogram is the oracle's (Alg. 3) on the same gradient bits
    lay = b.layout()
    nb = 16 * lay["k"]
    h_ref = np.zeros(nb, dtype=np.uint64)
    periods = b.periods
    for i, g in enumerate(g2):
        if offs is not None:
            base = sum(sizes[:i])
            sel = offs[(offs >= base) & (offs <= base + sizes[i])] - base
        else:
            sel = np.arange(0, sizes[i] + 1, periods[i], dtype=np.int64)
        oracle.histogram_blocks(grad_bits(g), sel, nb, h_ref)
    np.testing.assert_array_equal(hb, h_ref)
    assert not torch.equal(b.read(gf.STATE_CB_ENC), b.read(gf.STATE_CB_DEC))
    for t in (3, 4):   # the new codebook encodes at 3, and is used for both at 4
        g = gr(t)
        a.step(pa, g, *HP, t)
        b.step(pb, g, *HP, t)
        _assert_same(_arrays(a, pa), _arrays(b, pb), f"{name} step {t}")


def test_step_fit_histogram_is_read_only():
    dev = _dev()
    g = [_grad(4096, 5, False, dev)]
    st = gf.GefenState(g)
    h = st.read(gf.STATE_HIST)
    assert h.numel() == 16 * st.k and int(h.sum()) == 4096   # the init fit's histogram
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.write(gf.STATE_HIST, h)
