"""GPU parity of the secondary kernels: block inference (Alg. 2), the normalised
histogram and the exact DP codebook (Alg. 3, App. D), against the float64 oracle.

Bars: periods exact (ties excepted: a deciding comparison within 1e-9 relative);
scores within 1e-9 relative (parallel float64 sums); histogram counts exact; DP
codebook, cost and status bit-identical (same float64 operations in the same order).
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _bits(g):
    from parity import grad_bits
    return grad_bits(g)


def _deciding_margin(divs, scores, period):
    """Smallest relative gap among the comparisons that decide the chosen period."""
    s = np.asarray(scores)
    margins = []
    for i in range(1, len(s) - 1):
        for j in (i - 1, i + 1):
            den = max(abs(s[i]), abs(s[j]), 1e-300)
            margins.append(abs(s[i] - s[j]) / den)
    return min(margins) if margins else 1.0


def _row_grad(rows, cols, seed, dtype, dev, heads=0):
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    z = torch.randn(rows, cols, generator=gen, device=dev)
    sc = torch.exp(torch.empty(rows, device=dev).uniform_(np.log(1e-3), 0, generator=gen))
    if heads:
        hs = torch.exp(torch.empty(rows // heads, device=dev).uniform_(np.log(1e-2), 0,
                                                                       generator=gen))
        sc = sc * hs.repeat_interleave(heads)
    return (z * sc[:, None]).to(dtype).reshape(-1)


CASES = [
    ("rows_768", (64, 768), torch.float32, 0),
    ("rows_2048_bf16", (96, 2048), torch.bfloat16, 0),
    ("heads_64", (256, 128), torch.float32, 64),
    ("rows_odd", (50, 999), torch.float32, 0),
    ("big_p", (4, 200_000), torch.float32, 0),          # sub-chunked block sums
    ("vector_1d", (1, 3072), torch.float32, 0),
]


@pytest.mark.parametrize("name,shape,dtype,heads", CASES)
def test_partition_scores_and_period(name, shape, dtype, heads):
    dev = _dev()
    g = _row_grad(shape[0], shape[1], sum(map(ord, name)), dtype, dev, heads)
    d_gpu, s_gpu, p_gpu = gf.partition_scores(g, 1e-8)
    d_ref, s_ref, p_ref = oracle.partition(_bits(g), 1e-8)
    np.testing.assert_array_equal(d_gpu, d_ref)
    np.testing.assert_allclose(s_gpu, s_ref, rtol=1e-9, atol=1e-300)
    if p_gpu != p_ref:
        assert _deciding_margin(d_ref, s_ref, p_ref) <= 1e-9, (p_gpu, p_ref)
    if dtype == torch.float32 and heads == 0 and shape[0] > 1:
        assert p_gpu == shape[1]


@pytest.mark.parametrize("n", [1, 97, 7919, 1 << 16])
def test_partition_degenerate_sizes(n):
    dev = _dev()
    g = torch.randn(n, device=dev)
    _, _, p = gf.partition_scores(g, 1e-8)
    assert p == oracle.partition(_bits(g), 1e-8)[2]
    c = torch.full((n,), 0.5, device=dev)
    assert gf.partition_scores(c, 1e-8)[2] == 1


def test_histogram_exact_uniform_and_explicit():
    dev = _dev()
    from parity import Run
    # uniform periods across the kernel classes, bf16 and fp32
    specs = [(2048, 7, torch.bfloat16), (768, 9, torch.float32), (3, 500, torch.float32),
             (40000, 2, torch.bfloat16), (4, 333, torch.float32)]
    params, grads, pers = [], [], []
    for i, (p, nb, dt) in enumerate(specs):
        n = p * nb
        params.append(torch.zeros(n, device=dev))
        g = torch.distributions.StudentT(3.0).sample((n,)).to(dev).to(dt)
        g.view(nb, p)[1] = 0   # a zero block is skipped
        grads.append(g)
        pers.append(p)
    run = Run(params, grads, period_override=pers)
    nb_bins = 16 * run.k
    h_ref = np.zeros(nb_bins, dtype=np.uint64)
    for i, g in enumerate(grads):
        oracle.histogram_blocks(_bits(g), run.offsets[i], nb_bins, h_ref)
    h_gpu = run.state.histogram(grads).cpu().numpy().view(np.uint64)
    np.testing.assert_array_equal(h_gpu, h_ref)


@pytest.mark.parametrize("k,nbins,fill", [(256, 4096, 0.6), (256, 4096, 1.0), (16, 256, 0.8),
                                          (256, 4096, 0.03), (16, 256, 0.02), (4, 64, 1.0)])
def test_dp_codebook_bit_identical(k, nbins, fill):
    dev = _dev()
    rng = np.random.default_rng(int(k * 1000 + nbins + fill * 100))
    hist = np.zeros(nbins, dtype=np.uint64)
    nz = rng.random(nbins) < fill
    hist[nz] = rng.integers(1, 10**6, size=int(nz.sum())).astype(np.uint64)
    hist[0] = max(hist[0], 1)
    hist[-1] = max(hist[-1], 1)
    cb_ref, cost_ref, _, st_ref = oracle.dp_codebook(hist, k)
    h = torch.from_numpy(hist.view(np.int64)).to(dev)
    cb, cost, st = gf.dp_codebook(h, k)
    assert st == st_ref
    np.testing.assert_array_equal(cb.cpu().numpy(), cb_ref)
    assert cost == cost_ref


def test_dp_from_gradient_histogram():
    """Full-size DP (k = 256, 4096 bins) on a realistic block-normalised histogram."""
    dev = _dev()
    x = torch.distributions.StudentT(3.0).sample((4000, 512))
    x = x / x.abs().amax(dim=1, keepdim=True)
    hist = torch.histc(x.reshape(-1), bins=4096, min=-1, max=1).to(torch.int64)
    hist_np = hist.numpy().astype(np.uint64)
    cb_ref, cost_ref, _, st_ref = oracle.dp_codebook(hist_np, 256)
    cb, cost, st = gf.dp_codebook(hist.to(dev), 256)
    assert st == st_ref == 0
    np.testing.assert_array_equal(cb.cpu().numpy(), cb_ref)
    assert cost == cost_ref


@pytest.mark.parametrize("gdtype", [torch.float32, torch.bfloat16])
def test_stream_mix_moves_every_byte(gdtype):
    """The streaming-ceiling pass (measurement support) touches every element: in each
    full 4-element vector lanes 0 and 3 gain the gradient, the ragged tail gains it
    element by element, and every code byte flips its low bit."""
    dev = _dev()
    n = 3 * 1024 + 4 * 77 + 3
    rng = np.random.default_rng(5)
    th0 = rng.standard_normal(n).astype(np.float32)
    g = torch.from_numpy(rng.standard_normal(n).astype(np.float32)).to(gdtype)
    c0 = rng.integers(0, 256, n, dtype=np.uint8)
    theta = torch.from_numpy(th0).to(dev)
    codes = torch.from_numpy(c0).to(dev)
    gf.stream_mix(theta, g.to(dev), codes)
    torch.cuda.synchronize()
    gd = g.float().numpy()
    ref = th0.copy()
    full = n // 4 * 4
    ref[0:full:4] += gd[0:full:4]
    ref[3:full:4] += gd[3:full:4]
    ref[full:] += gd[full:]
    np.testing.assert_array_equal(theta.cpu().numpy(), ref)
    np.testing.assert_array_equal(codes.cpu().numpy(), c0 ^ 1)
