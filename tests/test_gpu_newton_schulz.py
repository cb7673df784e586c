"""The library's Newton-Schulz iterations (appendix "Gefen-Muon"; gefen_newton_schulz, the
matrix-core products gefen_muon_step runs) against the oracle, on the GPU.

Teacher-forced per iteration: the library's own X_k goes into one library iteration and
into the oracle's (ns_gram, ns_poly, ns_combine in float64 with a bfloat16 rounding after
each product). The results may differ only where a float32 sum, taken in another order,
rounds to the neighbouring bfloat16 value -- the gate of the oracle's pin against
torch's bfloat16 Muon on the CPU (tests/test_oracle_muon.py): each difference within one
bfloat16 step of every intermediate product carried through the iteration
(ns_iteration_bound; torch stays within a tenth of it), and at most 1 % of the elements
(torch's own iterations reach 0.76 % against the oracle, a misplaced rounding 54-66 %).
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")

FLIP_FRACTION = 1e-2


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _x0(batch, m, n, seed, dev):
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    u = torch.randn(batch, m, n, generator=gen, device=dev)
    u = u * torch.exp(torch.empty(batch, m, 1, device=dev).uniform_(-3, 0, generator=gen))
    x = u.bfloat16()
    nrm = torch.linalg.vector_norm(x.float(), dim=(1, 2), keepdim=True).bfloat16()
    return (x.float() / nrm.float()).bfloat16()


def _f64(x):
    return x.float().cpu().numpy().astype(np.float64)


def _check_iteration(x_in, x_out, what):
    """x_in, x_out: float64 [m, n] (bfloat16 values)."""
    from test_oracle_muon import ns_iteration_bound
    a, b, c = oracle.MUON_NS_COEFFS
    poly = oracle.ns_poly(oracle.ns_gram(x_in), b, c)
    ref = oracle.ns_combine(x_in, poly, a)
    d = np.abs(x_out - ref)
    bound = ns_iteration_bound(x_in, poly, ref)
    assert (d <= bound).all(), (what, (d / np.maximum(bound, 1e-300)).max())
    frac = np.count_nonzero(d) / d.size
    assert frac <= FLIP_FRACTION, (what, frac)
    return frac


SHAPES = [(1, 64, 192), (1, 128, 128), (3, 96, 1000), (2, 130, 259), (1, 64, 4096),
          (4, 768, 3072), (1, 768, 50257), (1, 3, 5), (5, 40, 1008)]


@pytest.mark.parametrize("batch,m,n", SHAPES, ids=lambda v: str(v))
def test_each_iteration_teacher_forced(batch, m, n):
    """Five iterations, each from the library's previous result. Shapes cover the
    128-tile edges (130 x 259), several batch entries, a split Gram product over K (a lone
    64 x 4096 and the 768 x 50257 embedding), the GPT-2 small MLP shape and tiny ones."""
    dev = _dev()
    x = _x0(batch, m, n, seed=m * 31 + n, dev=dev)
    worst = 0.0
    for k in range(5):
        y = gf.newton_schulz(x, steps=1)
        torch.cuda.synchronize()
        xi, yo = _f64(x), _f64(y)
        for bi in range(batch):
            worst = max(worst, _check_iteration(xi[bi], yo[bi], f"{(batch, m, n)} it {k} b {bi}"))
        x = y
    print(f"{(batch, m, n)}: largest share of one-step flips {worst:.2e}")


def test_big_tile_iterations():
    """The 256 x 256 tile (one workgroup per CU, 4 x 4 accumulators per wave) and its
    split Gram: six 1024 x 2048 matrices take the big tile in the Gram product (split 4
    ways over K) and in the combine. Three iterations, teacher-forced, every batch entry."""
    dev = _dev()
    batch, m, n = 6, 1024, 2048
    x = _x0(batch, m, n, seed=11, dev=dev)
    worst = 0.0
    for k in range(3):
        y = gf.newton_schulz(x, steps=1)
        torch.cuda.synchronize()
        xi, yo = _f64(x), _f64(y)
        for bi in range(batch):
            worst = max(worst, _check_iteration(xi[bi], yo[bi], f"big tile it {k} b {bi}"))
        x = y
    print(f"big tile: largest share of one-step flips {worst:.2e}")


def test_steps_chain_bitwise():
    """Five iterations in one call equal five calls of one iteration, bit for bit, and a
    repeated call gives the same bits (no order-dependent accumulation)."""
    dev = _dev()
    for batch, m, n in [(2, 96, 1000), (1, 64, 4096), (3, 128, 384)]:
        x = _x0(batch, m, n, seed=7 + m, dev=dev)
        five = gf.newton_schulz(x, steps=5)
        y = x
        for _ in range(5):
            y = gf.newton_schulz(y, steps=1)
        again = gf.newton_schulz(x, steps=5)
        torch.cuda.synchronize()
        assert torch.equal(five.view(torch.int16), y.view(torch.int16)), (batch, m, n)
        assert torch.equal(five.view(torch.int16), again.view(torch.int16)), (batch, m, n)


def test_zero_steps_copy_and_vectors():
    dev = _dev()
    x = _x0(2, 17, 33, seed=3, dev=dev)
    y = gf.newton_schulz(x, steps=0)
    torch.cuda.synchronize()
    assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    # 1 x n: the vector kernel, same rounding points (the Gram product is a scalar)
    v = _x0(3, 1, 300, seed=4, dev=dev)
    out = gf.newton_schulz(v, steps=5)
    torch.cuda.synchronize()
    a, b, c = oracle.MUON_NS_COEFFS
    for bi in range(3):
        ref = _f64(v)[bi]
        for _ in range(5):
            ref = oracle.ns_combine(ref, oracle.ns_poly(oracle.ns_gram(ref), b, c), a)
        got = _f64(out)[bi]
        assert np.abs(got - ref).max() <= 0.03 * np.abs(ref).max()


def test_argument_errors():
    dev = _dev()
    x = torch.zeros(1, 8, 4, dtype=torch.bfloat16, device=dev)
    with pytest.raises(gf.GefenError, match="EINVAL"):
        gf.newton_schulz(x)                       # m > n
    x = torch.zeros(1, 4, 8, dtype=torch.bfloat16, device=dev)
    with pytest.raises(gf.GefenError, match="EINVAL"):
        gf.newton_schulz(x, steps=101)
    with pytest.raises(gf.GefenError, match="EINVAL"):
        gf.newton_schulz(x, coeffs=(float("nan"), 1.0, 1.0))
    with pytest.raises(TypeError):
        gf.newton_schulz(x.float())
