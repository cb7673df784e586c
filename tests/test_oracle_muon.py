"""Pins of the Gefen-Muon oracle (appendix "Gefen-Muon") against facts fixed outside it.

* bfloat16 rounding: torch's float32 -> bfloat16 conversion (a library routine).
* Newton-Schulz in float64: the iteration X <- a X + (b X X^T + c (X X^T)^2) X keeps the
  singular vectors and maps every normalised singular value through the odd quintic
  p(s) = a s + b s^3 + c s^5, so the result is U diag(p^k(s / ||X||_F)) V^T (SVD by
  numpy). A transposed operand, a coefficient in the wrong place or a dropped term
  breaks this on both the wide and the tall path.
* Codec with one element per block: m / s' = +-1 are the forced end entries, so the
  codes are lossless and the quantized buffer follows Muon's plain momentum recursion.
* Codec against the Gefen step oracle: both compute the same momentum, scale and codes
  (the step's codes are pinned separately).
* Whole step with lossless codes against torch.optim.Muon (CPU), within bfloat16
  rounding of the orthogonalised update.
* bfloat16 Newton-Schulz against torch's own implementation (the one torch.optim.Muon
  runs), on the CPU: each of the three products of an iteration, given torch's inputs,
  rounds where torch rounds (bit-equal except rare one-step flips from float32
  accumulation order); one whole iteration from the normalisation on; five iterations
  within the spread that accumulation order alone produces.
"""
import numpy as np
import pytest
import torch

import oracle
from torch.optim._muon import _zeropower_via_newtonschulz as torch_newton_schulz


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.uniform(-8, 8, 20000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, -1.00390625, 65504.0, 1e-40]])
    x32 = x.astype(np.float32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).float().numpy().astype(np.float64)
    np.testing.assert_array_equal(oracle.to_bf16(x32.astype(np.float64)), ref)


def _svd_closed_form(x, steps, coeffs):
    a, b, c = coeffs
    u, sv, vt = np.linalg.svd(x, full_matrices=False)
    s = sv / np.sqrt(np.sum(x * x))
    for _ in range(steps):
        s = a * s + b * s ** 3 + c * s ** 5
    return (u * s) @ vt


@pytest.mark.parametrize("rows,cols", [(8, 24), (24, 8), (16, 16), (1, 40), (40, 1), (33, 65)])
def test_newton_schulz_float64_is_the_singular_value_polynomial(rows, cols):
    rng = np.random.default_rng(rows * 100 + cols)
    x = rng.standard_normal((rows, cols)) * rng.uniform(0.1, 3.0, (rows, 1))
    for steps in (1, 2, 5):
        got = oracle.newton_schulz(x, rows, cols, steps=steps, bf16=False)
        ref = _svd_closed_form(x, steps, oracle.MUON_NS_COEFFS)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * max(1.0, np.abs(ref).max()))


def test_newton_schulz_bf16_stays_near_float64():
    rng = np.random.default_rng(7)
    rows, cols = 48, 96
    x = rng.standard_normal((rows, cols))
    o64 = oracle.newton_schulz(x, rows, cols, bf16=False)
    o16 = oracle.newton_schulz(x, rows, cols, bf16=True)
    assert np.all(o16 == oracle.to_bf16(o16))                 # results are bfloat16 values
    assert np.abs(o16 - o64).max() < 0.05 * np.abs(o64).max()


def test_newton_schulz_zero_matrix():
    o = oracle.newton_schulz(np.zeros(12), 3, 4)
    assert np.all(o == 0)


def _lossless_codebook(k=256):
    cb = np.linspace(-1.0, 1.0, k)
    return cb


@pytest.mark.parametrize("nesterov", [False, True])
def test_codec_block_size_one_is_muon_momentum(nesterov):
    """p = 1: every m / s' is +-1, so the stored buffer is exact and u follows Muon."""
    rng = np.random.default_rng(3)
    n, mu = 500, 0.95
    cb = _lossless_codebook()
    codes = np.zeros(n, dtype=np.uint8)
    s = np.zeros(n, dtype=np.float64)
    offs = np.arange(n + 1, dtype=np.int64)
    buf = np.zeros(n)
    for t in range(6):
        g = rng.standard_normal(n).astype(np.float32)
        gd = g.astype(np.float64)
        u = oracle.muon_codec_blocks(g, codes, s, offs, cb, cb, mu, nesterov)
        buf = mu * buf + (1.0 - mu) * gd
        ref = (1.0 - mu) * gd + mu * buf if nesterov else buf
        np.testing.assert_allclose(u, ref, rtol=1e-13, atol=1e-300)
        np.testing.assert_allclose(s, np.abs(buf), rtol=1e-13)
        assert set(np.unique(codes)) <= {0, 255}


def test_codec_matches_the_step_oracle():
    """Same momentum, scale and codes as the Gefen step with beta1 = mu."""
    rng = np.random.default_rng(4)
    p, nb, mu = 64, 30, 0.9
    n = p * nb
    offs = np.arange(0, n + 1, p, dtype=np.int64)
    h = np.zeros(4096, dtype=np.uint64)
    g0 = (rng.standard_normal(n) * np.repeat(np.exp(rng.uniform(-5, 0, nb)), p)).astype(np.float32)
    oracle.histogram_blocks(g0, offs, 4096, h)
    cb, _, _, _ = oracle.dp_codebook(h, 256)
    c1 = np.zeros(n, dtype=np.uint8)
    s1 = np.zeros(nb)
    c2 = c1.copy()
    s2 = s1.copy()
    v2 = np.zeros(nb)
    for t in range(1, 4):
        g = (rng.standard_normal(n) * np.repeat(np.exp(rng.uniform(-5, 0, nb)), p)).astype(np.float32)
        u = oracle.muon_codec_blocks(g, c1, s1, offs, cb, cb, mu, nesterov=False)
        m = np.zeros(n)
        oracle.step_blocks(np.zeros(n), g, c2, s2, v2, offs, cb, cb, 1e-3, mu, 0.999, 1e-8, 0.0,
                           t, m_out=m)
        np.testing.assert_array_equal(c1, c2)
        np.testing.assert_array_equal(s1, s2)
        np.testing.assert_array_equal(u, m)


@pytest.mark.parametrize("rows,cols", [(32, 48), (48, 32)])
def test_lossless_step_matches_torch_muon(rows, cols):
    """Block size 1 with nesterov: Gefen-Muon is Muon; compare with torch.optim.Muon on
    the CPU over three steps, within bfloat16 rounding of the orthogonalised update."""
    rng = np.random.default_rng(rows)
    n = rows * cols
    lr, mu, wd = 0.02, 0.95, 0.01
    theta0 = rng.standard_normal(n) * 0.02
    theta = theta0.copy()
    p_ref = torch.nn.Parameter(torch.tensor(theta0.reshape(rows, cols), dtype=torch.float32))
    opt = torch.optim.Muon([p_ref], lr=lr, momentum=mu, weight_decay=wd, nesterov=True)
    cb = _lossless_codebook()
    codes = np.zeros(n, dtype=np.uint8)
    s = np.zeros(n)
    offs = np.arange(n + 1, dtype=np.int64)
    scale = lr * oracle.muon_lr_scale(rows, cols)
    for _ in range(3):
        g = rng.standard_normal(n).astype(np.float32)
        oracle.muon_step(theta, g, codes, s, offs, rows, cols, cb, cb, lr, mu, wd, nesterov=True)
        p_ref.grad = torch.from_numpy(g.reshape(rows, cols).copy())
        opt.step()
    ref = p_ref.detach().double().numpy().reshape(-1)
    # each step's update is lr * scale * O with |O| <= ~1.2; the two bfloat16 pipelines
    # round differently (accumulation order and width), measured up to 0.8 % of one step
    assert np.abs(theta - ref).max() < 0.02 * scale
    assert np.abs(theta - theta0).max() > 10 * np.abs(theta - ref).max()


# ------------------------------------------------------------------ bf16 Newton-Schulz
NS_SHAPES = [(64, 256), (96, 96), (128, 384), (32, 1000), (200, 600)]
FLIP_FRACTION = 2e-3   # measured at most 1e-3 (4 of 4096 elements) per product here


def _torch_products(x, coeffs):
    """One iteration in torch's bfloat16 form: the products the Muon implementation calls."""
    a, b, c = coeffs
    gram = x @ x.T
    poly = torch.addmm(gram, gram, gram, beta=b, alpha=c)
    return gram, poly, torch.addmm(x, poly, x, beta=a)


def _check_product(got, ref, mag, k, what):
    """got, ref: bfloat16 values (float64 arrays). They may differ where a float32 sum of
    k terms of total magnitude `mag`, taken in another order, rounds to the neighbouring
    bfloat16 value: one step of 2^-7 relative at most, or the sum's own error where the
    terms cancel. Such flips must stay rare."""
    d = np.abs(got - ref)
    bound = 2.0 ** -7 * np.abs(ref) + k * 2.0 ** -24 * mag
    assert (d <= bound).all(), (what, (d / np.maximum(bound, 1e-300)).max())
    frac = np.count_nonzero(d) / d.size
    assert frac <= FLIP_FRACTION, (what, frac)
    return frac


def _normalised_bf16(u):
    x = torch.from_numpy(u).bfloat16()
    return x / x.norm().clamp(min=oracle.MUON_EPS)


@pytest.mark.parametrize("m,n", NS_SHAPES)
def test_ns_products_round_as_torch(m, n):
    """Teacher-forced: every product of five iterations, fed torch's own operands."""
    a, b, c = oracle.MUON_NS_COEFFS
    rng = np.random.default_rng(m * 7 + n)
    x = _normalised_bf16(rng.standard_normal((m, n)).astype(np.float32))
    for _ in range(5):
        gram, poly, xn = _torch_products(x, oracle.MUON_NS_COEFFS)
        xd, gd, pd = (t.double().numpy() for t in (x, gram, poly))
        _check_product(oracle.ns_gram(xd), gd, np.abs(xd) @ np.abs(xd).T, n, "gram")
        _check_product(oracle.ns_poly(gd, b, c), pd,
                       abs(b) * np.abs(gd) + abs(c) * (np.abs(gd) @ np.abs(gd)), m, "poly")
        _check_product(oracle.ns_combine(xd, pd, a), xn.double().numpy(),
                       abs(a) * np.abs(xd) + np.abs(pd) @ np.abs(xd), m, "combine")
        x = xn


def test_ns_product_pin_catches_rounding_slips():
    """The product pin is sharp enough to see a misplaced rounding: each variant below
    rounds one intermediate that torch keeps in float32, and differs from torch in far
    more elements than the pin allows."""
    a, b, c = oracle.MUON_NS_COEFFS
    r = oracle.to_bf16
    rng = np.random.default_rng(11)
    x = _normalised_bf16(rng.standard_normal((128, 384)).astype(np.float32))
    for _ in range(2):   # the second iteration's operands are no longer near-orthogonal
        gram, poly, xn = _torch_products(x, oracle.MUON_NS_COEFFS)
        x = xn
    xd, gd, pd = (t.double().numpy() for t in (x, gram, poly))
    gram2, poly2, xn2 = (t.double().numpy() for t in _torch_products(x, oracle.MUON_NS_COEFFS))
    slips = {
        "A A rounded before scaling": (r(b * gram2 + r(c * r(gram2 @ gram2))), poly2),
        "b A rounded before the sum": (r(r(b * gram2) + c * (gram2 @ gram2)), poly2),
        "B X rounded before a X is added": (r(r(a * xd) + r(poly2 @ xd)), xn2),
    }
    for what, (got, ref) in slips.items():
        frac = np.count_nonzero(got != ref) / got.size
        assert frac > 10 * FLIP_FRACTION, (what, frac)


@pytest.mark.parametrize("rows,cols", [(64, 256), (256, 64), (96, 96), (40, 1000)])
def test_ns_one_iteration_matches_torch(rows, cols):
    """From the float32 input on: orientation, bfloat16 norm, division, one iteration."""
    rng = np.random.default_rng(rows + 3 * cols)
    u = rng.standard_normal((rows, cols)).astype(np.float32)
    got = oracle.newton_schulz(u, rows, cols, steps=1)
    ref = torch_newton_schulz(torch.from_numpy(u), oracle.MUON_NS_COEFFS, 1,
                              oracle.MUON_EPS).double().numpy()
    assert got.shape == ref.shape
    m, n = min(rows, cols), max(rows, cols)
    x = oracle.ns_normalise(u, rows, cols)
    gram = oracle.ns_gram(x)
    a, b, c = oracle.MUON_NS_COEFFS
    poly = oracle.ns_poly(gram, b, c)
    mag = abs(a) * np.abs(x) + np.abs(poly) @ np.abs(x)
    _check_product(got if rows <= cols else got.T, ref if rows <= cols else ref.T,
                   (1 + 8 * m * 2.0 ** -7) * mag, n, "iteration")


@pytest.mark.parametrize("rows,cols", [(64, 256), (256, 64), (96, 96), (200, 600), (48, 1000)])
def test_ns_five_iterations_match_torch(rows, cols):
    """Muon's default five iterations: the rare flips of each product spread through the
    later products, so the results differ in many elements, but only by the amount that
    float32 accumulation order alone produces (torch against itself on a column-permuted
    input reaches 0.47 % in Frobenius norm and 1.6 % of the largest entry on 200 x 600)."""
    rng = np.random.default_rng(rows * cols)
    u = rng.standard_normal((rows, cols)).astype(np.float32)
    got = oracle.newton_schulz(u, rows, cols)
    ref = torch_newton_schulz(torch.from_numpy(u), oracle.MUON_NS_COEFFS, 5,
                              oracle.MUON_EPS).double().numpy()
    fro = np.sqrt(np.sum((got - ref) ** 2) / np.sum(ref ** 2))
    assert fro <= 1e-2, fro
    assert np.abs(got - ref).max() <= 3e-2 * np.abs(ref).max()
    assert np.all(got == oracle.to_bf16(got))


@pytest.mark.parametrize("m,n", [(64, 192), (128, 128), (96, 1000), (130, 259), (40, 1008)])
def test_ns_whole_iterations_teacher_forced_match_torch(m, n):
    """Whole iterations, each fed torch's previous result: the flips of one product
    spread through the next two, up to 0.76 % of the elements (64 x 192, fifth
    iteration, where the near-orthogonal X makes a X and B X cancel), each within the
    propagated bound of ns_iteration_bound; the GPU iterations are held to the same gate
    (tests/test_gpu_newton_schulz.py)."""
    a, b, c = oracle.MUON_NS_COEFFS
    rng = np.random.default_rng(m * 31 + n)
    u = rng.standard_normal((m, n)) * np.exp(rng.uniform(-3, 0, (m, 1)))
    x = torch.from_numpy(u.astype(np.float32)).bfloat16()
    x = (x.float() / x.float().norm().bfloat16().float()).bfloat16()
    for _ in range(6):
        xd = x.double().numpy()
        poly = oracle.ns_poly(oracle.ns_gram(xd), b, c)
        got = oracle.ns_combine(xd, poly, a)
        x = _torch_products(x, oracle.MUON_NS_COEFFS)[2]
        ref = x.double().numpy()
        d = np.abs(got - ref)
        assert (d <= ns_iteration_bound(xd, poly, ref)).all()
        assert np.count_nonzero(d) / d.size <= 1e-2


def ns_iteration_bound(x, poly, ref):
    """Largest difference one whole iteration may show between two implementations that
    round at the same points: one bfloat16 step in every element of the Gram and
    polynomial products, carried through the later products (|delta B| <= 2^-7 (|B| +
    |b| |A| + 2 |c| |A| |A|), times |X|), one step of the result, and the float32 error
    of its sum. Torch's iterations stay within a tenth of it."""
    a, b, c = oracle.MUON_NS_COEFFS
    n = x.shape[1]
    gram = oracle.ns_gram(x)
    ag = np.abs(gram)
    dpoly = 2.0 ** -7 * (np.abs(poly) + abs(b) * ag + 2 * abs(c) * (ag @ ag))
    mag = abs(a) * np.abs(x) + np.abs(poly) @ np.abs(x)
    return 2.0 ** -7 * np.abs(ref) + dpoly @ np.abs(x) + n * 2.0 ** -24 * mag
