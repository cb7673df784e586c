"""Pins for the oracle's optimizer step (Alg. 1; AdamW of Sec. 3, eqs. 1-5).

* Block size 1 reduces Gefen to AdamW: m/s' is exactly +-1 and both +-1 are forced
  codebook entries, so quantization is lossless. The oracle must then follow
  ``torch.optim.AdamW`` (float64, CPU) over 100 steps, with quantization on and off.
* Block size p > 1 with a gradient that is constant inside each block is again AdamW
  on one scalar per block (checked against ``torch.optim.AdamW``).
* Block size p > 1 with a fixed gradient whose in-block ratios are codebook entries:
  quantization is lossless, so m_t = (1 - beta1^t) g, v_t = (1 - beta2^t) mean_B g^2,
  and the parameters follow a closed-form geometric series.
* Invariants for arbitrary gradients: the shared moment is the EMA of the block mean
  of g^2, the new scale is the block absmax of the momentum recovered from the
  update, every code is a nearest entry, and the absmax element encodes to an end.
"""
import numpy as np
import pytest
import torch


def _dp_codebook(oracle, k=256, seed=0):
    rng = np.random.default_rng(seed)
    x = rng.standard_t(3, size=(500, 200))
    x = (x / np.abs(x).max(axis=1, keepdims=True)).reshape(-1)
    hist = np.histogram(x, bins=16 * k, range=(-1, 1))[0].astype(np.uint64)
    cb, _, _, st = oracle.dp_codebook(hist, k)
    assert st == 0
    return cb


def _close(a, ref, lr, u, rel):
    err = np.abs(a - ref)
    bound = rel * np.abs(ref) + rel * lr * np.abs(u) + 1e-300
    return float(np.max(err / bound))


@pytest.mark.parametrize("quantize", [True, False])
def test_block_size_one_is_adamw(oracle, quantize):
    rng = np.random.default_rng(1)
    n, T = 300, 100
    lr, b1, b2, eps, wd = 1e-3, 0.9, 0.999, 1e-8, 0.1
    cb = _dp_codebook(oracle, k=256)
    theta0 = rng.standard_normal(n) * 0.02
    grads = [rng.standard_normal(n) * np.exp(rng.uniform(-6, 0, n)) for _ in range(T)]
    grads32 = [g.astype(np.float32) for g in grads]

    th = theta0.copy()
    codes = np.zeros(n, dtype=np.uint8)
    s = np.zeros(n)
    v = np.zeros(n)
    m_full = np.zeros(n)

    p_t = torch.tensor(theta0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p_t], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd,
                            foreach=False)
    for t in range(1, T + 1):
        g = grads32[t - 1]
        oracle.step_uniform(th, g, codes, s, v, 1, cb, cb, lr, b1, b2, eps, wd, t,
                            quantize=quantize, m_full=None if quantize else m_full)
        p_t.grad = torch.tensor(g.astype(np.float64))
        opt.step()
        ref = p_t.detach().numpy()
        # theta floor: parameters near 0 are judged against the step size
        assert _close(th, ref, lr, np.ones(n), 1e-12) <= 1.0, t
    if quantize:
        # state mirrors AdamW's moments: s = |m|, v = second moment
        st = opt.state[p_t]
        np.testing.assert_allclose(s, np.abs(st["exp_avg"].numpy()), rtol=1e-12)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-12)


def test_blockwise_constant_gradient_is_scalar_adamw(oracle):
    rng = np.random.default_rng(2)
    p, nb, T = 16, 40, 30
    lr, b1, b2, eps, wd = 6e-4, 0.9, 0.95, 1e-8, 0.1
    cb = _dp_codebook(oracle, k=16, seed=3)
    theta_b = rng.standard_normal(nb) * 0.02
    th = np.repeat(theta_b, p)
    codes = np.zeros(nb * p, dtype=np.uint8)
    s = np.zeros(nb)
    v = np.zeros(nb)
    p_t = torch.tensor(theta_b, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p_t], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd,
                            foreach=False)
    for t in range(1, T + 1):
        gb = (rng.standard_normal(nb) * np.exp(rng.uniform(-5, 0, nb))).astype(np.float32)
        oracle.step_uniform(th, np.repeat(gb, p), codes, s, v, p, cb, cb, lr, b1, b2, eps,
                            wd, t)
        p_t.grad = torch.tensor(gb.astype(np.float64))
        opt.step()
        ref = np.repeat(p_t.detach().numpy(), p)
        assert _close(th, ref, lr, np.ones_like(th), 1e-12) <= 1.0, t


def test_lossless_codebook_closed_form(oracle):
    # Codebook holds the exact in-block ratios r_i of a fixed gradient g_i = G_B r_i.
    cb = np.array([-1.0, -0.5, -0.25, 0.0, 0.25, 0.5, 0.75, 1.0])
    rng = np.random.default_rng(4)
    p, nb, T = 12, 25, 40
    lr, b1, b2, eps, wd = 1e-3, 0.9, 0.999, 1e-8, 0.1
    ridx = rng.integers(0, cb.size, size=(nb, p))
    ridx[:, 0] = rng.choice([0, cb.size - 1], size=nb)   # absmax ratio +-1 in each block
    G = 2.0 ** -rng.integers(0, 11, size=nb)        # powers of two keep G * r exact
    g = (G[:, None] * cb[ridx]).astype(np.float32)
    gd = g.astype(np.float64)
    theta0 = rng.standard_normal((nb, p)) * 0.02
    th = theta0.reshape(-1).copy()
    codes = np.zeros(nb * p, dtype=np.uint8)
    s = np.zeros(nb)
    v = np.zeros(nb)
    for t in range(1, T + 1):
        oracle.step_uniform(th, g.reshape(-1), codes, s, v, p, cb, cb, lr, b1, b2, eps, wd,
                            t)
    meansq = np.mean(gd ** 2, axis=1)
    u = gd / (np.sqrt(meansq)[:, None] + eps)
    decay = 1.0 - lr * wd
    geo = sum(decay ** i for i in range(T))
    expect = theta0 * decay ** T - lr * u * geo
    assert _close(th, expect.reshape(-1), lr, u.reshape(-1), 1e-11) <= 1.0
    np.testing.assert_array_equal(codes, ridx.reshape(-1))
    np.testing.assert_allclose(s, (1 - b1 ** T) * np.abs(gd).max(axis=1), rtol=1e-13)
    np.testing.assert_allclose(v, (1 - b2 ** T) * meansq, rtol=1e-13)


@pytest.mark.parametrize("p,dtype", [(8, np.float32), (37, np.float32), (64, np.uint16)])
def test_random_gradient_invariants(oracle, p, dtype):
    rng = np.random.default_rng(p)
    nb, T, k = 30, 12, 256
    lr, b1, b2, eps, wd = 1e-3, 0.9, 0.999, 1e-8, 0.1
    cb = _dp_codebook(oracle, k=k, seed=p)
    n = nb * p
    th = rng.standard_normal(n) * 0.02
    codes = np.zeros(n, dtype=np.uint8)
    s = np.zeros(nb)
    v = np.zeros(nb)
    scale = np.repeat(np.exp(rng.uniform(np.log(1e-3), 0, nb)), p)
    for t in range(1, T + 1):
        g32 = (rng.standard_normal(n) * scale).astype(np.float32)
        if dtype == np.uint16:
            gin = (g32.view(np.uint32) >> 16).astype(np.uint16)
            gd = (gin.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        else:
            gin, gd = g32, g32.astype(np.float64)
        th_prev, v_prev = th.copy(), v.copy()
        oracle.step_uniform(th, gin, codes, s, v, p, cb, cb, lr, b1, b2, eps, wd, t)
        # shared second moment: EMA of the block mean of g^2
        meansq = (gd ** 2).reshape(nb, p).mean(axis=1)
        np.testing.assert_allclose((v - b2 * v_prev) / (1 - b2), meansq, rtol=1e-9)
        # momentum recovered from the parameter update
        vhat = v / (1 - b2 ** t)
        denom = np.repeat(np.sqrt(vhat) + eps, p)
        m = (th_prev * (1 - lr * wd) - th) * (1 - b1 ** t) * denom / lr
        mb = np.abs(m).reshape(nb, p)
        np.testing.assert_allclose(mb.max(axis=1), s, rtol=1e-7)
        # every code is a nearest entry of m / s'
        x = m / np.repeat(s, p)
        d = np.abs(x[:, None] - cb[None, :])
        best = d.min(axis=1)
        chosen = d[np.arange(n), codes]
        assert np.all(chosen <= best + 1e-7)
        # the absmax element of each block encodes to an end of the codebook
        amax = mb.argmax(axis=1) + np.arange(nb) * p
        assert np.all(np.isin(codes[amax], [0, k - 1]))


def test_zero_gradient_block(oracle):
    cb = np.linspace(-1, 1, 16)
    p, nb = 10, 3
    th = np.full(nb * p, 0.5)
    codes = np.full(nb * p, 7, dtype=np.uint8)
    s = np.zeros(nb)
    v = np.array([0.0, 2.0, 0.0])
    g = np.zeros(nb * p, dtype=np.float32)
    oracle.step_uniform(th, g, codes, s, v, p, cb, cb, 1e-2, 0.9, 0.999, 1e-8, 0.1, 3)
    assert np.all(codes == 0) and np.all(s == 0.0)
    np.testing.assert_allclose(v, [0.0, 0.999 * 2.0, 0.0], rtol=1e-15)
    np.testing.assert_allclose(th, 0.5 * (1 - 1e-2 * 0.1), rtol=1e-15)


def test_explicit_blocks_match_uniform(oracle):
    # The CSR entry point with offsets 0, p, 2p, ... must equal the uniform one.
    rng = np.random.default_rng(8)
    p, nb = 24, 10
    cb = _dp_codebook(oracle, k=16, seed=1)
    g = rng.standard_normal(p * nb).astype(np.float32)
    a = [rng.standard_normal(p * nb) * 0.02, np.zeros(p * nb, np.uint8), np.zeros(nb),
         np.zeros(nb)]
    b = [x.copy() for x in a]
    oracle.step_uniform(a[0], g, a[1], a[2], a[3], p, cb, cb, 1e-3, 0.9, 0.999, 1e-8, 0.1, 1)
    oracle.step_blocks(b[0], g, b[1], b[2], b[3], np.arange(0, p * nb + 1, p), cb, cb, 1e-3,
                       0.9, 0.999, 1e-8, 0.1, 1)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
