"""GPU parity of the Gefen step (Alg. 1) against the float64 oracle, through the C ABI.

Teacher-forced per step (see parity.py for the gates). Covers every kernel class:
uniform blocks held in registers (p % 4 == 0, p <= 8192), the two-pass streaming kernel
(odd, unaligned, irregular or large blocks), register runs of short explicit blocks and
the lane-per-block kernel (blocks of at most 32 elements), with fp32 and bf16
gradients, ragged last tiles, zero blocks, misaligned tensors, explicit block tables,
codebook refits and checkpoints.
"""
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


def _grad(n, seed, dtype, rows=None, dev=None):
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    g = torch.randn(n, generator=gen, device=dev)
    if rows:
        sc = torch.exp(torch.empty(rows, device=dev).uniform_(np.log(1e-3), 0, generator=gen))
        g = (g.view(rows, -1) * sc[:, None]).reshape(-1)
    return g.to(dtype)


HP = dict(lr=1e-3, betas=(0.9, 0.999), eps=1e-8, wd=0.1)


def _run_steps(run, grads_fn, steps, hp=HP, where=""):
    reps = []
    for t in range(1, steps + 1):
        grads = grads_fn(t)
        reps.append(run.teacher_forced_step(grads, hp["lr"], hp["betas"], hp["eps"], hp["wd"], t,
                                            where=f"{where} step {t}"))
    return reps


def test_tiny_config_end_to_end():
    """The tiny MLP configuration: periods, histogram, codebook and 10 steps."""
    from parity import Run, grad_bits
    dev = _dev()
    w = W.get("tiny")
    fields = W.scale_fields(w)
    params = W.init_params(w, dev)
    g1 = W.make_grads(w, fields, 1, dev)
    run = Run(params, g1)
    # periods: Alg. 2 on the same gradient bits
    for i, g in enumerate(g1):
        _, _, per = oracle.partition(grad_bits(g), 1e-8)
        assert run.periods[i] == per, (i, run.periods[i], per)
    # histogram and DP of the init fit
    nb = 16 * run.k
    h_ref = np.zeros(nb, dtype=np.uint64)
    for i, g in enumerate(g1):
        oracle.histogram_blocks(grad_bits(g), run.offsets[i], nb, h_ref)
    h_gpu = run.state.histogram(g1).cpu().numpy().view(np.uint64)
    np.testing.assert_array_equal(h_gpu, h_ref)
    cb_ref, cost_ref, _, st_ref = oracle.dp_codebook(h_ref, run.k)
    cb_gpu = run.state.read(gf.STATE_CB_DEC64).cpu().numpy()
    np.testing.assert_array_equal(cb_gpu, cb_ref)
    cost, st = run.state.fit_info()
    assert st == st_ref and cost == cost_ref
    _run_steps(run, lambda t: W.make_grads(w, fields, t, dev), w.steps,
               hp=dict(lr=w.lr, betas=w.betas, eps=w.eps, wd=w.wd), where="tiny")


# (period, number of blocks): every kernel class, ragged last tiles
PERIODS = [(1, 3000), (2, 700), (3, 513), (4, 1000), (8, 300), (12, 257), (20, 100),
           (32, 300), (36, 90), (64, 70), (96, 41), (100, 33), (768, 19), (2048, 9),
           (1024, 11), (3072, 5), (4096, 6), (6144, 3), (8192, 3), (999, 40), (5003, 9),
           (8196, 2), (12288, 2), (40000, 2),
           (200000, 2)]


@pytest.mark.parametrize("p,nb", PERIODS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_uniform_periods(p, nb, dtype):
    from parity import Run
    dev = _dev()
    n = p * nb
    theta = (torch.randn(n, device=dev) * 0.02).contiguous()
    g1 = _grad(n, 1, dtype, dev=dev)
    run = Run([theta], [g1], period_override=[p])
    assert run.periods == [p]
    _run_steps(run, lambda t: [_grad(n, 100 + t, dtype, dev=dev)], 3, where=f"p={p}")


def test_explicit_irregular_blocks():
    from parity import Run
    dev = _dev()
    rng = np.random.default_rng(3)
    sizes = np.concatenate([[1, 2, 5, 31, 32, 33, 64, 1000, 9000, 70000],
                            rng.integers(1, 40, size=300), rng.integers(40, 3000, size=60)])
    rng.shuffle(sizes)
    sizes = np.concatenate([sizes, [7]])
    n1 = int(sizes[:200].sum())
    n = int(sizes.sum())
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    # two tensors split on a block boundary
    params = [(torch.randn(n1, device=dev) * 0.02), (torch.randn(n - n1, device=dev) * 0.02)]
    gr = lambda t: [_grad(n1, 10 + t, torch.bfloat16, dev=dev),
                    _grad(n - n1, 50 + t, torch.bfloat16, dev=dev)]
    run = Run(params, gr(1), block_offsets=offs)
    _run_steps(run, gr, 3, where="explicit")


def test_misaligned_tensors():
    """Parameter and gradient views at odd element offsets (unaligned vector loads)."""
    from parity import Run
    dev = _dev()
    p, nb = 2048, 5
    n = p * nb
    pbuf = torch.randn(n + 3, device=dev) * 0.02
    theta = pbuf[1:1 + n]
    assert theta.data_ptr() % 16 != 0
    gbufs = {t: _grad(n + 1, 30 + t, torch.bfloat16, dev=dev) for t in range(1, 4)}
    gr = lambda t: [gbufs[t][1:]]
    run = Run([theta], gr(1), period_override=[p])
    _run_steps(run, gr, 3, where="misaligned")
    assert pbuf[0].item() == pbuf[0].item() and torch.isfinite(pbuf).all()


def test_zero_gradient_blocks():
    from parity import Run
    dev = _dev()
    p, nb = 768, 12
    n = p * nb
    theta = torch.randn(n, device=dev) * 0.02

    def gr(t):
        g = _grad(n, 60 + t, torch.float32, dev=dev)
        g.view(nb, p)[::3] = 0.0
        return [g]

    run = Run([theta], gr(1), period_override=[p])
    _run_steps(run, gr, 3, where="zero-blocks")
    s = run.state.read(gf.STATE_SCALE).cpu().numpy()
    assert (s[::3] == 0).all()
    codes = run.state.read(gf.STATE_CODES).cpu().numpy()[:n].reshape(nb, p)
    assert (codes[::3] == 0).all()


def test_block_size_one_matches_torch_adamw_free_running():
    """p = 1: Gefen is AdamW (m/s' = +-1 are codebook entries). Free-running, fp32."""
    dev = _dev()
    n = 50_000
    torch.manual_seed(0)
    theta0 = torch.randn(n, device=dev) * 0.02
    p_gef = theta0.clone()
    p_ref = theta0.clone().requires_grad_(True)
    lr, b1, b2, eps, wd = 1e-3, 0.9, 0.999, 1e-8, 0.1
    opt = torch.optim.AdamW([p_ref], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd,
                            foreach=False)
    grads = [_grad(n, 200 + t, torch.float32, dev=dev) *
             torch.exp(torch.linspace(-6, 0, n, device=dev)) for t in range(1, 51)]
    st = gf.GefenState([grads[0]], period_override=[1])
    for t in range(1, 51):
        st.step([p_gef], [grads[t - 1]], lr, (b1, b2), eps, wd, t)
        p_ref.grad = grads[t - 1].clone()
        opt.step()
    torch.cuda.synchronize()
    a = p_gef.double()
    b = p_ref.detach().double()
    err = (a - b).abs()
    assert (err <= 1e-5 * b.abs() + 1e-5 * lr).all(), float((err / (b.abs() + lr)).max())


def test_step_is_deterministic():
    dev = _dev()
    n = 8192 * 7
    theta0 = torch.randn(n, device=dev) * 0.02
    g1 = _grad(n, 5, torch.bfloat16, rows=7 * 4, dev=dev)
    st = gf.GefenState([g1])
    th = theta0.clone()
    for t in range(1, 4):
        st.step([th], [_grad(n, 5 + t, torch.bfloat16, rows=28, dev=dev)], 1e-3, (0.9, 0.999),
                1e-8, 0.1, t)
    ck = st.export()
    th_ck = th.clone()
    g = _grad(n, 99, torch.bfloat16, rows=28, dev=dev)
    outs = []
    for _ in range(2):
        st.import_(ck)
        th.copy_(th_ck)
        st.step([th], [g], 1e-3, (0.9, 0.999), 1e-8, 0.1, 4)
        outs.append((th.clone(), st.read(gf.STATE_CODES).clone(), st.read(gf.STATE_SCALE).clone(),
                     st.read(gf.STATE_V).clone()))
    for x, y in zip(*outs):
        assert torch.equal(x, y)


def test_buffer_cycling_matches_fixed_buffers():
    """The library caches a few device tensor tables keyed by buffer addresses; cycling
    through more parameter/gradient buffer sets than it caches (and back) gives results
    bit-identical to one fixed set of buffers that is refilled each step."""
    dev = _dev()
    w = W.get("tiny")
    fields = W.scale_fields(w)
    hp = (w.lr, w.betas, w.eps, w.wd)
    pa = W.init_params(w, dev)
    pb = [p.clone() for p in pa]
    g1 = W.make_grads(w, fields, 1, dev)
    grad_sets = [W.make_grads(w, fields, t, dev) for t in range(1, 8)]
    order = [0, 1, 2, 3, 4, 5, 6, 0, 1, 6, 5, 0, 0, 3]
    a = gf.GefenState(g1)
    b = gf.GefenState(g1)
    fixed = [g.clone() for g in g1]
    for t, k in enumerate(order, start=1):
        a.step(pa, grad_sets[k], *hp, t)
        for f, g in zip(fixed, grad_sets[k]):
            f.copy_(g)
        b.step(pb, fixed, *hp, t)
        if t == 9:                      # a histogram on an older buffer set in between
            assert torch.equal(a.histogram(grad_sets[2]), b.histogram(grad_sets[2]))
    for x, y in zip(pa, pb):
        assert torch.equal(x, y)
    for which in (gf.STATE_CODES, gf.STATE_SCALE, gf.STATE_V):
        assert torch.equal(a.read(which), b.read(which))


def test_checkpoint_resume_bitwise():
    dev = _dev()
    w = W.get("tiny")
    fields = W.scale_fields(w)
    hp = (w.lr, w.betas, w.eps, w.wd)
    pa = W.init_params(w, dev)
    g1 = W.make_grads(w, fields, 1, dev)
    a = gf.GefenState(g1)
    for t in range(1, 6):
        a.step(pa, W.make_grads(w, fields, t, dev), hp[0], hp[1], hp[2], hp[3], t)
    ck = a.export(device=torch.device("cpu"))
    pb = [p.clone() for p in pa]
    for t in range(6, 11):
        a.step(pa, W.make_grads(w, fields, t, dev), hp[0], hp[1], hp[2], hp[3], t)
    b = gf.GefenState(g1)
    b.import_(ck.to(dev))
    for t in range(6, 11):
        b.step(pb, W.make_grads(w, fields, t, dev), hp[0], hp[1], hp[2], hp[3], t)
    for x, y in zip(pa, pb):
        assert torch.equal(x, y)
    for which in (gf.STATE_CODES, gf.STATE_SCALE, gf.STATE_V):
        assert torch.equal(a.read(which), b.read(which))


def test_refit_encodes_with_new_codebook_then_decodes_with_it():
    from parity import Run
    dev = _dev()
    p, nb = 2048, 6
    n = p * nb
    theta = torch.randn(n, device=dev) * 0.02
    gr = lambda t: [_grad(n, 300 + t, torch.bfloat16, rows=nb, dev=dev) * (3.0 if t > 2 else 1.0)]
    run = Run([theta], gr(1), period_override=[p])
    _run_steps(run, gr, 2, where="pre-refit")
    old = run.state.read(gf.STATE_CB_DEC).clone()
    # heavy-tailed gradients give a different codebook
    gt = torch.distributions.StudentT(1.5).sample((n,)).to(dev).to(torch.bfloat16)
    run.state.fit_codebook([gt])
    new_enc = run.state.read(gf.STATE_CB_ENC)
    assert torch.equal(run.state.read(gf.STATE_CB_DEC), old)
    assert not torch.equal(new_enc, old)
    rep = run.teacher_forced_step(gr(3), 1e-3, (0.9, 0.999), 1e-8, 0.1, 3, where="refit step")
    assert torch.equal(run.state.read(gf.STATE_CB_DEC), new_enc)
    run.teacher_forced_step(gr(4), 1e-3, (0.9, 0.999), 1e-8, 0.1, 4, where="post-refit")
    # the refit codebook is the oracle's DP on the oracle histogram of the same bits
    from parity import grad_bits
    h = oracle.histogram_blocks(grad_bits(gt), run.offsets[0], 16 * run.k)
    cb_ref, _, _, _ = oracle.dp_codebook(h, run.k)
    np.testing.assert_array_equal(run.state.read(gf.STATE_CB_DEC64).cpu().numpy(), cb_ref)
    assert rep["codes"] == n


def test_guard_bands_and_code_padding():
    """Sentinels around the parameters and the padded tail of the code buffer."""
    dev = _dev()
    n = 2048 * 3 + 0
    buf = torch.full((n + 2 * 1024,), 12345.0, device=dev)
    theta = buf[1024:1024 + n]
    theta.normal_(0, 0.02)
    n2 = 777  # odd, generic kernel; code padding of 15 bytes
    buf2 = torch.full((n2 + 2 * 64,), -7.0, device=dev)
    theta2 = buf2[64:64 + n2]
    theta2.normal_(0, 0.02)
    g = [_grad(n, 1, torch.float32, rows=3, dev=dev), _grad(n2, 2, torch.float32, dev=dev)]
    st = gf.GefenState(g, period_override=[2048, 777])
    for t in range(1, 4):
        st.step([theta, theta2], g, 1e-3, (0.9, 0.999), 1e-8, 0.1, t)
    torch.cuda.synchronize()
    assert (buf[:1024] == 12345.0).all() and (buf[1024 + n:] == 12345.0).all()
    assert (buf2[:64] == -7.0).all() and (buf2[64 + n2:] == -7.0).all()
    lay = st.layout()
    codes = st.read(gf.STATE_CODES).cpu().numpy()
    assert (codes[lay["code_offsets"][0] + n:lay["code_offsets"][1]] == 0).all()
    assert (codes[lay["code_offsets"][1] + n2:lay["code_offsets"][2]] == 0).all()


def test_four_bit_codebook():
    from parity import Run
    dev = _dev()
    p, nb = 768, 10
    n = p * nb
    theta = torch.randn(n, device=dev) * 0.02
    gr = lambda t: [_grad(n, 400 + t, torch.float32, rows=nb, dev=dev)]
    run = Run([theta], gr(1), period_override=[p], code_bits=4)
    assert run.k == 16
    _run_steps(run, gr, 3, where="4-bit")


def test_argument_errors_on_device():
    dev = _dev()
    g = torch.randn(1024, device=dev)
    st = gf.GefenState([g], period_override=[64])
    th = torch.zeros(1024, device=dev)
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.step([th], [g], 1e-3, (0.9, 0.999), 1e-8, 0.0, 0)          # t < 1
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.step([th], [g], 1e-3, (1.0, 0.999), 1e-8, 0.0, 1)          # beta1 = 1
    with pytest.raises(gf.GefenError, match="EDTYPE"):
        st.step([th], [g.bfloat16()], 1e-3, (0.9, 0.999), 1e-8, 0.0, 1)
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.step([th[:512]], [g[:512]], 1e-3, (0.9, 0.999), 1e-8, 0.0, 1)
    with pytest.raises(gf.GefenError, match="EINVAL"):
        gf.GefenState([g], period_override=[1000])                    # does not divide


def test_mixed_tensors_share_one_launch():
    """Tensors of several periods and both gradient dtypes in one state: tiles of the
    smaller classes run inside the largest class's launch (generic path)."""
    from parity import Run
    dev = _dev()
    specs = [(2048, 12, torch.bfloat16), (768, 7, torch.float32), (12, 300, torch.bfloat16),
             (3, 500, torch.float32), (999, 6, torch.bfloat16), (40000, 2, torch.float32),
             (64, 100, torch.float32)]
    params = [torch.randn(p * nb, device=dev) * 0.02 for p, nb, _ in specs]
    gr = lambda t: [_grad(p * nb, 700 + 10 * i + t, dt, dev=dev)
                    for i, (p, nb, dt) in enumerate(specs)]
    run = Run(params, gr(1), period_override=[p for p, _, _ in specs])
    _run_steps(run, gr, 3, where="mixed")
    st = run.state
    st.profile_begin(1)
    st.step(params, gr(4), 1e-3, (0.9, 0.999), 1e-8, 0.1, 4)
    kinds = [c["kind"] for c in st.profile_end()]
    assert kinds.count("uniform_registers") == 1 and "split_block" in kinds, kinds


@pytest.mark.parametrize("code_bits", [8, 4])
def test_split_blocks_of_both_gradient_types(code_bits):
    """Blocks split over workgroups (periods above 65536) in tensors of both gradient
    types, interleaved: each type's split blocks form a launch of their own, so their
    workspace slots are numbered in launch order (numbered tensor by tensor, such a state
    used to be refused by the plan check). Teacher-forced, three steps, and every split
    block in the profile's split class."""
    from parity import Run
    dev = _dev()
    specs = [(70000, 3, torch.float32), (70001, 2, torch.bfloat16), (65540, 2, torch.float32),
             (2048, 4, torch.bfloat16)]
    params = [torch.randn(p * nb, device=dev) * 0.02 for p, nb, _ in specs]
    gr = lambda t: [_grad(p * nb, 4400 + 10 * i + t, dt, dev=dev)
                    for i, (p, nb, dt) in enumerate(specs)]
    run = Run(params, gr(1), period_override=[p for p, _, _ in specs], code_bits=code_bits)
    _run_steps(run, gr, 3, where=f"split blocks of both types {code_bits}-bit")
    st = run.state
    st.profile_begin(1)
    st.step(params, gr(4), 1e-3, (0.9, 0.999), 1e-8, 0.1, 4)
    split = [c for c in st.profile_end() if c["kind"] == "split_block"]
    assert sorted(c["grad_dtype"] for c in split) == ["bf16", "f32"], split


DEGENERATE = [
    # (lr, betas, eps, wd, first t): no momentum memory (m = g); no second-moment memory
    # (v = mean g^2 of this step); a pure decay step (lr = 0 leaves theta unchanged and
    # still updates codes, scales and v); eps = 0 with bias corrections at 1 (large t);
    # strong decay and balanced betas
    (1e-3, (0.0, 0.999), 1e-8, 0.1, 1),
    (1e-3, (0.9, 0.0), 1e-8, 0.0, 1),
    (0.0, (0.9, 0.999), 1e-8, 0.1, 1),
    (1e-2, (0.99, 0.9999), 0.0, 0.0, 1_000_000),
    (1e-3, (0.5, 0.5), 1e-3, 1.0, 1),
]


@pytest.mark.parametrize("lr,betas,eps,wd,t0", DEGENERATE)
def test_degenerate_hyperparameters(lr, betas, eps, wd, t0):
    """Edge settings of the step on every kernel class, one state per class so that
    nothing is folded into the leftover launch: register blocks (p = 64 and 2048),
    streamed (p = 33), lane per block (p = 5), split blocks (p = 70000), and the leftover
    launch (small classes beside a register class)."""
    from parity import Run
    dev = _dev()
    cases = [[(64, 300), (2048, 12)], [(33, 200)], [(5, 400)], [(70000, 2)],
             [(2048, 40), (33, 20), (5, 30)]]
    for ci, specs in enumerate(cases):
        params = [torch.randn(p * nb, device=dev) * 0.02 for p, nb in specs]
        gr = lambda t: [_grad(p * nb, 1000 * ci + 50 * i + t, torch.bfloat16, rows=nb, dev=dev)
                        for i, (p, nb) in enumerate(specs)]
        run = Run(params, gr(0), period_override=[p for p, _ in specs])
        before = [p.clone() for p in params]
        for t in range(t0, t0 + 3):
            run.teacher_forced_step(gr(t), lr, betas, eps, wd, t,
                                    where=f"case {ci} lr={lr} b={betas} t={t}")
        if lr == 0.0:
            for a, b in zip(params, before):
                assert torch.equal(a, b)


@pytest.mark.parametrize("code_bits", [8, 4])
def test_degenerate_codebook_fit(code_bits):
    """A first gradient whose block-normalised values fill only a few histogram bins
    (each block holds +-its absmax and a few fixed fractions of it): the init fit sees
    b < k non-empty bins, reports status 1, and installs the oracle's fallback codebook
    bit for bit: the DP over max(b, 2) entries, strictly increasing from -1 to +1, then
    padded with +1 (App. D has no feasible k-entry solution here). Steps with it, and
    after a refit on ordinary gradients, match the oracle."""
    from parity import Run, grad_bits
    dev = _dev()
    p, nb = 64, 200
    n = p * nb
    levels = torch.tensor([-1.0, -0.5, 0.25, 1.0], device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)
    pick = torch.randint(0, 4, (n,), generator=gen, device=dev)
    pick.view(nb, p)[:, 0] = 3     # every block reaches its absmax
    scales = torch.exp(torch.empty(nb, device=dev).uniform_(-5, 0, generator=gen))
    g0 = (levels[pick].view(nb, p) * scales[:, None]).reshape(-1).contiguous()
    theta = torch.randn(n, device=dev) * 0.02
    run = Run([theta], [g0], period_override=[p], code_bits=code_bits)
    k = run.k
    cost, status = run.state.fit_info()
    h = np.zeros(16 * k, dtype=np.uint64)
    oracle.histogram_blocks(grad_bits(g0), run.offsets[0], 16 * k, h)
    assert int((h > 0).sum()) < k
    cb_ref, cost_ref, _, st_ref = oracle.dp_codebook(h, k)
    assert status == st_ref == 1 and cost == cost_ref
    cb = run.state.read(gf.STATE_CB_DEC64).cpu().numpy()
    np.testing.assert_array_equal(cb, cb_ref)
    b = int((h > 0).sum())
    head = cb[:max(b, 2)]
    assert head[0] == -1.0 and head[-1] == 1.0 and (np.diff(head) > 0).all()
    assert (cb[max(b, 2):] == 1.0).all()
    # such a codebook (repeated +1 entries) round-trips through write and a checkpoint
    cb32 = run.state.read(gf.STATE_CB_DEC).clone()
    run.state.write(gf.STATE_CB_DEC, cb32)
    assert torch.equal(run.state.read(gf.STATE_CB_DEC), cb32)
    run.state.import_(run.state.export())
    np.testing.assert_array_equal(run.state.read(gf.STATE_CB_DEC64).cpu().numpy(), cb_ref)
    hp = (1e-3, (0.9, 0.999), 1e-8, 0.1)
    run.teacher_forced_step([g0], *hp, 1, where="degenerate fit t=1")
    g2 = _grad(n, 77, torch.float32, rows=nb, dev=dev)
    run.teacher_forced_step([g2], *hp, 2, where="degenerate fit t=2")
    run.state.fit_codebook([g2])
    _, status2 = run.state.fit_info()
    assert status2 == 0
    run.teacher_forced_step([g2], *hp, 3, where="after refit t=3")


def test_import_refuses_bad_checkpoints_and_leaves_the_state():
    """A checkpoint whose codebook decreases (two entries swapped), or whose header does
    not match the state, is refused before anything is written: the state exports the
    same bytes afterwards."""
    dev = _dev()
    cpu = torch.device("cpu")
    w = W.get("tiny")
    fields = W.scale_fields(w)
    hp = (w.lr, w.betas, w.eps, w.wd)
    pa = W.init_params(w, dev)
    st = gf.GefenState(W.make_grads(w, fields, 1, dev))
    for t in range(1, 4):
        st.step(pa, W.make_grads(w, fields, t, dev), *hp, t)
    good = st.export(device=cpu).numpy()
    k = st.k
    cb = st.read(gf.STATE_CB_DEC64, device=cpu).numpy()
    off = good.tobytes().find(cb.tobytes())
    assert off >= 0
    bad = good.copy()
    vals = bad[off:off + 8 * k].view(np.float64)
    vals[[1, 2]] = vals[[2, 1]]
    with pytest.raises(gf.GefenError, match="codebook"):
        st.import_(torch.from_numpy(bad).to(dev))
    assert np.array_equal(st.export(device=cpu).numpy(), good)
    bad = good.copy()
    bad[8] ^= 1                       # n_tensors in the header
    with pytest.raises(gf.GefenError, match="does not match"):
        st.import_(torch.from_numpy(bad).to(dev))
    assert np.array_equal(st.export(device=cpu).numpy(), good)
    st.import_(torch.from_numpy(good).to(dev))
    assert np.array_equal(st.export(device=cpu).numpy(), good)


@pytest.mark.parametrize("code_bits", [8, 4])
def test_explicit_blocks_are_deterministic(code_bits):
    """Explicit irregular blocks take every kernel class (one lane per small block, one
    workgroup per block, a huge block split over workgroups; with 4-bit codes, nibbles
    shared across blocks and stored by atomic XOR). From one checkpoint, a refit and two
    steps give bitwise the same parameters, codes, scales and second moments twice."""
    dev = _dev()
    rng = np.random.default_rng(17)
    sizes = np.concatenate([[1, 3, 33, 70000, 9000], rng.integers(1, 40, size=200),
                            rng.integers(40, 5000, size=80)])
    rng.shuffle(sizes)
    n = int(sizes.sum())
    n1 = int(sizes[:150].sum())
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    gr = lambda t: [_grad(n1, 300 + t, torch.bfloat16, dev=dev),
                    _grad(n - n1, 400 + t, torch.bfloat16, dev=dev)]
    p0 = [torch.randn(n1, device=dev) * 0.02, torch.randn(n - n1, device=dev) * 0.02]
    st = gf.GefenState(gr(1), block_offsets=offs, code_bits=code_bits)
    ps = [p.clone() for p in p0]
    for t in range(1, 4):
        st.step(ps, gr(t), 1e-3, (0.9, 0.999), 1e-8, 0.1, t)
    ck = st.export()
    p_ck = [p.clone() for p in ps]
    outs = []
    for _ in range(2):
        st.import_(ck)
        for a, b in zip(ps, p_ck):
            a.copy_(b)
        st.fit_codebook(gr(4))
        for t in (4, 5):
            st.step(ps, gr(t), 1e-3, (0.9, 0.999), 1e-8, 0.1, t)
        torch.cuda.synchronize()
        outs.append([p.clone() for p in ps] +
                    [st.read(w).clone() for w in (gf.STATE_CODES, gf.STATE_SCALE, gf.STATE_V,
                                                  gf.STATE_CB_DEC)])
    for i, (x, y) in enumerate(zip(*outs)):
        assert torch.equal(x, y), i


@pytest.mark.parametrize("code_bits", [8, 4])
def test_explicit_block_class_edges(code_bits):
    """Explicit blocks at the edges of the kernel classes: 32 and 33 elements (one lane
    per block against one workgroup per block), 65536 and 65537 (one workgroup against a
    block split over workgroups), with odd neighbours so that 4-bit codes share bytes
    across every edge. Teacher-forced parity against the oracle over three steps."""
    from parity import Run
    dev = _dev()
    sizes = np.array([32, 33, 65536, 1, 65537, 31, 33, 32, 4097, 65536, 7, 65537, 3],
                     dtype=np.int64)
    n = int(sizes.sum())
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    params = [torch.randn(n, device=dev) * 0.02]
    gr = lambda t: [_grad(n, 500 + t, torch.bfloat16, dev=dev)]
    run = Run(params, gr(1), block_offsets=offs, code_bits=code_bits)
    _run_steps(run, gr, 3, where=f"class edges {code_bits}-bit")


def test_uniform_long_period_streamed():
    """A uniform period just above the register kernel's limit with enough blocks
    (4096) to stay in the one-workgroup-per-block kernel rather than being split: every
    block of an 8196 x 4096 tensor, teacher-forced against the oracle."""
    from parity import Run
    dev = _dev()
    p, nb = 8196, 4096
    n = p * nb
    params = [torch.randn(n, device=dev) * 0.02]
    gr = lambda t: [_grad(n, 700 + t, torch.bfloat16, rows=nb, dev=dev)]
    run = Run(params, gr(1), period_override=[p])
    _run_steps(run, gr, 2, where="p=8196 x 4096")
    run.state.profile_begin(1)
    run.state.step(params, gr(3), HP["lr"], HP["betas"], HP["eps"], HP["wd"], 3)
    assert [k["kind"] for k in run.state.profile_end()] == ["streamed_block"]


def _single_block_sizes(seed):
    """Explicit block sizes of one workgroup each (2043 to 32769 elements, with the
    powers of two and their successors), register runs and small blocks around them."""
    rng = np.random.default_rng(seed)
    sizes = np.concatenate([[2043, 4096, 4097, 8192, 8193, 16384, 16385, 32768, 32769, 1, 5,
                             33, 2042],
                            rng.integers(2043, 32769, size=24), rng.integers(33, 2043, size=8)])
    rng.shuffle(sizes)
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)


@pytest.mark.parametrize("code_bits", [8, 4])
@pytest.mark.parametrize("gdt", [torch.bfloat16, torch.float32])
def test_single_blocks(gdt, code_bits):
    """Explicit blocks of 2043 to 32769 elements, one per workgroup, beside register runs
    and small blocks: three steps teacher-forced against the oracle."""
    from parity import Run
    dev = _dev()
    offs = _single_block_sizes(41 + code_bits)
    n = int(offs[-1])
    params = [torch.randn(n, device=dev) * 0.02]
    gr = lambda t: [_grad(n, 4100 + t, gdt, dev=dev)]
    run = Run(params, gr(1), block_offsets=offs, code_bits=code_bits)
    _run_steps(run, gr, 3, where=f"single blocks {code_bits}-bit {gdt}")


@pytest.mark.parametrize("code_bits", [8, 4])
def test_single_blocks_misaligned(code_bits):
    """Explicit single blocks on parameter and gradient views at odd element offsets.
    Teacher-forced, three steps."""
    from parity import Run
    dev = _dev()
    offs = _single_block_sizes(7)[:12]
    n = int(offs[-1])
    pbuf = torch.randn(n + 3, device=dev) * 0.02
    theta = pbuf[1:1 + n]
    assert theta.data_ptr() % 16 != 0
    gbufs = {t: _grad(n + 1, 4200 + t, torch.bfloat16, dev=dev) for t in range(1, 4)}
    run = Run([theta], [gbufs[1][1:]], block_offsets=offs, code_bits=code_bits)
    _run_steps(run, lambda t: [gbufs[t][1:]], 3, where=f"single blocks misaligned {code_bits}")


def test_tiny_tensors_inferred():
    """Tensors of 1 to 12 elements (a scalar parameter, primes, small composites) beside a
    normal matrix, both gradient dtypes, periods inferred on the GPU: each period equals
    the oracle's Alg. 2 result on the same bits, and three steps match the oracle."""
    from parity import Run, grad_bits
    dev = _dev()
    sizes = [1, 2, 3, 5, 7, 4, 6, 12, 2048 * 6]
    dts = [torch.float32, torch.bfloat16] * 4 + [torch.bfloat16]
    params = [torch.randn(n, device=dev) * 0.02 for n in sizes]
    gr = lambda t: [_grad(n, 900 + 7 * i + t, dt, rows=6 if n > 12 else None, dev=dev)
                    for i, (n, dt) in enumerate(zip(sizes, dts))]
    g1 = gr(1)
    run = Run(params, g1)
    for i, g in enumerate(g1):
        _, _, per = oracle.partition(grad_bits(g), 1e-8)
        assert run.periods[i] == per, (sizes[i], run.periods[i], per)
    _run_steps(run, gr, 3, where="tiny tensors")
