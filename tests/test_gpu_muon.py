"""Gefen-Muon (appendix "Gefen-Muon") on the GPU against the oracle, through the C ABI.

Teacher-forced per step: before each step the oracle takes the library's codes, scales,
codebooks and parameters. Three stages are checked:

* codec: codes and scales with the gates of the Gefen step (ties at midpoints excepted);
* the bfloat16 momentum matrix U (state array 6): within one bfloat16 rounding of the
  oracle's float64 value, plus a cancellation floor for the float32 momentum;
* orthogonalisation and update: the library's O (recovered from the parameter change,
  O = (theta * decay - theta') / (lr * scale)) against the oracle's bfloat16
  Newton-Schulz of the library's own U, free-running over Muon's five iterations. Both
  round every product to bfloat16 at the same points (each single iteration is pinned
  element by element in tests/test_gpu_newton_schulz.py); over five iterations the rare
  one-step flips of float32 accumulation order spread, so the gate is the oracle's own
  pin against torch's bfloat16 Muon on the CPU: 1 % of ||O|| in Frobenius norm, 3 % of
  max |O| per element (plus the float32 rounding of the parameter update).
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


def _grad(rows, cols, seed, dtype, dev):
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    g = torch.randn(rows, cols, generator=gen, device=dev)
    sc = torch.exp(torch.empty(rows, 1, device=dev).uniform_(np.log(1e-3), 0, generator=gen))
    return (g * sc).reshape(-1).to(dtype)


class MuonRun:
    def __init__(self, shapes, dtype, dev, seed=0, code_bits=8, block_offsets=None,
                 period_override=None):
        from parity import Run
        self.shapes = shapes
        self.dtype = dtype
        self.dev = dev
        self.seed = seed
        self.params = [torch.randn(r * c, device=dev) * 0.02 for r, c in shapes]
        g1 = self.grads(0)
        self.run = Run(self.params, g1, block_offsets=block_offsets, code_bits=code_bits,
                       period_override=period_override)
        self.st = self.run.state
        self.st.muon_init([r for r, _ in shapes])

    def grads(self, t):
        return [_grad(r, c, self.seed + 1000 * i + t, self.dtype, self.dev)
                for i, (r, c) in enumerate(self.shapes)]

    def step(self, t, lr=0.02, mu=0.95, wd=0.01, nesterov=True, where=""):
        from parity import grad_bits, unpack_codes
        run = self.run
        grads = self.grads(t)
        pre = run.snapshot()
        self.st.muon_step(self.params, grads, lr, mu, wd, nesterov)
        post = run.snapshot()
        u_all = self.st.read(gf.STATE_MUON_U).cpu().numpy().view(np.uint16)
        u_all = (u_all.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        cb_dec, cb_enc = pre["cb_dec"], pre["cb_enc"]
        worst = {"o_max": 0.0, "o_fro": 0.0, "ties": 0}
        for i, (R, C) in enumerate(self.shapes):
            n = R * C
            offs = run.offsets[i]
            codes = pre["codes"][i].copy()
            s = pre["s"][i].copy()
            g = grad_bits(grads[i])
            u_ref = oracle.muon_codec_blocks(g, codes, s, offs, cb_dec, cb_enc, mu, nesterov)
            # codec: scales and codes
            gd = grads[i].double().cpu().numpy()
            sizes = np.diff(offs)
            blk = np.repeat(np.arange(sizes.size), sizes)
            prev = np.abs(cb_dec[pre["codes"][i]] * pre["s"][i][blk])
            mag = mu * prev + (1 - mu) * np.abs(gd)
            bmag = np.zeros(sizes.size)
            np.maximum.at(bmag, blk, mag)
            ds = np.abs(post["s"][i] - s)
            assert (ds <= 1e-6 * s + 1e-6 * bmag).all(), f"{where} tensor {i}: scale"
            bad = np.nonzero(post["codes"][i] != codes)[0]
            if bad.size:
                m_ref = oracle.muon_codec_blocks(g, pre["codes"][i].copy(), pre["s"][i].copy(),
                                                 offs, cb_dec, cb_enc, mu, False)
                x = m_ref[bad] / np.where(s[blk[bad]] > 0, s[blk[bad]], 1.0)
                a, b = post["codes"][i][bad].astype(int), codes[bad].astype(int)
                assert (np.abs(a - b) == 1).all(), f"{where} tensor {i}: non-adjacent code"
                midp = 0.5 * (cb_enc[np.minimum(a, b)] + cb_enc[np.maximum(a, b)])
                delta = 1e-6 * np.maximum(1.0, bmag[blk[bad]] / np.where(s[blk[bad]] > 0,
                                                                          s[blk[bad]], 1.0))
                assert (np.abs(x - midp) <= delta).all(), f"{where} tensor {i}: code"
                worst["ties"] += bad.size
            # bfloat16 momentum matrix
            c0 = run.code_off[i]
            u_gpu = u_all[c0:c0 + n]
            tol_u = 2.0 ** -8 * np.abs(u_ref) + 2e-6 * (mag + np.abs(gd))
            assert (np.abs(u_gpu - u_ref) <= tol_u).all(), f"{where} tensor {i}: U"
            # orthogonalisation + update
            o_ref = oracle.newton_schulz(u_gpu, R, C).reshape(-1)
            decay = 1.0 - lr * wd
            step = lr * oracle.muon_lr_scale(R, C)
            th_pre = pre["theta"][i]
            o_gpu = (th_pre * decay - post["theta"][i]) / step
            scale_o = max(np.abs(o_ref).max(), 1e-30)
            d = np.abs(o_gpu - o_ref)
            noise = 4e-7 * (np.abs(th_pre) + np.abs(post["theta"][i])) / step
            assert (d <= 0.03 * scale_o + noise).all(), (where, i, d.max() / scale_o)
            fro = np.sqrt(np.sum(d ** 2)) / max(np.sqrt(np.sum(o_ref ** 2)), 1e-30)
            fro_noise = np.sqrt(np.sum(noise ** 2)) / max(np.sqrt(np.sum(o_ref ** 2)), 1e-30)
            assert fro <= 0.01 + fro_noise, (where, i, fro)
            worst["o_max"] = max(worst["o_max"], d.max() / scale_o)
            worst["o_fro"] = max(worst.get("o_fro", 0.0), fro)
        return worst


SHAPES = [[(64, 192)], [(192, 64)], [(128, 128)], [(1, 300)], [(300, 1)], [(3, 5)],
          [(64, 128), (128, 64), (64, 128), (1, 77), (64, 128), (128, 64), (96, 96)],
          # lone tall-skinny matrices: the Gram product is split over K (even chunks; a
          # remainder chunk)
          [(64, 4096)], [(5000, 48)],
          # tall matrices with ragged edges (rows not a multiple of 8 or of the 64-row
          # tile; columns not a multiple of 8), two of one shape batched together
          [(1003, 40), (77, 9), (1003, 40), (130, 129)],
          # tall and wide tensors of one wide shape share a batch (1008 x 40 is stored
          # transposed, 40 x 1008 as it is); 1 x n and n x 1 share the vector kernel
          [(1008, 40), (40, 1008), (1, 50), (50, 1), (1008, 40)],
          # lone wide tall-skinny matrix whose K does not split evenly (remainder chunk)
          [(48, 5000)]]


@pytest.mark.parametrize("shapes", SHAPES, ids=lambda s: "+".join(f"{r}x{c}" for r, c in s))
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_muon_parity_shapes(shapes, dtype):
    dev = _dev()
    mr = MuonRun(shapes, dtype, dev, seed=len(shapes))
    for t in range(1, 4):
        mr.step(t, where=f"t={t}")


@pytest.mark.parametrize("seed", range(12))
def test_muon_random_models(seed):
    """Seeded random models: up to eight tensors of random sides (vectors, tiny, square,
    tall and wide, with repeats and the other orientation of a shape, so that groups batch
    tensors of both orientations and the lanes get several groups), either gradient type,
    both code widths; two steps against the oracle."""
    dev = _dev()
    rng = np.random.default_rng(900 + seed)
    shapes = []
    for _ in range(int(rng.integers(1, 6))):
        kind = int(rng.integers(5))
        if kind == 0:
            r, c = (1, int(rng.integers(2, 900))) if rng.integers(2) else (int(rng.integers(2, 900)), 1)
        elif kind == 1:
            r, c = int(rng.integers(2, 24)), int(rng.integers(2, 24))
        elif kind == 2:
            r, c = int(rng.integers(8, 64)), int(rng.integers(500, 3000))
        else:
            r, c = int(rng.integers(16, 400)), int(rng.integers(16, 400))
        shapes += [(r, c)] * int(rng.integers(1, 3))
        if rng.integers(2):
            shapes.append((c, r))
    shapes = shapes[:8]
    dtype = torch.bfloat16 if rng.integers(2) else torch.float32
    code_bits = int(rng.choice([8, 4]))
    mr = MuonRun(shapes, dtype, dev, seed=seed, code_bits=code_bits)
    for t in (1, 2):
        mr.step(t, where=f"seed {seed} {shapes} {code_bits}-bit t={t}")


@pytest.mark.parametrize("code_bits", [8, 4])
@pytest.mark.parametrize("nesterov", [True, False])
def test_muon_code_widths_and_nesterov(code_bits, nesterov):
    dev = _dev()
    mr = MuonRun([(96, 160), (160, 96), (1, 160)], torch.bfloat16, dev, seed=5,
                 code_bits=code_bits)
    for t in range(1, 4):
        mr.step(t, nesterov=nesterov, where=f"cb{code_bits} nesterov={nesterov} t={t}")


def test_muon_explicit_blocks_and_refit():
    dev = _dev()
    rng = np.random.default_rng(9)
    shapes = [(48, 100), (100, 48)]
    n = sum(r * c for r, c in shapes)
    sizes = np.concatenate([rng.integers(1, 40, 60), rng.integers(40, 600, 14)])
    sizes = sizes[np.cumsum(sizes) < n - 4800]
    bounds = np.concatenate([[0], np.cumsum(sizes)])
    bounds = np.unique(np.concatenate([bounds, [4800, n]]))
    mr = MuonRun(shapes, torch.float32, dev, seed=9, block_offsets=bounds.astype(np.int64))
    mr.step(1, where="explicit t=1")
    mr.step(2, where="explicit t=2")
    mr.st.fit_codebook(mr.grads(2))
    mr.step(3, where="explicit after refit")
    mr.step(4, where="explicit t=4")


def test_muon_gpt2_mlp_shape():
    """One GPT-2 small MLP pair at full size (768 x 3072 and 3072 x 768)."""
    dev = _dev()
    mr = MuonRun([(768, 3072), (3072, 768)], torch.float32, dev, seed=11)
    w = mr.step(1, where="gpt2 mlp t=1")
    w = mr.step(2, where="gpt2 mlp t=2")
    print("worst O deviation (max, mean) / max|O|:", w)


def test_muon_three_lanes_against_the_oracle():
    """A model whose groups fill all three lanes: four 1024 x 2048 matrices (three wide,
    one tall; lane 0), four 768 x 2304 ones (lane 1), both long enough to count for more
    than their launches and with split-K Grams, and the latency-bound small matrices and
    vectors (lane 2). Every tensor against the oracle, teacher-forced, two steps."""
    dev = _dev()
    shapes = ([(1024, 2048)] * 3 + [(2048, 1024)] + [(768, 2304)] * 4 +
              [(64, 128), (128, 64), (1, 300), (96, 96), (300, 1)])
    mr = MuonRun(shapes, torch.bfloat16, dev, seed=31)
    for t in (1, 2):
        w = mr.step(t, where=f"three lanes t={t}")
    print("worst O deviation (max, mean) / max|O|:", w)


def test_muon_lanes_are_deterministic():
    """The shape groups run on three concurrent streams; the same state and inputs give
    the same parameters bit for bit in two runs from scratch (no race between the lanes
    and no order-dependent accumulation), including the split-K Gram, the vector kernel,
    tall and wide parts and groups on every lane."""
    dev = _dev()
    shapes = [(5000, 48), (64, 128), (128, 64), (1, 77), (96, 96), (300, 1), (64, 128),
              (768, 3072), (3072, 768), (1024, 2048), (1024, 2048), (2048, 1024), (1024, 2048),
              (768, 2304), (768, 2304), (768, 2304), (768, 2304)]
    runs = []
    for _ in range(2):
        torch.manual_seed(21)
        ps = [torch.randn(r * c, device=dev) * 0.02 for r, c in shapes]
        gs = [[_grad(r, c, 100 * t + i, torch.bfloat16, dev) for i, (r, c) in enumerate(shapes)]
              for t in range(4)]
        st = gf.GefenState(gs[0])
        st.muon_init([r for r, _ in shapes])
        for t in range(4):
            st.muon_step(ps, gs[t], 0.02, 0.95, 0.01, True)
        torch.cuda.synchronize()
        runs.append([p.clone() for p in ps])
        st.close()
    for i, (a, b) in enumerate(zip(*runs)):
        assert torch.equal(a, b), f"tensor {i} {shapes[i]}"


def test_muon_lossless_block_size_one_matches_torch_muon():
    """Block size 1: the stored momentum is exact, so Gefen-Muon is Muon; free-running
    against torch.optim.Muon on the GPU (both bfloat16 Newton-Schulz)."""
    dev = _dev()
    R, C = 96, 256
    torch.manual_seed(3)
    theta0 = torch.randn(R * C, device=dev) * 0.02
    p_gef = theta0.clone()
    p_ref = torch.nn.Parameter(theta0.clone().reshape(R, C))
    lr, mu, wd = 0.02, 0.95, 0.01
    opt = torch.optim.Muon([p_ref], lr=lr, momentum=mu, weight_decay=wd, nesterov=True)
    gs = [torch.randn(R * C, device=dev) for _ in range(4)]
    st = gf.GefenState([gs[0]], period_override=[1])
    st.muon_init([R])
    for g in gs:
        st.muon_step([p_gef], [g], lr, mu, wd, True)
        p_ref.grad = g.reshape(R, C).clone()
        opt.step()
    torch.cuda.synchronize()
    step = lr * oracle.muon_lr_scale(R, C)
    diff = (p_gef - p_ref.detach().reshape(-1)).abs().max().item()
    moved = (p_gef - theta0).abs().max().item()
    assert diff < 0.03 * step, (diff / step)
    assert moved > 10 * diff


def test_muon_argument_errors():
    dev = _dev()
    g = torch.randn(12 * 8, device=dev)
    p = torch.zeros_like(g)
    st = gf.GefenState([g])
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.muon_step([p], [g], 0.02)                      # before muon_init
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.muon_init([5])                                 # 5 does not divide 96
    st.muon_init([12])
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.muon_init([12])                                # second call
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.muon_step([p], [g], 0.02, momentum=1.0)
    with pytest.raises(gf.GefenError, match="EINVAL"):
        st.muon_step([p], [g], 0.02, ns_eps=0.0)
    st.muon_step([p], [g], 0.02)
    torch.cuda.synchronize()
    assert torch.isfinite(p).all()


def test_muon_large_k_embedding_shape():
    """A GPT-2 1B token-embedding shape (2048 x 50257: the Gram product has K = 50257,
    where the GEMM library picks split-K solutions that need workspace). Lossless codes
    (block size 1); against torch.optim.Muon on the GPU for two steps."""
    dev = _dev()
    R, C = 50257, 2048
    torch.manual_seed(5)
    theta0 = torch.randn(R * C, device=dev) * 0.02
    p_gef = theta0.clone()
    p_ref = torch.nn.Parameter(theta0.clone().reshape(R, C))
    lr, mu, wd = 0.02, 0.95, 0.01
    opt = torch.optim.Muon([p_ref], lr=lr, momentum=mu, weight_decay=wd, nesterov=True)
    gs = [torch.randn(R * C, device=dev) for _ in range(2)]
    st = gf.GefenState([gs[0]], period_override=[1])
    st.muon_init([R])
    for g in gs:
        st.muon_step([p_gef], [g], lr, mu, wd, True)
        p_ref.grad = g.reshape(R, C).clone()
        opt.step()
    torch.cuda.synchronize()
    step = lr * oracle.muon_lr_scale(R, C)
    diff = (p_gef - p_ref.detach().reshape(-1)).abs().max().item()
    assert torch.isfinite(p_gef).all()
    assert diff < 0.03 * step, (diff / step)


def test_muon_gpt2_1b_shapes():
    """The GPT-2 1B shapes (292 tensors, 1.31e9 parameters; a batch of 48 MLP matrices of
    2048 x 8192, tall and wide together, and the 50257 x 2048 embedding) run a whole
    Gefen-Muon step. One matrix of each large shape group is checked against the oracle,
    teacher-forced on the library's own U: the embedding, an MLP up- and down-projection,
    an attention projection and a fused QKV matrix."""
    import workloads as W
    from parity import grad_bits
    dev = _dev()
    w = W.get("gpt2_1b")
    fields = W.scale_fields(w)
    params = W.init_params(w, dev)
    g1 = W.make_grads(w, fields, 1, dev)
    st = gf.GefenState(g1, eps_part=w.eps)
    rows = [t.rows for t in w.tensors]
    st.muon_init(rows)
    lay = st.layout()
    pre = [p.detach().clone() for p in params]
    lr, mu, wd = 0.02, 0.95, 0.01
    st.muon_step(params, g1, lr, mu, wd, True)
    torch.cuda.synchronize()
    u_all = st.read(gf.STATE_MUON_U).cpu().numpy().view(np.uint16)
    u_all = (u_all.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    names = [t.name for t in w.tensors]
    pick = [names.index(nm) for nm in ("wte", "h0.mlp.c_fc.weight", "h0.mlp.c_proj.weight",
                                        "h5.attn.c_proj.weight", "h11.attn.c_attn.weight")]
    decay = 1.0 - lr * wd
    for i in pick:
        R = w.tensors[i].rows
        C = w.tensors[i].numel // R
        c0 = lay["code_offsets"][i]
        u = u_all[c0:c0 + R * C]
        o_ref = oracle.newton_schulz(u, R, C).reshape(-1)
        step = lr * oracle.muon_lr_scale(R, C)
        th0 = pre[i].double().cpu().numpy().reshape(-1)
        th1 = params[i].detach().double().cpu().numpy().reshape(-1)
        o_gpu = (th0 * decay - th1) / step
        d = np.abs(o_gpu - o_ref)
        noise = 4e-7 * (np.abs(th0) + np.abs(th1)) / step
        assert (d <= 0.03 * np.abs(o_ref).max() + noise).all(), (names[i], d.max())
        fro = np.sqrt(np.sum(d ** 2) / np.sum(o_ref ** 2))
        assert fro <= 0.01 + np.sqrt(np.sum(noise ** 2) / np.sum(o_ref ** 2)), (names[i], fro)
        print(f"{names[i]} ({R} x {C}): O within {fro:.2e} (Frobenius) of the oracle")
    for p in params:
        assert torch.isfinite(p).all()
    st.close()


def test_gefen_muon_front_end_matches_the_state_calls():
    """The optimizer-style front end makes exactly the calls of the state API: init from
    the first gradients, muon_init with each parameter's rows, then muon_step."""
    dev = _dev()
    shapes = [(64, 96), (96, 64), (77,)]
    torch.manual_seed(4)
    p0 = [torch.randn(*s, device=dev) * 0.02 for s in shapes]
    gs = [[torch.randn(*s, device=dev) for s in shapes] for _ in range(3)]
    ps = [torch.nn.Parameter(p.clone()) for p in p0]
    opt = gf.GefenMuon(ps, lr=0.02, weight_decay=0.01)
    for g in gs:
        for p, gi in zip(ps, g):
            p.grad = gi
        opt.step()
    ref = [p.clone().reshape(-1) for p in p0]
    st = gf.GefenState([g.reshape(-1) for g in gs[0]])
    st.muon_init([s[0] if len(s) == 2 else 1 for s in shapes])
    for g in gs:
        st.muon_step(ref, [gi.reshape(-1) for gi in g], 0.02, 0.95, 0.01, True)
    torch.cuda.synchronize()
    for a, b in zip(ps, ref):
        assert torch.equal(a.detach().reshape(-1), b)


def test_steps_on_a_side_stream_match_the_default_stream():
    """Everything the library enqueues follows the caller's stream: the Gefen step and
    Gefen-Muon (whose second lane forks from that stream and joins back) on a
    non-default torch stream give bitwise the results of the default stream."""
    dev = _dev()
    shapes = [(64, 96), (96, 64), (77, 1), (128, 128)]
    gs = [[_grad(r, c, 40 * t + i, torch.bfloat16, dev) for i, (r, c) in enumerate(shapes)]
          for t in range(3)]
    out = {}
    side = torch.cuda.Stream()
    for name, stream in (("default", None), ("side", side)):
        torch.manual_seed(12)
        p_step = [torch.randn(r * c, device=dev) * 0.02 for r, c in shapes]
        p_muon = [p.clone() for p in p_step]
        torch.cuda.synchronize()
        ctx = torch.cuda.stream(stream) if stream is not None else torch.cuda.stream(
            torch.cuda.current_stream())
        with ctx:
            a = gf.GefenState(gs[0])
            b = gf.GefenState(gs[0])
            b.muon_init([r for r, _ in shapes])
            for t in range(3):
                a.step(p_step, gs[t], 1e-3, (0.9, 0.999), 1e-8, 0.1, t + 1)
                b.muon_step(p_muon, gs[t], 0.02, 0.95, 0.01, True)
        torch.cuda.synchronize()
        out[name] = [p.clone() for p in p_step + p_muon]
    for i, (x, y) in enumerate(zip(out["default"], out["side"])):
        assert torch.equal(x, y), i



# Kept as the record of a removed experiment; see the skip reason.
SKIP_TUNE = pytest.mark.skip(
    reason="the rocBLAS solution search for the Newton-Schulz products (gefen_muon_tune) "
           "was removed: its one GPU run took an illegal memory access inside a library "
           "solution it timed, whose cause was not found")


@SKIP_TUNE
def test_muon_tuned_products_match_oracle():
    """Steps after gefen_muon_tune (rocBLAS solutions chosen by timing) still match the
    oracle, teacher-forced: a batched wide group holding tall and wide GPT-2 MLP
    matrices, a square group and a lone 256 x 4096 matrix whose Gram product is split
    over K. The search never reports a chosen time above the library's."""
    dev = _dev()
    mr = MuonRun([(768, 3072), (3072, 768), (768, 768), (256, 4096)], torch.float32, dev,
                 seed=31)
    res = mr.st.muon_tune()
    assert 0.0 < res["tuned_us"] <= res["default_us"], res
    for t in (1, 2):
        w = mr.step(t, where=f"tuned t={t}")
    print("tuned products (us):", res, "worst O deviation:", w)


@SKIP_TUNE
def test_muon_tuned_steps_are_deterministic():
    """With the tuned solutions fixed, the same state and inputs give bitwise the same
    parameters (no solution that accumulates with atomics): three steps, a checkpoint
    restore, the same three steps again."""
    dev = _dev()
    shapes = [(768, 3072), (3072, 768), (768, 768), (256, 4096)]
    torch.manual_seed(41)
    p0 = [torch.randn(r * c, device=dev) * 0.02 for r, c in shapes]
    gs = [[_grad(r, c, 100 * t + i, torch.bfloat16, dev) for i, (r, c) in enumerate(shapes)]
          for t in range(3)]
    st = gf.GefenState(gs[0])
    st.muon_init([r for r, _ in shapes])
    st.muon_tune()
    ckpt = st.export()
    out = []
    for rep in range(2):
        if rep:
            st.import_(ckpt)
        ps = [p.clone() for p in p0]
        for t in range(3):
            st.muon_step(ps, gs[t], 0.02, 0.95, 0.01, True)
        torch.cuda.synchronize()
        out.append(ps)
    for i, (a, b) in enumerate(zip(*out)):
        assert torch.equal(a, b), f"tensor {i} {shapes[i]}"


@SKIP_TUNE
def test_muon_tune_before_init_is_refused():
    dev = _dev()
    g = torch.randn(1024, device=dev)
    st = gf.GefenState([g])
    with pytest.raises(gf.GefenError, match="gefen_muon_init"):
        st.muon_tune()
