"""Free-running report: the library and the oracle each run Gefen (Alg. 1) on their own
from the same start, with no state exchanged after it.

Both start from the library's state after init (the periods of Alg. 2 and the codebook of
Alg. 3, which the other tests pin to the oracle bit for bit; codes, scales and second
moments zero) and the same parameters, and take the same gradient bits every step. The
oracle then runs in float64 on its own state, the library in float32 on its own. Per
step the report gives the share of codes that differ, the largest parameter difference
(absolute, and relative to the largest parameter magnitude of its tensor), and the
largest relative differences of the block scales and second moments.

Not gated (only finiteness is asserted): a tie that float32 decides the other way
changes one momentum by a codebook gap times the scale, and the two runs then drift
apart by construction -- the reason the parity tests are teacher-forced. The report
shows how far they drift on the model workloads. For the two large models the oracle
runs a fixed subset of tensors (every kind of tensor of the first layers): the step is
independent per block once the codebook is fixed, so a subset runs exactly as it would
inside the whole model, which the library steps whole.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

gf = pytest.importorskip("paper_2606_13894_amd")

# (workload, code bits, steps, tensor indices the oracle runs; None: all)
CASES = [
    ("tiny", 8, 10, None),
    ("tiny", 4, 10, None),
    ("gpt2_125m", 8, 10, [1, 2, 3, 4, 5, 6, 10, 12]),
    ("llama3_1p5b", 8, 6, [1, 2, 3, 4, 8, 9]),
]


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda", 0)


def _snap(run, idx):
    """The library's parameters, codes, scales and second moments of tensors idx."""
    from parity import unpack_codes
    torch.cuda.synchronize()
    codes = unpack_codes(run.state.read(gf.STATE_CODES).cpu().numpy(), run.k)
    scale = run.state.read(gf.STATE_SCALE).cpu().numpy().astype(np.float64)
    v = run.state.read(gf.STATE_V).cpu().numpy().astype(np.float64)
    out = {"theta": {}, "codes": {}, "s": {}, "v": {}}
    for i in idx:
        n = run.numels[i]
        out["theta"][i] = run.params[i].detach().reshape(-1).cpu().numpy().astype(np.float64)
        out["codes"][i] = codes[run.code_off[i]:run.code_off[i] + n].copy()
        out["s"][i] = scale[run.blk_idx[i]:run.blk_idx[i + 1]].copy()
        out["v"][i] = v[run.blk_idx[i]:run.blk_idx[i + 1]].copy()
    return out


@pytest.mark.parametrize("name,code_bits,steps,subset", CASES,
                         ids=[f"{c[0]}-{c[1]}bit" for c in CASES])
def test_free_running_report(name, code_bits, steps, subset):
    from parity import Run, grad_bits
    dev = _dev()
    w = W.get(name)
    fields = W.scale_fields(w)
    params = W.init_params(w, dev)
    g1 = W.make_grads(w, fields, 1, dev)
    run = Run(params, g1, code_bits=code_bits)
    idx = list(range(len(params))) if subset is None else subset
    start = _snap(run, idx)
    cb_dec = run.state.read(gf.STATE_CB_DEC).cpu().numpy().astype(np.float64)
    cb_enc = run.state.read(gf.STATE_CB_ENC).cpu().numpy().astype(np.float64)
    # the oracle's own state: the start, in float64
    th = {i: start["theta"][i].copy() for i in idx}
    cq = {i: start["codes"][i].copy() for i in idx}
    s = {i: start["s"][i].copy() for i in idx}
    v = {i: start["v"][i].copy() for i in idx}
    assert not any(c.any() for c in cq.values())
    lr, (b1, b2), eps, wd = w.lr, w.betas, w.eps, w.wd
    rows = []
    for t in range(1, steps + 1):
        g = g1 if t == 1 else W.make_grads(w, fields, t, dev)
        run.step(g, lr, (b1, b2), eps, wd, t)
        for i in idx:
            oracle.step_blocks(th[i], grad_bits(g[i]), cq[i], s[i], v[i], run.offsets[i],
                               cb_dec, cb_enc, lr, b1, b2, eps, wd, t)
        post = _snap(run, idx)
        n = mism = 0
        d_abs = d_rel = s_rel = v_rel = 0.0
        for i in idx:
            tg, to = post["theta"][i], th[i]
            assert np.isfinite(tg).all() and np.isfinite(to).all(), (name, t, i)
            n += tg.size
            mism += int(np.count_nonzero(post["codes"][i] != cq[i]))
            d = np.abs(tg - to)
            d_abs = max(d_abs, float(d.max()))
            d_rel = max(d_rel, float(d.max() / max(np.abs(to).max(), 1e-30)))
            for ref, got, acc in ((s[i], post["s"][i], "s"), (v[i], post["v"][i], "v")):
                e = np.abs(got - ref) / np.maximum(np.abs(ref), 1e-30)
                e = float(e[ref != 0].max()) if (ref != 0).any() else 0.0
                if acc == "s":
                    s_rel = max(s_rel, e)
                else:
                    v_rel = max(v_rel, e)
        rows.append((t, mism / n, d_abs, d_rel, s_rel, v_rel))
        del g
    print(f"\nfree-running {name} {code_bits}-bit, {len(idx)} tensors, "
          f"{sum(th[i].size for i in idx)} elements")
    print(" step  code mismatch  max|dtheta|  max|dtheta|/max|theta|  max rel ds  max rel dv")
    for t, mr, da, dr, sr, vr in rows:
        print(f" {t:4d}  {mr:13.3e}  {da:11.3e}  {dr:22.3e}  {sr:10.3e}  {vr:10.3e}")
    del run, params, g1
    torch.cuda.empty_cache()
