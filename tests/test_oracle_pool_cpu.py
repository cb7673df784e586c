"""The parallel oracle harness of the full-size GPU tests (tests/oracle_pool.py), on the
CPU: a step whose 'library' state is the oracle's own result passes every gate in every
worker; one wrong code or parameter in the checked state is reported with its tensor
and blocks; partition tasks return the oracle's periods."""
import numpy as np

import oracle
import oracle_pool


def _job(tmp_path, rng):
    shapes = [(64, 40), (1, 300), (7, 128)]      # period, blocks
    numel = [p * nb for p, nb in shapes]
    elem_off = np.concatenate([[0], np.cumsum(numel)]).astype(np.int64)
    blk = np.concatenate([[0], np.cumsum([nb for _, nb in shapes])]).astype(np.int64)
    n, nbt = int(elem_off[-1]), int(blk[-1])
    g0 = rng.standard_normal(4096).astype(np.float32)
    h = oracle.histogram_uniform(g0, 64, 4096)
    cb, _, _, _ = oracle.dp_codebook(h, 256)
    theta = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g = (rng.standard_normal(n) * 0.1).astype(np.float32)
    codes = rng.integers(0, 256, n).astype(np.uint8)
    s = rng.uniform(0.01, 1, nbt).astype(np.float32)
    v = rng.uniform(0.01, 1, nbt).astype(np.float32)
    hp = {"lr": 1e-3, "b1": 0.9, "b2": 0.999, "eps": 1e-8, "wd": 0.1, "t": 4}
    post = {"theta": theta.copy(), "codes": codes.copy(), "s": s.copy(), "v": v.copy()}
    job = str(tmp_path)
    tasks, sizes = [], []
    for i, (p, nb) in enumerate(shapes):
        offs = np.arange(0, p * nb + 1, p, dtype=np.int64)
        oracle_pool.save(job, f"offs_{i}", offs)
        sl, bl = slice(elem_off[i], elem_off[i + 1]), slice(blk[i], blk[i + 1])
        th = theta[sl].astype(np.float64)
        c = codes[sl].copy()
        s_ = s[bl].astype(np.float64)
        v_ = v[bl].astype(np.float64)
        oracle.step_blocks(th, g[sl], c, s_, v_, offs, cb, cb, hp["lr"], hp["b1"], hp["b2"],
                           hp["eps"], hp["wd"], hp["t"])
        post["theta"][sl] = th.astype(np.float32)
        post["codes"][sl] = c
        post["s"][bl] = s_.astype(np.float32)
        post["v"][bl] = v_.astype(np.float32)
        for b0 in range(0, nb, 16):
            tasks.append({"kind": "step", "tensor": i, "b0": b0, "b1": min(nb, b0 + 16)})
            sizes.append(min(nb, b0 + 16) - b0)
    for name, a in (("theta_pre", theta), ("codes_pre", codes), ("s_pre", s), ("v_pre", v),
                    ("grad", g), ("cb_dec", cb), ("cb_enc", cb)):
        oracle_pool.save(job, name, a)
    meta = {"elem_off": elem_off.tolist(), "blk_off": blk.tolist(), "hp": hp,
            "numel": numel, "eps_part": 1e-8}
    return job, meta, tasks, sizes, post, shapes, elem_off


def _save_post(job, post):
    for k, a in post.items():
        oracle_pool.save(job, f"{k}_post", a)


def test_pool_passes_an_exact_state_and_reports_planted_errors(tmp_path):
    rng = np.random.default_rng(3)
    job, meta, tasks, sizes, post, shapes, elem_off = _job(tmp_path, rng)
    _save_post(job, post)
    res = oracle_pool.run(job, meta, tasks, sizes, 3, timeout=300)
    assert len(res) == len(tasks) and all(r["ok"] for r in res)
    assert sum(r["result"]["codes"] for r in res) == elem_off[-1]
    # a code two entries away, in tensor 2, block 9 (elements 63..69)
    bad = {k: a.copy() for k, a in post.items()}
    j = int(elem_off[2]) + 9 * 7 + 3
    bad["codes"][j] = (int(bad["codes"][j]) + 2) % 256
    _save_post(job, bad)
    res = oracle_pool.run(job, meta, tasks, sizes, 3, timeout=300)
    fails = [r for r in res if not r["ok"]]
    assert len(fails) == 1 and fails[0]["task"]["tensor"] == 2 and fails[0]["task"]["b0"] == 0
    # a parameter off by 1e-4 relative in tensor 0
    bad = {k: a.copy() for k, a in post.items()}
    bad["theta"][100] *= 1.0 + 1e-4
    _save_post(job, bad)
    res = oracle_pool.run(job, meta, tasks, sizes, 3, timeout=300)
    fails = [r for r in res if not r["ok"]]
    assert len(fails) == 1 and fails[0]["task"]["tensor"] == 0
    assert "theta gate" in fails[0]["error"]


def test_pool_partition_tasks(tmp_path):
    rng = np.random.default_rng(4)
    job, meta, _, _, _, shapes, elem_off = _job(tmp_path, rng)
    g = np.concatenate([(rng.standard_normal((nb, p)) * np.exp(rng.uniform(-6, 0, (nb, 1))))
                        .astype(np.float32).reshape(-1) for p, nb in shapes])
    oracle_pool.save(job, "grad", g)
    tasks = [{"kind": "partition", "tensor": i} for i in range(len(shapes))]
    res = oracle_pool.run(job, meta, tasks, [1, 1, 1], 2, timeout=300)
    for r in res:
        i = r["task"]["tensor"]
        gi = g[elem_off[i]:elem_off[i + 1]]
        _, scores, per = oracle.partition(gi, 1e-8)
        assert r["result"]["period"] == per
        np.testing.assert_array_equal(np.array(r["result"]["scores"]), scores)


def test_code_gate_accepts_rounding_ties_and_refuses_other_codes():
    """The code gate of tests/gates.py: a block of one element whose momentum cancels
    exactly in real arithmetic (bf16 gradients, g_2 = -0.9 g_1, beta1 = 0.9) holds
    rounding noise on both sides, so either end code is a tie; a far code for a
    well-conditioned element is refused."""
    import gates
    import pytest
    cb = np.linspace(-1.0, 1.0, 256)
    b1 = 0.9
    g1, g2 = 0.205078125, -0.1845703125          # bf16 values, g2 = -0.9 g1 exactly
    s_pre = np.array([abs(np.float32(0.1) * np.float32(g1))], dtype=np.float64)
    codes_pre = np.array([255], dtype=np.uint8)
    th = np.array([0.5])
    cq, s, v = codes_pre.copy(), s_pre.copy(), np.array([0.01])
    m = np.zeros(1)
    offs = np.array([0, 1], dtype=np.int64)
    g = np.array([g2], dtype=np.float32)
    oracle.step_blocks(th, g, cq, s, v, offs, cb, cb, 1e-3, b1, 0.999, 1e-8, 0.0, 2, m_out=m)
    assert abs(m[0]) < 1e-15                      # float64 noise of an exact zero
    post_codes = np.array([255 - int(cq[0])], dtype=np.uint8)   # the other end
    post_s = np.array([1e-10])
    args = (np.array([0.5]), codes_pre, s_pre, th.copy(), post_codes, post_s, v.copy(),
            th, cq, s, v, m, g.astype(np.float64), offs, cb, cb, 1e-3, (b1, 0.999), 1e-8,
            0.0, 2)
    rep = gates.check_tensor(*args)
    assert rep["code_ties"] == 1
    # a well-conditioned element: a code two entries away is refused
    g = np.array([0.3], dtype=np.float32)
    th = np.array([0.5])
    cq, s, v, m = codes_pre.copy(), s_pre.copy(), np.array([0.01]), np.zeros(1)
    oracle.step_blocks(th, g, cq, s, v, offs, cb, cb, 1e-3, b1, 0.999, 1e-8, 0.0, 2, m_out=m)
    bad = np.array([int(cq[0]) - 2], dtype=np.uint8)
    with pytest.raises(AssertionError, match="outside the tie window"):
        gates.check_tensor(np.array([0.5]), codes_pre, s_pre, th.copy(), bad, s.copy(),
                           v.copy(), th, cq, s, v, m, g.astype(np.float64), offs, cb, cb,
                           1e-3, (b1, 0.999), 1e-8, 0.0, 2)
